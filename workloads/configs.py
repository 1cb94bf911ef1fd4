"""Synthetic workload shapes and value distributions.

The shapes follow the two MoE models the paper evaluates (DeepSeek-V2-Lite and
Moonlight-16B-A3B: 27 layers, 64 routed + 2 shared experts, top-6; Section 4.1,
Table 1) plus a tiny fp32 layer for fast checks.  Trained weights and prompt
sets are not available, so every tensor is drawn from the seeded counter-based
streams in ``workloads.rng``.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

SOFTMAX = 0
SIGMOID = 1
F32 = 0
BF16 = 1
Q4_0 = 2    # blocks of 32 weights: 4-bit codes and an fp16 scale (18 bytes per block)


@dataclass(frozen=True)
class MoECfg:
    """One MoE layer: router, routed experts, shared path and draft expert."""

    name: str
    cfg_id: int
    hidden: int
    n_experts: int
    top_k: int
    inter: int              # routed expert intermediate size
    n_shared: int           # number of shared experts
    shared_each: int        # intermediate size of each shared expert
    draft_inter: int        # intermediate size of the draft expert
    score_func: int         # SOFTMAX or SIGMOID
    norm_topk: bool         # renormalise the top-k gates to sum to one
    wdtype: int             # F32, BF16 or Q4_0 expert weights
    weight_std: float       # routed / shared / draft expert weights
    router_std: float       # fp32 router weights
    bias_std: float = 0.0   # per-expert router bias (0 = no bias)
    routed_scale: float = 1.0
    gamma: float = 1.0      # draft-expert scale
    t_verify: int = 9
    x_std: float = 1.0

    @property
    def shared_inter(self) -> int:
        return self.n_shared * self.shared_each

    @property
    def welem(self) -> int:
        return 4 if self.wdtype == F32 else 2

    def expert_elems(self, inter: int | None = None) -> int:
        i = self.inter if inter is None else inter
        return 3 * i * self.hidden

    def mat_bytes(self, rows: int, cols: int) -> int:
        """Bytes of one [rows, cols] weight matrix in this layer's format."""
        if self.wdtype == Q4_0:
            return rows * cols * 9 // 16   # cols / 32 blocks of 16 code bytes + a 2-byte scale
        return rows * cols * self.welem

    def expert_bytes(self, inter: int | None = None) -> int:
        i = self.inter if inter is None else inter
        return 2 * self.mat_bytes(i, self.hidden) + self.mat_bytes(self.hidden, i)


@dataclass(frozen=True)
class ModelCfg:
    """A stacked decoder without attention: dense layer 0, then MoE layers."""

    name: str
    cfg_id: int
    moe: MoECfg
    n_moe_layers: int
    dense_inter: int
    vocab: int
    k_draft: int            # K: number of drafted tokens per step
    emb_std: float = 1.0
    lm_std: float = 0.02
    eps: float = 1e-6
    zipf_s: float = 0.0     # 0 = no popularity skew
    zipf_lam: float = 0.0   # scale of the Zipf router bias (tests/golden/calibrate_zipf.py)
    cache_slots: int = 0    # 0 = every expert resident in HBM


# Tiny single layer, fp32 weights; 1000-vocab bf16 head for the accept check.
CFG1 = MoECfg(
    name="tiny-fp32", cfg_id=1, hidden=256, n_experts=8, top_k=2, inter=128,
    n_shared=1, shared_each=128, draft_inter=64, score_func=SOFTMAX,
    norm_topk=True, wdtype=F32, weight_std=0.02, router_std=0.02, t_verify=5,
)
CFG1_VOCAB = 1000
CFG1_K = 4

# DeepSeek-V2-Lite-shaped layer: softmax top-6 of 64, gates not renormalised.
CFG2 = MoECfg(
    name="v2lite", cfg_id=2, hidden=2048, n_experts=64, top_k=6, inter=1408,
    n_shared=2, shared_each=1408, draft_inter=1408, score_func=SOFTMAX,
    norm_topk=False, wdtype=BF16, weight_std=0.02, router_std=0.1, t_verify=9,
)

# Moonlight-16B-A3B-shaped layer: sigmoid scores, per-expert selection bias,
# renormalised top-6 gates; block length swept over 5, 9, 17.
CFG3 = MoECfg(
    name="moonlight", cfg_id=3, hidden=2048, n_experts=64, top_k=6, inter=1408,
    n_shared=2, shared_each=1408, draft_inter=1408, score_func=SIGMOID,
    norm_topk=True, wdtype=BF16, weight_std=0.02, router_std=0.02, bias_std=0.1,
    t_verify=9,
)
CFG3_T = (5, 9, 17)

# Full draft+verify step: dense layer 0 + 26 V2-Lite MoE layers, K=8, V=102400.
CFG4 = ModelCfg(
    name="v2lite-step", cfg_id=4, moe=replace(CFG2, cfg_id=4), n_moe_layers=26,
    dense_inter=10944, vocab=102400, k_draft=8,
)

# Offload stress: Zipf(1.1) expert popularity through a router bias, K=16,
# 16 HBM cache slots per layer over a pinned host pool.
CFG5 = ModelCfg(
    name="v2lite-offload", cfg_id=5, moe=replace(CFG2, cfg_id=5), n_moe_layers=26,
    dense_inter=10944, vocab=102400, k_draft=16, zipf_s=1.1, zipf_lam=2.7449, cache_slots=16,
)


def scaled_model(base: ModelCfg, *, n_moe_layers: int | None = None, vocab: int | None = None,
                 dense_inter: int | None = None, k_draft: int | None = None,
                 moe: MoECfg | None = None, name: str | None = None) -> ModelCfg:
    """A smaller model with the same per-layer structure (for fast parity runs)."""
    return replace(
        base,
        name=name or base.name + "-small",
        n_moe_layers=base.n_moe_layers if n_moe_layers is None else n_moe_layers,
        vocab=base.vocab if vocab is None else vocab,
        dense_inter=base.dense_inter if dense_inter is None else dense_inter,
        k_draft=base.k_draft if k_draft is None else k_draft,
        moe=base.moe if moe is None else moe,
    )


# The tiny layer and the V2-Lite layer with Q4_0 expert weights (the mobile platform's format,
# Section 4.1): routed, shared and draft experts 4.5 bits per weight.
CFG1_Q4 = replace(CFG1, name="tiny-q4", cfg_id=7, wdtype=Q4_0)
CFG2_Q4 = replace(CFG2, name="v2lite-q4", cfg_id=6, wdtype=Q4_0)
# The offload stack with Q4_0 experts (the paper's mobile pairing of the 4.5-bit
# format with offloaded experts); same seeds, routers and Zipf biases as CFG5.
CFG5_Q4 = replace(CFG5, name="v2lite-offload-q4", moe=replace(CFG5.moe, wdtype=Q4_0))

ALL_LAYER_CFGS = {"cfg1": CFG1, "cfg2": CFG2, "cfg3": CFG3}
