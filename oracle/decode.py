"""Plain fp64 CPU oracle of the decoding step built from the MoE layer oracle.

TEST INFRASTRUCTURE ONLY (same rule as ``oracle.moe``).

The stacked model is a pre-norm residual stack without attention (attention
and its KV cache are outside the hot path; the paper keeps them resident,
Section 4.1): ``h <- Emb[token]``, ``h <- h + Dense(RMSNorm(h))`` for layer 0,
``h <- h + MoE_l(RMSNorm(h))`` for the MoE layers, then a final RMSNorm and the
LM head.  Without attention a block position depends only on its own token,
so the drafter's next token is the argmax of the draft logits of the previous
draft token, and the verifier scores all K+1 positions in one pass
(Algorithm 1: draft loop, verify, accept).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable

import numpy as np

from . import moe


@dataclass
class LayerWeights:
    """fp64 weights of one MoE layer (routed experts through a lookup)."""

    w_router: np.ndarray
    bias: np.ndarray | None
    routed: Callable[[int], tuple]
    shared: list
    draft: tuple | None
    gamma: float
    top_k: int
    score_func: int
    norm_topk: bool
    routed_scale: float = 1.0


@dataclass
class ModelWeights:
    emb: Callable[[int], np.ndarray]       # token -> fp64 [H]
    dense: tuple                           # (G, U, D) of layer 0
    layers: list                           # LayerWeights of MoE layers 1..L
    lm_head: np.ndarray                    # fp64 [V, H]
    eps: float = 1e-6
    draft_topr: int = 1                    # routed experts per draft layer (Eq. 5: 1)


@dataclass
class Trace:
    """Per-layer record of a forward pass (inputs to each MoE layer and routing)."""

    moe_inputs: list = field(default_factory=list)   # normed x entering each MoE layer
    idx: list = field(default_factory=list)
    gate: list = field(default_factory=list)
    moe_out: list = field(default_factory=list)
    final_h: np.ndarray | None = None
    logits: np.ndarray | None = None


def forward(model: ModelWeights, tokens, mode: str = "target", trace: Trace | None = None):
    """Logits [T, V] of the stack for each token; ``mode`` selects Eq. (4) or Eq. (5)."""
    toks = [int(t) for t in np.asarray(tokens).ravel()]
    h = np.stack([model.emb(t) for t in toks]).astype(np.float64)
    h = h + moe.swiglu(moe.rmsnorm(h, model.eps), *model.dense)
    for lw in model.layers:
        x = moe.rmsnorm(h, model.eps)
        if mode == "target":
            y, idx, gate = moe.moe_target(x, lw.w_router, lw.bias, lw.routed, lw.shared,
                                          lw.top_k, lw.score_func, lw.norm_topk, lw.routed_scale)
        elif mode == "draft":
            y, idx, gate = moe.moe_draft(x, lw.w_router, lw.bias, lw.routed, lw.shared, lw.draft,
                                         lw.gamma, lw.top_k, lw.score_func, lw.norm_topk,
                                         lw.routed_scale, model.draft_topr)
        else:
            raise ValueError(mode)
        if trace is not None:
            trace.moe_inputs.append(x)
            trace.idx.append(idx)
            trace.gate.append(gate)
            trace.moe_out.append(y)
        h = h + y
    hn = moe.rmsnorm(h, model.eps)
    logits = hn @ model.lm_head.T
    if trace is not None:
        trace.final_h = hn
        trace.logits = logits
    return logits


def spec_step(model: ModelWeights, last_token: int, k_draft: int, traces: list | None = None):
    """One exact draft-then-verify step (Algorithm 1 with a fixed draft length K).

    Drafts d_1..d_K with the fixed-footprint drafter, verifies the block
    [c, d_1..d_K] with the target in one pass and accepts the target-consistent
    prefix.  Returns (drafts, n, bonus, target_argmax); the emitted tokens are
    drafts[:n] followed by the bonus token.  With ``traces`` (a list), the
    Trace of each of the K draft passes and then of the verify pass is appended.
    """
    def traced():
        if traces is None:
            return None
        traces.append(Trace())
        return traces[-1]

    drafts = []
    cur = int(last_token)
    for _ in range(k_draft):
        cur = int(moe.argmax_first(forward(model, [cur], "draft", traced()))[0])
        drafts.append(cur)
    logits = forward(model, [int(last_token)] + drafts, "target", traced())
    n, bonus, t = moe.accept_len(logits, drafts)
    return drafts, n, bonus, t


def greedy_ar(model: ModelWeights, last_token: int, n_steps: int):
    """Plain greedy autoregressive decoding with the target, one token per pass."""
    out = []
    cur = int(last_token)
    for _ in range(n_steps):
        cur = int(moe.argmax_first(forward(model, [cur], "target"))[0])
        out.append(cur)
    return out


def single_layer_logits(x, y, lm_head, eps: float = 1e-6):
    """Teacher-forced logits of one layer: W_lm RMSNorm(x + y) per block position."""
    return moe.rmsnorm(np.asarray(x, np.float64) + y, eps) @ lm_head.T
