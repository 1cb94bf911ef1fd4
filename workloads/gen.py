"""CPU-side generation of every synthetic tensor, one seeded stream per tensor.

Layout conventions (shared by both sides, since they describe the inputs):

* An expert block is one contiguous stream of ``3*I*H`` values laid out as
  ``[G: I x H][U: I x H][D: H x I]``, each matrix row-major ``[out, in]``.
* The shared path of a layer is one such block with ``I = n_shared * I_each``
  (the shared experts concatenated along the intermediate dimension).
* Router weights are fp32 ``[N, H]``; biases fp32 ``[N]``.
* Embedding and LM head are bf16 ``[V, H]``.

Key fields: ``(cfg_id, redraw, tag, layer, index)``.  Single-layer configs use
layer 0.  In a stacked model layer 0 is the dense layer and MoE layers are
1..L.  Activation rows carry their own redraw counter so that a test can
resample one token without touching the others.
"""
from __future__ import annotations

import numpy as np

from . import rng
from .configs import BF16, F32, Q4_0, MoECfg, ModelCfg


def _weights(cfg_id: int, redraw: int, tag: str, layer: int, index: int, n: int,
             std: float, wdtype: int) -> np.ndarray:
    key = rng.key_for(cfg_id, redraw, tag, layer, index)
    if wdtype == BF16:
        return rng.normal_bf16(key, n, std)
    return rng.normal_f32(key, n, std)


def q4_keys(cfg_id: int, redraw: int, tag: str, layer: int, index: int, part: int):
    """Stream keys of the codes and the scales of matrix `part` (G 0, U 1, D 2)."""
    base = (cfg_id, redraw, rng.TAGS[tag], layer, index, 100 + part)
    return rng.stream_key(*base, 0), rng.stream_key(*base, 1)


def q4_matrix(kc: int, ks: int, rows: int, cols: int) -> np.ndarray:
    """One Q4_0 matrix as bytes: every row's codes (cols / 2 bytes per row,
    block b of a row at byte 16 b: element j of the block in the low nibble of
    byte j, element j + 16 in its high nibble), then every row's fp16 scales
    (cols / 32 per row)."""
    codes = rng.bytes_u8(kc, rows * cols // 2)
    scales = rng.q4_scale_bits(ks, rows * cols // 32).view(np.uint8)
    return np.concatenate([codes, scales])


def _q4_block(cfg_id: int, redraw: int, tag: str, layer: int, index: int, inter: int,
              hidden: int) -> np.ndarray:
    shapes = ((inter, hidden), (inter, hidden), (hidden, inter))
    return np.concatenate([q4_matrix(*q4_keys(cfg_id, redraw, tag, layer, index, p), r, c)
                           for p, (r, c) in enumerate(shapes)])


def _block(cfg: MoECfg, tag: str, layer: int, index: int, inter: int, redraw: int):
    if cfg.wdtype == Q4_0:
        return _q4_block(cfg.cfg_id, redraw, tag, layer, index, inter, cfg.hidden)
    return _weights(cfg.cfg_id, redraw, tag, layer, index, cfg.expert_elems(inter),
                    cfg.weight_std, cfg.wdtype)


def routed_block(cfg: MoECfg, layer: int, e: int, redraw: int = 0) -> np.ndarray:
    """Flat ``[G|U|D]`` block of routed expert ``e`` (uint16 bf16 bits, fp32, or
    Q4_0 bytes: the three matrices one after the other, each as q4_matrix)."""
    return _block(cfg, "routed", layer, e, cfg.inter, redraw)


def shared_block(cfg: MoECfg, layer: int, redraw: int = 0) -> np.ndarray:
    return _block(cfg, "shared", layer, 0, cfg.shared_inter, redraw)


def draft_block(cfg: MoECfg, layer: int, redraw: int = 0) -> np.ndarray:
    return _block(cfg, "draft", layer, 0, cfg.draft_inter, redraw)


def dense_block(model: ModelCfg, redraw: int = 0) -> np.ndarray:
    m = model.moe
    return _weights(model.cfg_id, redraw, "dense", 0, 0, 3 * model.dense_inter * m.hidden,
                    m.weight_std, BF16)


def router_weight(cfg: MoECfg, layer: int, redraw: int = 0) -> np.ndarray:
    key = rng.key_for(cfg.cfg_id, redraw, "router", layer, 0)
    return rng.normal_f32(key, cfg.n_experts * cfg.hidden, cfg.router_std).reshape(
        cfg.n_experts, cfg.hidden)


def router_bias(cfg: MoECfg, layer: int, redraw: int = 0) -> np.ndarray | None:
    if cfg.bias_std == 0.0:
        return None
    key = rng.key_for(cfg.cfg_id, redraw, "bias", layer, 0)
    return rng.normal_f32(key, cfg.n_experts, cfg.bias_std)


def zipf_bias(model: ModelCfg, layer: int, lam: float, redraw: int = 0) -> np.ndarray:
    """Router bias b_e = lam * (-s * ln r_e), r_e a seeded permutation of 1..N.

    Added to the softmax logits it makes expert popularity fall off with rank
    like a Zipf law of exponent s (lam is calibrated separately).
    """
    n = model.moe.n_experts
    key = rng.key_for(model.cfg_id, redraw, "perm", layer, 0)
    order = np.argsort(rng.uniform_f64(key, n), kind="stable")
    rank = np.empty(n, dtype=np.int64)
    rank[order] = np.arange(1, n + 1)
    return (lam * (-model.zipf_s * np.log(rank.astype(np.float64)))).astype(np.float32)


def x_rows(cfg: MoECfg, n_rows: int, block: int = 0, redraws=None) -> np.ndarray:
    """Activation rows ``[n_rows, H]`` fp32; row t uses its own redraw counter."""
    out = np.empty((n_rows, cfg.hidden), dtype=np.float32)
    for t in range(n_rows):
        r = 0 if redraws is None else int(redraws[t])
        key = rng.key_for(cfg.cfg_id, r, "x", block, t)
        out[t] = rng.normal_f32(key, cfg.hidden, cfg.x_std)
    return out


def embedding(model: ModelCfg, redraw: int = 0) -> np.ndarray:
    key = rng.key_for(model.cfg_id, redraw, "emb", 0, 0)
    return rng.normal_bf16(key, model.vocab * model.moe.hidden, model.emb_std).reshape(
        model.vocab, model.moe.hidden)


def lm_head(cfg_id: int, vocab: int, hidden: int, std: float = 0.02, redraw: int = 0) -> np.ndarray:
    key = rng.key_for(cfg_id, redraw, "lm", 0, 0)
    return rng.normal_bf16(key, vocab * hidden, std).reshape(vocab, hidden)


def start_token(model: ModelCfg, redraw: int = 0, index: int = 0) -> int:
    key = rng.key_for(model.cfg_id, redraw, "token", 0, index)
    return int(rng.uniform_int(key, 1, model.vocab)[0])


def split_block(block: np.ndarray, inter: int, hidden: int):
    """Views (G [I,H], U [I,H], D [H,I]) into a flat expert block."""
    n = inter * hidden
    return (block[:n].reshape(inter, hidden), block[n:2 * n].reshape(inter, hidden),
            block[2 * n:3 * n].reshape(hidden, inter))


__all__ = [
    "routed_block", "shared_block", "draft_block", "dense_block", "router_weight",
    "router_bias", "zipf_bias", "x_rows", "embedding", "lm_head", "start_token",
    "split_block", "F32", "BF16",
]
