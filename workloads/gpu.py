"""Device-side fills of the synthetic streams (bit-identical to ``workloads.rng``).

Large weight sets (a 64-expert layer is 1.1 GB in bf16, a 26-layer model
29 GB) are drawn directly in HBM by ``libdesynth.so`` instead of being copied
from the host.  Small tensors (activations, routers, biases) come from the
CPU generator and are copied.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

from . import gen, rng
from .configs import BF16, Q4_0, MoECfg, ModelCfg

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdesynth.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with `python -m workloads.build`")
        lib = ctypes.CDLL(path)
        lib.synth_fill_normal.restype = ctypes.c_int
        lib.synth_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                          ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                          ctypes.c_void_p]
        for name in ("synth_fill_bytes", "synth_fill_q4scale"):
            fn = getattr(lib, name)
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                           ctypes.c_void_p]
        _LIB = lib
    return _LIB


def fill_normal(out: torch.Tensor, key: int, std: float, start: int = 0) -> torch.Tensor:
    """Fill a contiguous device tensor (float32, or uint16/int16 holding bf16 bits)."""
    assert out.is_cuda and out.is_contiguous()
    bf16 = out.dtype in (torch.int16, torch.uint16, torch.bfloat16)
    assert bf16 or out.dtype == torch.float32
    rc = _lib().synth_fill_normal(out.data_ptr(), out.numel(), int(bf16), key, start,
                                  float(std) / rng.IH_STD, torch.cuda.current_stream().cuda_stream)
    if rc != 0:
        raise RuntimeError(f"synth_fill_normal failed ({rc})")
    return out


def _wtensor(n: int, wdtype: int, device) -> torch.Tensor:
    return torch.empty(n, dtype=torch.int16 if wdtype == BF16 else torch.float32, device=device)


def _call(name, *args):
    rc = getattr(_lib(), name)(*args, torch.cuda.current_stream().cuda_stream)
    if rc != 0:
        raise RuntimeError(f"{name} failed ({rc})")


def fill_q4_block(out: torch.Tensor, cfg: MoECfg, tag: str, layer: int, index: int, inter: int,
                  redraw: int = 0) -> torch.Tensor:
    """A Q4_0 [G|U|D] block (uint8 device tensor), bit-identical to gen's."""
    assert out.is_cuda and out.is_contiguous() and out.dtype == torch.uint8
    H = cfg.hidden
    off = 0
    for part, (r, c) in enumerate(((inter, H), (inter, H), (H, inter))):
        kc, ks = gen.q4_keys(cfg.cfg_id, redraw, tag, layer, index, part)
        nc, ns = r * c // 2, r * c // 32
        _call("synth_fill_bytes", out[off:].data_ptr(), nc, kc, 0)
        _call("synth_fill_q4scale", out[off + nc:].data_ptr(), ns, ks, 0)
        off += nc + 2 * ns
    return out


def _block(cfg: MoECfg, tag: str, layer: int, index: int, inter: int, device, redraw: int):
    if cfg.wdtype == Q4_0:
        out = torch.empty(cfg.expert_bytes(inter), dtype=torch.uint8, device=device)
        return fill_q4_block(out, cfg, tag, layer, index, inter, redraw)
    out = _wtensor(cfg.expert_elems(inter), cfg.wdtype, device)
    return fill_normal(out, rng.key_for(cfg.cfg_id, redraw, tag, layer, index), cfg.weight_std)


def routed_experts(cfg: MoECfg, layer: int, device="cuda", redraw: int = 0,
                   n_experts: int | None = None) -> torch.Tensor:
    """[N, block] expert blocks, expert e in row e (the resident layout)."""
    n = cfg.n_experts if n_experts is None else n_experts
    if cfg.wdtype == Q4_0:
        out = torch.empty(n, cfg.expert_bytes(), dtype=torch.uint8, device=device)
        for e in range(n):
            fill_q4_block(out[e], cfg, "routed", layer, e, cfg.inter, redraw)
        return out
    out = _wtensor(n * cfg.expert_elems(), cfg.wdtype, device).view(n, -1)
    for e in range(n):
        fill_normal(out[e], rng.key_for(cfg.cfg_id, redraw, "routed", layer, e), cfg.weight_std)
    return out


def shared_block(cfg: MoECfg, layer: int, device="cuda", redraw: int = 0) -> torch.Tensor:
    return _block(cfg, "shared", layer, 0, cfg.shared_inter, device, redraw)


def draft_block(cfg: MoECfg, layer: int, device="cuda", redraw: int = 0) -> torch.Tensor:
    return _block(cfg, "draft", layer, 0, cfg.draft_inter, device, redraw)


def dense_block(model: ModelCfg, device="cuda", redraw: int = 0) -> torch.Tensor:
    out = _wtensor(3 * model.dense_inter * model.moe.hidden, BF16, device)
    return fill_normal(out, rng.key_for(model.cfg_id, redraw, "dense", 0, 0), model.moe.weight_std)


def embedding(model: ModelCfg, device="cuda", redraw: int = 0) -> torch.Tensor:
    out = _wtensor(model.vocab * model.moe.hidden, BF16, device).view(model.vocab, -1)
    return fill_normal(out, rng.key_for(model.cfg_id, redraw, "emb", 0, 0), model.emb_std)


def lm_head(cfg_id: int, vocab: int, hidden: int, std: float = 0.02, device="cuda",
            redraw: int = 0) -> torch.Tensor:
    out = torch.empty(vocab * hidden, dtype=torch.int16, device=device).view(vocab, hidden)
    return fill_normal(out, rng.key_for(cfg_id, redraw, "lm", 0, 0), std)


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def router(cfg: MoECfg, layer: int, device="cuda", redraw: int = 0) -> torch.Tensor:
    return to_device(gen.router_weight(cfg, layer, redraw), device)


def model_tensors(model: ModelCfg, device="cuda", redraw: int = 0) -> dict:
    """Every weight of a stacked model, resident in HBM.

    MoE layer l (1..L) uses the layer-l streams of the per-layer generators;
    layer 0 is the dense layer.  Returns {"emb", "dense", "lm", "layers"}, each
    layer a dict with "router", "bias", "routed", "shared", "draft"."""
    m = model.moe
    layers = []
    for l in range(1, model.n_moe_layers + 1):
        b = gen.router_bias(m, l, redraw)
        if model.zipf_s > 0:
            b = gen.zipf_bias(model, l, model.zipf_lam, redraw)
        layers.append(dict(
            router=router(m, l, device, redraw),
            bias=None if b is None else to_device(b, device),
            routed=routed_experts(m, l, device, redraw),
            shared=shared_block(m, l, device, redraw) if m.shared_inter else None,
            draft=draft_block(m, l, device, redraw) if m.draft_inter else None,
        ))
    return dict(
        emb=embedding(model, device, redraw),
        dense=dense_block(model, device, redraw) if model.dense_inter else None,
        lm=lm_head(model.cfg_id, model.vocab, m.hidden, model.lm_std, device, redraw),
        layers=layers,
    )
