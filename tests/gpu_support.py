"""Device-side counterparts of the test layers (GPU tests only)."""
from __future__ import annotations

import numpy as np
import torch

import paper_2607_24434_amd as de
from workloads import configs, gpu as wgpu

from support import OracleLayer


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device")


def desc_of(cfg: configs.MoECfg, **over):
    kw = dict(hidden=cfg.hidden, n_experts=cfg.n_experts, top_k=cfg.top_k, inter=cfg.inter,
              shared_inter=cfg.shared_inter, draft_inter=cfg.draft_inter,
              score_func=cfg.score_func, norm_topk=cfg.norm_topk, routed_scale=cfg.routed_scale,
              wdtype=cfg.wdtype)
    kw.update(over)
    return de.make_desc(**kw)


class DevLayer:
    """Resident device weights of one generated layer (GPU-filled streams)."""

    def __init__(self, cfg: configs.MoECfg, layer: int = 0, redraw: int = 0, bias=None,
                 device="cuda"):
        self.cfg = cfg
        self.routed = wgpu.routed_experts(cfg, layer, device, redraw)
        self.shared = wgpu.shared_block(cfg, layer, device, redraw) if cfg.shared_inter else None
        self.draft = wgpu.draft_block(cfg, layer, device, redraw) if cfg.draft_inter else None
        self.router = wgpu.router(cfg, layer, device, redraw)
        self.bias = None if bias is None else torch.from_numpy(np.asarray(bias, np.float32)).to(device)
        self.desc = desc_of(cfg)
        self.stride = cfg.expert_bytes()
        self.table = de.make_table(self.routed, self.stride, None, cfg.n_experts)
        self.device = device

    def ws(self, T: int) -> torch.Tensor:
        return de.workspace(self.desc, T, self.device)


_LAYERS: dict = {}


def layer_pair(cfg: configs.MoECfg, layer: int = 0):
    key = (cfg.name, cfg.cfg_id, layer)
    if key not in _LAYERS:
        orc = OracleLayer(cfg, layer)
        dev = DevLayer(cfg, layer, bias=orc.bias_f32)
        _LAYERS[key] = (orc, dev)
    return _LAYERS[key]


def f32(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def i32(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


def verify_outputs(dev: DevLayer, x_dev: torch.Tensor, T: int, epi=None, y=None):
    cfg = dev.cfg
    d = x_dev.device
    out = dict(
        y=torch.empty(T, cfg.hidden, dtype=torch.float32, device=d) if y is None else y,
        idx=torch.empty(T, cfg.top_k, dtype=torch.int32, device=d),
        gate=torch.empty(T, cfg.top_k, dtype=torch.float32, device=d),
        nu=torch.empty(1, dtype=torch.int32, device=d),
        uids=torch.empty(cfg.n_experts, dtype=torch.int32, device=d),
        offs=torch.empty(cfg.n_experts + 1, dtype=torch.int32, device=d),
        tok=torch.empty(T * cfg.top_k, dtype=torch.int32, device=d),
        glist=torch.empty(T * cfg.top_k, dtype=torch.float32, device=d),
        ppos=torch.empty(T, cfg.top_k, dtype=torch.int32, device=d),
    )
    de.de_verify_layer(dev.desc, T, x_dev, dev.router, dev.bias, dev.table, dev.shared, out["y"],
                       out["idx"], out["gate"], out["nu"], out["uids"], out["offs"], out["tok"],
                       out["glist"], out["ppos"], ws=dev.ws(T), epi=epi)
    return out
