#!/usr/bin/env python3
"""Benchmark of the DraftExpert MoE draft/verify hot path on one MI355X.

Workload: one DeepSeek-V2-Lite-shaped MoE layer (H=2048, 64 routed SwiGLU
experts of I=1408, 2 shared experts, softmax top-6, bf16 expert weights, fp32
router, one draft expert of I=1408) with K=8 drafts.  One step is the whole hot
path over one block:

  * 8 draft-layer passes (Eq. 5), one position each;
  * one verify-layer pass over the 9-position block (Eq. 4: routing, union,
    grouped SwiGLU over the union, shared path);
  * the 102400-vocab bf16 LM head over the 8 draft positions and the 9 verify
    positions (teacher-forced, RMSNorm(x + y) as in a one-layer model) and the
    greedy accept length (Algorithm 1).

Weights are drawn in HBM before timing.  Every layer call in a step uses a
different copy of the layer weights (8 copies rotated), so no call finds its
weights in the 256 MB Infinity Cache left behind by the previous one.

Reported: ``value`` = achieved GB/s over the union expert weights of the verify
layer (n_union x 17,301,504 B / verify-layer time), plus per-stage times, a
``roofline`` object for the dominant kernel (the grouped gate/up GEMV of the
verify layer, timed live with HIP events around its launch) and the CPU
oracle's rate on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

METRIC = "verify-layer µs + achieved HBM GB/s over union expert weights (K=8, V2-Lite shape)"
PEAK_HBM_GBS = 8000.0

# HBM bytes per launch of the verify-layer gate/up kernel, from two rocprofv3
# --pmc runs of this benchmark (FETCH_SIZE, then WRITE_SIZE; summary and scale
# factors in profiles/verify_layer_v2lite_T9.md).  Valid only for the kernel
# sources they were measured on: reported as null once those change.
PMC_TRAFFIC = {
    "bytes_per_launch": 463.53e6,
    "vs_algorithmic": 1.004,
    "union_mean": 38.0,
    "sources": ["paper_2607_24434_amd/csrc/grouped_swiglu.hip",
                "paper_2607_24434_amd/csrc/grouped_core.h",
                "paper_2607_24434_amd/csrc/topk_union.h",
                "paper_2607_24434_amd/csrc/de_common.h"],
    "sha256": "87cb95446bf41797167802e6d934f5cf9c65f6a9e217c7886e25d26cd1eb4193",
}


def pmc_traffic():
    """The measured per-launch traffic when the kernel sources are unchanged, else None."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    h = hashlib.sha256()
    try:
        for f in PMC_TRAFFIC["sources"]:
            with open(os.path.join(root, f), "rb") as fh:
                h.update(fh.read())
    except OSError:
        return None
    return PMC_TRAFFIC["bytes_per_launch"] if h.hexdigest() == PMC_TRAFFIC["sha256"] else None


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=30)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--copies", type=int, default=8)
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--no-probe", action="store_true", help="skip the HBM read-ceiling probe")
    p.add_argument("--no-full-step", action="store_true",
                   help="skip the 26-layer draft+verify step measurement")
    p.add_argument("--full-steps", type=int, default=12)
    p.add_argument("--no-offload", action="store_true",
                   help="skip the expert-cache (offload) step measurement")
    p.add_argument("--offload-steps", type=int, default=3)
    p.add_argument("--no-verify-side", action="store_true",
                   help="skip the truncation / prefetch comparison on the offload stack")
    p.add_argument("--no-q4", action="store_true",
                   help="skip the Q4_0-weight layer measurement")
    p.add_argument("--no-draft-side", action="store_true",
                   help="skip the drafter comparison (top-r against DraftExpert) on the offload stack")
    p.add_argument("--no-cfg3", action="store_true",
                   help="skip the Moonlight-shaped block-length sweep (T = 1, 5, 9, 17)")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported (the library "
              f"has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_24434_amd as de
    from workloads import configs, gen
    from workloads import gpu as wgpu

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    dev = "cuda"
    cfg = configs.CFG2
    K = 8
    T = K + 1
    H = cfg.hidden
    V = configs.CFG4.vocab
    R = args.copies

    desc = de.make_desc(H, cfg.n_experts, cfg.top_k, cfg.inter, cfg.shared_inter,
                        cfg.draft_inter, cfg.score_func, cfg.norm_topk, cfg.routed_scale,
                        cfg.wdtype)
    stride = cfg.expert_bytes()
    copies = []
    for c in range(R):
        routed = wgpu.routed_experts(cfg, 0, dev, redraw=c)
        copies.append(dict(
            routed=routed,
            table=de.make_table(routed, stride, None, cfg.n_experts),
            shared=wgpu.shared_block(cfg, 0, dev, redraw=c),
            draft=wgpu.draft_block(cfg, 0, dev, redraw=c),
            router=wgpu.router(cfg, 0, dev, redraw=c),
        ))
    w_lm = wgpu.lm_head(configs.CFG4.cfg_id, V, H, configs.CFG4.lm_std, dev)
    x_ver = wgpu.to_device(gen.x_rows(cfg, T, block=0), dev)
    x_dr = wgpu.to_device(gen.x_rows(cfg, K, block=1), dev)

    ws = de.workspace(desc, T, dev)
    aws = de.accept_workspace(K, V, dev)
    y_dr = torch.empty(K, H, dtype=torch.float32, device=dev)
    n_dr = torch.empty(K, H, dtype=torch.float32, device=dev)
    pred = torch.empty(K, cfg.top_k, dtype=torch.int32, device=dev)
    y_ver = torch.empty(T, H, dtype=torch.float32, device=dev)
    n_ver = torch.empty(T, H, dtype=torch.float32, device=dev)
    lg_dr = torch.empty(K, V, dtype=torch.float32, device=dev)
    lg_ver = torch.empty(T, V, dtype=torch.float32, device=dev)
    dtok = torch.empty(K, dtype=torch.int32, device=dev)
    tmax = torch.empty(T, dtype=torch.int32, device=dev)
    acc_dummy = torch.empty(2, dtype=torch.int32, device=dev)
    total = args.warmup + args.steps
    nu_all = torch.zeros(total, dtype=torch.int32, device=dev)
    acc_all = torch.zeros(total, 2, dtype=torch.int32, device=dev)
    zero_tok = torch.zeros(K, dtype=torch.int32, device=dev)

    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def step(s, evs, phases=False):
        base = s * (K + 1)
        evs["s0"].record()
        for i in range(K):
            cp = copies[(base + i) % R]
            epi = de.make_epilogue(residual=x_dr[i:i + 1], normed=n_dr[i:i + 1])
            de.de_draft_layer(desc, 1, x_dr[i:i + 1], cp["router"], None, cp["table"], cp["shared"],
                              cp["draft"], cfg.gamma, y_dr[i:i + 1], pred[i:i + 1], None, ws, epi=epi)
        evs["d1"].record()
        de.de_lm_head(K, H, V, n_dr, w_lm, lg_dr)
        de.de_accept_len(K - 1, V, lg_dr, zero_tok, dtok, acc_dummy, aws)  # row argmax = drafts
        evs["v0"].record()
        cp = copies[(base + K) % R]
        if phases:
            de.de_time_next_phase(de.DE_PHASE_GATEUP, evs["g0"], evs["g1"])
            de.de_time_next_phase(de.DE_PHASE_DOWN, evs["p0"], evs["p1"])
        de.de_verify_layer(desc, T, x_ver, cp["router"], None, cp["table"], cp["shared"], y_ver,
                           n_union=nu_all[s:s + 1], ws=ws,
                           epi=de.make_epilogue(residual=x_ver, normed=n_ver))
        evs["v1"].record()
        de.de_lm_head(T, H, V, n_ver, w_lm, lg_ver)
        de.de_accept_len(K, V, lg_ver, dtok, tmax, acc_all[s], aws)
        evs["s1"].record()

    names = ["s0", "d1", "v0", "v1", "s1", "g0", "g1", "p0", "p1"]
    for s in range(args.warmup):
        step(s, {n: ev() for n in names})
    torch.cuda.synchronize()

    rec = [{n: ev() for n in names} for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, rec[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0

    # Kernel durations for the roofline: the same steps again, with HIP events
    # recorded around the grouped gate/up and down launches of the verify layer
    # on the library's stream.  They are kept out of the timed steps above
    # because the extra event records add gaps between the layer's kernels.
    prec = [{n: ev() for n in names} for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(args.warmup + i, prec[i], phases=True)
    torch.cuda.synchronize()

    nu = nu_all[args.warmup:].cpu().numpy().astype(np.int64)
    accs = acc_all[args.warmup:].cpu().numpy()
    step_ms = [r["s0"].elapsed_time(r["s1"]) for r in rec]
    draft_ms = [r["s0"].elapsed_time(r["d1"]) / K for r in rec]
    ver_ms = [r["v0"].elapsed_time(r["v1"]) for r in rec]
    gu_ms = [r["g0"].elapsed_time(r["g1"]) for r in prec]
    dn_ms = [r["p0"].elapsed_time(r["p1"]) for r in prec]

    eb = stride
    union_bytes = nu * eb
    value = float(union_bytes.sum() / (sum(ver_ms) * 1e-3) / 1e9)
    # Algorithmic bytes of one gate/up launch: G and U of every union expert and
    # of the shared path, the block's activations read once and A written once.
    gu_bytes = (nu * 2 * cfg.inter * H * 2 + 2 * cfg.shared_inter * H * 2 + T * H * 4
                + (T * cfg.top_k * cfg.inter + T * cfg.shared_inter) * 4)
    gu_gbs = float(gu_bytes.sum() / (sum(gu_ms) * 1e-3) / 1e9)
    dn_bytes = (nu * cfg.inter * H * 2 + cfg.shared_inter * H * 2
                + (T * cfg.top_k * cfg.inter + T * cfg.shared_inter) * 4 + (T * cfg.top_k + T) * H * 4)
    dn_gbs = float(dn_bytes.sum() / (sum(dn_ms) * 1e-3) / 1e9)

    del copies
    torch.cuda.empty_cache()
    q4 = None
    if not args.no_q4:
        q4 = q4_layer(args, de, configs, gen, wgpu, torch, np, 1e3 * statistics.median(ver_ms))
    sweep = None if args.no_cfg3 else cfg3_sweep(args, de, configs, gen, wgpu, torch, np)
    full = None if args.no_full_step else full_step(args, de, configs, gen, wgpu, torch, np)
    offload = None if args.no_offload else offload_step(args, de, configs, gen, wgpu, torch, np)

    probe_gbs = None
    if not args.no_probe:
        nbytes = 4 << 30
        buf = torch.empty(nbytes // 2, dtype=torch.int16, device=dev)
        wgpu.fill_normal(buf, 12345, 1.0)
        sink = torch.zeros(1, dtype=torch.float32, device=dev)
        for _ in range(2):
            de.de_stream_probe(buf, nbytes, sink)
        e0, e1 = ev(), ev()
        reps = 10
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            de.de_stream_probe(buf, nbytes, sink)
        e1.record()
        torch.cuda.synchronize()
        probe_gbs = nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del buf

    cpu = None
    cpu_extra = None
    if not args.no_cpu:
        cpu = cpu_baseline(cfg, gen.x_rows(cfg, T, block=0), args.cpu_seconds)
        cpu_extra = cpu_baseline_extras(configs, gen, args.cpu_seconds / 3)

    med = statistics.median
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(med(step_ms), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "v2lite-moe-layer-K8: H=2048, 64 routed + 2 shared SwiGLU experts (I=1408), "
                        "softmax top-6, draft expert I=1408, bf16 expert weights, fp32 router and "
                        "activations; 8 draft positions + 9-position verify block; 102400-vocab bf16 "
                        "LM head; 8 rotated weight copies",
            "hidden": H, "n_experts": cfg.n_experts, "top_k": cfg.top_k, "inter": cfg.inter,
            "shared_inter": cfg.shared_inter, "draft_inter": cfg.draft_inter, "k_draft": K,
            "verify_block": T, "vocab": V, "weights": "bf16",
        },
        "union_hbm_frac": round(value / PEAK_HBM_GBS, 4),
        "verify_layer_us": round(1e3 * med(ver_ms), 2),
        "verify_layer_us_p10_p90": [round(1e3 * float(np.percentile(ver_ms, 10)), 2),
                                    round(1e3 * float(np.percentile(ver_ms, 90)), 2)],
        "draft_layer_us": round(1e3 * med(draft_ms), 2),
        "gateup_us": round(1e3 * med(gu_ms), 2),
        "down_us": round(1e3 * med(dn_ms), 2),
        "down_gbs": round(dn_gbs, 1),
        "union_mean": round(float(nu.mean()), 2),
        "accept_mean": round(float(accs[:, 0].mean()), 3),
        "wall_s_timed": round(wall, 4),
        "hbm_read_ceiling_gbs": None if probe_gbs is None else round(probe_gbs, 1),
        "roofline": {
            "kernel": "gateup_kernel (verify layer)",
            "bound": "hbm",
            "achieved": round(gu_gbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(gu_gbs / PEAK_HBM_GBS, 4),
            "traffic": pmc_traffic(),
            "traffic_vs_algorithmic": PMC_TRAFFIC["vs_algorithmic"] if pmc_traffic() else None,
            "algorithmic_bytes_per_launch": int(round(float(gu_bytes.mean()))),
        },
        "q4_layer": q4,
        "cfg3_sweep": sweep,
        "full_step": full,
        "offload_step": offload,
        "cpu_baseline": cpu,
        "cpu_baseline_extra": cpu_extra,
    }
    print(json.dumps(out), flush=True)


def q4_layer(args, de, configs, gen, wgpu, torch, np, bf16_verify_us):
    """The V2-Lite layer with Q4_0 expert weights (routed, shared and draft;
    4,866,048 bytes per expert instead of 17,301,504): the 9-position verify
    layer and a draft layer, on rotated weight copies, with the grouped
    kernels timed by HIP events in separate steps."""
    cfg = configs.CFG2_Q4
    dev = "cuda"
    H, T, R = cfg.hidden, 9, args.copies
    desc = de.make_desc(H, cfg.n_experts, cfg.top_k, cfg.inter, cfg.shared_inter,
                        cfg.draft_inter, cfg.score_func, cfg.norm_topk, cfg.routed_scale,
                        cfg.wdtype)
    eb = cfg.expert_bytes()
    copies = []
    for c in range(R):
        routed = wgpu.routed_experts(cfg, 0, dev, redraw=c)
        copies.append(dict(routed=routed, table=de.make_table(routed, eb, None, cfg.n_experts),
                           shared=wgpu.shared_block(cfg, 0, dev, redraw=c),
                           draft=wgpu.draft_block(cfg, 0, dev, redraw=c),
                           router=wgpu.router(cfg, 0, dev, redraw=c)))
    x = wgpu.to_device(gen.x_rows(cfg, T, block=0), dev)
    ws = de.workspace(desc, T, dev)
    y = torch.empty(T, H, dtype=torch.float32, device=dev)
    steps = args.warmup + args.steps
    nu = torch.zeros(steps, dtype=torch.int32, device=dev)

    def ev():
        # Recorded once here so that torch accepts them; the library records
        # the phase events again around its launches.
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def verify(i, e=None):
        cp = copies[i % R]
        if e is not None:
            de.de_time_next_phase(de.DE_PHASE_GATEUP, e[0], e[1])
            de.de_time_next_phase(de.DE_PHASE_DOWN, e[2], e[3])
        de.de_verify_layer(desc, T, x, cp["router"], None, cp["table"], cp["shared"], y,
                           n_union=nu[i:i + 1], ws=ws)

    def draft(i):
        cp = copies[i % R]
        de.de_draft_layer(desc, 1, x[:1], cp["router"], None, cp["table"], cp["shared"],
                          cp["draft"], cfg.gamma, y[:1], None, None, ws)

    for i in range(args.warmup):
        verify(i)
        draft(i)
    torch.cuda.synchronize()
    vt, dt, ph = [], [], []
    for i in range(args.warmup, steps):
        a, b, c, d = ev(), ev(), ev(), ev()
        a.record()
        verify(i)
        b.record()
        draft(i)
        c.record()
        vt.append((a, b))
        dt.append((b, c))
    for i in range(args.warmup, steps):
        e = [ev() for _ in range(4)]
        verify(i, e)
        ph.append(e)
    torch.cuda.synchronize()
    med = statistics.median
    ver_ms = [a.elapsed_time(b) for a, b in vt]
    n = nu[args.warmup:].cpu().numpy().astype(np.int64)
    gu_ms = [e[0].elapsed_time(e[1]) for e in ph]
    dn_ms = [e[2].elapsed_time(e[3]) for e in ph]
    mb = cfg.mat_bytes
    gu_bytes = (n * 2 * mb(cfg.inter, H) + 2 * mb(cfg.shared_inter, H) + T * H * 4
                + (T * cfg.top_k * cfg.inter + T * cfg.shared_inter) * 4)
    dn_bytes = (n * mb(H, cfg.inter) + mb(H, cfg.shared_inter)
                + (T * cfg.top_k * cfg.inter + T * cfg.shared_inter) * 4 + (T * cfg.top_k + T) * H * 4)
    gu_gbs = float(gu_bytes.sum() / (sum(gu_ms) * 1e-3) / 1e9)
    value = float((n * eb).sum() / (sum(ver_ms) * 1e-3) / 1e9)
    res = {
        "workload": "v2lite-moe-layer-q4_0: the V2-Lite layer (H=2048, 64 routed + 2 shared "
                    "experts of I=1408, top-6, draft expert I=1408) with Q4_0 expert weights "
                    "(18-byte blocks of 32 weights), 9-position verify block, fp32 activations",
        "expert_bytes": eb,
        "verify_layer_us": round(1e3 * med(ver_ms), 2),
        "draft_layer_us": round(1e3 * med([a.elapsed_time(b) for a, b in dt]), 2),
        "gateup_us": round(1e3 * med(gu_ms), 2),
        "down_us": round(1e3 * med(dn_ms), 2),
        "union_mean": round(float(n.mean()), 2),
        "union_gbs": round(value, 1),
        "union_frac_of_peak": round(value / PEAK_HBM_GBS, 4),
        "gateup_gbs": round(gu_gbs, 1),
        "gateup_frac_of_peak": round(gu_gbs / PEAK_HBM_GBS, 4),
        "down_gbs": round(float(dn_bytes.sum() / (sum(dn_ms) * 1e-3) / 1e9), 1),
        "verify_speedup_vs_bf16": round(bf16_verify_us / (1e3 * med(ver_ms)), 3),
    }
    del copies
    torch.cuda.empty_cache()
    return res


def full_step(args, de, configs, gen, wgpu, torch, np):
    """Decode with the full V2-Lite-shaped stack: dense layer 0 + 26 MoE layers,
    K = 8 drafts per step, 102400-vocab head.  Steps run back to back on the
    device (each step's bonus token is the next step's last committed token,
    copied on the device), so the timed region has no host synchronisation."""
    model = configs.CFG4
    m = model.moe
    K, Lyr, V, H = model.k_draft, model.n_moe_layers, model.vocab, m.hidden
    dev = "cuda"
    t0 = time.perf_counter()
    t = wgpu.model_tensors(model, dev)
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    dm = de.DeviceModel(desc, t["layers"], V, t["emb"], t["lm"], t["dense"], model.dense_inter,
                        de.DE_BF16, model.eps, m.gamma, K + 1, dev)
    torch.cuda.synchronize()
    fill_s = time.perf_counter() - t0
    W, S = 2, args.full_steps
    n_all = W + S
    blocks = torch.zeros(n_all, K + 1, dtype=torch.int32, device=dev)
    amax = torch.empty(n_all, K + 1, dtype=torch.int32, device=dev)
    outs = torch.empty(n_all, 2, dtype=torch.int32, device=dev)
    nus = torch.empty(n_all, Lyr, dtype=torch.int32, device=dev)
    blocks[0, 0] = gen.start_token(model)

    def run(i):
        dm.spec_step(blocks[i], amax[i], outs[i], nus[i])
        if i + 1 < n_all:
            blocks[i + 1, :1].copy_(outs[i, 1:])

    for i in range(W):
        run(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(W, n_all):
        run(i)
    e1.record()
    torch.cuda.synchronize()
    step_ms = e0.elapsed_time(e1) / S

    # The two halves of a step, timed apart: one draft position, one verify block.
    lg = torch.empty(K + 1, V, dtype=torch.float32, device=dev)
    am = torch.empty(K + 1, dtype=torch.int32, device=dev)
    reps = 6
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    def ev_rec():
        e = torch.cuda.Event(enable_timing=True)
        e.record()  # torch reads only events it has recorded once
        return e

    # The persistent launch of each draft position's MoE layers, bracketed by
    # the library's phase timer.
    pev = [[ev_rec() for _ in range(2)] for _ in range(reps)]
    ev[0].record()
    for i in range(reps):
        de.de_time_next_phase(de.DE_PHASE_DRAFT_PASS, pev[i][0], pev[i][1])
        dm.forward(blocks[W + i % S, :1], de.DE_DRAFT, lg[:1], am[:1])
    ev[1].record()
    for i in range(reps):
        dm.forward(blocks[W + i % S], de.DE_TARGET, lg, am)
    ev[2].record()
    torch.cuda.synchronize()
    draft_ms = ev[0].elapsed_time(ev[1]) / reps
    pass_us = statistics.median(1e3 * p[0].elapsed_time(p[1]) for p in pev)
    verify_ms = ev[1].elapsed_time(ev[2]) / reps

    o = outs[W:].cpu().numpy()
    nu = nus[W:].cpu().numpy().astype(np.float64)
    emitted = int((o[:, 0] + 1).sum())
    eb = m.expert_bytes()
    shared_b = m.expert_bytes(m.shared_inter)
    draft_b = m.expert_bytes(m.draft_inter)
    router_b = m.n_experts * H * 4
    dense_b = 3 * model.dense_inter * H * 2
    head_b = V * H * 2
    draft_bytes = dense_b + Lyr * (router_b + shared_b + eb + draft_b) + head_b
    verify_bytes = dense_b + Lyr * (router_b + shared_b) + float(nu.sum(axis=1).mean()) * eb + head_b
    step_bytes = K * draft_bytes + verify_bytes
    res = {
        "workload": "v2lite-step-K8: dense layer 0 (I=10944) + 26 V2-Lite MoE layers, K=8 drafts "
                    "(shared + top-1 + draft expert), one 9-position verify block, 102400-vocab "
                    "bf16 LM head, greedy accept; random weights, so acceptance is that of an "
                    "untrained drafter",
        "steps": S,
        "ms_per_step": round(step_ms, 3),
        "tokens_per_s": round(emitted / (S * step_ms * 1e-3), 2),
        "accept_mean": round(float(o[:, 0].mean()), 3),
        "tokens_per_s_if_all_accepted": round((K + 1) / (step_ms * 1e-3), 2),
        "draft_position_ms": round(draft_ms, 3),
        "draft_pass_us": round(pass_us, 1),
        "draft_layer_in_position_us": round(pass_us / Lyr, 2),
        "verify_block_ms": round(verify_ms, 3),
        "union_mean_per_layer": round(float(nu.mean()), 2),
        "union_per_layer_min_max": [int(nu.min()), int(nu.max())],
        "step_gb": round(step_bytes / 1e9, 3),
        "step_hbm_gbs": round(step_bytes / (step_ms * 1e-3) / 1e9, 1),
        "step_hbm_frac": round(step_bytes / (step_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "weights_fill_s": round(fill_s, 2),
    }
    del dm, t
    torch.cuda.empty_cache()
    return res


def offload_step(args, de, configs, gen, wgpu, torch, np):
    """The skewed-routing offload workload: the 26-layer stack with Zipf(1.1)
    router biases, K = 16, routed experts in pinned host memory behind a
    16-slot HBM cache per layer.  One cold step, then warm steps back to back
    (each continuing from the previous bonus token); the cache counts of the
    warm steps are reported."""
    model = configs.CFG5
    m = model.moe
    K, Lyr, N, V = model.k_draft, model.n_moe_layers, m.n_experts, model.vocab
    dev = "cuda"
    t = wgpu.model_tensors(model, dev)
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    eb = m.expert_bytes()
    host = torch.empty(Lyr * N * eb, dtype=torch.uint8, pin_memory=True)
    hv = host.view(Lyr, N, eb)
    for l in range(Lyr):
        hv[l].copy_(t["layers"][l]["routed"].view(torch.uint8).view(N, eb))
        t["layers"][l]["routed"] = None  # the device copy is dropped: experts live in host memory
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    # The resident tables are never read by the cached step; a placeholder slot
    # table keeps the model description valid.
    cache = de.ExpertCache(Lyr, N, model.cache_slots, eb, host, device=dev)
    layers = []
    for l in range(Lyr):
        d = dict(t["layers"][l])
        d["table"] = cache.table(l)
        layers.append(d)
    dm = de.DeviceModel(desc, layers, V, t["emb"], t["lm"], t["dense"], model.dense_inter,
                        de.DE_BF16, model.eps, m.gamma, K + 1, dev)
    S = args.offload_steps
    blocks = torch.zeros(S + 1, K + 1, dtype=torch.int32, device=dev)
    amax = torch.empty(S + 1, K + 1, dtype=torch.int32, device=dev)
    outs = torch.empty(S + 1, 2, dtype=torch.int32, device=dev)
    nus = torch.empty(S + 1, Lyr, dtype=torch.int32, device=dev)
    blocks[0, 0] = gen.start_token(model)

    def run(i):
        de.de_spec_step_cached(dm.model, cache, K, blocks[i], amax[i], outs[i], nus[i], None,
                               dm.ws)
        if i + 1 <= S:
            blocks[i + 1, :1].copy_(outs[i, 1:])

    t_cold = time.perf_counter()
    run(0)  # cold
    torch.cuda.synchronize()
    cold_ms = 1e3 * (time.perf_counter() - t_cold)
    cold = cache.stats()
    cache_t0 = time.perf_counter()
    base = cache.stats()
    for i in range(1, S + 1):
        run(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - cache_t0
    st = cache.stats()
    d = {k: st[k] - base[k] for k in st}
    o = outs[1:].cpu().numpy()
    nu = nus[1:].cpu().numpy().astype(np.float64)
    res = {
        "workload": "v2lite-offload-K16: dense layer 0 + 26 V2-Lite MoE layers with Zipf(1.1) "
                    "router biases, K=16 drafts, 17-position verify block, routed experts "
                    "(28.8 GB) in pinned host memory, 16 HBM slots per layer, draft-router "
                    "prefetch; random weights",
        "steps": S,
        "ms_per_step": round(1e3 * wall / S, 2),
        "tokens_per_s": round(float((o[:, 0] + 1).sum()) / wall, 2),
        "accept_mean": round(float(o[:, 0].mean()), 3),
        "union_mean_per_layer": round(float(nu.mean()), 2),
        "prefetch_hit_rate": round(d["prefetch_used"] / max(1, d["prefetch_issued"]), 4),
        "prefetch_waste_rate": round(d["prefetch_wasted"] / max(1, d["prefetch_issued"]), 4),
        "verify_coverage": round(d["verify_hits"] / max(1, d["verify_needed"]), 4),
        "draft_top1_hit_rate": round(d["draft_hits"] / max(1, d["draft_needed"]), 4),
        "stall_us_per_step": round(d["stall_us"] / S, 1),
        "verify_layer_us": round(d["verify_layer_us"] / max(1, d["verify_layers"]), 1),
        "draft_layer_us": round(d["draft_layer_us"] / max(1, d["draft_layers"]), 1),
        "host_to_hbm_gb_per_step": round(d["bytes_copied"] / S / 1e9, 3),
        "host_to_hbm_gbs": round(d["bytes_copied"] / wall / 1e9, 2),
        "counts": {k: d[k] for k in de.CACHE_COUNTS},
        "cold_step_ms": round(cold_ms, 2),
        "cold_bytes_gb": round(cold["bytes_copied"] / 1e9, 3),
    }
    if not args.no_verify_side:
        res["verify_side"] = verify_side(args, de, model, dm, cache, gen, torch, np)
    if not args.no_draft_side:
        res["draft_side"] = draft_side(args, de, model, dm, layers, t, cache, gen, torch, np)
    cache.close()
    del dm, t, host
    torch.cuda.empty_cache()
    return res


# Confidence threshold of the truncation rows: every token of the random-weight
# stack is far less confident (its largest draft probability is about 1e-3).
TRUNC_TAU = 0.5


def verify_side(args, de, model, dm, cache, gen, torch, np):
    """Verify-side cost control on the offload stack: fixed K against
    confidence-expansion truncation (cache-derived budget), without and with
    draft-router prefetch, each verify pass's cost relative to one-token
    autoregressive decoding through the same cache.  Every policy starts from
    an empty cache, runs one untimed step, then `offload_steps` steps back to
    back; the verify cost is the time of the verify pass's MoE layers
    (copy waits included) per step."""
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    S = args.offload_steps
    dev = "cuda"
    policies = [  # name, k_max, tau, budget, prefetch
        ("ar", 0, 0.0, 0, False),
        ("fixed_k", K, 0.0, 0, False),
        ("conf_exp", K, TRUNC_TAU, de.DE_BUDGET_CACHE, False),
        ("conf_exp_prefetch", K, TRUNC_TAU, de.DE_BUDGET_CACHE, True),
        ("fixed_k_prefetch", K, 0.0, 0, True),
    ]
    rows = {}
    for name, kmax, tau, budget, pf in policies:
        cache.reset()
        block = torch.zeros(kmax + 1, dtype=torch.int32, device=dev)
        amax = torch.empty(kmax + 1, dtype=torch.int32, device=dev)
        outv = torch.empty(2, dtype=torch.int32, device=dev)
        pred = torch.empty(max(1, kmax), L, k, dtype=torch.int32, device=dev)
        q = torch.empty(max(1, kmax), dtype=torch.float32, device=dev)
        block[0] = gen.start_token(model)
        kept, acc, qs = [], [], []

        def one():
            nd = dm.spec_step_trunc(block, amax, outv, pred, q, tau, budget, 0, cache=cache,
                                    prefetch=pf)
            o = outv.cpu().tolist()
            if kmax > 0:
                qs.extend(q[:min(kmax, nd + 1)].cpu().tolist())
            block[0] = o[1]
            return nd, o[0]

        one()
        base = cache.stats()
        t0 = time.perf_counter()
        for _ in range(S):
            nd, n = one()
            kept.append(nd)
            acc.append(n)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        st = cache.stats()
        d = {key: st[key] - base[key] for key in st}
        rows[name] = {
            "k_max": kmax, "tau": tau, "budget": "cache" if budget < 0 else budget,
            "prefetch": pf,
            "drafts_kept_mean": round(float(np.mean(kept)), 2),
            "accept_mean": round(float(np.mean(acc)), 3),
            "verify_ms_per_step": round(d["verify_layer_us"] / S / 1e3, 2),
            "draft_ms_per_step": round(d["draft_layer_us"] / S / 1e3, 2),
            "stall_ms_per_step": round(d["stall_us"] / S / 1e3, 2),
            "ms_per_step": round(1e3 * wall / S, 2),
            "tokens_per_s": round(float(sum(a + 1 for a in acc)) / wall, 2),
            "prefetch_hit_rate": round(d["prefetch_used"] / max(1, d["prefetch_issued"]), 4),
            "prefetch_waste_rate": round(d["prefetch_wasted"] / max(1, d["prefetch_issued"]), 4),
            "host_to_hbm_gb_per_step": round(d["bytes_copied"] / S / 1e9, 3),
            "q_below_tau": (round(float(np.mean(np.asarray(qs) < tau)), 3) if qs and tau > 0
                            else None),
        }
    ar = rows["ar"]["verify_ms_per_step"]
    for r in rows.values():
        r["verify_cost_vs_ar"] = round(r["verify_ms_per_step"] / ar, 2) if ar > 0 else None
    return rows


def draft_side(args, de, model, dm, layers, t, cache, gen, torch, np):
    """Draft-side cost on the offload stack: the shared + top-r self-drafters
    (r = 1, 2, 3, no draft expert) against DraftExpert's shared + top-1 +
    draft-expert path, K = 4 drafts per step, no verifier prefetch.  Reported:
    the drafter's MoE-layer time per draft token (copy waits included)
    relative to top-1, the unique layer-experts the drafter itself requests
    per block, and the verify pass's cost relative to one-token decoding."""
    K, L, k, V = 4, model.n_moe_layers, model.moe.top_k, model.vocab
    S = args.offload_steps
    dev = "cuda"
    m = model.moe
    drafters = [("top1", 1, False), ("top2", 2, False), ("top3", 3, False),
                ("draftexpert", 1, True)]
    rows = {}
    for name, r, with_draft in drafters:
        ls = layers if with_draft else [dict(l, draft=None, gamma=0.0) for l in layers]
        dmr = de.DeviceModel(dm.desc, ls, V, t["emb"], t["lm"], t["dense"], model.dense_inter,
                             de.DE_BF16, model.eps, m.gamma, K + 1, dev, draft_topr=r)
        cache.reset()
        block = torch.zeros(K + 1, dtype=torch.int32, device=dev)
        amax = torch.empty(K + 1, dtype=torch.int32, device=dev)
        outv = torch.empty(2, dtype=torch.int32, device=dev)
        pred = torch.empty(K, L, k, dtype=torch.int32, device=dev)
        q = torch.empty(K, dtype=torch.float32, device=dev)
        block[0] = gen.start_token(model)
        uniq = []

        def one():
            dmr.spec_step_trunc(block, amax, outv, pred, q, 0.0, 0, 0, cache=cache,
                                prefetch=False)
            p = pred.cpu().numpy()
            uniq.append(len({(l, int(e)) for i in range(K) for l in range(L)
                             for e in p[i, l, :r]}))
            block[0] = int(outv[1].item())

        one()
        uniq.clear()
        base = cache.stats()
        t0 = time.perf_counter()
        for _ in range(S):
            one()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        st = cache.stats()
        d = {key: st[key] - base[key] for key in st}
        rows[name] = {
            "routed_experts_per_layer": r, "draft_expert": with_draft,
            "draft_ms_per_token": round(d["draft_layer_us"] / (S * K) / 1e3, 3),
            "drafter_layer_experts_per_block": round(float(np.mean(uniq)), 1),
            "draft_hit_rate": round(d["draft_hits"] / max(1, d["draft_needed"]), 4),
            "verify_ms_per_step": round(d["verify_layer_us"] / S / 1e3, 2),
            "ms_per_step": round(1e3 * wall / S, 2),
            "host_to_hbm_gb_per_step": round(d["bytes_copied"] / S / 1e9, 3),
        }
        del dmr
    top1 = rows["top1"]["draft_ms_per_token"]
    for r in rows.values():
        r["draft_cost_vs_top1"] = round(r["draft_ms_per_token"] / top1, 3) if top1 > 0 else None
    return rows


def cfg3_sweep(args, de, configs, gen, wgpu, torch, np):
    """Union growth and verify bandwidth against block length (§2.3, Eq. 3) on
    the Moonlight-shaped layer (sigmoid router with a selection bias, top-6
    renormalised gates, bf16 experts): for T = 1 (one-token decoding) and each
    block length K + 1 in {5, 9, 17}, the verify layer over blocks of fresh
    activations on rotated weight copies (union mean, µs, GB/s over the
    union's expert bytes, fraction of the 8 TB/s peak, cost relative to T = 1),
    and the V2-Lite stack's dense layer 0 (I = 10944, bf16) at the same T,
    whose weights are read once whatever the block length."""
    cfg = configs.CFG3
    dev = "cuda"
    H, R = cfg.hidden, args.copies
    desc = de.make_desc(H, cfg.n_experts, cfg.top_k, cfg.inter, cfg.shared_inter,
                        cfg.draft_inter, cfg.score_func, cfg.norm_topk, cfg.routed_scale,
                        cfg.wdtype)
    eb = cfg.expert_bytes()
    copies = []
    for c in range(R):
        routed = wgpu.routed_experts(cfg, 0, dev, redraw=c)
        copies.append(dict(routed=routed, table=de.make_table(routed, eb, None, cfg.n_experts),
                           shared=wgpu.shared_block(cfg, 0, dev, redraw=c),
                           router=wgpu.router(cfg, 0, dev, redraw=c),
                           bias=wgpu.to_device(gen.router_bias(cfg, 0, redraw=c), dev)))
    n_blocks = 8
    steps, warm = args.steps, args.warmup

    def timed(T, call):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(steps)]
        for i in range(warm + steps):
            if i >= warm:
                evs[i - warm][0].record()
            call(i)
            if i >= warm:
                evs[i - warm][1].record()
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]

    moe_rows = []
    for T in (1,) + tuple(configs.CFG3_T):
        xs = [wgpu.to_device(gen.x_rows(cfg, T, block=100 + b), dev) for b in range(n_blocks)]
        ws = de.workspace(desc, T, dev)
        y = torch.empty(T, H, dtype=torch.float32, device=dev)
        nrm = torch.empty(T, H, dtype=torch.float32, device=dev)
        nu = torch.zeros(warm + steps, dtype=torch.int32, device=dev)

        def call(i):
            cp, x = copies[i % R], xs[i % n_blocks]
            de.de_verify_layer(desc, T, x, cp["router"], cp["bias"], cp["table"], cp["shared"], y,
                               n_union=nu[i:i + 1], ws=ws,
                               epi=de.make_epilogue(residual=x, normed=nrm))

        ms = timed(T, call)
        n = nu[warm:].cpu().numpy().astype(np.int64)
        gbs = float(n.sum() * eb / (sum(ms) * 1e-3) / 1e9)
        moe_rows.append({"T": T, "union_mean": round(float(n.mean()), 2),
                         "union_min_max": [int(n.min()), int(n.max())],
                         "verify_us": round(1e3 * statistics.median(ms), 2),
                         "union_gbs": round(gbs, 1), "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4)})
        del ws, xs
    del copies
    torch.cuda.empty_cache()
    base = moe_rows[0]["verify_us"]
    for r in moe_rows:
        r["cost_vs_T1"] = round(r["verify_us"] / base, 3)

    model = configs.CFG4
    I = model.dense_inter
    dense = [wgpu.dense_block(model, dev, redraw=c) for c in range(R)]
    wbytes = 3 * I * H * 2
    dense_rows = []
    for T in (1,) + tuple(configs.CFG3_T):
        x = wgpu.to_device(gen.x_rows(cfg, T, block=200), dev)
        y = torch.empty(T, H, dtype=torch.float32, device=dev)
        ws = torch.empty(de.de_dense_workspace_bytes(T, H, I), dtype=torch.uint8, device=dev)
        ms = timed(T, lambda i: de.de_dense_swiglu(T, H, I, de.DE_BF16, x, dense[i % R], y, ws))
        us = 1e3 * statistics.median(ms)
        gbs = wbytes / (us * 1e-6) / 1e9
        dense_rows.append({"T": T, "us": round(us, 2), "gbs": round(gbs, 1),
                           "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4)})
    del dense
    torch.cuda.empty_cache()
    for r in dense_rows:
        r["cost_vs_T1"] = round(r["us"] / dense_rows[0]["us"], 3)
    return {
        "workload": "moonlight-moe-layer: H=2048, 64 routed + 2 shared SwiGLU experts (I=1408), "
                    "sigmoid router with a N(0, 0.1) selection bias, top-6 renormalised gates, "
                    "bf16 experts; 8 blocks of fresh activations per T, 8 rotated weight copies; "
                    "dense: V2-Lite layer 0 (I=10944, bf16, 134.5 MB)",
        "moe_verify": moe_rows,
        "dense_layer": dense_rows,
    }


def _time_runs(run, budget_s, max_runs=20):
    """Median seconds of run() over repeated calls within budget_s (at least one)."""
    times = []
    t_end = time.perf_counter() + budget_s
    while True:
        t0 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t0)
        if time.perf_counter() > t_end or len(times) >= max_runs:
            break
    return statistics.median(times), len(times)


def cpu_baseline_extras(configs, gen, budget_s):
    """The oracle on the host cores for the other legs, each on a bounded
    sample: the V2-Lite draft layer (one position, Eq. 5), the Moonlight-shaped
    verify layer at T = 17 (Eq. 4), and one V2-Lite K = 8 decode step composed
    from timed oracle parts (Algorithm 1: per draft position the dense layer,
    26 draft layers and the LM head at T = 1; then the dense layer, 26 verify
    layers and the LM head at T = 9)."""
    import numpy as np

    from oracle import moe

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        cores = len(os.sched_getaffinity(0))

    def layer_parts(cfg, x, with_draft):
        w_router = gen.router_weight(cfg, 0).astype(np.float64)
        bias = gen.router_bias(cfg, 0)
        idx, _, _ = moe.route_topk(x, w_router, bias, cfg.top_k, cfg.score_func, cfg.norm_topk)
        members = sorted(set(int(e) for e in np.asarray(idx).ravel()))
        raw = {e: gen.routed_block(cfg, 0, e) for e in members}
        shared_raw = gen.shared_block(cfg, 0)
        draft_raw = gen.draft_block(cfg, 0) if with_draft else None
        return w_router, bias, members, raw, shared_raw, draft_raw

    def verify_run(cfg, x):
        w_router, bias, members, raw, shared_raw, _ = layer_parts(cfg, x, False)

        def run():
            shared = moe.split_shared(shared_raw, cfg.n_shared, cfg.shared_each, cfg.hidden)
            routed = {}

            def get(e):
                if e not in routed:
                    routed[e] = moe.split_expert(raw[e], cfg.inter, cfg.hidden)
                return routed[e]
            moe.moe_target(x, w_router, bias, get, shared, cfg.top_k, cfg.score_func,
                           cfg.norm_topk)
        return run, len(members)

    def draft_run(cfg, x):
        w_router, bias, _, raw, shared_raw, draft_raw = layer_parts(cfg, x, True)

        def run():
            shared = moe.split_shared(shared_raw, cfg.n_shared, cfg.shared_each, cfg.hidden)
            draft = moe.split_expert(draft_raw, cfg.draft_inter, cfg.hidden)
            moe.moe_draft(x, w_router, bias, lambda e: moe.split_expert(raw[e], cfg.inter, cfg.hidden),
                          shared, draft, cfg.gamma, cfg.top_k, cfg.score_func, cfg.norm_topk)
        return run

    out = {}
    cfg2 = configs.CFG2
    x1 = gen.x_rows(cfg2, 1, block=1).astype(np.float64)
    t_draft, n = _time_runs(draft_run(cfg2, x1), budget_s / 3)
    out["cfg2_draft_layer"] = {
        "value": round(t_draft * 1e3, 2), "unit": "ms per draft layer", "cores": int(cores),
        "kind": "oracle",
        "sample": f"fp64 oracle draft layer (shared + top-1 + draft expert, one position) on the "
                  f"V2-Lite shape, bf16 weights in host memory, median of {n} runs"}
    cfg3 = configs.CFG3
    x17 = gen.x_rows(cfg3, 17, block=100).astype(np.float64)
    run17, nu17 = verify_run(cfg3, x17)
    t17, n = _time_runs(run17, budget_s / 3)
    out["cfg3_verify_T17"] = {
        "value": round(nu17 * cfg3.expert_bytes() / t17 / 1e9, 4), "unit": "GB/s", "cores": int(cores),
        "kind": "oracle",
        "sample": f"fp64 oracle verify layer (T=17, |U|={nu17}) on the Moonlight shape, "
                  f"median {t17 * 1e3:.1f} ms over {n} runs"}
    # The V2-Lite step from its parts.
    model = configs.CFG4
    m = model.moe
    x9 = gen.x_rows(m, 9, block=0).astype(np.float64)
    run9, _ = verify_run(m, x9)
    t9, _ = _time_runs(run9, budget_s / 6, max_runs=3)
    t1, _ = _time_runs(draft_run(m, gen.x_rows(m, 1, block=1).astype(np.float64)), budget_s / 12,
                       max_runs=5)
    dense_raw = gen.dense_block(model)
    lm = moe.to_f64(gen.lm_head(model.cfg_id, model.vocab, m.hidden, model.lm_std))

    def dense_run(x):
        def run():
            g, u, d = moe.split_expert(dense_raw, model.dense_inter, m.hidden)
            moe.swiglu(x, g, u, d)
        return run

    dense_run(x9[:1])()  # first touch of the dense weights
    td1, _ = _time_runs(dense_run(x9[:1]), budget_s / 12, max_runs=3)
    td9, _ = _time_runs(dense_run(x9), budget_s / 12, max_runs=3)
    th1, _ = _time_runs(lambda: x9[:1] @ lm.T, budget_s / 12, max_runs=5)
    th9, _ = _time_runs(lambda: x9 @ lm.T, budget_s / 12, max_runs=5)
    L, K = model.n_moe_layers, model.k_draft
    step = K * (td1 + L * t1 + th1) + td9 + L * t9 + th9
    out["cfg4_step"] = {
        "value": round(1.0 / step, 5), "unit": "tokens/s at one token per step", "cores": int(cores),
        "kind": "oracle",
        "step_s": round(step, 2),
        "sample": f"composed from timed fp64 oracle parts: draft layer {t1 * 1e3:.1f} ms, verify "
                  f"layer (T=9) {t9 * 1e3:.1f} ms, dense layer {td1 * 1e3:.1f} / {td9 * 1e3:.1f} ms "
                  f"and LM head {th1 * 1e3:.1f} / {th9 * 1e3:.1f} ms at T=1 / 9; step = "
                  f"{K} x (dense + {L} draft layers + head) + dense + {L} verify layers + head"}
    return out


def cpu_baseline(cfg, x, budget_s):
    """The oracle's verify layer on the host cores, weights already in memory."""
    import numpy as np

    from oracle import moe
    from workloads import gen

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        cores = len(os.sched_getaffinity(0))
    w_router = gen.router_weight(cfg, 0).astype(np.float64)
    idx, gate, _ = moe.route_topk(x, w_router, None, cfg.top_k, cfg.score_func, cfg.norm_topk)
    members = sorted(set(int(e) for e in idx.ravel()))
    raw = {e: gen.routed_block(cfg, 0, e) for e in members}
    shared_raw = gen.shared_block(cfg, 0)

    def run():
        shared = moe.split_shared(shared_raw, cfg.n_shared, cfg.shared_each, cfg.hidden)
        routed = {}

        def get(e):
            if e not in routed:
                routed[e] = moe.split_expert(raw[e], cfg.inter, cfg.hidden)
            return routed[e]
        moe.moe_target(x, w_router, None, get, shared, cfg.top_k, cfg.score_func, cfg.norm_topk)

    times = []
    t_end = time.perf_counter() + budget_s
    while True:
        t0 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t0)
        if time.perf_counter() > t_end or len(times) >= 50:
            break
    t = statistics.median(times)
    # The same layer on one thread (a quarter of the budget, at least one run).
    single = []
    try:
        from threadpoolctl import threadpool_limits
        t_end = time.perf_counter() + budget_s / 4
        with threadpool_limits(limits=1):
            while True:
                t0 = time.perf_counter()
                run()
                single.append(time.perf_counter() - t0)
                if time.perf_counter() > t_end or len(single) >= 10:
                    break
    except Exception:  # noqa: BLE001
        single = []
    host = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            host = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = ",".join(sorted({i.get("internal_api", "?") for i in threadpool_info()})) or "none"
    except Exception:  # noqa: BLE001
        blas = "unknown"
    one = (f"; one thread: median {statistics.median(single) * 1e3:.1f} ms over {len(single)} runs"
           if single else "")
    return {
        "value": round(len(members) * cfg.expert_bytes() / t / 1e9, 4),
        "unit": "GB/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": f"fp64 oracle verify layer (T={x.shape[0]}, |U|={len(members)}) on the V2-Lite "
                  f"shape, bf16 weights in host memory, {len(times)} runs, median {t * 1e3:.1f} ms"
                  f"{one}; {host}, NumPy {np.__version__}, BLAS {blas}",
    }


if __name__ == "__main__":
    main()
