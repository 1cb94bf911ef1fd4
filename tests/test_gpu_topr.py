"""The shared + top-r self-drafter on the GPU against the oracle (Eq. 5 with
r routed experts; the baseline of Section 1 and Table 3).

Layer: outputs within 1e-5 (fp32 weights) / 1e-4 (bf16) of the fp64 oracle
for r in {2, 3, k}, with and without the draft expert, predictions
bit-exact; r = 1 equals the fixed-footprint layer bit for bit; r outside
[1, k] is rejected.  Stack: a top-2 drafter's step against the oracle step,
a top-k drafter without draft experts accepts every draft, and the cached
top-2 step equals the resident one with counts equal to the simulation of an
r = 2 drafter.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from gpu_support import f32, layer_pair, require_gpu
from oracle import moe
from oracle.cache_sim import CacheSim
from support import OracleModel, gapped_x, rel_err
from workloads import configs, gen
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu

CASES = [("cfg1", configs.CFG1, 1, 2, True), ("cfg1", configs.CFG1, 3, 2, False),
         ("cfg2", configs.CFG2, 1, 2, False), ("cfg2", configs.CFG2, 1, 3, False),
         ("cfg2", configs.CFG2, 3, 6, True), ("cfg3", configs.CFG3, 5, 3, True)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,cfg,T,r,with_draft", CASES,
                         ids=[f"{c[0]}-T{c[2]}-r{c[3]}-{'draft' if c[4] else 'nodraft'}"
                              for c in CASES])
def test_draft_layer_topr_matches_oracle(name, cfg, T, r, with_draft):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=2)
    gamma = cfg.gamma if with_draft else 0.0
    y_o, idx_o, _ = moe.moe_draft(x, orc.w_router, orc.bias, orc.routed, orc.shared,
                                  orc.draft if with_draft else None, gamma, cfg.top_k,
                                  cfg.score_func, cfg.norm_topk, cfg.routed_scale, r=r)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    pidx = torch.empty(T, cfg.top_k, dtype=torch.int32, device="cuda")
    de.de_draft_layer_topr(dev.desc, T, f32(x), dev.router, dev.bias, dev.table, dev.shared,
                           dev.draft if with_draft else None, gamma, r, y, pidx, None, dev.ws(T))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(pidx.cpu().numpy(), idx_o)
    tol = 1e-5 if cfg.wdtype == configs.F32 else 1e-4
    assert rel_err(y.cpu().numpy(), y_o) <= tol


def test_top1_equals_fixed_footprint_layer_and_bad_r_is_rejected():
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, 1, block=3)
    ws = dev.ws(1)
    y0 = torch.empty(1, cfg.hidden, dtype=torch.float32, device="cuda")
    y1 = torch.empty_like(y0)
    de.de_draft_layer(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table, dev.shared,
                      dev.draft, 1.0, y0, None, None, ws)
    de.de_draft_layer_topr(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table, dev.shared,
                           dev.draft, 1.0, 1, y1, None, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
    for r in (0, cfg.top_k + 1):
        with pytest.raises(de.DEError):
            de.de_draft_layer_topr(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table,
                                   dev.shared, None, 0.0, r, y1, None, None, ws)


TINY = configs.scaled_model(configs.CFG4, n_moe_layers=3, vocab=1000, dense_inter=256, k_draft=4,
                            moe=replace(configs.CFG1, cfg_id=41, gamma=6.0), name="tiny-stack")
OFF = replace(configs.scaled_model(configs.CFG5, n_moe_layers=2, vocab=8192, dense_inter=1408,
                                   k_draft=4, name="v2lite-offload-small"), cache_slots=4)


def _device_model(model, r, no_draft=False):
    m = model.moe
    t = wgpu.model_tensors(model)
    layers = t["layers"]
    if no_draft:
        layers = [dict(l, draft=None, gamma=0.0) for l in layers]
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    return de.DeviceModel(desc, layers, model.vocab, t["emb"], t["lm"], t["dense"],
                          model.dense_inter, de.DE_BF16, model.eps, m.gamma, model.k_draft + 1,
                          draft_topr=r), t


def _oracle(model, r, no_draft=False):
    om = OracleModel(model)
    w = om.weights
    if no_draft:
        w = replace(w, layers=[replace(lw, draft=None, gamma=0.0) for lw in w.layers])
    return om, replace(w, draft_topr=r)


def _step(dm, model, c, cache=None):
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    block = dm.new_block(K, c)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
    if cache is None:
        dm.spec_step(block, amax, out, nu, pred)
    else:
        de.de_spec_step_cached(dm.model, cache, K, block, amax, out, nu, pred, dm.ws)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (block, amax, out, nu, pred)]


def _gapped(om, w, K, redraw0=0):
    from oracle import decode
    for rr in range(redraw0, redraw0 + 8):
        c = gen.start_token(om.cfg, redraw=rr)
        traces: list = []
        res = decode.spec_step(w, c, K, traces)
        if all(om.trace_gaps_ok(tr) for tr in traces):
            return c, res, traces
    raise RuntimeError("no gapped start token")


def test_top2_drafter_step_matches_oracle():
    model = TINY
    om, w = _oracle(model, 2)
    dm, _ = _device_model(model, 2)
    c, (drafts, n, bonus, t), traces = _gapped(om, w, model.k_draft)
    block, amax, out, nu, pred = _step(dm, model, c)
    print(f"start {c}: drafts {drafts} n {n} bonus {bonus}", flush=True)
    assert block[1:].tolist() == drafts
    assert amax.tolist() == [int(v) for v in t]
    assert out.tolist() == [n, bonus]
    want_pred = np.stack([np.stack([np.asarray(i)[0] for i in tr.idx])
                          for tr in traces[:model.k_draft]])
    np.testing.assert_array_equal(pred, want_pred)


def test_top_k_drafter_without_draft_experts_accepts_every_draft():
    model = TINY
    dm, _ = _device_model(model, model.moe.top_k, no_draft=True)
    for rr in range(3):
        block, amax, out, nu, pred = _step(dm, model, gen.start_token(model, redraw=rr))
        assert out[0] == model.k_draft


def test_cached_top2_step_equals_resident_and_simulation():
    model = OFF
    K, L, N, r = model.k_draft, model.n_moe_layers, model.moe.n_experts, 2
    om, w = _oracle(model, r)
    dm, t = _device_model(model, r)
    eb = model.moe.expert_bytes()
    host = torch.empty(L * N * eb, dtype=torch.uint8, pin_memory=True)
    hv = host.view(L, N, eb)
    for l in range(L):
        hv[l].copy_(t["layers"][l]["routed"].view(torch.uint8).view(N, eb))
    torch.cuda.synchronize()
    cache = de.ExpertCache(L, N, model.cache_slots, eb, host)
    sim = CacheSim(L, N, model.cache_slots, eb)
    c, (drafts, n, bonus, _), traces = _gapped(om, w, K)
    res = _step(dm, model, c)
    got = _step(dm, model, c, cache=cache)
    for a, b, name in zip(got, res, ("block", "argmax", "out", "n_union", "pred")):
        assert np.array_equal(a, b), name
    assert got[0][1:].tolist() == drafts and got[2].tolist() == [n, bonus]
    draft_topk = [[np.asarray(traces[i].idx[l])[0] for l in range(L)] for i in range(K)]
    verify_topk = [np.asarray(traces[K].idx[l]) for l in range(L)]
    sim.step(draft_topk, verify_topk, r=r)
    st = cache.stats()
    for name in de.CACHE_COUNTS:
        assert st[name] == sim.counts[name], name
    assert st["draft_needed"] == K * L * r
    cache.close()
