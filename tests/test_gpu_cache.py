"""The offloaded step on the GPU: routed experts in pinned host memory behind
the expert cache.

A cached step must give the same bits as the resident step (prefetching and
chunked verification change no semantics), and its cache bookkeeping must
equal the oracle simulation replayed on the oracle's own routing decisions.
Small case: 2 V2-Lite-shaped layers with Zipf-biased routers, 4 slots per
layer (so the verify union is requested in several chunks), two consecutive
steps (cold, then warm cache).  Full case: the 26-layer skewed-routing stack
with K = 16 and 16 slots per layer, cached against resident.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from oracle.cache_sim import CacheSim
from support import OracleModel
from workloads import configs, gen
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu

SMALL = configs.scaled_model(configs.CFG5, n_moe_layers=2, vocab=8192, dense_inter=1408,
                             k_draft=4, name="v2lite-offload-small")
SMALL = replace(SMALL, cache_slots=4)


def build(model):
    m = model.moe
    t = wgpu.model_tensors(model)
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    dm = de.DeviceModel(desc, t["layers"], model.vocab, t["emb"], t["lm"], t["dense"],
                        model.dense_inter, de.DE_BF16, model.eps, m.gamma, model.k_draft + 1)
    eb = m.expert_bytes()
    L, N = model.n_moe_layers, m.n_experts
    host = torch.empty(L * N * eb, dtype=torch.uint8, pin_memory=True)
    hv = host.view(L, N, eb)
    for l in range(L):
        hv[l].copy_(t["layers"][l]["routed"].view(torch.uint8).view(N, eb))
    torch.cuda.synchronize()
    cache = de.ExpertCache(L, N, model.cache_slots, eb, host)
    return dm, cache


def run_step(dm, model, c, cached=None):
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    block = dm.new_block(K, c)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
    if cached is None:
        dm.spec_step(block, amax, out, nu, pred)
    else:
        de.de_spec_step_cached(dm.model, cached, K, block, amax, out, nu, pred, dm.ws)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (block, amax, out, nu, pred)]


def test_cached_step_equals_resident_and_bookkeeping_equals_oracle():
    model = SMALL
    K, L = model.k_draft, model.n_moe_layers
    om = OracleModel(model)
    dm, cache = build(model)
    sim = CacheSim(L, model.moe.n_experts, model.cache_slots, model.moe.expert_bytes())
    for r0 in (0, 5):
        c, drafts, n, bonus, t, traces = om.gapped_step(K, redraw0=r0)
        print(f"start {c}: drafts {drafts} n {n} bonus {bonus}", flush=True)
        res = run_step(dm, model, c)
        got = run_step(dm, model, c, cached=cache)
        for a, b, name in zip(got, res, ("block", "argmax", "out", "n_union", "pred")):
            assert np.array_equal(a, b), name
        assert got[0][1:].tolist() == drafts and got[2].tolist() == [n, bonus]
        draft_topk = [[np.asarray(traces[i].idx[l])[0] for l in range(L)] for i in range(K)]
        verify_topk = [np.asarray(traces[K].idx[l]) for l in range(L)]
        sim.step(draft_topk, verify_topk)
        st = cache.stats()
        print({k: st[k] for k in st}, flush=True)
        for name in de.CACHE_COUNTS:
            assert st[name] == sim.counts[name], name
        assert st["draft_layers"] == K * L * (1 if r0 == 0 else 2)
        assert st["verify_layers"] == L * (1 if r0 == 0 else 2)
    cache.close()


def test_q4_cached_step_equals_resident():
    """Q4_0 experts through the cache: the cached step (slot copies of 4.87 MB
    blocks, chunked verification when the union exceeds the slots) equals the
    resident step bit for bit."""
    model = replace(SMALL, moe=configs.CFG5_Q4.moe, name="v2lite-offload-q4-small")
    K = model.k_draft
    dm, cache = build(model)
    for r in range(2):
        c = gen.start_token(model, redraw=r)
        res = run_step(dm, model, c)
        got = run_step(dm, model, c, cached=cache)
        for a, b, name in zip(got, res, ("block", "argmax", "out", "n_union", "pred")):
            assert np.array_equal(a, b), name
    st = cache.stats()
    print(f"q4 cached: stats {st}", flush=True)
    assert st["bytes_copied"] == (st["prefetch_issued"] + st["demand_loads"]) * model.moe.expert_bytes()
    assert st["draft_needed"] == 2 * K * model.n_moe_layers
    cache.close()


def test_full_offload_stack_cached_equals_resident():
    model = configs.CFG5
    K, L = model.k_draft, model.n_moe_layers
    dm, cache = build(model)
    for r in range(2):
        c = gen.start_token(model, redraw=r)
        res = run_step(dm, model, c)
        got = run_step(dm, model, c, cached=cache)
        for a, b, name in zip(got, res, ("block", "argmax", "out", "n_union", "pred")):
            assert np.array_equal(a, b), name
        st = cache.stats()
        nu = got[3]
        print(f"start {c}: n {got[2][0]} union mean {nu.mean():.1f} stats {st}", flush=True)
    eb = model.moe.expert_bytes()
    assert st["draft_needed"] == 2 * K * L
    assert st["bytes_copied"] == (st["prefetch_issued"] + st["demand_loads"]) * eb
    assert st["prefetch_used"] + st["prefetch_wasted"] <= st["prefetch_issued"]
    assert st["verify_hits"] <= st["verify_needed"]
    cache.close()
    del dm
    torch.cuda.empty_cache()
