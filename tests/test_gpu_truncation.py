"""Confidence-expansion truncation on the GPU against the oracle (Section 3.4,
Eqs. 12-14; Algorithm 1).

The confidence kernel is compared with the fp64 oracle on fp32 logits
(relative 1e-5; aligned and unaligned rows, -inf and NaN logits); the
expansion kernel bit-exact against the oracle's set arithmetic over token
sequences (fixed and cache-derived budgets, several words per layer, more
layers than threads, out-of-range ids); the truncated step of a small stack
against the oracle's truncated step, with thresholds placed away from every
token's confidence so that fp32 and fp64 take the same decisions; and the
cached truncated step against the resident one and the cache simulation.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from oracle import truncation
from oracle.cache_sim import CacheSim
from support import OracleModel
from workloads import configs, gen
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu

TINY = configs.scaled_model(configs.CFG4, n_moe_layers=3, vocab=1000, dense_inter=256, k_draft=4,
                            moe=replace(configs.CFG1, cfg_id=41, gamma=6.0), name="tiny-stack")
OFF = replace(configs.scaled_model(configs.CFG5, n_moe_layers=2, vocab=8192, dense_inter=1408,
                                   k_draft=4, name="v2lite-offload-small"), cache_slots=4)


@pytest.mark.parametrize("T,V", [(3, 102400), (5, 1000), (4, 1003), (1, 1)])
def test_confidence_matches_oracle(T, V):
    rng = np.random.default_rng(T * 7 + V)
    lg = rng.normal(0, 4, (T, V)).astype(np.float32)
    if V > 8:
        lg[0, :V // 2] = -np.inf
        lg[-1, 3] = np.nan
    dev = torch.from_numpy(lg).cuda()
    q = torch.empty(T, dtype=torch.float32, device="cuda")
    de.de_confidence(T, V, dev, q)
    torch.cuda.synchronize()
    want = truncation.confidence(np.nan_to_num(lg.astype(np.float64), nan=-np.inf))
    np.testing.assert_allclose(q.cpu().numpy(), want, rtol=1e-5)


def test_confidence_of_an_empty_row_is_nan():
    lg = torch.full((1, 300), -float("inf"), device="cuda")
    q = torch.empty(1, device="cuda")
    de.de_confidence(1, 300, lg, q)
    torch.cuda.synchronize()
    assert torch.isnan(q).all()


def _oracle_pairs(pred, N):
    return {(l, int(e)) for l in range(pred.shape[0]) for e in pred[l] if 0 <= e < N}


@pytest.mark.parametrize("L,N,k,budget,slots", [
    (26, 64, 6, 20, 0), (26, 64, 6, de.DE_BUDGET_CACHE, 16), (5, 256, 16, 7, 0),
    (300, 100, 3, de.DE_BUDGET_CACHE, 5), (1, 1, 1, 0, 0)])
def test_expansion_matches_oracle(L, N, k, budget, slots):
    rng = np.random.default_rng(L * 1000 + N)
    words = (N + 63) // 64
    uhat = torch.full((L, words), -1, dtype=torch.int64, device="cuda")  # stale: `first` ignores it
    out = torch.empty(5, dtype=torch.int32, device="cuda")
    qd = torch.empty(1, dtype=torch.float32, device="cuda")
    tau = 0.5
    want_set: set = set()
    # Skewed draws so that later tokens add few pairs and some are kept.
    pool = rng.choice(N, size=min(N, k + 2), replace=False)
    for i in range(7):
        src = pool if i % 2 else np.arange(N)
        pred = np.stack([rng.choice(src, k, replace=False) for _ in range(L)]).astype(np.int32)
        q = float(rng.choice([0.2, 0.9]))
        qd.fill_(q)
        de.de_expansion(L, k, N, torch.from_numpy(pred).cuda(), uhat, i == 0, qd, tau, budget,
                        slots, out)
        torch.cuda.synchronize()
        stop, delta, b, want_set = truncation.decide(q, want_set, _oracle_pairs(pred, N), tau,
                                                     budget, L, slots)
        assert out.cpu().tolist() == [delta, int(stop), b, len(want_set), 0], i
        bits = uhat.cpu().numpy().view(np.uint64)
        got_set = {(l, w * 64 + j) for l in range(L) for w in range(words) for j in range(64)
                   if (int(bits[l, w]) >> j) & 1}
        assert got_set == want_set, i


def test_expansion_counts_out_of_range_ids():
    pred = torch.tensor([[0, 70], [-1, 3]], dtype=torch.int32, device="cuda")
    uhat = torch.zeros(2, 1, dtype=torch.int64, device="cuda")
    out = torch.empty(5, dtype=torch.int32, device="cuda")
    q = torch.ones(1, device="cuda")
    de.de_expansion(2, 2, 64, pred, uhat, True, q, 0.5, 0, 0, out)
    torch.cuda.synchronize()
    assert out.cpu().tolist() == [2, 0, 0, 2, 2]


def test_expansion_rejects_bad_arguments():
    t = torch.zeros(8, dtype=torch.int64, device="cuda")
    q = torch.ones(1, device="cuda")
    for args in [(0, 1, 8), (2, 1, 257), (2, 9, 8)]:
        with pytest.raises(de.DEError):
            de.de_expansion(*args, t, t, True, q, 0.5, 0, 0, t)
    with pytest.raises(de.DEError):
        de.de_expansion(2, 1, 8, t, t, True, q, float("nan"), 0, 0, t)
    with pytest.raises(de.DEError):
        de.de_expansion(2, 1, 8, t, t, True, q, 0.5, -2, 0, t)


_MODELS: dict = {}


def _device_model(model):
    if model.name not in _MODELS:
        _MODELS.clear()
        m = model.moe
        t = wgpu.model_tensors(model)
        desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter,
                            m.draft_inter, m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
        _MODELS[model.name] = (de.DeviceModel(desc, t["layers"], model.vocab, t["emb"], t["lm"],
                                              t["dense"], model.dense_inter, de.DE_BF16,
                                              model.eps, m.gamma, model.k_draft + 1), t)
    return _MODELS[model.name]


def _gapped_start(om, k_max, redraw0):
    """A start token whose never-stopping run has gapped decisions everywhere;
    returns (token, q of the k_max evaluated tokens)."""
    for r in range(redraw0, redraw0 + 8):
        c = gen.start_token(om.cfg, redraw=r)
        traces: list = []
        res = truncation.truncated_step(om.weights, c, k_max, 0.0, 0, traces=traces)
        if all(om.trace_gaps_ok(tr) for tr in traces):
            return c, res["q"]
    raise RuntimeError("no gapped start token")


def _mids(q):
    """Thresholds between consecutive confidences (lowest first), each at a
    relative distance above 1e-3 from every q."""
    qs = sorted(q)
    return [0.5 * (a + b) for a, b in zip(qs, qs[1:]) if b - a > 2e-3 * b]


def _policies(q, L, k, n_mid):
    """(tau, budget) pairs: never stop, stop at the first token, the strict
    boundary of a fixed budget, and stops set by the q order."""
    pol = [(0.0, 0), (2.0, 0), (2.0, L * k)]
    for m in _mids(q)[:n_mid]:
        pol += [(m, 0), (m, L * k // 2), (m, truncation.BUDGET_CACHE)]
    return pol


def _run_trunc(dm, model, c, tau, budget, slots, cache=None, prefetch=True):
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    block = dm.new_block(K, c)
    amax = torch.full((K + 1,), -7, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.full((K, L, k), -7, dtype=torch.int32, device="cuda")
    q = torch.full((K,), -1.0, dtype=torch.float32, device="cuda")
    tr = torch.full((K, 4), -7, dtype=torch.int32, device="cuda")
    nd = dm.spec_step_trunc(block, amax, out, pred, q, tau, budget, slots, cache=cache,
                            n_union=nu, trace=tr, prefetch=prefetch)
    torch.cuda.synchronize()
    return nd, [x.cpu().numpy() for x in (block, amax, out, nu, pred, q, tr)]


@pytest.mark.parametrize("model,redraw0,n_mid", [(TINY, 0, 2), (TINY, 4, 2), (OFF, 0, 1)],
                         ids=["tiny-a", "tiny-b", "v2lite-2layer"])
def test_truncated_step_matches_oracle(model, redraw0, n_mid):
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    om = OracleModel(model)
    dm, _ = _device_model(model)
    c, qall = _gapped_start(om, K, redraw0)
    slots = 4
    stops_seen = set()
    for tau, budget in _policies(qall, L, k, n_mid):
        traces: list = []
        r = truncation.truncated_step(om.weights, c, K, tau, budget, slots=slots, traces=traces)
        nd, (block, amax, out, nu, pred, q, tr) = _run_trunc(dm, model, c, tau, budget, slots)
        ne = len(r["q"])
        print(f"start {c} tau {tau:.4g} B {budget}: kept {nd} evaluated {ne} n {r['n']}",
              flush=True)
        stops_seen.add(nd)
        assert nd == len(r["drafts"])
        assert block[1:nd + 1].tolist() == r["drafts"]
        assert amax[:nd + 1].tolist() == [int(v) for v in r["target_argmax"]]
        assert out.tolist() == [r["n"], r["bonus"]]
        np.testing.assert_allclose(q[:ne], r["q"], rtol=1e-5)
        assert tr[:ne].tolist() == [[d, int(s), b, z] for d, s, b, z in
                                    zip(r["delta"], r["stop"], r["budget"], r["set_size"])]
        assert (tr[ne:] == -7).all() and (q[ne:] == -1.0).all()
        want_pred = np.stack([np.stack([np.asarray(i)[0] for i in t.idx]) for t in traces[:ne]])
        np.testing.assert_array_equal(pred[:ne], want_pred)
        assert nu.tolist() == [len(set(np.asarray(i).ravel().tolist())) for i in traces[-1].idx]
    assert 0 in stops_seen and K in stops_seen


def test_cached_truncated_step_equals_resident_and_simulation():
    model = OFF
    K, L, k, N = model.k_draft, model.n_moe_layers, model.moe.top_k, model.moe.n_experts
    om = OracleModel(model)
    dm, t = _device_model(model)
    eb = model.moe.expert_bytes()
    host = torch.empty(L * N * eb, dtype=torch.uint8, pin_memory=True)
    hv = host.view(L, N, eb)
    for l in range(L):
        hv[l].copy_(t["layers"][l]["routed"].view(torch.uint8).view(N, eb))
    torch.cuda.synchronize()
    cache = de.ExpertCache(L, N, model.cache_slots, eb, host)
    sim = CacheSim(L, N, model.cache_slots, eb)
    c, qall = _gapped_start(om, K, 0)
    # Below every confidence but the lowest: the least confident token stops
    # when it adds pairs, the others are kept.
    mids = _mids(qall)
    tau = mids[0] if mids else 2.0
    for budget, prefetch in ((0, True), (truncation.BUDGET_CACHE, True), (0, False)):
        traces: list = []
        r = truncation.truncated_step(om.weights, c, K, tau, budget, slots=model.cache_slots,
                                      traces=traces)
        nd_res, res = _run_trunc(dm, model, c, tau, budget, model.cache_slots)
        issued = cache.stats()["prefetch_issued"]
        nd, got = _run_trunc(dm, model, c, tau, budget, 0, cache=cache, prefetch=prefetch)
        assert nd == nd_res == len(r["drafts"])
        for a, b, name in zip(got, res, ("block", "argmax", "out", "n_union", "pred", "q",
                                         "trace")):
            assert np.array_equal(a, b), name
        ne = len(r["q"])
        draft_topk = [[np.asarray(traces[i].idx[l])[0] for l in range(L)] for i in range(ne)]
        verify_topk = [np.asarray(traces[-1].idx[l]) for l in range(L)]
        # Without prefetching no token starts a copy before verification.
        sim.step_truncated(draft_topk, nd if prefetch else 0, verify_topk)
        st = cache.stats()
        print(f"B {budget} prefetch {prefetch}: kept {nd} of {ne} evaluated; {st}", flush=True)
        if not prefetch:
            assert st["prefetch_issued"] == issued
        for name in de.CACHE_COUNTS:
            assert st[name] == sim.counts[name], name
    cache.close()
