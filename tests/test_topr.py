"""Pins of the shared + top-r drafter in the oracle (the training-free
self-drafting baseline of Section 1 and Table 3: Eq. 5 with r routed experts
and no draft expert).

r = k with no draft expert is the target layer (Eq. 4), the difference from
the target is the Eq. 6 residual over the experts ranked r+1..k, a stack whose
drafter equals its target accepts every draft, and the cache simulation's
drafter requests r experts per layer.
"""
from dataclasses import replace

import numpy as np
import pytest

from oracle import cache_sim, decode, moe
from support import OracleLayer, OracleModel, gapped_x
from workloads import configs, gen


def _layer():
    return OracleLayer(configs.CFG1, 0)


def test_top_k_drafter_without_draft_expert_is_the_target():
    ol = _layer()
    c = ol.cfg
    x, _ = gapped_x(ol, 4)
    yt, it, gt = ol.target(x)
    yd, idx, gate = moe.moe_draft(x, ol.w_router, ol.bias, ol.routed, ol.shared, None, 0.0,
                                  c.top_k, c.score_func, c.norm_topk, c.routed_scale, r=c.top_k)
    np.testing.assert_array_equal(idx, it)
    np.testing.assert_allclose(yd, yt, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("r", [1, 2])
def test_top_r_residual_is_the_lower_ranked_experts(r):
    ol = _layer()
    c = ol.cfg
    x, _ = gapped_x(ol, 3, block=1)
    yt, _, _ = ol.target(x)
    yd, idx, gate = moe.moe_draft(x, ol.w_router, ol.bias, ol.routed, ol.shared, None, 0.0,
                                  c.top_k, c.score_func, c.norm_topk, c.routed_scale, r=r)
    want = np.zeros_like(yt)
    for t in range(x.shape[0]):
        for j in range(r, c.top_k):
            g, u, d = ol.routed(int(idx[t, j]))
            xt = x[t].astype(np.float64)
            h = (xt @ g.T) / (1 + np.exp(-(xt @ g.T))) * (xt @ u.T)
            want[t] += gate[t, j] * (h @ d.T)
    np.testing.assert_allclose(yt - yd, want, rtol=1e-9, atol=1e-13)


def test_r_out_of_range_is_rejected():
    ol = _layer()
    c = ol.cfg
    x, _ = gapped_x(ol, 1)
    for r in (0, c.top_k + 1):
        with pytest.raises(ValueError):
            moe.moe_draft(x, ol.w_router, ol.bias, ol.routed, ol.shared, None, 0.0, c.top_k,
                          c.score_func, c.norm_topk, c.routed_scale, r=r)


def test_stack_whose_drafter_is_its_target_accepts_every_draft():
    model = configs.scaled_model(configs.CFG4, n_moe_layers=2, vocab=1000, dense_inter=256,
                                 k_draft=3, moe=replace(configs.CFG1, cfg_id=43),
                                 name="tiny-topk-drafter")
    om = OracleModel(model)
    w = om.weights
    layers = [replace(lw, draft=None, gamma=0.0) for lw in w.layers]
    w = replace(w, layers=layers, draft_topr=model.moe.top_k)
    drafts, n, bonus, t = decode.spec_step(w, gen.start_token(model), 3)
    assert n == 3
    assert drafts + [bonus] == decode.greedy_ar(w, gen.start_token(model), 4)


def test_cache_sim_drafter_requests_r_experts():
    rng = np.random.default_rng(9)
    draft = [[rng.choice(10, 4, replace=False).tolist() for _ in range(3)] for _ in range(2)]
    verify = [[rng.choice(10, 4, replace=False).tolist() for _ in range(3)] for _ in range(3)]
    for r in (1, 2, 4):
        sim = cache_sim.CacheSim(3, 10, 6)
        sim.step(draft, verify, r=r)
        assert sim.counts["draft_needed"] == 2 * 3 * r
    a, b = cache_sim.CacheSim(3, 10, 6), cache_sim.CacheSim(3, 10, 6)
    a.step(draft, verify, r=2)
    b.step_truncated(draft, 2, verify, r=2)
    assert a.counts == b.counts and a.slot == b.slot
