"""Pins of the truncation oracle (Section 3.4, Eqs. 12-14; Algorithm 1).

Each check ties ``oracle.truncation`` to something other than itself: a
library softmax, closed forms of the first token's expansion and of the
cache-derived budget, brute-force set unions from the traces, the special
cases that reduce to the fixed-K step or to one greedy target step, the strict
inequality of Eq. 14 at its boundary, and exactness against greedy decoding.
"""
from dataclasses import replace

import numpy as np
import pytest
import scipy.special

from oracle import cache_sim, decode, truncation
from support import OracleModel
from workloads import configs, gen

TINY = configs.scaled_model(configs.CFG4, n_moe_layers=3, vocab=1000, dense_inter=256, k_draft=4,
                            moe=replace(configs.CFG1, cfg_id=41, gamma=6.0), name="tiny-stack")
L, K = TINY.n_moe_layers, TINY.moe.top_k
_OM = {}


def om():
    if "m" not in _OM:
        _OM["m"] = OracleModel(TINY)
    return _OM["m"]


def test_confidence_library_and_closed_forms():
    rng = np.random.default_rng(5)
    lg = rng.normal(0, 3, (6, 777))
    np.testing.assert_allclose(truncation.confidence(lg),
                               scipy.special.softmax(lg, axis=1).max(axis=1), rtol=1e-13)
    assert truncation.confidence(np.full(1000, 2.5))[0] == pytest.approx(1e-3, rel=1e-14)
    row = np.zeros(500)
    row[123] = 7.0
    assert truncation.confidence(row)[0] == pytest.approx(1 / (1 + 499 * np.exp(-7.0)), rel=1e-13)
    # Shift invariance and range.
    q = truncation.confidence(lg)
    np.testing.assert_allclose(truncation.confidence(lg + 100.0), q, rtol=1e-13)
    assert np.all((q > 0) & (q <= 1))


def test_cache_budget_closed_form():
    assert truncation.cache_budget(set(), 26, 16) == 26 * 16
    s = {(0, 1), (0, 2), (3, 9)}
    assert truncation.cache_budget(s, 4, 2) == 0 + 2 + 2 + 1
    assert truncation.cache_budget({(1, e) for e in range(40)}, 2, 16) == 16


def test_first_token_expansion_is_layers_times_k():
    c = gen.start_token(TINY)
    r = truncation.truncated_step(om().weights, c, 1, tau=0.0, budget=0)
    assert r["delta"] == [L * K]
    assert r["set_size"] == [L * K]


def test_never_stopping_equals_fixed_k_step():
    c = gen.start_token(TINY)
    traces = []
    r = truncation.truncated_step(om().weights, c, 4, tau=0.0, budget=0, traces=traces)
    drafts, n, bonus, t = decode.spec_step(om().weights, c, 4)
    assert r["drafts"] == drafts and r["n"] == n and r["bonus"] == bonus
    assert r["stop"] == [False] * 4
    # Brute force: the set after each token is the union of the pairs so far.
    seen = set()
    for i, tr in enumerate(traces[:4]):
        before = len(seen)
        for l, idx in enumerate(tr.idx):
            for e in np.asarray(idx).ravel():
                seen.add((l, int(e)))
        assert r["delta"][i] == len(seen) - before
        assert r["set_size"][i] == len(seen)
    assert sum(r["delta"]) == len(seen)


def test_stop_at_first_token_is_one_greedy_step():
    c = gen.start_token(TINY)
    r = truncation.truncated_step(om().weights, c, 4, tau=2.0, budget=0)
    assert r["drafts"] == [] and r["stop"] == [True] and r["n"] == 0
    assert r["bonus"] == decode.greedy_ar(om().weights, c, 1)[0]
    # The stopped token's pairs never enter the set.
    assert r["set_size"] == [0]


def test_eq14_boundary_is_strict():
    c = gen.start_token(TINY)
    # Every token is uncertain (q < 2); Delta_1 = L k exactly.
    below = truncation.truncated_step(om().weights, c, 3, tau=2.0, budget=L * K - 1)
    assert below["stop"] == [True] and below["drafts"] == []
    at = truncation.truncated_step(om().weights, c, 3, tau=2.0, budget=L * K)
    # No later token can add more than L k pairs either.
    assert at["stop"] == [False] * 3 and len(at["drafts"]) == 3
    # A confident token is kept whatever its expansion: tau below every q.
    conf = truncation.truncated_step(om().weights, c, 3, tau=min(at["q"]) * 0.5, budget=0)
    assert conf["stop"] == [False] * 3


def test_cache_budget_mode():
    c = gen.start_token(TINY)
    r = truncation.truncated_step(om().weights, c, 3, tau=2.0, budget=truncation.BUDGET_CACHE,
                                  slots=0)
    assert r["budget"] == [0] and r["stop"] == [True]
    r = truncation.truncated_step(om().weights, c, 3, tau=2.0, budget=truncation.BUDGET_CACHE,
                                  slots=TINY.moe.n_experts)
    assert r["budget"][0] == L * TINY.moe.n_experts
    assert r["stop"][0] is False
    # Later budgets follow the closed form from the set before each token.
    assert r["budget"][1] == L * TINY.moe.n_experts - r["set_size"][0]


@pytest.mark.parametrize("tau,budget", [(0.3, 2), (0.9, 4), (0.6, truncation.BUDGET_CACHE)])
def test_truncated_step_is_exact(tau, budget):
    c = gen.start_token(TINY, redraw=2)
    r = truncation.truncated_step(om().weights, c, 4, tau=tau, budget=budget, slots=4)
    emitted = r["drafts"][:r["n"]] + [r["bonus"]]
    assert emitted == decode.greedy_ar(om().weights, c, r["n"] + 1)
    kept = len(r["drafts"])
    assert r["stop"] == [False] * kept + ([True] if kept < 4 else [])


def test_cache_sim_truncated_order_matches_fixed_k_when_all_kept():
    rng = np.random.default_rng(3)
    draft = [[rng.choice(12, 3, replace=False).tolist() for _ in range(2)] for _ in range(3)]
    verify = [[rng.choice(12, 3, replace=False).tolist() for _ in range(4)] for _ in range(2)]
    a, b = cache_sim.CacheSim(2, 12, 4), cache_sim.CacheSim(2, 12, 4)
    a.step(draft, verify)
    b.step_truncated(draft, 3, verify)
    assert a.counts == b.counts and a.slot == b.slot
    # A stopped last token requests its top-1 experts but prefetches nothing.
    c1, c2 = cache_sim.CacheSim(2, 12, 4), cache_sim.CacheSim(2, 12, 4)
    c1.step_truncated(draft, 2, verify)
    c2.step_truncated(draft[:2], 2, verify)
    assert c1.counts["prefetch_issued"] == c2.counts["prefetch_issued"]
    assert c1.counts["draft_needed"] == c2.counts["draft_needed"] + 2
