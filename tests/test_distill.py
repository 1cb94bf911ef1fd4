"""Pins of the self-distillation signals oracle (Section 3.3, Eqs. 6-10).

The residual target against the lower-ranked experts' terms computed
directly (Eq. 6); KL against SciPy's relative entropy, zero for equal
distributions, and the temperature scaling of Eq. 8 in closed form; the
token term against SciPy's log-softmax; router distributions summing to one;
and a stack whose drafter equals its target, where every divergence is zero.
"""
from dataclasses import replace

import numpy as np
import pytest
import scipy.special

from oracle import decode, distill, moe
from support import OracleLayer, OracleModel, gapped_x
from workloads import configs, gen


def test_residual_target_is_the_lower_ranked_experts():
    ol = OracleLayer(configs.CFG1, 0)
    c = ol.cfg
    x, _ = gapped_x(ol, 3, block=4)
    m = distill.residual_target(x, ol.layer_weights())
    idx, gate, _ = ol.route(x)
    want = np.zeros_like(m)
    for t in range(3):
        xt = x[t].astype(np.float64)
        for j in range(1, c.top_k):
            g, u, d = ol.routed(int(idx[t, j]))
            h = xt @ g.T
            want[t] += gate[t, j] * ((h / (1 + np.exp(-h)) * (xt @ u.T)) @ d.T)
    np.testing.assert_allclose(m, want, rtol=1e-9, atol=1e-14)


def test_kl_against_scipy_and_zero_for_equal_rows():
    rng = np.random.default_rng(2)
    p = scipy.special.softmax(rng.normal(size=(4, 50)), axis=1)
    q = scipy.special.softmax(rng.normal(size=(4, 50)), axis=1)
    np.testing.assert_allclose(distill.kl_rows(p, q),
                               scipy.special.rel_entr(p, q).sum(axis=1), rtol=1e-12)
    np.testing.assert_allclose(distill.kl_rows(p, p), 0.0, atol=1e-15)
    assert np.all(distill.kl_rows(p, q) > 0)


def test_logit_kl_temperature_closed_form():
    # Two logits: p = sigmoid(a / tau), q = sigmoid(b / tau).
    a, b, tau = 1.3, -0.4, 2.0
    p, q = 1 / (1 + np.exp(-a / tau)), 1 / (1 + np.exp(-b / tau))
    want = tau * tau * (p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q)))
    got = distill.logit_kl(np.array([[a, 0.0]]), np.array([[b, 0.0]]), tau)[0]
    assert got == pytest.approx(want, rel=1e-12)


def test_token_ce_against_scipy():
    rng = np.random.default_rng(3)
    zt, zd = rng.normal(size=(5, 300)), rng.normal(size=(5, 300))
    want = -scipy.special.log_softmax(zd, axis=1)[np.arange(5), zt.argmax(axis=1)]
    np.testing.assert_allclose(distill.token_ce(zt, zd), want, rtol=1e-12)


@pytest.mark.parametrize("score_func", [moe.SOFTMAX, moe.SIGMOID])
def test_router_distribution_sums_to_one(score_func):
    rng = np.random.default_rng(4)
    z = rng.normal(size=(3, 64))
    r = distill.router_distribution(z, rng.normal(size=64), score_func)
    np.testing.assert_allclose(r.sum(axis=1), 1.0, rtol=1e-14)
    if score_func == moe.SOFTMAX:
        b = rng.normal(size=64)
        np.testing.assert_allclose(distill.router_distribution(z, b, score_func),
                                   scipy.special.softmax(z + b, axis=1), rtol=1e-13)


def test_divergences_vanish_when_the_drafter_is_the_target():
    model = configs.scaled_model(configs.CFG4, n_moe_layers=2, vocab=1000, dense_inter=256,
                                 k_draft=3, moe=replace(configs.CFG1, cfg_id=45),
                                 name="tiny-distill")
    w = OracleModel(model).weights
    w = replace(w, layers=[replace(lw, draft=None, gamma=0.0) for lw in w.layers],
                draft_topr=model.moe.top_k)
    toks = [gen.start_token(model, redraw=r) for r in range(4)]
    s = distill.distill_signals(w, toks, tau=1.5)
    assert s["m_star"].shape == (2, 4, model.moe.hidden)
    np.testing.assert_allclose(s["router_kl"], 0.0, atol=1e-12)
    np.testing.assert_allclose(s["logit_kl"], 0.0, atol=1e-12)
    # CE is then minus the log of the largest target probability.
    q = scipy.special.softmax(s["target_logits"], axis=1).max(axis=1)
    np.testing.assert_allclose(s["token_ce"], -np.log(q), rtol=1e-10)
    assert np.abs(s["m_star"]).max() > 0
