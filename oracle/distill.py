"""Plain fp64 oracle of the self-distillation signals (Section 3.3, Eqs. 6-10)
as by-products of teacher-forced target and draft passes over a block.

TEST INFRASTRUCTURE ONLY (same rule as ``oracle.moe``).

The training itself is outside the path; what the runtime can emit for it is
computed here from its definition:

* the residual target of Eq. 6 per MoE layer and position: the target layer's
  output minus its shared path and its top-1 expert's gated term, i.e. what
  the draft expert is trained to supply (Eq. 7 compares gamma E^d with it);
* the router agreement of Eq. 10 per layer and position: the KL divergence
  from the target's router distribution at the target's hidden state to the
  draft path's router distribution at the draft hidden state of the same
  position;
* the logit distillation term of Eq. 8 per position (temperature tau, scaled
  by tau^2) and the token term of Eq. 9 (cross entropy of the draft logits
  against the target's argmax token).

Readings: the router distribution R_l is softmax(z + b) for softmax routers
and, for sigmoid routers, the sigmoid scores normalised to sum to one (Eq. 10
needs a distribution); positions are teacher-forced, so the draft pass at
position t reads the same token as the target pass (the stack has no
attention, so a position depends only on its token).
"""
from __future__ import annotations

import numpy as np

from . import decode, moe


def residual_target(x, lw: decode.LayerWeights) -> np.ndarray:
    """m* of Eq. 6 for each row of the layer input x: y* - S(x) - g_e1 E_e1(x)."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    y, idx, gate = moe.moe_target(x, lw.w_router, lw.bias, lw.routed, lw.shared, lw.top_k,
                                  lw.score_func, lw.norm_topk, lw.routed_scale)
    m = y - moe.shared_path(x, lw.shared)
    for t in range(x.shape[0]):
        g, u, d = lw.routed(int(idx[t, 0]))
        m[t] -= gate[t, 0] * moe.swiglu(x[t:t + 1], g, u, d)[0]
    return m


def router_distribution(z, bias, score_func: int) -> np.ndarray:
    """R_l from router logits z [T, N]: softmax(z + b), or normalised sigmoid(z)."""
    z = np.atleast_2d(np.asarray(z, dtype=np.float64))
    if score_func == moe.SOFTMAX:
        zb = z + (0.0 if bias is None else np.asarray(bias, dtype=np.float64))
        e = np.exp(zb - zb.max(axis=1, keepdims=True))
        return e / e.sum(axis=1, keepdims=True)
    s = 1.0 / (1.0 + np.exp(-z))
    return s / s.sum(axis=1, keepdims=True)


def kl_rows(p, q) -> np.ndarray:
    """sum_i p_i (log p_i - log q_i) per row (terms with p_i = 0 are zero)."""
    p = np.atleast_2d(np.asarray(p, dtype=np.float64))
    q = np.atleast_2d(np.asarray(q, dtype=np.float64))
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(p > 0, p * (np.log(p) - np.log(q)), 0.0)
    return t.sum(axis=1)


def softmax_rows(z) -> np.ndarray:
    z = np.atleast_2d(np.asarray(z, dtype=np.float64))
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def logit_kl(z_target, z_draft, tau: float) -> np.ndarray:
    """Eq. 8 per position: tau^2 KL(softmax(z*/tau) || softmax(z^d/tau))."""
    return tau * tau * kl_rows(softmax_rows(np.asarray(z_target) / tau),
                               softmax_rows(np.asarray(z_draft) / tau))


def token_ce(z_target, z_draft) -> np.ndarray:
    """Eq. 9 per position: -log softmax(z^d)[argmax z*] (argmax on fp32, ties low)."""
    t = moe.argmax_first(z_target)
    zd = np.atleast_2d(np.asarray(z_draft, dtype=np.float64))
    mx = zd.max(axis=1)
    lse = mx + np.log(np.exp(zd - mx[:, None]).sum(axis=1))
    return lse - zd[np.arange(zd.shape[0]), t]


def distill_signals(model: decode.ModelWeights, tokens, tau: float = 1.0) -> dict:
    """The signals of Eqs. 6-10 for the positions `tokens`, from one target and
    one draft pass: m_star [L, T, H], router_kl [L, T], logit_kl [T],
    token_ce [T] (plus the two passes' logits)."""
    tt, td = decode.Trace(), decode.Trace()
    z_t = decode.forward(model, tokens, "target", tt)
    z_d = decode.forward(model, tokens, "draft", td)
    m_star, rkl = [], []
    for l, lw in enumerate(model.layers):
        m_star.append(residual_target(tt.moe_inputs[l], lw))
        zt, _, _ = moe.router_scores(tt.moe_inputs[l], lw.w_router, lw.bias, lw.score_func)
        zd, _, _ = moe.router_scores(td.moe_inputs[l], lw.w_router, lw.bias, lw.score_func)
        rkl.append(kl_rows(router_distribution(zt, lw.bias, lw.score_func),
                           router_distribution(zd, lw.bias, lw.score_func)))
    return dict(m_star=np.stack(m_star) if m_star else np.zeros((0,)),
                router_kl=np.stack(rkl) if rkl else np.zeros((0,)),
                logit_kl=logit_kl(z_t, z_d, tau), token_ce=token_ce(z_t, z_d),
                target_logits=z_t, draft_logits=z_d)
