"""Plain fp64 oracle of confidence-expansion truncation of the draft loop
(Section 3.4, Eqs. 12-14; Algorithm 1).

TEST INFRASTRUCTURE ONLY (same rule as ``oracle.moe``): imported by tests/,
the smoke check and the CPU baseline, never by the product path.

For draft token i the controller has a confidence q_i from the draft logits
and the verifier experts the draft router predicts in every MoE layer l.  The
predicted block-level verifier set is the union of those (layer, expert)
pairs over the kept tokens; the token's marginal expansion Delta_i is how many
pairs it would add.  Drafting stops before appending token i when
q_i < tau and Delta_i > B_i (Eq. 14); the stopped token is not verified.

Readings taken here (the paper leaves them open):

* q_i is the largest softmax probability of token i's draft logits, taken in
  fp64 here from the logits the drafter produced;
* the predicted experts of token i in layer l are the draft router's top-k at
  that layer (the list the drafter already computes for the draft gate);
* B_i is either a fixed count of layer-experts, or derived from the expert
  cache as the room the predicted set still has in it:
  B_i = sum_l max(0, S - |set before token i, layer l|), S slots per layer.
"""
from __future__ import annotations

import numpy as np

from . import decode, moe

BUDGET_CACHE = -1   # B_i from the cache slots instead of a fixed count


def confidence(logits) -> np.ndarray:
    """q per row: the largest softmax probability, 1 / sum_v exp(l_v - max_v l)."""
    lg = np.atleast_2d(np.asarray(logits, dtype=np.float64))
    mx = lg.max(axis=1, keepdims=True)
    return 1.0 / np.exp(lg - mx).sum(axis=1)


def predicted_pairs(idx_per_layer) -> set:
    """The (layer, expert) pairs one draft token predicts: its top-k in each layer."""
    return {(l, int(e)) for l, idx in enumerate(idx_per_layer)
            for e in np.asarray(idx).ravel().tolist()}


def cache_budget(uhat: set, n_layers: int, slots: int) -> int:
    """B_i derived from the cache: the slots per layer not yet claimed by the set."""
    per_layer = [0] * n_layers
    for l, _ in uhat:
        per_layer[l] += 1
    return sum(max(0, slots - c) for c in per_layer)


def decide(q: float, uhat: set, pairs: set, tau: float, budget: int, n_layers: int,
           slots: int = 0):
    """Eq. 14 for one token: (stop, delta, B_i, the set after the token).

    The returned set is the old one when the token is stopped."""
    grown = uhat | pairs
    delta = len(grown) - len(uhat)
    b = cache_budget(uhat, n_layers, slots) if budget == BUDGET_CACHE else int(budget)
    stop = bool(q < tau and delta > b)
    return stop, delta, b, (uhat if stop else grown)


def truncated_step(model: decode.ModelWeights, last_token: int, k_max: int, tau: float,
                   budget: int, slots: int = 0, traces: list | None = None) -> dict:
    """One exact step of Algorithm 1 with truncation: draft up to k_max tokens,
    stop by Eq. 14, verify the kept drafts with the target, accept greedily.

    Returns a dict: drafts (kept), n, bonus, target_argmax, and per evaluated
    token (the stopped one included) q, delta, budget, stop, set_size.  With
    ``traces`` the Trace of every draft pass, then of the verify pass, is
    appended."""
    n_layers = len(model.layers)
    uhat: set = set()
    drafts: list = []
    rec = {"q": [], "delta": [], "budget": [], "stop": [], "set_size": []}
    cur = int(last_token)
    for _ in range(k_max):
        tr = decode.Trace()
        logits = decode.forward(model, [cur], "draft", tr)
        if traces is not None:
            traces.append(tr)
        v = int(moe.argmax_first(logits)[0])
        q = float(confidence(logits)[0])
        stop, delta, b, uhat = decide(q, uhat, predicted_pairs(tr.idx), tau, budget, n_layers,
                                      slots)
        for key, val in (("q", q), ("delta", delta), ("budget", b), ("stop", stop),
                         ("set_size", len(uhat))):
            rec[key].append(val)
        if stop:
            break
        drafts.append(v)
        cur = v
    vt = decode.Trace() if traces is not None else None
    logits = decode.forward(model, [int(last_token)] + drafts, "target", vt)
    if traces is not None:
        traces.append(vt)
    n, bonus, t = moe.accept_len(logits, drafts)
    return dict(drafts=drafts, n=n, bonus=bonus, target_argmax=t, **rec)
