"""Calibrates the router-bias scale of the skewed-routing workload.

The bias of MoE layer l is b_e = lam * (-s * ln r_e), r_e a seeded rank
permutation of the experts (workloads.gen.zipf_bias), added to the softmax
router logits.  lam is chosen by bisection so that, over 1e5 activation rows
drawn like the workload's (N(0, 1)), the least-squares slope of
log(selection share) against log(rank) is -s.  Selections are counted with
the oracle's top-k.  Writes zipf_lambda.json next to this file.

Run: python tests/golden/calibrate_zipf.py
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import moe  # noqa: E402
from workloads import configs, gen  # noqa: E402

N_TOKENS = 100_000
LAYER = 1
BLOCK = 9001  # activation stream reserved for this calibration


def rank_of(model, layer):
    """Rank r_e (1 = most favoured) implied by the bias at any lam > 0."""
    b = gen.zipf_bias(model, layer, 1.0)
    order = np.argsort(-b.astype(np.float64), kind="stable")
    r = np.empty(model.moe.n_experts, dtype=np.int64)
    r[order] = np.arange(1, model.moe.n_experts + 1)
    return r


def slope(model, x, w, lam, layer=LAYER):
    m = model.moe
    b = gen.zipf_bias(model, layer, lam)
    counts = np.zeros(m.n_experts)
    for i in range(0, x.shape[0], 10_000):
        idx, _, _ = moe.route_topk(x[i:i + 10_000], w, b, m.top_k, m.score_func, m.norm_topk)
        counts += np.bincount(idx.ravel(), minlength=m.n_experts)
    share = counts / counts.sum()
    r = rank_of(model, layer)
    keep = share > 0
    A = np.stack([np.log(r[keep]), np.ones(keep.sum())], axis=1)
    coef, *_ = np.linalg.lstsq(A, np.log(share[keep]), rcond=None)
    return float(coef[0]), share


def main():
    model = configs.CFG5
    m = model.moe
    x = gen.x_rows(m, N_TOKENS, block=BLOCK).astype(np.float64)
    w = gen.router_weight(m, LAYER).astype(np.float64)
    lo, hi = 0.0, 4.0
    target = -model.zipf_s
    s_hi, _ = slope(model, x, w, hi)
    assert s_hi < target, "upper bracket too small"
    for _ in range(30):
        mid = 0.5 * (lo + hi)
        s_mid, _ = slope(model, x, w, mid)
        if s_mid > target:
            lo = mid
        else:
            hi = mid
    lam = round(0.5 * (lo + hi), 4)
    s_fin, share = slope(model, x, w, lam)
    out = {"lam": lam, "slope": round(s_fin, 4), "target_slope": target, "tokens": N_TOKENS,
           "layer": LAYER, "top_share": round(float(share.max()), 4),
           "note": "selection share of the most favoured expert saturates below 1/k"}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "zipf_lambda.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


if __name__ == "__main__":
    main()
