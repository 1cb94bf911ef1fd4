"""Writes cfg4_step.json: one exact draft-then-verify step of the full-size
V2-Lite-shaped stack (dense layer 0 with I = 10944, 26 MoE layers, K = 8,
102400-vocab head), computed by the fp64 oracle alone (Algorithm 1 with a
fixed draft length).

The start token is the first of the generator's start-token stream (redraw
counter 0, 1, ...) for which every routing decision of every pass (each
layer's top-k keys, down to the (k+1)-th, and every row argmax of the logits)
has a margin above 1e-4, so that fp32 rounding on the GPU cannot flip a
decision.  Stored: the start token and its redraw counter, the drafts, the
target argmax, n and the bonus token, the verify union size of every MoE layer,
the drafter's top-k in every layer at every draft position, and a sample of
the logits (each row's 8 largest entries and 24 seeded random columns) of the
verify pass and of the first draft pass.

Run from the repository root: python tests/golden/make_cfg4_step.py
(about 3 minutes per candidate start token on one host core).
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

from oracle import decode  # noqa: E402
from support import OracleModel  # noqa: E402
from workloads import configs, gen  # noqa: E402

OUT = os.path.join(HERE, "cfg4_step.json")
N_TOP, N_RAND = 8, 24


def logit_sample(logits: np.ndarray, seed: int):
    rows = []
    r = np.random.default_rng(seed)
    for j, row in enumerate(np.atleast_2d(logits)):
        top = np.argsort(-row, kind="stable")[:N_TOP]
        rnd = r.choice(row.size, N_RAND, replace=False)
        cols = np.unique(np.concatenate([top, rnd]))
        rows.append({"cols": cols.tolist(), "vals": [float(row[c]) for c in cols]})
    return rows


def main(max_tries: int = 12):
    model = configs.CFG4
    t0 = time.time()
    om = OracleModel(model)
    print(f"oracle model ready in {time.time() - t0:.0f} s", flush=True)
    K = model.k_draft
    for redraw in range(max_tries):
        c = gen.start_token(model, redraw=redraw)
        t1 = time.time()
        traces: list = []
        drafts, n, bonus, t = decode.spec_step(om.weights, c, K, traces)
        ok = [om.trace_gaps_ok(tr) for tr in traces]
        print(f"redraw {redraw}: start {c} drafts {drafts} n {n} bonus {bonus} gaps {ok} "
              f"({time.time() - t1:.0f} s)", flush=True)
        if not all(ok):
            continue
        ver = traces[-1]
        out = {
            "model": model.name, "redraw": redraw, "start": int(c), "k_draft": K,
            "drafts": [int(d) for d in drafts], "n": int(n), "bonus": int(bonus),
            "target_argmax": [int(v) for v in t],
            "n_union": [len(set(np.asarray(i).ravel().tolist())) for i in ver.idx],
            "pred_idx": [[np.asarray(i)[0].tolist() for i in tr.idx] for tr in traces[:K]],
            "verify_logits": logit_sample(ver.logits, 4),
            "draft0_logits": logit_sample(traces[0].logits, 5),
        }
        with open(OUT, "w") as f:
            json.dump(out, f)
        print("wrote", OUT, flush=True)
        return
    raise SystemExit("no gapped start token within the tries")


if __name__ == "__main__":
    main()
