"""The LM head of a block of positions on the matrix cores (§3.3: the target's
logits at every block position) against the fp64 oracle product and against
the vector-ALU row-dot, on the GPU.

The matrix-core path splits each fp32 activation exactly into three bf16 parts,
so every product is exact; only the fp32 summation order differs from the
row-dot.  Integer-valued weights and activations make every partial sum exact,
so there both paths must match the exact dot product bit for bit: a wrong
operand or output lane layout cannot pass that.  Blocks of 5 to 12 positions
take the matrix cores; 1, 2 and 13 positions check the row-dot fallback.
"""
import os

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de

from gpu_support import require_gpu
from support import rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _restore_env():
    require_gpu()
    old = os.environ.get("DE_LMHEAD_MFMA")
    yield
    if old is None:
        os.environ.pop("DE_LMHEAD_MFMA", None)
    else:
        os.environ["DE_LMHEAD_MFMA"] = old


def run(T, H, V, x, w_bf16, mfma):
    os.environ["DE_LMHEAD_MFMA"] = "1" if mfma else "0"
    out = torch.full((T, V), float("nan"), dtype=torch.float32, device="cuda")
    de.de_lm_head(T, H, V, torch.from_numpy(x).cuda(), w_bf16.view(torch.int16), out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("T,H,V", [(5, 32, 16), (6, 64, 17), (9, 256, 1000), (12, 128, 4099),
                                   (9, 2048, 102400), (5, 2048, 1), (2, 64, 33)])
def test_integer_products_are_exact(T, H, V):
    r = np.random.default_rng(T * 1000 + V)
    w = r.integers(-8, 9, size=(V, H)).astype(np.float32)
    x = r.integers(-8, 9, size=(T, H)).astype(np.float32)
    want = x.astype(np.int64) @ w.astype(np.int64).T
    wt = torch.from_numpy(w).to(torch.bfloat16).cuda()
    for mfma in (True, False):
        got = run(T, H, V, x, wt, mfma)
        np.testing.assert_array_equal(got, want.astype(np.float32), err_msg=f"mfma={mfma}")


@pytest.mark.parametrize("T,H,V", [(5, 2048, 4096), (9, 2048, 102400), (12, 1024, 3001),
                                   (13, 256, 500), (2, 2048, 2048), (1, 2048, 2048)])
def test_matches_oracle_and_row_dot(T, H, V):
    r = np.random.default_rng(7 * T + H + V)
    w64 = (r.standard_normal((V, H)) * 0.02).astype(np.float32)
    wt = torch.from_numpy(w64).to(torch.bfloat16).cuda()
    w64 = wt.float().cpu().numpy().astype(np.float64)  # the bf16 values the GPU reads
    # Activations with a wide spread of magnitudes, so the three bf16 parts all matter.
    x = (r.standard_normal((T, H)) * np.exp(r.uniform(-6, 6, size=(T, H)))).astype(np.float32)
    want = x.astype(np.float64) @ w64.T
    got_m = run(T, H, V, x, wt, True)
    got_v = run(T, H, V, x, wt, False)
    em, ev = rel_err(got_m, want), rel_err(got_v, want)
    print(f"T={T} H={H} V={V}: rel err matrix cores {em:.2e}, row-dot {ev:.2e}", flush=True)
    assert em <= 1e-5 and ev <= 1e-5
    assert np.isfinite(got_m).all()


def test_nonfinite_activation_stays_nonfinite():
    T, H, V = 5, 256, 64
    r = np.random.default_rng(3)
    w = (r.standard_normal((V, H)) * 0.02).astype(np.float32)
    wt = torch.from_numpy(w).to(torch.bfloat16).cuda()
    x = r.standard_normal((T, H)).astype(np.float32)
    x[1, 7] = np.inf
    x[2, 9] = np.nan
    x[3, 0] = 3.4e38  # rounds up to infinity in bf16; the split keeps it finite
    got = run(T, H, V, x, wt, True)
    ref = run(T, H, V, x, wt, False)
    assert np.isfinite(got[0]).all()
    assert not np.isfinite(got[1]).any() and not np.isfinite(got[2]).any()
    np.testing.assert_array_equal(np.isfinite(got), np.isfinite(ref))
    assert rel_err(got[3], ref[3]) <= 1e-5
