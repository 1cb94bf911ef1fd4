"""The verify layer as one launch, on the GPU.

de_verify_layer runs the layer of a bf16 block of 2..9 positions (V2-Lite
and Moonlight shapes) as one launch whose blocks exchange the gate/up outputs
and the down partials as (value, launch epoch) words.  Every value is computed
by the same operations as in the separate launches, so each output must equal
theirs bit for bit (DE_VERIFY_FUSED=1 selects the single launch, which is
off by default, and 0 the separate launches); the
oracle comparisons of the layer (test_gpu_layer.py) cover both paths at their
shapes.  Covered here: the block lengths the launch serves at its edges, long
runs of calls on one workspace (every call must see only its own words),
alternating block lengths, the epilogue, a needed expert without a slot and
the phase timer.
"""
import os

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from workloads import configs

from gpu_support import f32, layer_pair, require_gpu, verify_outputs
from support import gapped_x, rel_err

pytestmark = pytest.mark.gpu

NOT_RESIDENT = -5
KEYS = ["y", "idx", "gate", "nu", "uids", "offs", "tok", "glist", "ppos"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    with launch_mode("1"):
        yield
    torch.cuda.synchronize()


class launch_mode:
    """DE_VERIFY_FUSED=value for the duration (the library reads it at each call)."""

    def __init__(self, value):
        self.value = value

    def __enter__(self):
        self.old = os.environ.get("DE_VERIFY_FUSED")
        os.environ["DE_VERIFY_FUSED"] = self.value

    def __exit__(self, *exc):
        if self.old is None:
            del os.environ["DE_VERIFY_FUSED"]
        else:
            os.environ["DE_VERIFY_FUSED"] = self.old


def same_bits(a, b):
    a = a.cpu().numpy()
    b = b.cpu().numpy()
    assert a.dtype == b.dtype
    return np.array_equal(a.view(np.uint8), b.view(np.uint8))


def outputs_equal(got, want, T):
    n = int(want["nu"].item())
    assert int(got["nu"].item()) == n
    for k in KEYS:
        g, w = got[k], want[k]
        if k == "uids":
            g, w = g[:n], w[:n]
        elif k == "offs":
            g, w = g[:n + 1], w[:n + 1]
        assert same_bits(g, w), k


@pytest.mark.parametrize("cfg,T", [(configs.CFG2, 2), (configs.CFG2, 5), (configs.CFG2, 8),
                                   (configs.CFG2, 9), (configs.CFG3, 5), (configs.CFG3, 9)],
                         ids=["cfg2-T2", "cfg2-T5", "cfg2-T8", "cfg2-T9", "cfg3-T5", "cfg3-T9"])
def test_single_launch_equals_separate_launches(cfg, T):
    orc, dev = layer_pair(cfg)
    assert de.de_verify_single_launch(dev.desc, T)
    x, _ = gapped_x(orc, T, block=0)
    xd = f32(x)
    print(f"{cfg.name} T={T}: single launch", flush=True)
    got = verify_outputs(dev, xd, T)
    torch.cuda.synchronize()
    with launch_mode("0"):
        assert not de.de_verify_single_launch(dev.desc, T)
        want = verify_outputs(dev, xd, T)
    torch.cuda.synchronize()
    outputs_equal(got, want, T)
    # ... and the layer itself against the oracle.
    assert rel_err(got["y"].cpu().numpy(), orc.target(x)[0]) < 1e-4


def test_off_by_default():
    _, dev = layer_pair(configs.CFG2)
    del os.environ["DE_VERIFY_FUSED"]
    try:
        assert not de.de_verify_single_launch(dev.desc, 9)
    finally:
        os.environ["DE_VERIFY_FUSED"] = "1"


def test_block_lengths_served():
    """The single launch serves the V2-Lite layer at T = 2..9 (the staged
    rows of a sweep fit a CU's LDS); other lengths use the separate launches."""
    _, dev = layer_pair(configs.CFG2)
    served = [T for T in range(1, 65) if de.de_verify_single_launch(dev.desc, T)]
    assert served == list(range(2, 10))


def test_single_launch_with_epilogue():
    cfg, T = configs.CFG2, 9
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=1)
    xd = f32(x)
    res = f32(np.random.default_rng(7).standard_normal((T, cfg.hidden)))
    outs = []
    for fused in (True, False):
        normed = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        epi = de.make_epilogue(residual=res, normed=normed, eps=1e-6)
        if fused:
            o = verify_outputs(dev, xd, T, epi=epi)
        else:
            with launch_mode("0"):
                o = verify_outputs(dev, xd, T, epi=epi)
        torch.cuda.synchronize()
        o["normed"] = normed
        outs.append(o)
    outputs_equal(outs[0], outs[1], T)
    assert same_bits(outs[0]["normed"], outs[1]["normed"])


def test_residual_target_after_single_launch():
    """The Eq. 6 target reads the plain routed partials the launch also writes."""
    cfg, T = configs.CFG2, 9
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=2)
    xd = f32(x)
    got = []
    for fused in (True, False):
        ws = dev.ws(T)
        y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        m = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        if fused:
            de.de_verify_layer(dev.desc, T, xd, dev.router, dev.bias, dev.table, dev.shared, y,
                               ws=ws)
        else:
            with launch_mode("0"):
                de.de_verify_layer(dev.desc, T, xd, dev.router, dev.bias, dev.table, dev.shared, y,
                                   ws=ws)
        de.de_residual_target(dev.desc, T, ws, m)
        torch.cuda.synchronize()
        got.append(m)
    assert same_bits(got[0], got[1])


def test_many_calls_on_one_workspace():
    """Forty calls on one workspace with fresh inputs each time, alternating two
    block lengths: each must equal the separate launches on the same input (a
    word of an earlier call never passes for this call's)."""
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    rng = np.random.default_rng(11)
    ws = {T: dev.ws(T) for T in (5, 9)}
    for i in range(40):
        T = 9 if i % 3 else 5
        x = rng.standard_normal((T, cfg.hidden)).astype(np.float32)
        xd = f32(x)
        y1 = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        y0 = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        nu = torch.empty(1, dtype=torch.int32, device="cuda")
        de.de_verify_layer(dev.desc, T, xd, dev.router, dev.bias, dev.table, dev.shared, y1,
                           n_union=nu, ws=ws[T])
        with launch_mode("0"):
            de.de_verify_layer(dev.desc, T, xd, dev.router, dev.bias, dev.table, dev.shared, y0,
                               ws=dev.ws(T))
        torch.cuda.synchronize()
        assert same_bits(y1, y0), (i, T)
    assert de.de_layer_status(ws[5]) == 0
    assert de.de_layer_status(ws[9]) == 0


def test_single_launch_reports_missing_expert():
    cfg, T = configs.CFG2, 9
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    idx_o, _, _ = orc.route(x)
    missing = int(idx_o[2, 3])
    slots = torch.arange(cfg.n_experts, dtype=torch.int32, device="cuda")
    slots[missing] = -1
    tab = de.make_table(dev.routed, dev.stride, slots, cfg.n_experts)
    ys = []
    for fused in (True, False):
        ws = dev.ws(T)
        y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        if fused:
            de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, tab, dev.shared, y, ws=ws)
        else:
            with launch_mode("0"):
                de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, tab, dev.shared, y,
                                   ws=ws)
        assert de.de_layer_status(ws) == NOT_RESIDENT
        assert de.de_layer_status(ws) == 0
        ys.append(y)
    assert same_bits(ys[0], ys[1])


def test_layer_phase_timer_brackets_the_launch():
    cfg, T = configs.CFG2, 9
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for ev in e:
        ev.record()
    de.de_time_next_phase(de.DE_PHASE_LAYER, e[0], e[1])
    verify_outputs(dev, f32(x), T)
    torch.cuda.synchronize()
    ms = e[0].elapsed_time(e[1])
    print(f"single launch: {1e3 * ms:.1f} us", flush=True)
    assert 0.0 < ms < 50.0
