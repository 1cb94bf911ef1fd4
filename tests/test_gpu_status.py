"""Device-side conditions surfaced at the boundary, on the GPU.

A routed expert that a layer needs but whose slot is outside [0, n_slots)
cannot be loaded by a layer call (Section 3.5 and Algorithm 1 load a missed
expert on demand; only the expert cache does that).  The call leaves the
expert's term out of y, with zero partials so that nothing stale from an
earlier call is summed, and de_layer_status then returns DE_ERR_NOT_RESIDENT.
The expected y is the oracle's layer with that expert's weights set to zero.
A token id outside the vocabulary reaches no embedding row: its rows are NaN
and the status reports it.  None of these cases reads or writes out of
bounds: the kernels skip the work.
"""
import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from oracle import moe
from workloads import configs
from workloads import gpu as wgpu

from gpu_support import f32, i32, layer_pair, require_gpu
from support import gapped_x, rel_err

pytestmark = pytest.mark.gpu

NOT_RESIDENT = -5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def table_without(dev, e_missing):
    slots = torch.arange(dev.cfg.n_experts, dtype=torch.int32, device="cuda")
    if e_missing is not None:
        slots[e_missing] = -1
    return de.make_table(dev.routed, dev.stride, slots, dev.cfg.n_experts), slots


def zeroed(orc, e_missing):
    def routed(e):
        g, u, d = orc.routed(e)
        if e == e_missing:
            return np.zeros_like(g), np.zeros_like(u), np.zeros_like(d)
        return g, u, d
    return routed


@pytest.mark.parametrize("cfg,T", [(configs.CFG1, 5), (configs.CFG2, 9)], ids=["cfg1-T5", "cfg2-T9"])
def test_verify_layer_reports_missing_expert(cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    idx_o, _, _ = orc.route(x)
    missing = int(idx_o[0, 1])
    ws = dev.ws(T)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    nu = torch.empty(1, dtype=torch.int32, device="cuda")
    # A complete call first, so that the workspace holds every partial of the
    # full layer: the call with the hole must not pick any of them up.
    full, _ = table_without(dev, None)
    de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, full, dev.shared, y,
                       n_union=nu, ws=ws)
    assert de.de_layer_status(ws) == 0
    y_full = orc.target(x)[0]
    assert rel_err(y.cpu().numpy(), y_full) < 1e-4
    tab, _ = table_without(dev, missing)
    de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, tab, dev.shared, y,
                       n_union=nu, ws=ws)
    assert de.de_layer_status(ws) == NOT_RESIDENT
    assert de.de_layer_status(ws) == 0          # read and cleared
    want = moe.moe_target(x, orc.w_router, orc.bias, zeroed(orc, missing), orc.shared, cfg.top_k,
                          cfg.score_func, cfg.norm_topk, cfg.routed_scale)[0]
    err = rel_err(y.cpu().numpy(), want)
    print(f"{cfg.name}: expert {missing} missing, rel err {err:.2e}", flush=True)
    assert err < 1e-4
    assert int(nu.item()) == len(set(idx_o.ravel().tolist()))
    # The complete table again: no status, the full output.
    de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, full, dev.shared, y, ws=ws)
    assert de.de_layer_status(ws) == 0
    assert rel_err(y.cpu().numpy(), y_full) < 1e-4


def test_expert_absent_but_unneeded_is_not_reported():
    cfg, T = configs.CFG2, 9
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    idx_o, _, _ = orc.route(x)
    unused = sorted(set(range(cfg.n_experts)) - set(idx_o.ravel().tolist()))[0]
    tab, _ = table_without(dev, unused)
    ws = dev.ws(T)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, tab, dev.shared, y, ws=ws)
    assert de.de_layer_status(ws) == 0
    assert rel_err(y.cpu().numpy(), orc.target(x)[0]) < 1e-4


def test_draft_layer_reports_missing_top1():
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, 1, block=1)
    idx_o, _, _ = orc.route(x)
    e1 = int(idx_o[0, 0])
    tab, _ = table_without(dev, e1)
    ws = dev.ws(1)
    y = torch.empty(1, cfg.hidden, dtype=torch.float32, device="cuda")
    pred = torch.empty(1, cfg.top_k, dtype=torch.int32, device="cuda")
    de.de_draft_layer(dev.desc, 1, f32(x), dev.router, dev.bias, tab, dev.shared, dev.draft,
                      cfg.gamma, y, pred, None, ws)
    assert de.de_layer_status(ws) == NOT_RESIDENT
    want = moe.moe_draft(x, orc.w_router, orc.bias, zeroed(orc, e1), orc.shared, orc.draft,
                         cfg.gamma, cfg.top_k, cfg.score_func, cfg.norm_topk, cfg.routed_scale)[0]
    assert rel_err(y.cpu().numpy(), want) < 1e-4
    np.testing.assert_array_equal(pred.cpu().numpy(), idx_o)


def test_grouped_swiglu_reports_missing_member():
    cfg, T = configs.CFG1, 5
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    idx_o, gate_o, _ = orc.route(x)
    u = moe.expert_union(idx_o, gate_o)
    missing = int(u["union_ids"][-1])
    tab, _ = table_without(dev, missing)
    ws = dev.ws(T)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    n = np.full(cfg.n_experts + 1, u["offsets"][-1], np.int32)
    n[:len(u["offsets"])] = u["offsets"]
    uid = np.full(cfg.n_experts, -1, np.int32)
    uid[:u["n_union"]] = u["union_ids"]
    de.de_grouped_swiglu(dev.desc, T, f32(x), tab, i32([u["n_union"]]), i32(uid), i32(n),
                         i32(u["tok_list"]), f32(u["gate_list"]), i32(u["pair_pos"]), dev.shared, y,
                         ws)
    assert de.de_layer_status(ws) == NOT_RESIDENT
    want = moe.moe_target(x, orc.w_router, orc.bias, zeroed(orc, missing), orc.shared, cfg.top_k,
                          cfg.score_func, cfg.norm_topk, cfg.routed_scale)[0]
    assert rel_err(y.cpu().numpy(), want) < 1e-5


def test_embed_reports_out_of_range_token():
    V, H = 1000, 256
    emb = torch.randn(V, H, device="cuda").to(torch.bfloat16).view(torch.int16)
    toks = i32([3, V, -1, 999])
    h = torch.zeros(4, H, dtype=torch.float32, device="cuda")
    hn = torch.zeros(4, H, dtype=torch.float32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    de.de_embed_gather(4, H, V, toks, emb, h, hn, 1e-6, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 2
    hc = h.cpu()
    assert torch.isnan(hc[1]).all() and torch.isnan(hc[2]).all() and torch.isnan(hn.cpu()[1]).all()
    want = emb.view(torch.bfloat16).float().cpu()
    assert torch.equal(hc[0], want[3]) and torch.equal(hc[3], want[999])


def test_model_status_reports_bad_token_and_missing_expert():
    from test_gpu_model import V2_SMALL, device_model
    dm = device_model(V2_SMALL, 1)
    logits = torch.empty(1, V2_SMALL.vocab, dtype=torch.float32, device="cuda")
    dm.forward(i32([V2_SMALL.vocab + 5]), de.DE_TARGET, logits)
    assert de.de_model_status(dm.model, dm.ws) == -1
    dm.forward(i32([7]), de.DE_TARGET, logits)
    assert de.de_model_status(dm.model, dm.ws) == 0
    assert torch.isfinite(logits).all()
