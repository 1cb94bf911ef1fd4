"""Q4_0 expert weights on the GPU against the oracle (the 4.5-bit block format
of the paper's mobile platform, Section 4.1; a dequantise-in-the-dot-product
variant of the grouped gate/up and down).

The GPU fill of Q4_0 blocks equals the CPU generator bit for bit.  Layer
outputs are compared with the fp64 oracle, which dequantises the same bytes
exactly (relative 1e-4, as for bf16 weights); routing, union and lists stay
bit-exact.  Cases: the tiny layer, the V2-Lite layer at T = 1, 9 (activations
staged in LDS) and 17 (read from global memory), the draft layer, and a
two-layer Q4_0 stack's draft-then-verify step.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from gpu_support import f32, layer_pair, require_gpu, verify_outputs
from oracle import moe
from support import OracleModel, gapped_x, rel_err
from workloads import configs, gen
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu

CASES = [("cfg1q4-T5", configs.CFG1_Q4, 5), ("cfg2q4-T1", configs.CFG2_Q4, 1),
         ("cfg2q4-T9", configs.CFG2_Q4, 9), ("cfg2q4-T17", configs.CFG2_Q4, 17)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def test_q4_fill_matches_cpu_generator():
    c = configs.CFG2_Q4
    dev = wgpu.routed_experts(c, 0, n_experts=4)
    for e in (0, 3):
        assert np.array_equal(dev[e].cpu().numpy(), gen.routed_block(c, 0, e))
    assert np.array_equal(wgpu.shared_block(c, 0).cpu().numpy(), gen.shared_block(c, 0))
    assert np.array_equal(wgpu.draft_block(c, 0).cpu().numpy(), gen.draft_block(c, 0))


@pytest.mark.parametrize("name,cfg,T", CASES, ids=[c[0] for c in CASES])
def test_q4_verify_layer(name, cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    y_o, idx_o, gate_o = orc.target(x)
    uo = moe.expert_union(idx_o, gate_o)
    out = verify_outputs(dev, f32(x), T)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["idx"].cpu().numpy(), idx_o)
    assert int(out["nu"].item()) == uo["n_union"]
    np.testing.assert_array_equal(out["tok"].cpu().numpy(), uo["tok_list"])
    err = rel_err(out["y"].cpu().numpy(), y_o)
    print(f"[q4 verify {name}] union={uo['n_union']} rel_err={err:.3e}", flush=True)
    assert err <= 1e-4


@pytest.mark.parametrize("cfg,T", [(configs.CFG1_Q4, 1), (configs.CFG2_Q4, 1),
                                   (configs.CFG2_Q4, 3)])
def test_q4_draft_layer(cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=1)
    y_o, idx_o, _ = orc.draft_out(x)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    pidx = torch.empty(T, cfg.top_k, dtype=torch.int32, device="cuda")
    de.de_draft_layer(dev.desc, T, f32(x), dev.router, dev.bias, dev.table, dev.shared, dev.draft,
                      cfg.gamma, y, pidx, None, dev.ws(T))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(pidx.cpu().numpy(), idx_o)
    assert rel_err(y.cpu().numpy(), y_o) <= 1e-4


def test_q4_rejects_rows_that_are_not_whole_blocks():
    c = configs.CFG1_Q4
    for over in (dict(hidden=c.hidden + 8), dict(inter=c.inter - 16), dict(draft_inter=48)):
        kw = dict(hidden=c.hidden, n_experts=c.n_experts, top_k=c.top_k, inter=c.inter,
                  shared_inter=c.shared_inter, draft_inter=c.draft_inter,
                  score_func=c.score_func, norm_topk=c.norm_topk, routed_scale=c.routed_scale,
                  wdtype=de.DE_Q4_0)
        kw.update(over)
        assert de.LIB.de_check_desc(de.make_desc(**kw)) != 0


def test_q4_stack_step_matches_oracle():
    model = configs.scaled_model(configs.CFG4, n_moe_layers=2, vocab=8192, dense_inter=1408,
                                 k_draft=2, moe=replace(configs.CFG2_Q4, cfg_id=44),
                                 name="v2lite-q4-stack")
    om = OracleModel(model)
    c, drafts, n, bonus, t, traces = om.gapped_step(model.k_draft)
    m = model.moe
    tens = wgpu.model_tensors(model)
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    dm = de.DeviceModel(desc, tens["layers"], model.vocab, tens["emb"], tens["lm"], tens["dense"],
                        model.dense_inter, de.DE_BF16, model.eps, m.gamma, model.k_draft + 1)
    K, L = model.k_draft, model.n_moe_layers
    block = dm.new_block(K, c)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    dm.spec_step(block, amax, out, nu)
    torch.cuda.synchronize()
    print(f"start {c}: drafts {drafts} n {n} bonus {bonus}", flush=True)
    assert block[1:].cpu().tolist() == drafts
    assert amax.cpu().tolist() == [int(v) for v in t]
    assert out.cpu().tolist() == [n, bonus]
    assert nu.cpu().tolist() == [len(set(np.asarray(i).ravel().tolist())) for i in traces[-1].idx]
