"""The persistent draft pass (one launch for a draft position's MoE layers,
Eq. 5) against the separate gate/up, down and combine launches, on the GPU.

Both paths do the same fp32 operations in the same order, so every output
must be identical bit for bit: the draft logits of a position, its argmax,
the drafter's top-k in every layer, and a whole draft-then-verify step.  The
environment variable DE_DRAFT_PERSISTENT=0 selects the separate launches,
and DE_PD_COOPERATIVE=1 a cooperative launch of the persistent kernel (same
bits as the default plain launch).
Stacks: the 2-layer V2-Lite stack (also against the fp64 oracle), the same
stack without draft experts, a Moonlight-style stack (sigmoid router with a
selection bias, renormalised gates), a 34-layer stack of small bf16 layers
(two launches of at most 32 layers), and the full 26-layer V2-Lite stack.
"""
import os
from dataclasses import replace

import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from workloads import configs, gen
from workloads import gpu as wgpu

from gpu_support import require_gpu
from support import OracleModel, rel_err

pytestmark = pytest.mark.gpu

V2_SMALL = configs.scaled_model(configs.CFG4, n_moe_layers=2, vocab=8192, dense_inter=1408,
                                k_draft=2, name="v2lite-stack-small")
MOON_SMALL = configs.scaled_model(configs.CFG4, n_moe_layers=3, vocab=4096, dense_inter=1408,
                                  k_draft=3, moe=replace(configs.CFG3, cfg_id=43),
                                  name="moonlight-stack-small")
# Small bf16 layers (H 512, 16 experts of I 256, top-2, 2 x 256 shared, draft 256)
# in a stack longer than one launch holds.
DEEP = configs.scaled_model(
    configs.CFG4, n_moe_layers=34, vocab=2048, dense_inter=512, k_draft=3,
    moe=replace(configs.CFG2, cfg_id=44, hidden=512, n_experts=16, top_k=2, inter=256,
                shared_each=256, draft_inter=256),
    name="deep-small-stack")


@pytest.fixture(autouse=True)
def _restore_env():
    require_gpu()
    names = ("DE_DRAFT_PERSISTENT", "DE_PD_COOPERATIVE")
    old = {n: os.environ.get(n) for n in names}
    yield
    for n, v in old.items():
        if v is None:
            os.environ.pop(n, None)
        else:
            os.environ[n] = v


def device_model(model, max_block, no_draft=False):
    m = model.moe
    t = wgpu.model_tensors(model)
    if no_draft:
        for lw in t["layers"]:
            lw["draft"] = None
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    return de.DeviceModel(desc, t["layers"], model.vocab, t["emb"], t["lm"], t["dense"],
                          model.dense_inter, de.DE_BF16, model.eps, m.gamma, max_block)


def both_paths(fn):
    out = []
    for flag in ("1", "0"):
        os.environ["DE_DRAFT_PERSISTENT"] = flag
        out.append(fn())
        torch.cuda.synchronize()
    return out


def draft_and_step(model, dm, tokens):
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k

    def run():
        res = []
        for t in tokens:
            lg = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
            am = torch.empty(1, dtype=torch.int32, device="cuda")
            dm.forward(torch.tensor([t], dtype=torch.int32, device="cuda"), de.DE_DRAFT, lg, am)
            res.append((lg, am))
        block = dm.new_block(K, tokens[0])
        amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
        out = torch.empty(2, dtype=torch.int32, device="cuda")
        nu = torch.empty(L, dtype=torch.int32, device="cuda")
        pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
        dm.spec_step(block, amax, out, nu, pred)
        # A draft forward right after a verify pass (another block length on
        # the same workspace).
        lg2 = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
        dm.forward(block[:1], de.DE_DRAFT, lg2)
        assert de.de_model_status(dm.model, dm.ws) == 0
        return res, block, amax, out, nu, pred, lg2

    (r1, *s1), (r0, *s0) = both_paths(run)
    for (l1, m1), (l0, m0) in zip(r1, r0):
        assert torch.equal(l1, l0) and torch.equal(m1, m0)
    for a, b in zip(s1, s0):
        assert torch.equal(a, b)
    return r1, s1


@pytest.mark.parametrize("name,model,no_draft", [
    ("v2lite-2layer", V2_SMALL, False),
    ("v2lite-2layer-no-draft-expert", V2_SMALL, True),
    ("moonlight-3layer", MOON_SMALL, False),
    ("small-34layer", DEEP, False),
], ids=lambda v: v if isinstance(v, str) else "")
def test_persistent_draft_equals_separate_launches(name, model, no_draft):
    dm = device_model(model, model.k_draft + 1, no_draft)
    toks = [gen.start_token(model, redraw=r) for r in range(3)]
    (res, (block, amax, out, nu, pred, lg2)) = draft_and_step(model, dm, toks)
    print(f"{name}: drafts {block.cpu().tolist()} n,bonus {out.cpu().tolist()}", flush=True)
    if name == "v2lite-2layer":
        # Against the fp64 oracle: the first position's draft logits, and the
        # drafter's routing at every draft position of the step.
        om = OracleModel(model)
        from oracle import decode
        tr = decode.Trace()
        want = decode.forward(om.weights, [toks[0]], "draft", tr)
        err = rel_err(res[0][0].cpu().numpy(), want)
        print(f"{name}: draft logits rel err vs oracle {err:.2e}", flush=True)
        assert err < 1e-4
        np.testing.assert_array_equal(pred[0].cpu().numpy(),
                                      np.stack([np.asarray(i)[0] for i in tr.idx]))
    del dm
    torch.cuda.empty_cache()


def test_persistent_draft_full_stack_equals_separate_launches():
    model = configs.CFG4
    dm = device_model(model, model.k_draft + 1)
    toks = [gen.start_token(model, redraw=r) for r in range(2)]
    _, (block, amax, out, nu, pred, lg2) = draft_and_step(model, dm, toks)
    print(f"full stack: drafts {block.cpu().tolist()} n,bonus {out.cpu().tolist()}", flush=True)
    del dm
    torch.cuda.empty_cache()


def test_cooperative_launch_equals_plain_launch():
    """The persistent kernel launched cooperatively (DE_PD_COOPERATIVE=1) and
    plainly (the default) writes the same bits: a whole step and the draft
    logits of a second start token."""
    model = V2_SMALL
    dm = device_model(model, model.k_draft + 1)
    os.environ["DE_DRAFT_PERSISTENT"] = "1"
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    res = []
    for coop in ("0", "1"):
        os.environ["DE_PD_COOPERATIVE"] = coop
        block = dm.new_block(K, gen.start_token(model))
        amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
        out = torch.empty(2, dtype=torch.int32, device="cuda")
        nu = torch.empty(L, dtype=torch.int32, device="cuda")
        pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
        dm.spec_step(block, amax, out, nu, pred)
        lg = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
        dm.forward(torch.tensor([gen.start_token(model, redraw=1)], dtype=torch.int32,
                                device="cuda"), de.DE_DRAFT, lg)
        torch.cuda.synchronize()
        assert de.de_model_status(dm.model, dm.ws) == 0
        res.append((block, amax, out, nu, pred, lg))
    for a, b in zip(*res):
        assert torch.equal(a, b)
    del dm
    torch.cuda.empty_cache()


def test_draft_pass_phase_timer():
    """DE_PHASE_DRAFT_PASS brackets the persistent launch of a draft forward
    (and nothing when the separate launches run)."""
    model = V2_SMALL
    dm = device_model(model, model.k_draft + 1)
    tok = torch.tensor([gen.start_token(model)], dtype=torch.int32, device="cuda")
    lg = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
    os.environ["DE_DRAFT_PERSISTENT"] = "1"
    e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for ev in e:
        ev.record()  # torch reads only events it has recorded once
    e[0].record()
    de.de_time_next_phase(de.DE_PHASE_DRAFT_PASS, e[1], e[2])
    dm.forward(tok, de.DE_DRAFT, lg)
    e[3].record()
    torch.cuda.synchronize()
    inner = e[1].elapsed_time(e[2])
    outer = e[0].elapsed_time(e[3])
    print(f"draft pass {1e3 * inner:.1f} us of a {1e3 * outer:.1f} us forward", flush=True)
    assert 0.0 < inner < outer
    del dm
    torch.cuda.empty_cache()
