"""The stacked model's draft-then-verify step on the GPU against the oracle.

Small stacks (3 tiny fp32 layers; 2 V2-Lite-shaped layers) are compared with
the fp64 oracle step: drafts, target argmax, accept length, bonus, the verify
union size of every layer and the drafter's predicted experts bit-exact, the
verify logits within 1e-4 relative.  The full 26-layer V2-Lite stack
(102400-vocab head, K = 8) is checked through properties that hold at any
size: the emitted tokens equal greedy target decoding, and a step is
deterministic.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

from support import OracleModel, rel_err
from workloads import configs
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu

# A tiny fp32 stack whose drafter (gamma 6) often disagrees with the target,
# so the start tokens below give accept lengths 4, 1 and 2 of K = 4.
TINY = configs.scaled_model(configs.CFG4, n_moe_layers=3, vocab=1000, dense_inter=256, k_draft=4,
                            moe=replace(configs.CFG1, cfg_id=41, gamma=6.0), name="tiny-stack")
V2_SMALL = configs.scaled_model(configs.CFG4, n_moe_layers=2, vocab=8192, dense_inter=1408,
                                k_draft=2, name="v2lite-stack-small")
SMALL = [("tiny-3layer-K4-a", TINY, 0), ("tiny-3layer-K4-b", TINY, 3),
         ("tiny-3layer-K4-c", TINY, 6), ("v2lite-2layer-K2", V2_SMALL, 0)]


def device_model(model: configs.ModelCfg, max_block: int):
    import paper_2607_24434_amd as de
    m = model.moe
    t = wgpu.model_tensors(model)
    desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter, m.draft_inter,
                        m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
    return de.DeviceModel(desc, t["layers"], model.vocab, t["emb"], t["lm"], t["dense"],
                          model.dense_inter, de.DE_BF16, model.eps, m.gamma, max_block)


_ORACLES: dict = {}
_DEVICE: dict = {}


@pytest.mark.parametrize("name,model,redraw0", SMALL, ids=[s[0] for s in SMALL])
def test_spec_step_matches_oracle(name, model, redraw0):
    import paper_2607_24434_amd as de
    K = model.k_draft
    L = model.n_moe_layers
    k = model.moe.top_k
    if model.name not in _ORACLES:
        _ORACLES[model.name] = OracleModel(model)
    om = _ORACLES[model.name]
    c, drafts, n, bonus, t, traces = om.gapped_step(K, redraw0=redraw0)
    print(f"{name}: start {c} drafts {drafts} n {n} bonus {bonus}", flush=True)
    if model.name not in _DEVICE:
        _DEVICE.clear()
        _DEVICE[model.name] = device_model(model, K + 1)
    dm = _DEVICE[model.name]
    block = dm.new_block(K, c)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
    dm.spec_step(block, amax, out, nu, pred)
    torch.cuda.synchronize()
    assert block[1:].cpu().tolist() == drafts
    assert amax.cpu().tolist() == [int(v) for v in t]
    assert out.cpu().tolist() == [n, bonus]
    ver = traces[-1]
    assert nu.cpu().tolist() == [len(set(np.asarray(i).ravel().tolist())) for i in ver.idx]
    want_pred = np.stack([np.stack([np.asarray(i)[0] for i in tr.idx]) for tr in traces[:K]])
    np.testing.assert_array_equal(pred.cpu().numpy(), want_pred)
    # Verify logits through the forward call on the same block.
    logits = torch.empty(K + 1, model.vocab, dtype=torch.float32, device="cuda")
    am2 = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    dm.forward(block, de.DE_TARGET, logits, am2)
    torch.cuda.synchronize()
    err = rel_err(logits.cpu().numpy(), ver.logits)
    print(f"{name}: verify logits rel err {err:.2e}", flush=True)
    assert err < 1e-4
    assert torch.equal(am2, amax)
    # Draft logits of the first position.
    dl = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
    dm.forward(block[:1], de.DE_DRAFT, dl)
    torch.cuda.synchronize()
    assert rel_err(dl.cpu().numpy(), traces[0].logits) < 1e-4


@pytest.fixture(scope="module")
def full_model():
    model = configs.CFG4
    dm = device_model(model, model.k_draft + 1)
    yield model, dm
    del dm
    torch.cuda.empty_cache()


def test_full_stack_spec_step_emits_greedy_tokens(full_model):
    from workloads import gen
    model, dm = full_model
    K, L = model.k_draft, model.n_moe_layers
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.empty(K, L, model.moe.top_k, dtype=torch.int32, device="cuda")
    for r in range(3):
        c = gen.start_token(model, redraw=r)
        block = dm.new_block(K, c)
        dm.spec_step(block, amax, out, nu, pred)
        torch.cuda.synchronize()
        n, bonus = out.cpu().tolist()
        emitted = block[1:n + 1].cpu().tolist() + [bonus]
        toks = torch.zeros(n + 2, dtype=torch.int32, device="cuda")
        toks[0] = c
        dm.greedy(toks)
        torch.cuda.synchronize()
        print(f"start {c}: n {n} emitted {emitted} union {nu.cpu().tolist()}", flush=True)
        assert toks[1:].cpu().tolist() == emitted
        assert 0 <= n <= K
        u = nu.cpu().numpy()
        assert np.all(u >= model.moe.top_k) and np.all(u <= min(model.moe.n_experts, (K + 1) * 6))
        p = pred.cpu().numpy()
        assert p.min() >= 0 and p.max() < model.moe.n_experts
        assert all(len(set(row.tolist())) == model.moe.top_k for row in p.reshape(-1, 6))


def test_full_stack_step_is_deterministic(full_model):
    from workloads import gen
    model, dm = full_model
    K = model.k_draft
    res = []
    for _ in range(2):
        block = dm.new_block(K, gen.start_token(model, redraw=7))
        amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
        out = torch.empty(2, dtype=torch.int32, device="cuda")
        nu = torch.empty(model.n_moe_layers, dtype=torch.int32, device="cuda")
        dm.spec_step(block, amax, out, nu)
        torch.cuda.synchronize()
        res.append((block.cpu().tolist(), amax.cpu().tolist(), out.cpu().tolist(), nu.cpu().tolist()))
    assert res[0] == res[1]


_CHAIN: dict = {}


def _chain_model():
    """The 2-layer V2-Lite stack for blocks of up to 64 positions, with its tensors."""
    if "dm" not in _CHAIN:
        import paper_2607_24434_amd as de
        model = V2_SMALL
        m = model.moe
        t = wgpu.model_tensors(model)
        desc = de.make_desc(m.hidden, m.n_experts, m.top_k, m.inter, m.shared_inter,
                            m.draft_inter, m.score_func, m.norm_topk, m.routed_scale, m.wdtype)
        _CHAIN.update(t=t, desc=desc, dm=de.DeviceModel(
            desc, t["layers"], model.vocab, t["emb"], t["lm"], t["dense"], model.dense_inter,
            de.DE_BF16, model.eps, m.gamma, 64))
    return _CHAIN["t"], _CHAIN["desc"], _CHAIN["dm"]


@pytest.mark.parametrize("mode", ["target", "draft"])
@pytest.mark.parametrize("T", [4, 8, 16, 64])
def test_chained_forward_equals_layer_calls(T, mode):
    """The stacked forward chains its launches (each combine also computes the
    next layer's router logits, in blocks that all read the position's
    residual row while one of them writes the output row).  It must give the
    same bits as the same stack run through the public layer calls one by
    one, at block lengths whose blocks of one position can share an XCD."""
    import paper_2607_24434_amd as de
    t, desc, dm = _chain_model()
    model, m = V2_SMALL, V2_SMALL.moe
    H, V = m.hidden, model.vocab
    dmode = de.DE_TARGET if mode == "target" else de.DE_DRAFT
    toks = torch.from_numpy(np.random.default_rng(T).integers(0, V, T).astype(np.int32)).cuda()
    chained = torch.empty(T, V, dtype=torch.float32, device="cuda")
    dm.forward(toks, dmode, chained)
    assert de.de_model_status(dm.model, dm.ws) == 0
    # The same stack, one public call per stage, ping-pong buffers.
    h = [torch.empty(T, H, dtype=torch.float32, device="cuda") for _ in range(2)]
    n = [torch.empty(T, H, dtype=torch.float32, device="cuda") for _ in range(2)]
    de.de_embed_gather(T, H, V, toks, t["emb"], h[0], n[0], model.eps)
    dws = torch.zeros(de.de_dense_workspace_bytes(T, H, model.dense_inter), dtype=torch.uint8,
                      device="cuda")
    de.de_dense_swiglu(T, H, model.dense_inter, de.DE_BF16, n[0], t["dense"], h[1], dws,
                       epi=de.make_epilogue(residual=h[0], normed=n[1], eps=model.eps))
    cur = 1
    ws = de.workspace(desc, T)
    stride = m.expert_bytes()
    for lw in t["layers"]:
        tab = de.make_table(lw["routed"], stride, None, m.n_experts)
        epi = de.make_epilogue(residual=h[cur], normed=n[1 - cur], eps=model.eps)
        if mode == "target":
            de.de_verify_layer(desc, T, n[cur], lw["router"], lw["bias"], tab, lw["shared"],
                               h[1 - cur], ws=ws, epi=epi)
        else:
            de.de_draft_layer(desc, T, n[cur], lw["router"], lw["bias"], tab, lw["shared"],
                              lw["draft"], m.gamma, h[1 - cur], None, None, ws, epi=epi)
        cur = 1 - cur
    calls = torch.empty(T, V, dtype=torch.float32, device="cuda")
    de.de_lm_head(T, H, V, n[cur], t["lm"], calls)
    torch.cuda.synchronize()
    assert de.de_layer_status(ws) == 0
    assert torch.equal(chained, calls)


def test_full_stack_step_matches_oracle(full_model):
    """The full-size step (dense layer 0 with I = 10944, 26 V2-Lite MoE layers,
    K = 8, 102400-vocab head) against the fp64 oracle's step from the same
    start token, stored by tests/golden/make_cfg4_step.py (the oracle alone;
    about 3 minutes per candidate start token on the CPU).  Drafts, target
    argmax, n, bonus, every layer's verify union size and the drafter's top-k
    in every layer at every draft position are exact; sampled logits (each
    row's 8 largest entries and 24 seeded columns) of the verify pass and of
    the first draft position are within 1e-4 of the sample's largest
    magnitude."""
    import json
    import os
    import paper_2607_24434_amd as de
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "cfg4_step.json")))
    model, dm = full_model
    K, L, k = model.k_draft, model.n_moe_layers, model.moe.top_k
    assert g["k_draft"] == K and g["model"] == model.name
    block = dm.new_block(K, g["start"])
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    nu = torch.empty(L, dtype=torch.int32, device="cuda")
    pred = torch.empty(K, L, k, dtype=torch.int32, device="cuda")
    dm.spec_step(block, amax, out, nu, pred)
    torch.cuda.synchronize()
    print(f"start {g['start']}: drafts {block[1:].cpu().tolist()} n,bonus {out.cpu().tolist()}",
          flush=True)
    assert block[1:].cpu().tolist() == g["drafts"]
    assert amax.cpu().tolist() == g["target_argmax"]
    assert out.cpu().tolist() == [g["n"], g["bonus"]]
    assert nu.cpu().tolist() == g["n_union"]
    np.testing.assert_array_equal(pred.cpu().numpy(), np.asarray(g["pred_idx"]))

    def check(logits, sample, what):
        lg = logits.cpu().numpy()
        worst = 0.0
        for j, row in enumerate(sample):
            got = lg[j, row["cols"]]
            want = np.asarray(row["vals"])
            worst = max(worst, float(np.max(np.abs(got - want)) / np.max(np.abs(want))))
        print(f"{what}: sampled logits rel err {worst:.2e}", flush=True)
        assert worst < 1e-4

    lv = torch.empty(K + 1, model.vocab, dtype=torch.float32, device="cuda")
    dm.forward(block, de.DE_TARGET, lv)
    ld = torch.empty(1, model.vocab, dtype=torch.float32, device="cuda")
    dm.forward(block[:1], de.DE_DRAFT, ld)
    torch.cuda.synchronize()
    check(lv, g["verify_logits"], "verify")
    check(ld, g["draft0_logits"], "draft position 0")
