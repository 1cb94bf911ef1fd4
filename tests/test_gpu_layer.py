"""GPU parity of one MoE layer through the C ABI against the fp64 oracle.

Integer results (top-k ids, the union, token lists, pair positions) must be
bit-exact; they are decided on inputs whose selection keys are at least 1e-4
apart, far above the fp32 logit error (about 1e-6).  Floating results:

* layer outputs: max|y - y*| / max|y*| <= 1e-5 for fp32 weights and <= 1e-4
  for bf16 weights.  bf16 weights are upconverted exactly and activations
  stay fp32, so only fp32 summation order differs from the fp64 oracle: the
  relative error of a length-n fp32 dot is bounded by about n * 2^-24
  (1.2e-4 for n = 2048) and is about 1e-6 in practice.  Both bounds are well
  inside the 1e-2 (bf16) / 1e-5 (fp32) acceptance of the method.
* gates: |g - g*| <= 2e-6 + 1e-5 |g*| (fp32 softmax / sigmoid).
"""
import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from oracle import moe
from workloads import configs, gen, rng
from workloads import gpu as wgpu

from gpu_support import DevLayer, f32, i32, layer_pair, require_gpu, verify_outputs
from support import OracleLayer, gapped_x, rel_err

pytestmark = pytest.mark.gpu

CASES = [
    ("cfg1-T5", configs.CFG1, 5),
    ("cfg2-T9", configs.CFG2, 9),
    ("cfg3-T5", configs.CFG3, 5),
    ("cfg3-T9", configs.CFG3, 9),
    ("cfg3-T17", configs.CFG3, 17),
    # The largest block the ABI takes: 64-bit position masks up to bit 63,
    # positions read from global memory, eight positions per selecting wave.
    ("cfg1-T64", configs.CFG1, 64),
    ("cfg2-T64", configs.CFG2, 64),
]
IDS = [c[0] for c in CASES]


def y_tol(cfg):
    return 1e-5 if cfg.wdtype == configs.F32 else 1e-4


def gate_close(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert np.all(np.abs(got - want) <= 2e-6 + 1e-5 * np.abs(want)), np.max(np.abs(got - want))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------------ generator

def test_gpu_fill_matches_cpu_generator():
    c2 = configs.CFG2
    dev = torch.empty(c2.expert_elems(), dtype=torch.int16, device="cuda")
    wgpu.fill_normal(dev, rng.key_for(2, 0, "routed", 0, 5), c2.weight_std)
    cpu = gen.routed_block(c2, 0, 5)
    assert np.array_equal(dev.cpu().numpy().view(np.uint16), cpu)
    c1 = configs.CFG1
    dev = torch.empty(1000, dtype=torch.float32, device="cuda")
    key = rng.key_for(1, 3, "routed", 0, 2)
    wgpu.fill_normal(dev, key, 0.02, start=777)
    assert np.array_equal(dev.cpu().numpy(), rng.normal_f32_ref(key, 1000, 0.02, start=777))


# ------------------------------------------------------------------ routing

@pytest.mark.parametrize("name,cfg,T", CASES, ids=IDS)
def test_route_topk(name, cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    idx_o, gate_o, _ = orc.route(x)
    idx = torch.empty(T, cfg.top_k, dtype=torch.int32, device="cuda")
    gate = torch.empty(T, cfg.top_k, dtype=torch.float32, device="cuda")
    de.de_route_topk(dev.desc, T, f32(x), dev.router, dev.bias, idx, gate, dev.ws(T))
    np.testing.assert_array_equal(idx.cpu().numpy(), idx_o)
    gate_close(gate.cpu().numpy(), gate_o)


def _planted_keys(r, N, k):
    """Distinct logits in [-2, 2) on a 4/N grid (exact in fp32), then equal
    pairs planted at the top, across the k-th place and at random."""
    v = (r.permutation(N) - N // 2) * (4.0 / N)
    order = np.argsort(-v, kind="stable")
    j = int(r.integers(N))
    if j != order[0]:
        v[j] = v[order[0]]
    if k < N:
        order = np.argsort(-v, kind="stable")
        v[order[k]] = v[order[k - 1]]
    a, b = r.choice(N, 2, replace=False)
    v[b] = v[a]
    return v


@pytest.mark.parametrize("N,k,score", [(33, 6, 0), (64, 6, 0), (64, 8, 1), (65, 6, 0),
                                       (128, 16, 1), (256, 8, 0), (256, 1, 1), (8, 8, 0)])
def test_route_topk_planted_ties(N, k, score):
    """Selection order with exactly equal keys: larger key first, ties to the
    lower expert id, against the oracle's stable sort.  Position t's input is
    the unit vector e_t, so its logits are router column t exactly on both
    sides.  Covers one candidate per lane (N <= 64) and more (N > 64)."""
    T, H = 5, 256
    r = np.random.default_rng(1000 * N + 10 * k + score)
    w = np.zeros((N, H), np.float32)
    for t in range(T):
        w[:, t] = _planted_keys(r, N, k)
    x = np.zeros((T, H), np.float32)
    x[np.arange(T), np.arange(T)] = 1.0
    idx_o, gate_o, _ = moe.route_topk(x, w, None, k, score, False)
    desc = de.make_desc(H, N, k, 64, 64, 64, score, 0, 1.0, de.DE_BF16)
    idx = torch.empty(T, k, dtype=torch.int32, device="cuda")
    gate = torch.empty(T, k, dtype=torch.float32, device="cuda")
    de.de_route_topk(desc, T, f32(x), f32(w), None, idx, gate, de.workspace(desc, T))
    np.testing.assert_array_equal(idx.cpu().numpy(), idx_o)
    gate_close(gate.cpu().numpy(), gate_o)


# ------------------------------------------------------------------ union

def union_case(T, k, N, seed):
    r = np.random.default_rng(seed)
    idx = np.stack([r.permutation(N)[:k] for _ in range(T)]).astype(np.int32)
    gate = r.random((T, k)).astype(np.float32)
    return idx, gate


@pytest.mark.parametrize("T,k,N,seed", [(1, 6, 64, 0), (9, 6, 64, 1), (17, 6, 64, 2), (5, 2, 8, 3),
                                        (64, 1, 64, 4), (64, 32, 256, 5), (33, 8, 16, 6),
                                        (64, 6, 64, 7), (3, 4, 4, 8)])
def test_expert_union_bit_exact(T, k, N, seed):
    idx, gate = union_case(T, k, N, seed)
    want = moe.expert_union(idx, gate)
    nu = torch.empty(1, dtype=torch.int32, device="cuda")
    uids = torch.empty(N, dtype=torch.int32, device="cuda")
    offs = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    tok = torch.empty(T * k, dtype=torch.int32, device="cuda")
    gl = torch.empty(T * k, dtype=torch.float32, device="cuda")
    pp = torch.empty(T, k, dtype=torch.int32, device="cuda")
    de.de_expert_union(T, k, N, i32(idx), f32(gate), nu, uids, offs, tok, gl, pp)
    n = want["n_union"]
    assert int(nu.item()) == n
    u = uids.cpu().numpy()
    np.testing.assert_array_equal(u[:n], want["union_ids"])
    assert (u[n:] == -1).all()
    o = offs.cpu().numpy()
    np.testing.assert_array_equal(o[:n + 1], want["offsets"])
    assert (o[n:] == T * k).all()
    np.testing.assert_array_equal(tok.cpu().numpy(), want["tok_list"])
    np.testing.assert_array_equal(gl.cpu().numpy(), want["gate_list"].astype(np.float32))
    np.testing.assert_array_equal(pp.cpu().numpy(), want["pair_pos"])


@pytest.mark.parametrize("bad", ["dup", "neg", "big"])
def test_expert_union_rejects_invalid_ids(bad):
    T, k, N = 4, 3, 16
    idx, gate = union_case(T, k, N, 11)
    if bad == "dup":
        idx[2, 2] = idx[2, 0]
    elif bad == "neg":
        idx[1, 1] = -3
    else:
        idx[3, 0] = N
    nu = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    bufs = [torch.zeros(n, dtype=torch.int32, device="cuda") for n in (N, N + 1, T * k)]
    gl = torch.zeros(T * k, dtype=torch.float32, device="cuda")
    pp = torch.zeros(T * k, dtype=torch.int32, device="cuda")
    de.de_expert_union(T, k, N, i32(idx), f32(gate), nu, bufs[0], bufs[1], bufs[2], gl, pp)
    assert int(nu.item()) == -1


# ------------------------------------------------------------------ verify layer (Eq. 4)

@pytest.mark.parametrize("name,cfg,T", CASES, ids=IDS)
def test_verify_layer(name, cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    print(f"[verify {name}] T={T}", flush=True)
    y_o, idx_o, gate_o = orc.target(x)
    uo = moe.expert_union(idx_o, gate_o)
    out = verify_outputs(dev, f32(x), T)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["idx"].cpu().numpy(), idx_o)
    gate_close(out["gate"].cpu().numpy(), gate_o)
    n = uo["n_union"]
    assert int(out["nu"].item()) == n
    np.testing.assert_array_equal(out["uids"].cpu().numpy()[:n], uo["union_ids"])
    np.testing.assert_array_equal(out["offs"].cpu().numpy()[:n + 1], uo["offsets"])
    np.testing.assert_array_equal(out["tok"].cpu().numpy(), uo["tok_list"])
    gate_close(out["glist"].cpu().numpy(), uo["gate_list"])
    np.testing.assert_array_equal(out["ppos"].cpu().numpy(), uo["pair_pos"])
    err = rel_err(out["y"].cpu().numpy(), y_o)
    print(f"[verify {name}] union={n} rel_err={err:.3e}", flush=True)
    assert err <= y_tol(cfg)


@pytest.mark.parametrize("name,cfg,T", CASES[:2], ids=IDS[:2])
def test_verify_layer_is_deterministic(name, cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    a = verify_outputs(dev, f32(x), T)["y"].clone()
    b = verify_outputs(dev, f32(x), T)["y"]
    assert torch.equal(a, b)


def test_verify_layer_epilogue_residual_and_norm():
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    T = 9
    x, _ = gapped_x(orc, T, block=0)
    y_o, _, _ = orc.target(x)
    h = gen.x_rows(cfg, T, block=7) * 3.0
    h_dev = f32(h)
    normed = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    epi = de.make_epilogue(residual=h_dev, normed=normed, eps=1e-6)
    out = verify_outputs(dev, f32(x), T, epi=epi, y=h_dev)  # residual aliases y
    want = h.astype(np.float64) + y_o
    assert rel_err(out["y"].cpu().numpy(), want) <= y_tol(cfg)
    assert rel_err(normed.cpu().numpy(), moe.rmsnorm(want, 1e-6)) <= y_tol(cfg)


def test_verify_layer_through_permuted_slot_table_is_bitwise_equal():
    # Experts stored in a permuted slot pool, found through slot_of_expert.
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    T = 9
    x, _ = gapped_x(orc, T, block=0)
    ref = verify_outputs(dev, f32(x), T)["y"].clone()
    perm = np.random.default_rng(5).permutation(cfg.n_experts)
    pool = torch.empty_like(dev.routed)
    pool[torch.from_numpy(perm).cuda().long()] = dev.routed   # expert e in slot perm[e]
    table = de.make_table(pool, dev.stride, i32(perm), cfg.n_experts)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    de.de_verify_layer(dev.desc, T, f32(x), dev.router, dev.bias, table, dev.shared, y, ws=dev.ws(T))
    assert torch.equal(y, ref)
    del pool


# ------------------------------------------------------------------ grouped SwiGLU from a given union

@pytest.mark.parametrize("name,cfg,T", CASES[:3], ids=IDS[:3])
def test_grouped_swiglu_from_oracle_union(name, cfg, T):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=0)
    y_o, idx_o, gate_o = orc.target(x)
    u = moe.expert_union(idx_o, gate_o)
    N = cfg.n_experts
    uids = np.full(N, -1, np.int32)
    uids[:u["n_union"]] = u["union_ids"]
    offs = np.full(N + 1, T * cfg.top_k, np.int32)
    offs[:u["n_union"] + 1] = u["offsets"]
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    de.de_grouped_swiglu(dev.desc, T, f32(x), dev.table, i32([u["n_union"]]), i32(uids), i32(offs),
                         i32(u["tok_list"]), f32(u["gate_list"]), i32(u["pair_pos"]), dev.shared, y,
                         dev.ws(T))
    assert rel_err(y.cpu().numpy(), y_o) <= y_tol(cfg)


# ------------------------------------------------------------------ draft layer (Eq. 5)

DRAFT_CASES = [("cfg1", configs.CFG1, 1), ("cfg2", configs.CFG2, 1), ("cfg3", configs.CFG3, 1),
               ("cfg1-T5", configs.CFG1, 5)]


@pytest.mark.parametrize("name,cfg,T", DRAFT_CASES, ids=[c[0] for c in DRAFT_CASES])
@pytest.mark.parametrize("variant", ["draft", "no-draft", "gamma0.5"])
def test_draft_layer(name, cfg, T, variant):
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=1)
    gamma = 0.5 if variant == "gamma0.5" else cfg.gamma
    with_draft = variant != "no-draft"
    y_o, idx_o, gate_o = orc.draft_out(x, gamma=gamma, with_draft=with_draft)
    y = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    pidx = torch.empty(T, cfg.top_k, dtype=torch.int32, device="cuda")
    pgate = torch.empty(T, cfg.top_k, dtype=torch.float32, device="cuda")
    de.de_draft_layer(dev.desc, T, f32(x), dev.router, dev.bias, dev.table, dev.shared,
                      dev.draft if with_draft else None, gamma, y, pidx, pgate, dev.ws(T))
    np.testing.assert_array_equal(pidx.cpu().numpy(), idx_o)
    gate_close(pgate.cpu().numpy(), gate_o)
    assert rel_err(y.cpu().numpy(), y_o) <= y_tol(cfg)


@pytest.mark.parametrize("name,cfg,T", DRAFT_CASES + [("cfg2-T5", configs.CFG2, 5)],
                         ids=[c[0] for c in DRAFT_CASES] + ["cfg2-T5"])
def test_draft_layer_without_predictions(name, cfg, T):
    """Without the predicted lists the layer may select only the leading
    expert (when no top-k renormalisation needs the rest): the output equals
    the oracle's and, bit for bit, that of the call with the lists."""
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, T, block=1)
    y_o, _, _ = orc.draft_out(x)
    ws = dev.ws(T)
    y0 = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    y1 = torch.empty_like(y0)
    pidx = torch.empty(T, cfg.top_k, dtype=torch.int32, device="cuda")
    de.de_draft_layer(dev.desc, T, f32(x), dev.router, dev.bias, dev.table, dev.shared, dev.draft,
                      cfg.gamma, y0, None, None, ws)
    de.de_draft_layer(dev.desc, T, f32(x), dev.router, dev.bias, dev.table, dev.shared, dev.draft,
                      cfg.gamma, y1, pidx, None, ws)
    assert rel_err(y0.cpu().numpy(), y_o) <= y_tol(cfg)
    assert torch.equal(y0, y1)


@pytest.mark.parametrize("name,cfg", [("cfg2", configs.CFG2), ("cfg3", configs.CFG3)],
                         ids=["cfg2", "cfg3"])
@pytest.mark.parametrize("variant", ["draft", "no-draft", "in-place"])
def test_single_draft_layer_persistent_equals_separate(name, cfg, variant, monkeypatch):
    """A one-position draft layer runs as one persistent launch unless
    DE_PD_SINGLE=0: both paths write the same bits (output, RMSNorm epilogue,
    predicted lists and gates, the router logits left in the workspace)."""
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, 1, block=2)
    h = gen.x_rows(cfg, 1, block=6)
    ws = dev.ws(1)
    draft = None if variant == "no-draft" else dev.draft
    res = []
    for flag in ("1", "0"):
        monkeypatch.setenv("DE_PD_SINGLE", flag)
        res_in = f32(h)
        y = res_in if variant == "in-place" else torch.empty(1, cfg.hidden, dtype=torch.float32,
                                                             device="cuda")
        normed = torch.empty(1, cfg.hidden, dtype=torch.float32, device="cuda")
        pidx = torch.empty(1, cfg.top_k, dtype=torch.int32, device="cuda")
        pgate = torch.empty(1, cfg.top_k, dtype=torch.float32, device="cuda")
        z = torch.empty(1, cfg.n_experts, dtype=torch.float32, device="cuda")
        epi = de.make_epilogue(residual=res_in, normed=normed)
        de.de_draft_layer(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table, dev.shared, draft,
                          cfg.gamma, y, pidx, pgate, ws, epi=epi)
        de.de_layer_router_logits(dev.desc, 1, ws, z)
        torch.cuda.synchronize()
        assert de.de_layer_status(ws) == 0
        res.append((y.clone(), normed, pidx, pgate, z))
    for a, b in zip(*res):
        assert torch.equal(a, b)
    y_o, idx_o, _ = orc.draft_out(x, with_draft=draft is not None)
    np.testing.assert_array_equal(res[0][2].cpu().numpy(), idx_o)
    assert rel_err(res[0][0].cpu().numpy() - h, y_o) <= y_tol(cfg)


def test_draft_layer_zero_draft_expert_equals_no_draft():
    cfg = configs.CFG2
    orc, dev = layer_pair(cfg)
    x, _ = gapped_x(orc, 1, block=1)
    ws = dev.ws(1)
    y0 = torch.empty(1, cfg.hidden, dtype=torch.float32, device="cuda")
    y1 = torch.empty_like(y0)
    zero = torch.zeros_like(dev.draft)
    de.de_draft_layer(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table, dev.shared, None, 1.0,
                      y0, None, None, ws)
    de.de_draft_layer(dev.desc, 1, f32(x), dev.router, dev.bias, dev.table, dev.shared, zero, 1.0,
                      y1, None, None, ws)
    assert torch.equal(y0, y1)


# ------------------------------------------------------------------ dense layer, norm, embedding

def test_dense_swiglu_with_epilogue():
    H, I, T = 2048, 10944, 9
    key = rng.key_for(4, 0, "dense", 0, 0)
    w_cpu = rng.normal_bf16(key, 3 * I * H, 0.02)
    w = torch.empty(3 * I * H, dtype=torch.int16, device="cuda")
    wgpu.fill_normal(w, key, 0.02)
    x = gen.x_rows(configs.CFG2, T, block=3)
    h = gen.x_rows(configs.CFG2, T, block=4)
    g, u, d = moe.split_expert(w_cpu, I, H)
    want = h.astype(np.float64) + moe.swiglu(x, g, u, d)
    y = f32(h)
    normed = torch.empty(T, H, dtype=torch.float32, device="cuda")
    ws = torch.empty(de.de_dense_workspace_bytes(T, H, I), dtype=torch.uint8, device="cuda")
    de.de_dense_swiglu(T, H, I, de.DE_BF16, f32(x), w, y, ws,
                       epi=de.make_epilogue(residual=y, normed=normed, eps=1e-6))
    assert rel_err(y.cpu().numpy(), want) <= 1e-4
    assert rel_err(normed.cpu().numpy(), moe.rmsnorm(want)) <= 1e-4


def test_rmsnorm_and_embedding():
    V, H, T = 1000, 256, 7
    key = rng.key_for(1, 0, "emb", 0, 0)
    emb = wgpu.fill_normal(torch.empty(V * H, dtype=torch.int16, device="cuda"), key, 1.0)
    emb_cpu = moe.to_f64(rng.normal_bf16(key, V * H, 1.0)).reshape(V, H)
    toks = np.array([0, 999, 5, 5, 123, 400, 998], np.int32)
    h = torch.empty(T, H, dtype=torch.float32, device="cuda")
    hn = torch.empty_like(h)
    de.de_embed_gather(T, H, V, i32(toks), emb, h, hn, 1e-6)
    np.testing.assert_array_equal(h.cpu().numpy(), emb_cpu[toks].astype(np.float32))
    assert rel_err(hn.cpu().numpy(), moe.rmsnorm(emb_cpu[toks])) <= 1e-6
    out = torch.empty_like(h)
    de.de_rmsnorm(T, H, h, 1e-6, out)
    assert rel_err(out.cpu().numpy(), moe.rmsnorm(emb_cpu[toks])) <= 1e-6


# ------------------------------------------------------------------ LM head and acceptance

@pytest.mark.parametrize("V,H,T", [(1000, 256, 5), (102400, 2048, 9), (1000, 256, 1)])
def test_lm_head_and_argmax(V, H, T):
    key = rng.key_for(9, 0, "lm", 0, 0)
    w = wgpu.fill_normal(torch.empty(V * H, dtype=torch.int16, device="cuda"), key, 0.02)
    w64 = moe.to_f64(rng.normal_bf16(key, V * H, 0.02)).reshape(V, H)
    x = moe.rmsnorm(gen.x_rows(configs.CFG2 if H == 2048 else configs.CFG1, T, block=5)).astype(np.float32)
    want = x.astype(np.float64) @ w64.T
    logits = torch.empty(T, V, dtype=torch.float32, device="cuda")
    de.de_lm_head(T, H, V, f32(x), w, logits)
    got = logits.cpu().numpy()
    assert rel_err(got, want) <= 1e-4
    amax = torch.empty(T, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    de.de_accept_len(T - 1, V, logits, i32(np.zeros(max(T - 1, 1), np.int32)), amax, out,
                     de.accept_workspace(T - 1, V))
    top2 = np.sort(want, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 1e-4
    np.testing.assert_array_equal(amax.cpu().numpy()[clear], np.argmax(want, axis=1)[clear])


@pytest.mark.parametrize("K", [0, 1, 4, 8, 16])
@pytest.mark.parametrize("V", [1000, 1003, 102400])
def test_accept_len_planted_prefix(K, V):
    r = np.random.default_rng(1000 * K + V)
    logits = r.standard_normal((K + 1, V)).astype(np.float32)
    t = np.argmax(logits, axis=1)
    lg = f32(logits)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    ws = de.accept_workspace(K, V)
    for m in range(K + 1):
        drafts = t[:K].copy()
        if m < K:
            drafts[m] = (drafts[m] + 1) % V
        n_o, bonus_o, t_o = moe.accept_len(logits, drafts)
        de.de_accept_len(K, V, lg, i32(drafts) if K else None, amax, out, ws)
        o = out.cpu().numpy()
        assert (int(o[0]), int(o[1])) == (n_o, bonus_o) == (m, int(t[m]))
        np.testing.assert_array_equal(amax.cpu().numpy(), t_o)


@pytest.mark.parametrize("V", [1003, 8192])
def test_accept_len_more_drafts_than_threads(V):
    """K = 300 drafts: the first mismatch is found by a block of 256 threads
    over strided shares, so mismatches on either side of 256 are checked."""
    K = 300
    r = np.random.default_rng(V)
    logits = r.standard_normal((K + 1, V)).astype(np.float32)
    t = np.argmax(logits, axis=1)
    lg = f32(logits)
    amax = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    ws = de.accept_workspace(K, V)
    for m in (0, 1, 255, 256, 257, 299, 300):
        drafts = t[:K].copy()
        if m < K:
            drafts[m] = (drafts[m] + 1) % V
            drafts[min(m + 7, K - 1)] = (drafts[min(m + 7, K - 1)] + 1) % V
        n_o, bonus_o, t_o = moe.accept_len(logits, drafts)
        de.de_accept_len(K, V, lg, i32(drafts), amax, out, ws)
        o = out.cpu().numpy()
        assert (int(o[0]), int(o[1])) == (n_o, bonus_o) == (m, int(t[m]))
        np.testing.assert_array_equal(amax.cpu().numpy(), t_o)


def test_argmax_ties_go_to_lowest_index():
    V = 4096
    logits = np.zeros((3, V), np.float32)
    logits[0, [17, 900, 4000]] = 5.0
    logits[1, :] = 1.0
    logits[2, [V - 1]] = 2.0
    amax = torch.empty(3, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    de.de_accept_len(2, V, f32(logits), i32([17, 0]), amax, out, de.accept_workspace(2, V))
    np.testing.assert_array_equal(amax.cpu().numpy(), [17, 0, V - 1])
    assert out.cpu().tolist() == [2, V - 1]


@pytest.mark.parametrize("V", [4096, 4099])
def test_single_row_argmax_ties_and_nan(V):
    """K = 0 (one row, the draft loop's case): ties go to the lowest index and
    a NaN counts as -infinity, in 16-byte loads (V = 4096) and element loads
    (V = 4099); an all-NaN row gives index 0."""
    logits = np.zeros((1, V), np.float32)
    logits[0, 3] = np.nan
    logits[0, [11, 4000, V - 1]] = 7.0
    amax = torch.empty(1, dtype=torch.int32, device="cuda")
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    ws = de.accept_workspace(0, V)
    de.de_accept_len(0, V, f32(logits), None, amax, out, ws)
    assert int(amax.item()) == 11 and out.cpu().tolist() == [0, 11]
    nan_row = np.full((1, V), np.nan, np.float32)
    de.de_accept_len(0, V, f32(nan_row), None, amax, out, ws)
    assert int(amax.item()) == 0 and out.cpu().tolist() == [0, 0]
