"""Pins of the CPU oracle against what the paper and mathematics fix.

Every check here is independent of the oracle's own code: brute force in
pure Python, torch library routines in fp64, closed forms, invariants and
special cases.  A plausible slip in the oracle (a dropped term, a transposed
operand, a wrong index or sign, an off-by-one in acceptance) fails at least
one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decode, moe

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_layer(rng, H=24, N=7, I=10, n_shared=2, Id=6, router_std=0.5):
    w_router = rng.normal(0, router_std, (N, H))
    experts = [(rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (H, I)))
               for _ in range(N)]
    shared = [(rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (H, I)))
              for _ in range(n_shared)]
    draft = (rng.normal(0, 0.3, (Id, H)), rng.normal(0, 0.3, (Id, H)), rng.normal(0, 0.3, (H, Id)))
    return w_router, experts, shared, draft


def t64(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def torch_expert(x, g, u, d):
    """Library form of one SwiGLU expert (torch fp64)."""
    x = t64(np.atleast_2d(x))
    return (F.silu(x @ t64(g).T) * (x @ t64(u).T) @ t64(d).T).numpy()


# ------------------------------------------------------------------ P8 single expert

def test_swiglu_matches_torch_library_nonsquare():
    rng = np.random.default_rng(1)
    H, I = 13, 5  # non-square so a transposed operand cannot pass
    g, u, d = rng.normal(size=(I, H)), rng.normal(size=(I, H)), rng.normal(size=(H, I))
    x = rng.normal(size=(4, H))
    np.testing.assert_allclose(moe.swiglu(x, g, u, d), torch_expert(x, g, u, d), rtol=1e-13, atol=1e-13)


def test_silu_closed_form_values():
    # silu(0) = 0, silu(v) - silu(-v) = v, silu(large) ~ v
    v = np.array([0.0, 1.0, -1.0, 3.0, 40.0, -40.0])
    s = moe.silu(v)
    assert s[0] == 0.0
    assert abs((s[1] - s[2]) - 1.0) < 1e-15
    assert abs(s[1] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15
    assert abs(s[4] - 40.0) < 1e-12 and abs(s[5]) < 1e-15


# ------------------------------------------------------------------ P7 routing vs torch.topk

@pytest.mark.parametrize("score_func,norm", [(moe.SOFTMAX, False), (moe.SOFTMAX, True),
                                             (moe.SIGMOID, True), (moe.SIGMOID, False)])
def test_route_topk_matches_torch(score_func, norm):
    rng = np.random.default_rng(7 + score_func + 2 * norm)
    T, H, N, k = 11, 32, 16, 5
    x = rng.normal(size=(T, H))
    w = rng.normal(0, 0.4, (N, H))
    bias = rng.normal(0, 0.3, N) if score_func == moe.SIGMOID else None
    idx, gate, _ = moe.route_topk(x, w, bias, k, score_func, norm, routed_scale=1.7)
    z = t64(x) @ t64(w).T
    if score_func == moe.SOFTMAX:
        score = torch.softmax(z, dim=1)
        key = score
    else:
        score = torch.sigmoid(z)
        key = score + t64(bias)
    top = torch.topk(key, k, dim=1, largest=True, sorted=True)
    g = torch.gather(score, 1, top.indices)
    if norm:
        g = g / g.sum(dim=1, keepdim=True)
    np.testing.assert_array_equal(idx, top.indices.numpy())
    np.testing.assert_allclose(gate, 1.7 * g.numpy(), rtol=1e-13)


def test_softmax_bias_shifts_logits():
    # softmax(z + b) with b added to the logits (selection and gates follow it)
    rng = np.random.default_rng(3)
    x = rng.normal(size=(3, 8))
    w = rng.normal(size=(5, 8))
    b = np.array([0.0, 50.0, 0.0, 0.0, 0.0])
    idx, gate, (z, p, key) = moe.route_topk(x, w, b, 1, moe.SOFTMAX, False)
    assert (idx[:, 0] == 1).all()
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(gate[:, 0], torch.softmax(t64(z) + t64(b), 1)[:, 1].numpy(), rtol=1e-13)


def test_sigmoid_bias_steers_selection_only():
    # The bias picks the expert; the gate is the unbiased sigmoid (renormalised).
    rng = np.random.default_rng(4)
    x = rng.normal(size=(6, 8))
    w = rng.normal(0, 0.1, (5, 8))
    b = np.array([0.0, 0.0, 0.0, 10.0, 9.0])
    idx, gate, (z, s, _) = moe.route_topk(x, w, b, 2, moe.SIGMOID, True)
    assert (idx[:, 0] == 3).all() and (idx[:, 1] == 4).all()
    sg = 1.0 / (1.0 + np.exp(-z))
    np.testing.assert_allclose(gate[:, 0], sg[:, 3] / (sg[:, 3] + sg[:, 4]), rtol=1e-13)


def test_topk_ties_go_to_lower_index():
    w = np.zeros((6, 4))  # every logit is 0: a six-way tie
    x = np.ones((2, 4))
    idx, gate, _ = moe.route_topk(x, w, None, 3, moe.SOFTMAX, False)
    np.testing.assert_array_equal(idx, [[0, 1, 2], [0, 1, 2]])
    np.testing.assert_allclose(gate, 1.0 / 6.0, rtol=1e-15)


# ------------------------------------------------------------------ P3 gate invariants

@pytest.mark.parametrize("score_func", [moe.SOFTMAX, moe.SIGMOID])
def test_normalised_gates_sum_to_one(score_func):
    rng = np.random.default_rng(11)
    x = rng.normal(size=(20, 16))
    w = rng.normal(0, 1.0, (9, 16))
    idx, gate, (_, score, _) = moe.route_topk(x, w, None, 4, score_func, True)
    np.testing.assert_allclose(gate.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    assert (gate > 0).all()
    if score_func == moe.SOFTMAX:
        np.testing.assert_allclose(score.sum(axis=1), 1.0, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ P1 / P2 union brute force

def brute_union(idx, gate):
    T, k = len(idx), len(idx[0])
    members = []
    for t in range(T):
        for j in range(k):
            if idx[t][j] not in members:
                members.append(idx[t][j])
    members.sort()
    lists = {e: [(t, gate[t][j]) for t in range(T) for j in range(k) if idx[t][j] == e] for e in members}
    return members, lists


@pytest.mark.parametrize("T,N,k,seed", [(1, 8, 2, 0), (5, 8, 2, 1), (9, 64, 6, 2), (17, 64, 6, 3),
                                        (64, 256, 16, 4), (3, 4, 4, 5)])
def test_union_matches_brute_force(T, N, k, seed):
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.permutation(N)[:k] for _ in range(T)]).astype(np.int32)
    gate = rng.random((T, k))
    u = moe.expert_union(idx, gate)
    members, lists = brute_union(idx.tolist(), gate.tolist())
    assert u["n_union"] == len(members) <= min(N, T * k)
    np.testing.assert_array_equal(u["union_ids"], members)
    assert u["offsets"][0] == 0 and u["offsets"][-1] == T * k
    assert (np.diff(u["offsets"]) > 0).all()
    for pos, e in enumerate(members):
        a, b = u["offsets"][pos], u["offsets"][pos + 1]
        assert [int(t) for t in u["tok_list"][a:b]] == [t for t, _ in lists[e]]
        np.testing.assert_array_equal(u["gate_list"][a:b], [g for _, g in lists[e]])
    for t in range(T):
        for j in range(k):
            p = u["pair_pos"][t, j]
            assert u["tok_list"][p] == t
            owner = np.searchsorted(u["offsets"], p, side="right") - 1
            assert u["union_ids"][owner] == idx[t, j]
            assert u["gate_list"][p] == gate[t, j]


def test_union_size_matches_closed_form_under_uniform_routing():
    # E|U| = N (1 - (1 - k/N)^T) for i.i.d. uniform k-subsets (statistical).
    rng = np.random.default_rng(99)
    for N, k, T, want in [(64, 6, 9, 37.6), (8, 2, 5, 6.1), (64, 6, 17, 52.0)]:
        sizes = [moe.expert_union(np.stack([rng.permutation(N)[:k] for _ in range(T)]),
                                  np.ones((T, k)))["n_union"] for _ in range(2000)]
        closed = N * (1 - (1 - k / N) ** T)
        assert abs(closed - want) < 0.06
        assert abs(np.mean(sizes) - closed) < 4 * np.std(sizes) / math.sqrt(len(sizes)) + 0.05


# ------------------------------------------------------------------ Eq. (4) target layer

def test_target_with_all_experts_equals_dense_mixture():
    # k = N, softmax, no renormalisation: y = S(x) + sum_e p_e E_e(x) for every e.
    rng = np.random.default_rng(21)
    w, experts, shared, _ = rand_layer(rng, N=5)
    x = rng.normal(size=(4, 24))
    y, idx, gate = moe.moe_target(x, w, None, lambda e: experts[e], shared, 5, moe.SOFTMAX, False)
    p = torch.softmax(t64(x) @ t64(w).T, dim=1).numpy()
    want = sum(torch_expert(x, *s) for s in shared)
    want = want + sum(p[:, [e]] * torch_expert(x, *experts[e]) for e in range(5))
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)


def test_target_is_token_independent_and_permutation_equivariant():
    rng = np.random.default_rng(22)
    w, experts, shared, _ = rand_layer(rng, N=7)
    x = rng.normal(size=(5, 24))
    y, idx, _ = moe.moe_target(x, w, None, lambda e: experts[e], shared, 3, moe.SOFTMAX, True)
    for t in range(5):
        yt, _, _ = moe.moe_target(x[t:t + 1], w, None, lambda e: experts[e], shared, 3, moe.SOFTMAX, True)
        np.testing.assert_allclose(yt[0], y[t], rtol=1e-13, atol=1e-14)
    perm = rng.permutation(7)  # expert perm[i] becomes expert i
    yp, idxp, _ = moe.moe_target(x, w[perm], None, lambda e: experts[perm[e]], shared, 3,
                                 moe.SOFTMAX, True)
    np.testing.assert_allclose(yp, y, rtol=1e-13, atol=1e-14)
    np.testing.assert_array_equal(perm[idxp], idx)


def test_identical_experts_with_normalised_gates_collapse():
    # If every routed expert is the same E and gates sum to one, y = S(x) + E(x).
    rng = np.random.default_rng(23)
    w, experts, shared, _ = rand_layer(rng, N=6)
    x = rng.normal(size=(3, 24))
    y, _, _ = moe.moe_target(x, w, None, lambda e: experts[0], shared, 4, moe.SIGMOID, True)
    want = sum(torch_expert(x, *s) for s in shared) + torch_expert(x, *experts[0])
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ Eq. (5) draft layer, Eq. (6)

def torch_route(x, w, k):
    top = torch.topk(torch.softmax(t64(x) @ t64(w).T, 1), k, dim=1)
    return top.indices.numpy(), top.values.numpy()


def test_zero_draft_expert_is_shared_plus_top1():
    # P4: a zero draft expert (or gamma = 0) leaves S(x) + g_{e1} E_{e1}(x).
    rng = np.random.default_rng(31)
    w, experts, shared, draft = rand_layer(rng)
    x = rng.normal(size=(4, 24))
    ti, tv = torch_route(x, w, 3)
    want = sum(torch_expert(x, *s) for s in shared)
    want = want + np.stack([tv[t, 0] * torch_expert(x[t], *experts[ti[t, 0]])[0] for t in range(4)])
    zero = tuple(np.zeros_like(m) for m in draft)
    for dr, gamma in [(None, 1.0), (zero, 1.0), (draft, 0.0)]:
        y, idx, gate = moe.moe_draft(x, w, None, lambda e: experts[e], shared, dr, gamma, 3,
                                     moe.SOFTMAX, False)
        np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-13)
        np.testing.assert_array_equal(idx, ti)


def test_draft_expert_term_is_gamma_scaled():
    rng = np.random.default_rng(32)
    w, experts, shared, draft = rand_layer(rng)
    x = rng.normal(size=(2, 24))
    y0, _, _ = moe.moe_draft(x, w, None, lambda e: experts[e], shared, draft, 0.0, 3, moe.SOFTMAX, False)
    y1, _, _ = moe.moe_draft(x, w, None, lambda e: experts[e], shared, draft, 0.37, 3, moe.SOFTMAX, False)
    np.testing.assert_allclose(y1 - y0, 0.37 * torch_expert(x, *draft), rtol=1e-11, atol=1e-13)


def test_missing_residual_identity_eq6():
    # Eq. (6): y* - S - g_{e1} E_{e1} equals the remaining top-k experts' gated sum.
    rng = np.random.default_rng(33)
    w, experts, shared, _ = rand_layer(rng)
    x = rng.normal(size=(5, 24))
    ys, _, _ = moe.moe_target(x, w, None, lambda e: experts[e], shared, 4, moe.SOFTMAX, True)
    yd, _, _ = moe.moe_draft(x, w, None, lambda e: experts[e], shared, None, 1.0, 4, moe.SOFTMAX, True)
    top = torch.topk(torch.softmax(t64(x) @ t64(w).T, 1), 4, dim=1)
    g = (top.values / top.values.sum(1, keepdim=True)).numpy()
    rest = np.stack([sum(g[t, j] * torch_expert(x[t], *experts[top.indices[t, j]])[0] for j in range(1, 4))
                     for t in range(5)])
    np.testing.assert_allclose(ys - yd, rest, rtol=1e-11, atol=1e-13)


# ------------------------------------------------------------------ P10 shared concatenation

def test_shared_concatenation_equals_sum_of_experts():
    rng = np.random.default_rng(41)
    H, each, ns = 12, 5, 3
    block = rng.normal(size=3 * ns * each * H)
    parts = moe.split_shared(block, ns, each, H)
    G, U, D = moe.split_expert(block, ns * each, H)
    x = rng.normal(size=(4, H))
    np.testing.assert_allclose(moe.shared_path(x, parts), torch_expert(x, G, U, D), rtol=1e-12, atol=1e-13)
    # the pieces are the expected slices of the concatenated matrices
    np.testing.assert_array_equal(parts[1][0], G[each:2 * each])
    np.testing.assert_array_equal(parts[2][2], D[:, 2 * each:3 * each])


def test_bf16_upconversion_bit_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x7F7F], dtype=np.uint16)
    v = moe.to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 1.0 + 2 ** -7 and v[3] == 0.0
    assert v[4] == 0.0 and math.copysign(1, v[4]) == -1.0
    assert v[5] == float.fromhex("0x1.fe00000000000p+127")


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(5)
    h = rng.normal(size=(6, 40)) * 3
    want = F.rms_norm(t64(h), (40,), eps=1e-6).numpy()
    np.testing.assert_allclose(moe.rmsnorm(h, 1e-6), want, rtol=1e-13)


# ------------------------------------------------------------------ P6 acceptance

@pytest.mark.parametrize("K", [0, 1, 4, 8, 16])
def test_accept_len_planted_prefix(K):
    rng = np.random.default_rng(100 + K)
    V = 50
    for m in range(K + 1):
        logits = rng.normal(size=(K + 1, V))
        t = logits.argmax(axis=1)
        drafts = [int(t[i]) for i in range(K)]
        if m < K:
            drafts[m] = (drafts[m] + 1 + int(rng.integers(V - 1))) % V  # first mismatch at m
        for i in range(m + 1, K):
            drafts[i] = int(rng.integers(V))  # anything after the mismatch is irrelevant
        n, bonus, tt = moe.accept_len(logits, drafts)
        assert n == m
        assert bonus == int(t[m])
        np.testing.assert_array_equal(tt, t)


def test_argmax_ties_to_lowest_index():
    logits = np.array([[0.5, 2.0, 2.0, 1.0], [3.0, 3.0, 3.0, 3.0]])
    np.testing.assert_array_equal(moe.argmax_first(logits), [1, 0])


# ------------------------------------------------------------------ decode-level pins

def tiny_model(rng, H=16, N=6, k=2, I=8, L=2, V=40, draft_scale=0.3, k_route=None):
    layers = []
    for _ in range(L):
        w, experts, shared, draft = rand_layer(rng, H=H, N=N, I=I, n_shared=1, Id=4, router_std=0.8)
        layers.append(decode.LayerWeights(
            w_router=w, bias=None, routed=(lambda ex: (lambda e: ex[e]))(experts), shared=shared,
            draft=tuple(draft_scale * m for m in draft), gamma=1.0, top_k=k if k_route is None else k_route,
            score_func=moe.SOFTMAX, norm_topk=True))
    emb = rng.normal(size=(V, H))
    dense = (rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (I, H)), rng.normal(0, 0.3, (H, I)))
    return decode.ModelWeights(emb=lambda t: emb[t], dense=dense, layers=layers,
                               lm_head=rng.normal(size=(V, H)))


def test_forward_with_zero_blocks_is_norm_then_head():
    rng = np.random.default_rng(51)
    m = tiny_model(rng)
    zero = lambda t: tuple(np.zeros_like(a) for a in t)  # noqa: E731
    m.dense = zero(m.dense)
    for lw in m.layers:
        ex = lw.routed
        lw.routed = (lambda ex: (lambda e: zero(ex(e))))(ex)
        lw.shared = [zero(s) for s in lw.shared]
    toks = [3, 7, 7, 0]
    emb = np.stack([m.emb(t) for t in toks])
    want = F.rms_norm(t64(emb), (emb.shape[1],), eps=1e-6).numpy() @ m.lm_head.T
    np.testing.assert_allclose(decode.forward(m, toks, "target"), want, rtol=1e-12, atol=1e-12)


def test_forward_dense_only_layer():
    rng = np.random.default_rng(52)
    m = tiny_model(rng, L=0)
    toks = [1, 2]
    h = t64(np.stack([m.emb(t) for t in toks]))
    h = h + torch.from_numpy(torch_expert(F.rms_norm(h, (h.shape[1],), eps=1e-6).numpy(), *m.dense))
    want = F.rms_norm(h, (h.shape[1],), eps=1e-6).numpy() @ m.lm_head.T
    np.testing.assert_allclose(decode.forward(m, toks), want, rtol=1e-12, atol=1e-12)


def test_spec_step_emits_greedy_ar_tokens():
    # P15: the emitted tokens of an exact step equal n+1 steps of greedy AR.
    for seed in range(6):
        rng = np.random.default_rng(60 + seed)
        m = tiny_model(rng, draft_scale=1.0 if seed % 2 else 0.2)
        c = int(rng.integers(40))
        drafts, n, bonus, _ = decode.spec_step(m, c, 5)
        ar = decode.greedy_ar(m, c, n + 1)
        assert drafts[:n] + [bonus] == ar


def test_k1_zero_draft_accepts_everything():
    # P5: k = 1 with renormalised gates and no draft expert makes drafter == target.
    rng = np.random.default_rng(70)
    m = tiny_model(rng, k_route=1)
    for lw in m.layers:
        lw.draft = None
    for c in range(5):
        drafts, n, bonus, _ = decode.spec_step(m, c, 6)
        assert n == 6


# ------------------------------------------------------------------ P12 paper-printed shape facts

def test_v2lite_shape_facts_from_paper():
    facts = json.load(open(os.path.join(GOLDEN, "v2lite_shape_facts.json")))
    from workloads.configs import CFG4
    m = CFG4.moe
    assert CFG4.n_moe_layers + 1 == facts["layers"]
    assert m.n_experts == facts["routed_experts"] and m.n_shared == facts["shared_experts"]
    assert m.top_k == facts["top_k"]
    routed = CFG4.n_moe_layers * m.n_experts * 3 * m.hidden * m.inter
    assert routed == 14_394_851_328
    assert round(routed / 1e9, 1) == facts["routed_params_billion"]
    assert round(routed * 2 / 2 ** 30, 1) == facts["routed_bf16_gib"]
    assert round(100 * m.top_k / m.n_experts, 1) == facts["active_fraction_percent"]
    # the printed share is reachable with a non-routed size that rounds to the printed 2.4 GiB
    shares = [round(100 * routed / (routed + g * 2 ** 30 / 2), 1) for g in np.arange(2.35, 2.45, 0.001)]
    assert facts["routed_share_percent"] in shares


def test_expert_block_layout_roundtrip():
    # A block is [G (I x H) | U (I x H) | D (H x I)], each row-major [out, in].
    rng = np.random.default_rng(42)
    H, I = 7, 3
    G, U, D = rng.normal(size=(I, H)), rng.normal(size=(I, H)), rng.normal(size=(H, I))
    block = np.concatenate([G.ravel(), U.ravel(), D.ravel()])
    g, u, d = moe.split_expert(block, I, H)
    np.testing.assert_array_equal(g, G)
    np.testing.assert_array_equal(u, U)
    np.testing.assert_array_equal(d, D)
