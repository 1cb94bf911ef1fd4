"""Plain fp64 CPU oracle of one MoE layer: routing, union, target and draft forms.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  It shares no code with
the HIP path and is written for reading, not speed: per-token loops, the
textbook formulas, NumPy matmuls as the only library steps.

Notation follows the paper (Sections 2.1, 2.3 and 3.2):
``TopK_l(h)`` the router's top-k set (Eq. 1), ``U_l(B)`` the union of the top-k
sets over a block (Eq. 2 and Eq. 3), ``y*`` the target MoE output (Eq. 4) and
``y^d`` the fixed-footprint draft output (Eq. 5).

Readings where the paper is silent (each one is also listed in the design
notes): the router distribution R_l is softmax(z + b) or, for the sigmoid
router, sigmoid(z) selected by sigmoid(z) + b; the gate g_{l,e} is the score of
expert e, optionally renormalised over the top-k and scaled; the top-k is
ordered by descending selection key with ties to the lower expert index, and
the selection is made on the keys rounded to fp32 (the kernel's precision);
the draft gate g_{l,e1} is the target gate of the top-1 expert; an expert is a
SwiGLU ``D (silu(G x) * (U x))``.
"""
from __future__ import annotations

import numpy as np

from . import q4

SOFTMAX = 0
SIGMOID = 1


def to_f64(w: np.ndarray) -> np.ndarray:
    """Exact upconversion of stored weights: uint16 arrays are bf16 bit patterns."""
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return w.astype(np.float64)


def split_expert(block: np.ndarray, inter: int, hidden: int):
    """fp64 (G [I,H], U [I,H], D [H,I]) from a flat ``[G|U|D]`` expert block
    (uint8 blocks are Q4_0, dequantised by ``oracle.q4``)."""
    if np.asarray(block).dtype == np.uint8:
        return q4.split_expert(block, inter, hidden)
    w = to_f64(block)
    n = inter * hidden
    return (w[:n].reshape(inter, hidden), w[n:2 * n].reshape(inter, hidden),
            w[2 * n:3 * n].reshape(hidden, inter))


def split_shared(block: np.ndarray, n_shared: int, each: int, hidden: int):
    """The shared path stored as one concatenated block, returned as its n_shared experts.

    Expert s owns rows [s*I, (s+1)*I) of G and U and the same columns of D.
    """
    g, u, d = split_expert(block, n_shared * each, hidden)
    return [(g[s * each:(s + 1) * each], u[s * each:(s + 1) * each], d[:, s * each:(s + 1) * each])
            for s in range(n_shared)]


# ---------------------------------------------------------------- routing (Eq. 1)

def router_scores(x: np.ndarray, w_router: np.ndarray, bias, score_func: int):
    """Router logits z = W_r h, scores R_l(h) and selection keys for each token.

    softmax: scores = softmax(z + b) (b = 0 when absent); key = z + b, which
    orders experts exactly as the probabilities do.
    sigmoid: scores = sigmoid(z); key = sigmoid(z) + b (the bias only steers
    selection).
    Returns (z, scores, keys), each [T, N] fp64.
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    w = np.asarray(w_router, dtype=np.float64)
    b = np.zeros(w.shape[0]) if bias is None else np.asarray(bias, dtype=np.float64)
    z = x @ w.T
    if score_func == SOFTMAX:
        zb = z + b
        ex = np.exp(zb - zb.max(axis=1, keepdims=True))
        scores = ex / ex.sum(axis=1, keepdims=True)
        keys = zb
    elif score_func == SIGMOID:
        scores = 1.0 / (1.0 + np.exp(-z))
        keys = scores + b
    else:
        raise ValueError("unknown score function")
    return z, scores, keys


def route_topk(x, w_router, bias, top_k: int, score_func: int, norm_topk: bool,
               routed_scale: float = 1.0, decision_dtype=np.float32):
    """TopK_l(h) of Eq. (1) with the gates g_{l,e} of Eq. (4).

    Per token: the k experts with the largest selection keys, in descending
    key order, ties to the lower index (a stable sort of the negated keys).
    The comparison is made on the keys rounded to ``decision_dtype``.
    Returns idx [T,k] int32, gate [T,k] fp64 and the (z, scores, keys) triple.
    """
    z, scores, keys = router_scores(x, w_router, bias, score_func)
    kd = keys.astype(decision_dtype)
    idx = np.argsort(-kd, axis=1, kind="stable")[:, :top_k]
    gate = np.take_along_axis(scores, idx, axis=1)
    if norm_topk:
        gate = gate / gate.sum(axis=1, keepdims=True)
    gate = gate * routed_scale
    return idx.astype(np.int32), gate, (z, scores, keys)


# ---------------------------------------------------------------- union (Eq. 2, Eq. 3)

def expert_union(idx: np.ndarray, gate: np.ndarray):
    """U(B) = union over the block of each token's top-k set, with per-expert token lists.

    The union is listed in ascending expert id.  For each member e the token
    list holds every block position t whose top-k contains e, ascending in t,
    with the matching gate.  ``pair_pos[t, j]`` is the position of the pair
    (idx[t, j], t) in the concatenated lists and ``offsets`` delimit them.
    """
    idx = np.asarray(idx)
    T, k = idx.shape
    members = sorted(set(int(e) for e in idx.ravel()))
    tok_list: list[int] = []
    gate_list: list[float] = []
    offsets = [0]
    pair_pos = np.full((T, k), -1, dtype=np.int32)
    for e in members:
        for t in range(T):
            for j in range(k):
                if int(idx[t, j]) == e:
                    pair_pos[t, j] = len(tok_list)
                    tok_list.append(t)
                    gate_list.append(float(gate[t, j]))
        offsets.append(len(tok_list))
    return {
        "n_union": len(members),
        "union_ids": np.array(members, dtype=np.int32),
        "offsets": np.array(offsets, dtype=np.int32),
        "tok_list": np.array(tok_list, dtype=np.int32),
        "gate_list": np.array(gate_list, dtype=np.float64),
        "pair_pos": pair_pos,
    }


# ---------------------------------------------------------------- experts and layers

def silu(v: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return v / (1.0 + np.exp(-v))


def swiglu(x: np.ndarray, g: np.ndarray, u: np.ndarray, d: np.ndarray) -> np.ndarray:
    """One expert E(x) = D (silu(G x) * (U x)) for each row of x [T,H] -> [T,H]."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    return (silu(x @ g.T) * (x @ u.T)) @ d.T


def shared_path(x: np.ndarray, shared) -> np.ndarray:
    """S_l(h): the sum of the shared experts, each with weight one."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    out = np.zeros_like(x)
    for (g, u, d) in shared:
        out = out + swiglu(x, g, u, d)
    return out


def moe_target(x, w_router, bias, routed, shared, top_k: int, score_func: int,
               norm_topk: bool, routed_scale: float = 1.0):
    """Target MoE output of Eq. (4), token by token.

    y*_t = S(x_t) + sum over e in TopK(x_t) of g_{t,e} E_e(x_t).
    ``routed(e)`` returns expert e's fp64 (G, U, D); ``shared`` is the list of
    shared experts.  Returns (y [T,H], idx, gate).
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    idx, gate, _ = route_topk(x, w_router, bias, top_k, score_func, norm_topk, routed_scale)
    y = shared_path(x, shared)
    for t in range(x.shape[0]):
        for j in range(top_k):
            g, u, d = routed(int(idx[t, j]))
            y[t] += gate[t, j] * swiglu(x[t:t + 1], g, u, d)[0]
    return y, idx, gate


def moe_draft(x, w_router, bias, routed, shared, draft, gamma: float, top_k: int,
              score_func: int, norm_topk: bool, routed_scale: float = 1.0, r: int = 1):
    """Fixed-footprint draft output of Eq. (5), token by token.

    y^d_t = S(x_t) + g_{t,e1} E_{e1}(x_t) + gamma * E^d(x_t), where e1 is the
    expert with the largest selection key and g_{t,e1} is its target gate.
    ``draft`` is the draft expert's (G, U, D) or None (a zero draft expert).
    With r > 1 the routed term runs over the r experts with the largest keys,
    each with its target gate: the shared + top-r self-drafter the paper
    compares against (Section 1, Table 3), with gamma = 0.
    The full top-k is still returned: it is the draft router's prediction of
    the verifier's experts (Section 3.4).  Returns (y, idx, gate).
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    idx, gate, _ = route_topk(x, w_router, bias, top_k, score_func, norm_topk, routed_scale)
    if not 1 <= r <= top_k:
        raise ValueError("r must lie in [1, top_k]")
    y = shared_path(x, shared)
    for t in range(x.shape[0]):
        for j in range(r):
            g, u, d = routed(int(idx[t, j]))
            y[t] += gate[t, j] * swiglu(x[t:t + 1], g, u, d)[0]
        if draft is not None:
            y[t] += gamma * swiglu(x[t:t + 1], *draft)[0]
    return y, idx, gate


# ---------------------------------------------------------------- norm, head, acceptance

def rmsnorm(h: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """h / sqrt(mean(h^2) + eps) per row, unit gain."""
    h = np.atleast_2d(np.asarray(h, dtype=np.float64))
    return h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)


def argmax_first(logits: np.ndarray, decision_dtype=np.float32) -> np.ndarray:
    """Row-wise argmax on the logits rounded to ``decision_dtype``; ties to the lowest index."""
    return np.argmax(np.atleast_2d(logits).astype(decision_dtype), axis=1).astype(np.int32)


def accept_len(target_logits: np.ndarray, draft_tokens, decision_dtype=np.float32):
    """Greedy exact verification (Algorithm 1, verify and accept steps).

    Block position j = 0..K holds the last committed token (j = 0) and the
    drafts d_1..d_K; row j of ``target_logits`` is the target's prediction
    after position j, t_j = argmax.  The accepted prefix length n is the
    largest m <= K with d_i = t_{i-1} for every i <= m; the bonus token is t_n.
    Returns (n, bonus, t).
    """
    t = argmax_first(target_logits, decision_dtype)
    d = [int(v) for v in np.asarray(draft_tokens).ravel()]
    n = 0
    while n < len(d) and d[n] == int(t[n]):
        n += 1
    return n, int(t[n]), t
