"""Pin of the oracle's stacked forward with live (non-zero) MoE layers.

The oracle's model (``oracle.decode.forward``) is a pre-norm residual stack:
h = Emb[token]; h += Dense(RMSNorm(h)); h += MoE_l(RMSNorm(h)) for every MoE
layer (Eq. 4 for the target, Eq. 5 for the drafter); logits = W_lm RMSNorm(h).
Here the same stack is written out again with torch fp64 library operations
(``F.rms_norm``, ``torch.softmax`` + ``torch.topk``, ``F.silu``) over random
weights whose routing differs from token to token, and the two must agree to
rounding.  A misplaced pre-norm (a MoE layer applied to h instead of
RMSNorm(h)), a dropped residual, a transposed expert matrix, the wrong expert
or gate in the draft term, or a missing final norm changes the logits by far
more than the tolerance.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decode, moe

H, N, K, I, NS, ID, V = 32, 8, 2, 16, 2, 8, 50
EPS = 1e-6


def make_stack(seed: int, n_layers: int, norm_topk: bool, gamma: float):
    rng = np.random.default_rng(seed)

    def expert(inter):
        return (rng.normal(0, 0.3, (inter, H)), rng.normal(0, 0.3, (inter, H)),
                rng.normal(0, 0.3, (H, inter)))

    emb = rng.normal(0, 1.0, (V, H))
    dense = expert(24)
    layers = []
    for _ in range(n_layers):
        routed = [expert(I) for _ in range(N)]
        layers.append(dict(w_router=rng.normal(0, 0.5, (N, H)), routed=routed,
                           shared=[expert(I) for _ in range(NS)], draft=expert(ID)))
    lm = rng.normal(0, 0.2, (V, H))
    weights = decode.ModelWeights(
        emb=lambda t: emb[t], dense=dense,
        layers=[decode.LayerWeights(w_router=l["w_router"], bias=None,
                                    routed=(lambda e, r=l["routed"]: r[e]), shared=l["shared"],
                                    draft=l["draft"], gamma=gamma, top_k=K,
                                    score_func=moe.SOFTMAX, norm_topk=norm_topk)
                for l in layers],
        lm_head=lm, eps=EPS)
    return weights, dict(emb=emb, dense=dense, layers=layers, lm=lm)


def t64(a):
    return torch.as_tensor(np.asarray(a), dtype=torch.float64)


def expert_torch(x, gud):
    g, u, d = (t64(m) for m in gud)
    return (F.silu(x @ g.T) * (x @ u.T)) @ d.T


def reference_logits(raw, tokens, mode: str, norm_topk: bool, gamma: float):
    """The stack written with torch fp64 library calls, independent of the oracle's code."""
    h = t64(raw["emb"])[torch.as_tensor(tokens)]
    h = h + expert_torch(F.rms_norm(h, (H,), eps=EPS), raw["dense"])
    for l in raw["layers"]:
        x = F.rms_norm(h, (H,), eps=EPS)
        p = torch.softmax(x @ t64(l["w_router"]).T, dim=-1)
        top, idx = torch.topk(p, K, dim=-1)
        g = top / top.sum(dim=-1, keepdim=True) if norm_topk else top
        y = sum(expert_torch(x, s) for s in l["shared"])
        rows = []
        for t in range(x.shape[0]):
            xt = x[t:t + 1]
            if mode == "target":
                r = sum(g[t, j] * expert_torch(xt, l["routed"][int(idx[t, j])]) for j in range(K))
            else:
                r = (g[t, 0] * expert_torch(xt, l["routed"][int(idx[t, 0])])
                     + gamma * expert_torch(xt, l["draft"]))
            rows.append(r)
        h = h + y + torch.cat(rows, dim=0)
    return (F.rms_norm(h, (H,), eps=EPS) @ t64(raw["lm"]).T).numpy()


@pytest.mark.parametrize("mode", ["target", "draft"])
@pytest.mark.parametrize("n_layers,norm_topk,gamma,seed", [
    (1, False, 1.0, 11), (2, True, 0.7, 12), (2, False, 1.5, 13)])
def test_stacked_forward_matches_torch_composition(mode, n_layers, norm_topk, gamma, seed):
    weights, raw = make_stack(seed, n_layers, norm_topk, gamma)
    tokens = [3, 17, 17, 42, 0, 29]
    got = decode.forward(weights, tokens, mode)
    want = reference_logits(raw, tokens, mode, norm_topk, gamma)
    scale = np.max(np.abs(want))
    assert np.max(np.abs(got - want)) <= 1e-11 * scale
    # The routing is live: the tokens do not all pick the same experts, so a
    # wrong routed term cannot hide behind identical selections.
    tr = decode.Trace()
    decode.forward(weights, tokens, mode, tr)
    assert len({tuple(r) for r in np.asarray(tr.idx[0]).tolist()}) > 1


def test_moe_layers_change_the_logits():
    # The MoE contributions are not negligible: without them the logits move by
    # far more than the tolerance above, so the comparison exercises them.
    weights, raw = make_stack(14, 2, False, 1.0)
    tokens = [1, 2, 3, 4]
    full = decode.forward(weights, tokens, "target")
    bare = decode.ModelWeights(emb=weights.emb, dense=weights.dense, layers=[],
                               lm_head=weights.lm_head, eps=EPS)
    assert np.max(np.abs(full - decode.forward(bare, tokens, "target"))) > 1e-2 * np.max(np.abs(full))
