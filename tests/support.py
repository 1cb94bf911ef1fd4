"""Test helpers: oracle-side layer weights, gap resampling, error metrics.

Inputs for the oracle always come from the CPU generator; device tensors come
from the GPU fill of the same streams (checked bit-exact in the GPU tests).
"""
from __future__ import annotations

import functools

import numpy as np

from oracle import decode, moe
from workloads import configs, gen

GAP = 1e-4  # minimum selection-key gap of generated inputs (top-k boundaries)


def rel_err(got, want) -> float:
    """max |got - want| / max |want| (the layer-output error metric)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    den = np.max(np.abs(want))
    return float(np.max(np.abs(got - want)) / (den if den > 0 else 1.0))


def topk_gaps_ok(keys_row: np.ndarray, k: int, gap: float = GAP) -> bool:
    """Every gap among the k+1 largest keys exceeds ``gap`` (k/k+1 boundary included)."""
    s = np.sort(np.asarray(keys_row, dtype=np.float64))[::-1]
    m = min(k + 1, s.size)
    return bool(np.all(s[:m - 1] - s[1:m] > gap))


class OracleLayer:
    """fp64 weights of one generated MoE layer, expert blocks created on demand."""

    def __init__(self, cfg: configs.MoECfg, layer: int = 0, redraw: int = 0, bias=None):
        self.cfg = cfg
        self.layer = layer
        self.redraw = redraw
        self.w_router = gen.router_weight(cfg, layer, redraw).astype(np.float64)
        b = gen.router_bias(cfg, layer, redraw) if bias is None else bias
        self.bias_f32 = None if b is None else np.asarray(b, dtype=np.float32)
        self.bias = None if b is None else np.asarray(b, dtype=np.float32).astype(np.float64)
        self._shared = None
        self._draft = None

    @functools.lru_cache(maxsize=80)
    def routed(self, e: int):
        c = self.cfg
        return moe.split_expert(gen.routed_block(c, self.layer, e, self.redraw), c.inter, c.hidden)

    @property
    def shared(self):
        if self._shared is None:
            c = self.cfg
            self._shared = moe.split_shared(gen.shared_block(c, self.layer, self.redraw), c.n_shared,
                                            c.shared_each, c.hidden)
        return self._shared

    @property
    def draft(self):
        if self._draft is None:
            c = self.cfg
            self._draft = moe.split_expert(gen.draft_block(c, self.layer, self.redraw),
                                           c.draft_inter, c.hidden)
        return self._draft

    def route(self, x):
        c = self.cfg
        return moe.route_topk(x, self.w_router, self.bias, c.top_k, c.score_func, c.norm_topk,
                              c.routed_scale)

    def target(self, x):
        c = self.cfg
        return moe.moe_target(x, self.w_router, self.bias, self.routed, self.shared, c.top_k,
                              c.score_func, c.norm_topk, c.routed_scale)

    def draft_out(self, x, gamma=None, with_draft=True):
        c = self.cfg
        return moe.moe_draft(x, self.w_router, self.bias, self.routed, self.shared,
                             self.draft if with_draft else None, c.gamma if gamma is None else gamma,
                             c.top_k, c.score_func, c.norm_topk, c.routed_scale)

    def layer_weights(self) -> decode.LayerWeights:
        c = self.cfg
        return decode.LayerWeights(w_router=self.w_router, bias=self.bias, routed=self.routed,
                                   shared=self.shared, draft=self.draft, gamma=c.gamma,
                                   top_k=c.top_k, score_func=c.score_func, norm_topk=c.norm_topk,
                                   routed_scale=c.routed_scale)


def gapped_x(layer: OracleLayer, T: int, block: int = 0, max_redraw: int = 200):
    """Activation rows whose oracle selection keys all have top-k gaps > GAP.

    Rows are resampled one at a time (each row has its own redraw counter).
    Returns (x fp32 [T, H], redraws).
    """
    c = layer.cfg
    redraws = [0] * T
    x = gen.x_rows(c, T, block, redraws)
    for t in range(T):
        while True:
            _, _, (_, _, keys) = layer.route(x[t:t + 1])
            if topk_gaps_ok(keys[0], c.top_k):
                break
            redraws[t] += 1
            if redraws[t] > max_redraw:
                raise RuntimeError("could not draw a gapped activation row")
            x[t] = gen.x_rows(c, t + 1, block, redraws)[t]
    return x, redraws


class OracleModel:
    """fp64 weights of a generated stacked model (MoE layer l uses the layer-l streams)."""

    def __init__(self, model: configs.ModelCfg):
        m = model.moe
        self.cfg = model
        self.layers = [
            OracleLayer(m, l, bias=gen.zipf_bias(model, l, model.zipf_lam) if model.zipf_s > 0
                        else None)
            for l in range(1, model.n_moe_layers + 1)]
        emb = gen.embedding(model)
        dense = moe.split_expert(gen.dense_block(model), model.dense_inter, m.hidden)
        lm = moe.to_f64(gen.lm_head(model.cfg_id, model.vocab, m.hidden, model.lm_std))
        self.weights = decode.ModelWeights(
            emb=lambda t: moe.to_f64(emb[t]), dense=dense,
            layers=[ol.layer_weights() for ol in self.layers], lm_head=lm, eps=model.eps)

    def trace_gaps_ok(self, tr: decode.Trace, gap: float = GAP) -> bool:
        """Every routing decision and every row argmax of one pass has a margin > gap."""
        k = self.cfg.moe.top_k
        for ol, x in zip(self.layers, tr.moe_inputs):
            _, _, (_, _, keys) = ol.route(x)
            if not all(topk_gaps_ok(row, k, gap) for row in keys):
                return False
        lg = np.asarray(tr.logits, dtype=np.float32).astype(np.float64)
        return all(topk_gaps_ok(row, 1, gap) for row in lg)

    def gapped_step(self, K: int, tries: int = 6, redraw0: int = 0):
        """An oracle step from the first generated start token whose decisions are all gapped.

        Returns (start_token, drafts, n, bonus, target_argmax, traces)."""
        for r in range(redraw0, redraw0 + tries):
            c = gen.start_token(self.cfg, redraw=r)
            traces: list = []
            drafts, n, bonus, t = decode.spec_step(self.weights, c, K, traces)
            if all(self.trace_gaps_ok(tr) for tr in traces):
                return c, drafts, n, bonus, t, traces
        raise RuntimeError("no gapped start token found")
