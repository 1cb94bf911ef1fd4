"""The stacked model and the draft-then-verify step over device tensors.

Argument marshalling only: ``DeviceModel`` builds the ``de_model`` struct of
``include/draftexpert.h`` from resident weight tensors, owns a workspace, and
calls ``de_spec_step`` / ``de_model_forward`` / ``de_greedy_decode``, whose
launches all run in ``libdraftexpert.so``.
"""
from __future__ import annotations

import torch

from . import _lib as L


class DeviceModel:
    """A pre-norm residual stack (embedding, dense layer 0, MoE layers, LM head).

    ``layers`` is a list of dicts with "router" (fp32 [N, H]), "bias" (fp32
    [N] or None), "table" (an ``ExpertTable``) or "routed" (resident [N, block]
    tensor), "shared", "draft" and optionally "gamma".  ``draft_topr`` is the
    number of routed experts of every draft layer (1: Eq. 5).
    """

    def __init__(self, desc, layers, vocab, emb, lm_head, dense=None, dense_inter=0,
                 dense_wdtype=L.DE_BF16, eps=1e-6, gamma=1.0, max_block=17, device="cuda",
                 draft_topr=1):
        self.desc = desc
        self.vocab = int(vocab)
        self.n_layers = len(layers)
        stride = L.expert_bytes(desc.wdtype, desc.inter, desc.hidden)
        entries = []
        for l in layers:
            table = l.get("table")
            if table is None:
                table = L.make_table(l["routed"], stride, None, desc.n_experts)
            entries.append(dict(w_router=l["router"], bias=l.get("bias"), table=table,
                                shared_w=l.get("shared"), draft_w=l.get("draft"),
                                gamma=l.get("gamma", gamma)))
        self._keep = (layers, emb, lm_head, dense)
        self.model = L.make_model(desc, entries, vocab, emb, lm_head, dense, dense_inter,
                                  dense_wdtype, eps, draft_topr)
        rc = L.de_check_model(self.model)
        if rc != 0:
            L._check("de_check_model", rc)
        self.max_block = int(max_block)
        self.ws = L.model_workspace(self.model, self.max_block, device)
        self.device = device

    def spec_step(self, block, target_argmax, out, n_union=None, pred_idx=None, stream=None):
        K = block.numel() - 1
        L.de_spec_step(self.model, K, block, target_argmax, out, n_union, pred_idx, self.ws, stream)

    def spec_step_trunc(self, block, target_argmax, out, pred_idx, q, tau, budget, slots=0,
                        cache=None, n_union=None, trace=None, stream=None,
                        prefetch=True) -> int:
        """Algorithm 1 with confidence-expansion truncation; returns the kept draft count."""
        k_max = block.numel() - 1
        return L.de_spec_step_trunc(self.model, cache, k_max, tau, budget, slots, block,
                                    target_argmax, out, pred_idx, q, n_union, trace, self.ws,
                                    stream, prefetch)

    def distill(self, tokens, tau, m_star, router_kl, logit_kl, token_ce, stream=None):
        """The self-distillation signals (Eqs. 6-10) of teacher-forced positions."""
        L.de_distill_signals(self.model, tokens.numel(), tokens, tau, m_star, router_kl,
                             logit_kl, token_ce, self.ws, stream)

    def forward(self, tokens, mode, logits, argmax=None, n_union=None, stream=None):
        L.de_model_forward(self.model, tokens.numel(), tokens, mode, logits, argmax, n_union,
                           self.ws, stream)

    def greedy(self, tokens, stream=None):
        L.de_greedy_decode(self.model, tokens.numel() - 1, tokens, self.ws, stream)

    def new_block(self, K, last_token):
        b = torch.empty(K + 1, dtype=torch.int32, device=self.device)
        b[0] = int(last_token)
        return b
