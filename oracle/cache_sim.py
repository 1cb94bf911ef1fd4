"""Plain simulation of the expert cache of offloaded decoding (Section 3.5,
Algorithm 1): which experts sit in the accelerator cache C, which copies are
started, and the hit / waste / miss counts.

TEST INFRASTRUCTURE ONLY: imported by tests/ and nothing in the product path.

The paper fixes the sets (the cache C, the in-flight set P, the predicted
verifier sets of each draft token) and the rules that prefetches skip experts
in C or P and that verification loads misses on demand.  It gives no eviction
rule; this simulation takes the following reading, step by step:

* every layer has S slots; a copy takes the free slot with the lowest index,
  else the least recently used slot (ties to the lower index) whose expert is
  neither needed by the current request nor predicted for the current block;
  only an on-demand load may then fall back to a predicted (unneeded) expert;
  a prefetch with no such slot is dropped;
* an expert whose copy has started is in the cache from then on (a request
  for it waits for the copy, and counts as a hit);
* "use" times are requests and copies (a prefetch of a cached expert only
  marks it predicted);
* a prefetched expert counts as used when a verify request of its block needs
  it, and as wasted when it is evicted, or its block ends, first;
* the draft path requests its top-1 expert and then prefetches its whole
  top-k; verification requests its union in chunks of S members, the members
  in the cache first, then the others, each part in ascending id.

Timing (how long a request waits) is not simulated.
"""
from __future__ import annotations

DRAFT = 0
VERIFY = 1

COUNTS = ("prefetch_issued", "prefetch_used", "prefetch_wasted", "prefetch_skipped",
          "draft_needed", "draft_hits", "verify_needed", "verify_hits", "demand_loads",
          "evictions", "bytes_copied")


class CacheSim:
    def __init__(self, n_layers: int, n_experts: int, n_slots: int, expert_bytes: int = 1):
        self.L, self.N, self.S = n_layers, n_experts, n_slots
        self.expert_bytes = expert_bytes
        self.slot = [[None] * n_slots for _ in range(n_layers)]      # expert held by each slot
        self.last = [[0] * n_slots for _ in range(n_layers)]         # use time of each slot
        self.from_prefetch = [[False] * n_slots for _ in range(n_layers)]
        self.predicted = [set() for _ in range(n_layers)]
        self.clock = 0
        self.counts = {name: 0 for name in COUNTS}

    # -- state queries
    def slot_of(self, layer: int, e: int) -> int:
        row = self.slot[layer]
        return row.index(e) if e in row else -1

    def slot_table(self, layer: int) -> list:
        return [self.slot_of(layer, e) for e in range(self.N)]

    # -- the policy
    def _victim(self, layer: int, need: set, may_take_predicted: bool):
        row = self.slot[layer]
        for s in range(self.S):
            if row[s] is None:
                return s
        tiers = (False, True) if may_take_predicted else (False,)
        for predicted_tier in tiers:
            cands = [s for s in range(self.S)
                     if row[s] not in need and (row[s] in self.predicted[layer]) == predicted_tier]
            if cands:
                return min(cands, key=lambda s: (self.last[layer][s], s))
        return None

    def _copy(self, layer: int, e: int, s: int, prefetch: bool):
        old = self.slot[layer][s]
        if old is not None:
            self.counts["evictions"] += 1
            if self.from_prefetch[layer][s]:
                self.counts["prefetch_wasted"] += 1
        self.clock += 1
        self.slot[layer][s] = e
        self.last[layer][s] = self.clock
        self.from_prefetch[layer][s] = prefetch
        self.counts["bytes_copied"] += self.expert_bytes
        self.counts["prefetch_issued" if prefetch else "demand_loads"] += 1

    def begin_block(self):
        for layer in range(self.L):
            for s in range(self.S):
                if self.from_prefetch[layer][s]:
                    self.counts["prefetch_wasted"] += 1
                    self.from_prefetch[layer][s] = False
            self.predicted[layer] = set()

    def prefetch(self, layer: int, experts):
        experts = [int(e) for e in experts]
        self.predicted[layer].update(experts)
        for e in experts:
            if self.slot_of(layer, e) >= 0:
                continue
            s = self._victim(layer, set(), False)
            if s is None:
                self.counts["prefetch_skipped"] += 1
                continue
            self._copy(layer, e, s, True)

    def ensure(self, layer: int, need, purpose: int):
        need = [int(e) for e in need]
        assert 1 <= len(need) <= self.S and len(set(need)) == len(need)
        hits = 0
        for e in need:
            if self.slot_of(layer, e) >= 0:
                hits += 1
                continue
            self._copy(layer, e, self._victim(layer, set(need), True), False)
        key = "draft" if purpose == DRAFT else "verify"
        self.counts[key + "_needed"] += len(need)
        self.counts[key + "_hits"] += hits
        for e in need:
            s = self.slot_of(layer, e)
            self.clock += 1
            self.last[layer][s] = self.clock
            if purpose == VERIFY and self.from_prefetch[layer][s]:
                self.counts["prefetch_used"] += 1
                self.from_prefetch[layer][s] = False

    def verify_chunks(self, layer: int, union):
        """The verify requests of one layer's union: cached members first, then
        the others, each part ascending, cut into chunks of S."""
        members = sorted(set(int(e) for e in union))
        cached = [e for e in members if self.slot_of(layer, e) >= 0]
        rest = [e for e in members if self.slot_of(layer, e) < 0]
        order = cached + rest
        return [order[i:i + self.S] for i in range(0, len(order), self.S)]

    def verify_layer(self, layer: int, union):
        for chunk in self.verify_chunks(layer, union):
            self.ensure(layer, chunk, VERIFY)

    def draft_layer(self, layer: int, topk, r: int = 1):
        """The drafter's request (its r routed experts), then the prefetch of
        the whole top-k."""
        topk = [int(e) for e in topk]
        self.ensure(layer, topk[:r], DRAFT)
        self.prefetch(layer, topk)

    def step_truncated(self, draft_topk, n_kept: int, verify_topk, r: int = 1):
        """One offloaded step with truncation (Algorithm 1 in its own order):
        every evaluated draft token requests its r routed experts in each
        layer; only a kept token (the first n_kept) then prefetches its top-k
        in every layer, after the keep decision; the stopped token prefetches
        nothing."""
        self.begin_block()
        for i, per_layer in enumerate(draft_topk):
            for layer, topk in enumerate(per_layer):
                self.ensure(layer, [int(e) for e in topk[:r]], DRAFT)
            if i < n_kept:
                for layer, topk in enumerate(per_layer):
                    self.prefetch(layer, topk)
        for layer, lists in enumerate(verify_topk):
            self.verify_layer(layer, [e for row in lists for e in row])

    def step(self, draft_topk, verify_topk, r: int = 1):
        """One offloaded step: draft_topk[i][l] the drafter's top-k at draft
        position i in layer l; verify_topk[l] the verify block's [T, k] lists;
        the drafter requests its r routed experts."""
        self.begin_block()
        for per_layer in draft_topk:
            for layer, topk in enumerate(per_layer):
                self.draft_layer(layer, topk, r)
        for layer, lists in enumerate(verify_topk):
            self.verify_layer(layer, [e for row in lists for e in row])
