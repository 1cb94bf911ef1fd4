"""The expert cache: the oracle simulation pinned on hand-worked cases, then
the library's bookkeeping (host copies, no GPU) against the simulation on
random request sequences, counts and slot tables exact."""
import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from oracle.cache_sim import DRAFT, VERIFY, CacheSim

# ------------------------------------------------------------ simulation pins


def test_lru_evicts_least_recently_used():
    c = CacheSim(1, 8, 2)
    c.ensure(0, [3], DRAFT)
    c.ensure(0, [5], DRAFT)
    c.ensure(0, [3], DRAFT)      # 3 used after 5
    c.ensure(0, [6], DRAFT)      # evicts 5 (slot 1)
    assert c.slot_table(0)[3] == 0 and c.slot_table(0)[6] == 1 and c.slot_table(0)[5] == -1
    assert c.counts["demand_loads"] == 3 and c.counts["evictions"] == 1
    assert c.counts["draft_needed"] == 4 and c.counts["draft_hits"] == 1


def test_everything_fits_loads_each_expert_once():
    rng = np.random.default_rng(3)
    c = CacheSim(2, 6, 6)
    touched = set()
    for _ in range(40):
        layer = int(rng.integers(2))
        need = list(rng.choice(6, size=int(rng.integers(1, 4)), replace=False))
        c.ensure(layer, need, VERIFY)
        touched.update((layer, int(e)) for e in need)
    assert c.counts["demand_loads"] == len(touched)
    assert c.counts["evictions"] == 0
    assert c.counts["verify_needed"] - c.counts["verify_hits"] == len(touched)


def test_exact_predictions_are_all_used():
    # Predicting exactly the union, with room for it: every prefetch is used,
    # every verify request hits, nothing is wasted.
    c = CacheSim(1, 16, 8)
    c.begin_block()
    c.prefetch(0, [2, 9, 4])
    c.prefetch(0, [9, 11])
    c.verify_layer(0, [11, 2, 4, 9, 2])
    c.begin_block()
    k = c.counts
    assert k["prefetch_issued"] == 4 and k["prefetch_used"] == 4 and k["prefetch_wasted"] == 0
    assert k["verify_needed"] == 4 and k["verify_hits"] == 4 and k["demand_loads"] == 0


def test_disjoint_predictions_are_all_wasted():
    c = CacheSim(1, 16, 8)
    c.begin_block()
    c.prefetch(0, [1, 2, 3])
    c.verify_layer(0, [7, 8])
    c.begin_block()
    k = c.counts
    assert k["prefetch_used"] == 0 and k["prefetch_wasted"] == 3 and k["demand_loads"] == 2
    assert k["verify_hits"] == 0


def test_prefetch_never_evicts_predicted_and_skips_when_full():
    c = CacheSim(1, 10, 2)
    c.begin_block()
    c.prefetch(0, [4, 5, 6])
    assert c.counts["prefetch_issued"] == 2 and c.counts["prefetch_skipped"] == 1
    assert sorted(e for e in c.slot[0]) == [4, 5]


def test_demand_load_falls_back_to_predicted_but_never_needed():
    c = CacheSim(1, 10, 2)
    c.begin_block()
    c.prefetch(0, [4, 5])
    c.ensure(0, [5, 7], VERIFY)     # 4 is predicted but not needed: evicted for 7
    assert c.slot_table(0)[4] == -1 and c.slot_table(0)[7] >= 0 and c.slot_table(0)[5] >= 0
    assert c.counts["prefetch_wasted"] == 1 and c.counts["prefetch_used"] == 1


def test_verify_chunks_put_cached_members_first():
    c = CacheSim(1, 12, 3)
    c.ensure(0, [9], DRAFT)
    c.ensure(0, [2], DRAFT)
    chunks = c.verify_chunks(0, [1, 2, 5, 9, 11, 0])
    assert chunks == [[2, 9, 0], [1, 5, 11]]
    c.verify_layer(0, [1, 2, 5, 9, 11, 0])
    assert c.counts["verify_needed"] == 6 and c.counts["verify_hits"] == 2


# ---------------------------------------------- library bookkeeping vs simulation


def fake_cache(L, N, S, eb=64):
    host = torch.arange(L * N * eb, dtype=torch.int64).remainder(251).to(torch.uint8)
    return de.ExpertCache(L, N, S, eb, host, fake=True), host.view(L, N, eb)


def check_same(cache, sim, host, eb):
    got = cache.stats()
    for name in de.CACHE_COUNTS:
        want = sim.counts[name] * (eb if name == "bytes_copied" else 1)
        assert got[name] == want, name
    for layer in range(sim.L):
        table = cache.slots(layer)
        assert table == sim.slot_table(layer)
        pool = cache.slot_pool.view(sim.L, sim.S, cache.stride)
        for e, s in enumerate(table):
            if s >= 0:
                assert torch.equal(pool[layer, s, :eb], host[layer, e])


@pytest.mark.parametrize("seed,S", [(0, 1), (1, 2), (2, 4), (3, 6), (4, 8)])
def test_library_bookkeeping_matches_simulation(seed, S):
    rng = np.random.default_rng(seed)
    L, N, k, eb = 3, 8, 3, 64
    cache, host = fake_cache(L, N, S, eb)
    sim = CacheSim(L, N, S)
    for _ in range(6):
        K = int(rng.integers(1, 5))
        draft = [[list(rng.choice(N, size=k, replace=False)) for _ in range(L)] for _ in range(K)]
        verify = [[list(rng.choice(N, size=k, replace=False)) for _ in range(K + 1)]
                  for _ in range(L)]
        sim.begin_block()
        cache.begin_block()
        for per_layer in draft:
            for layer, topk in enumerate(per_layer):
                sim.draft_layer(layer, topk)
                cache.ensure(layer, [topk[0]], de.DE_NEED_DRAFT)
                cache.prefetch(layer, topk)
                check_same(cache, sim, host, eb)
        for layer, lists in enumerate(verify):
            union = [e for row in lists for e in row]
            for chunk in sim.verify_chunks(layer, union):
                sim.ensure(layer, chunk, VERIFY)
                cache.ensure(layer, chunk, de.DE_NEED_VERIFY)
                check_same(cache, sim, host, eb)
                # the layer's slot table marks exactly the chunk resident
                row = cache.slot_map.view(L, N)[layer].tolist()
                assert [e for e in range(N) if row[e] >= 0] == sorted(chunk)
    sim.begin_block()
    cache.begin_block()
    check_same(cache, sim, host, eb)
    k = cache.stats()
    assert k["prefetch_used"] + k["prefetch_wasted"] == k["prefetch_issued"]
    cache.reset()
    assert all(v == 0 for v in cache.stats().values())
    assert all(s == -1 for layer in range(L) for s in cache.slots(layer))


def test_cache_rejects_bad_arguments():
    cache, _ = fake_cache(2, 8, 3)
    with pytest.raises(de.DEError):
        cache.ensure(0, [1, 2, 3, 4], de.DE_NEED_VERIFY)      # more than the slots
    with pytest.raises(de.DEError):
        cache.ensure(0, [1, 1], de.DE_NEED_VERIFY)            # repeated id
    with pytest.raises(de.DEError):
        cache.ensure(0, [8], de.DE_NEED_DRAFT)                # id out of range
    with pytest.raises(de.DEError):
        cache.ensure(2, [1], de.DE_NEED_DRAFT)                # layer out of range
    with pytest.raises(de.DEError):
        cache.ensure(0, [1], 7)                               # unknown purpose
    with pytest.raises(de.DEError):
        cache.prefetch(0, [9])
    assert all(v == 0 for v in cache.stats().values())        # nothing was counted
    host = torch.zeros(2 * 8 * 64, dtype=torch.uint8)
    with pytest.raises(de.DEError):
        de.ExpertCache(2, 8, 9, 64, host, fake=True)          # more slots than experts
    with pytest.raises(de.DEError):
        de.ExpertCache(2, 8, 2, 60, host, fake=True)          # block not a multiple of 16


def test_zipf_bias_scale_is_the_recorded_calibration():
    # The skewed-routing workload's bias scale was fitted so that expert
    # selection share falls off with rank like rank^-1.1; a smaller sample of
    # a different activation stream reproduces the slope.
    import json
    import os
    import sys
    from workloads import configs, gen
    here = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
    rec = json.load(open(os.path.join(here, "zipf_lambda.json")))
    assert configs.CFG5.zipf_lam == rec["lam"]
    assert abs(rec["slope"] - rec["target_slope"]) < 0.01
    sys.path.insert(0, here)
    import calibrate_zipf as cz
    m = configs.CFG5.moe
    x = gen.x_rows(m, 20_000, block=9002).astype(np.float64)
    w = gen.router_weight(m, cz.LAYER).astype(np.float64)
    s, share = cz.slope(configs.CFG5, x, w, rec["lam"])
    assert abs(s + 1.1) < 0.05
    assert share.max() < 1.0 / m.top_k
