"""Checks of the seeded input generators (CPU side)."""
import numpy as np
import torch

from workloads import configs, gen, rng


def test_splitmix64_reference_values():
    # SplitMix64 seeded with 0: the first outputs of the published generator.
    out = rng.raw_bits(0, 0, 3)
    assert [int(v) for v in out] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_streams_are_deterministic_and_sliceable():
    k = rng.key_for(2, 0, "routed", 3, 17)
    a = rng.normal_f32(k, 10000, 0.02)
    b = rng.normal_f32(k, 10000, 0.02)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(rng.normal_f32(k, 500, 0.02, start=1234), a[1234:1734])
    assert not np.array_equal(a, rng.normal_f32(rng.key_for(2, 0, "routed", 3, 18), 10000, 0.02))
    assert not np.array_equal(a, rng.normal_f32(rng.key_for(2, 1, "routed", 3, 17), 10000, 0.02))


def test_normal_moments():
    v = rng.normal_f32(rng.key_for(9, 0, "x", 0, 0), 2_000_000, 0.5).astype(np.float64)
    assert abs(v.mean()) < 3 * 0.5 / np.sqrt(v.size)
    assert abs(v.std() - 0.5) < 2e-3
    # Irwin-Hall(4): bounded tails, excess kurtosis -0.3
    assert np.abs(v).max() <= 0.5 * 2 * np.sqrt(3) + 1e-6
    kurt = ((v - v.mean()) ** 4).mean() / v.var() ** 2
    assert abs(kurt - 2.7) < 0.02


def test_bf16_rounding_matches_torch():
    v = rng.normal_f32(rng.key_for(9, 0, "x", 1, 0), 100000, 3.0)
    v[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 65504.0]  # ties to even
    ours = rng.f32_to_bf16_bits(v)
    theirs = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, theirs)
    np.testing.assert_array_equal(rng.bf16_bits_to_f32(ours),
                                  torch.from_numpy(v).to(torch.bfloat16).float().numpy())


def test_block_shapes_and_dtypes():
    c = configs.CFG1
    assert gen.routed_block(c, 0, 3).dtype == np.float32
    assert gen.routed_block(c, 0, 3).size == 3 * c.inter * c.hidden
    assert gen.shared_block(c, 0).size == 3 * c.shared_inter * c.hidden
    assert gen.draft_block(c, 0).size == 3 * c.draft_inter * c.hidden
    assert gen.router_weight(c, 0).shape == (c.n_experts, c.hidden)
    assert gen.router_bias(c, 0) is None
    c3 = configs.CFG3
    assert gen.router_bias(c3, 0).shape == (c3.n_experts,)
    x = gen.x_rows(c, 5, block=0)
    x2 = gen.x_rows(c, 5, block=0, redraws=[0, 0, 1, 0, 0])
    np.testing.assert_array_equal(x[[0, 1, 3, 4]], x2[[0, 1, 3, 4]])
    assert not np.array_equal(x[2], x2[2])


def test_zipf_bias_is_a_rank_law():
    b = gen.zipf_bias(configs.CFG5, 1, lam=0.5)
    r = np.argsort(-b, kind="stable")
    ranks = np.empty(64, dtype=np.int64)
    ranks[r] = np.arange(1, 65)
    np.testing.assert_allclose(b, (-0.5 * 1.1 * np.log(ranks)).astype(np.float32), rtol=1e-6)
    assert sorted(ranks.tolist()) == list(range(1, 65))
