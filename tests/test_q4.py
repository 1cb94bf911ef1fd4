"""Pins of the Q4_0 dequantisation oracle (the 4.5-bit block format of the
paper's mobile platform, Section 4.1).

Hand-built blocks with known codes and scales, the nibble order, fp16 scale
decoding against NumPy's float16, the placement of every row and block, and
the size the paper states (18-byte blocks of 32 weights, 4.5 bits per
weight, about 3.6x fewer expert bytes than bf16).
"""
import numpy as np
import pytest

from oracle import moe, q4
from workloads import configs, gen


def _fp16_bits(v) -> np.ndarray:
    return np.asarray(v, dtype=np.float16).view(np.uint8)


def test_one_block_by_hand():
    codes = np.array([(j & 0xF) | ((15 - j) << 4) for j in range(16)], dtype=np.uint8)
    buf = np.concatenate([codes, _fp16_bits([0.5])])
    w = q4.dequant(buf, 1, 32)[0]
    want = [0.5 * (j - 8) for j in range(16)] + [0.5 * (7 - j) for j in range(16)]
    assert w.tolist() == want


@pytest.mark.parametrize("bits,value", [(0x3C00, 1.0), (0xB800, -0.5), (0x0001, 2.0 ** -24),
                                        (0x7BFF, 65504.0)])
def test_scale_decoding_matches_float16(bits, value):
    codes = np.full(16, 0x99, dtype=np.uint8)          # q = 9 in both nibbles: weight = d
    buf = np.concatenate([codes, np.array([bits], np.uint16).view(np.uint8)])
    w = q4.dequant(buf, 1, 32)[0]
    assert np.all(w == value)
    assert value == float(np.array([bits], np.uint16).view(np.float16)[0])


def test_row_and_block_placement():
    rows, cols = 3, 96
    nb = cols // 32
    codes = np.full(rows * cols // 2, 0x88, dtype=np.uint8)   # every weight 0
    scales = np.array([1 + 4 * r + b for r in range(rows) for b in range(nb)], np.float16)
    for r, b, j in [(0, 0, 0), (1, 2, 15), (2, 1, 7)]:
        buf_codes = codes.copy()
        buf_codes[r * cols // 2 + 16 * b + j] = 0x3A          # low nibble 10, high nibble 3
        w = q4.dequant(np.concatenate([buf_codes, scales.view(np.uint8)]), rows, cols)
        nz = np.argwhere(w != 0).tolist()
        assert nz == [[r, 32 * b + j], [r, 32 * b + 16 + j]]
        d = 1 + 4 * r + b
        assert w[r, 32 * b + j] == 2.0 * d and w[r, 32 * b + 16 + j] == -5.0 * d


def test_size_is_four_and_a_half_bits_per_weight():
    assert q4.matrix_bytes(1, 32) == 18
    c = configs.CFG2_Q4
    assert c.expert_bytes() == 3 * 2048 * 1408 * 9 // 16 == 4_866_048
    assert configs.CFG2.expert_bytes() / c.expert_bytes() == pytest.approx(32 / 9)
    assert round(32 / 9, 1) == 3.6


def test_generated_expert_splits_into_three_matrices():
    c = configs.CFG2_Q4
    blk = gen.routed_block(c, 0, 5)
    assert blk.dtype == np.uint8 and blk.size == c.expert_bytes()
    g, u, d = moe.split_expert(blk, c.inter, c.hidden)
    assert g.shape == (c.inter, c.hidden) and u.shape == g.shape and d.shape == (c.hidden, c.inter)
    # Codes are uniform 4-bit values and scales lie in [2^-8, 2^-7): every
    # weight is d (q - 8) with |q - 8| <= 8.
    for m in (g, u, d):
        assert np.all(np.abs(m) < 8 * 2.0 ** -7)
    assert 0.02 < float(np.std(d)) < 0.04
    # The second matrix is U, not a repeat of G.
    assert not np.array_equal(g, u)
