"""Plain fp64 dequantisation of Q4_0 expert weights (the 4.5-bit block format
of the mobile platform, Section 4.1).

TEST INFRASTRUCTURE ONLY (same rule as ``oracle.moe``).

A block holds 32 consecutive weights of a row: 16 bytes of 4-bit codes q
(byte j: weight j in its low nibble, weight j + 16 in its high nibble) and an
fp16 scale d; weight = d * (q - 8).  A matrix [rows, cols] (cols a multiple
of 32) stores every row's codes first (row r at byte r * cols / 2, block b of
the row at 16 b), then every row's scales (row r's at rows * cols / 2 +
r * cols / 16, one fp16 per block).  An expert block is [G][U][D] with G, U
[I, H] and D [H, I], each such a matrix.
"""
from __future__ import annotations

import numpy as np


def matrix_bytes(rows: int, cols: int) -> int:
    """18 bytes per 32 weights."""
    return rows * cols * 9 // 16


def dequant(buf, rows: int, cols: int) -> np.ndarray:
    """fp64 [rows, cols] from one matrix's bytes."""
    if cols % 32:
        raise ValueError("Q4_0 rows hold whole 32-weight blocks")
    buf = np.asarray(buf, dtype=np.uint8)
    nc = rows * cols // 2
    codes = buf[:nc].reshape(rows, cols // 32, 16)
    scales = buf[nc:nc + rows * cols // 16].view(np.float16).astype(np.float64)
    scales = scales.reshape(rows, cols // 32)
    lo = (codes & 0x0F).astype(np.float64) - 8.0      # weights 0..15 of each block
    hi = (codes >> 4).astype(np.float64) - 8.0        # weights 16..31
    q = np.concatenate([lo, hi], axis=2)               # [rows, blocks, 32] in weight order
    return (q * scales[:, :, None]).reshape(rows, cols)


def split_expert(block, inter: int, hidden: int):
    """fp64 (G [I,H], U [I,H], D [H,I]) from a Q4_0 expert block."""
    block = np.asarray(block, dtype=np.uint8)
    mg = matrix_bytes(inter, hidden)
    return (dequant(block[:mg], inter, hidden), dequant(block[mg:2 * mg], inter, hidden),
            dequant(block[2 * mg:2 * mg + matrix_bytes(hidden, inter)], hidden, inter))
