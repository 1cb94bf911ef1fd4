"""Counter-based synthetic number streams, bit-identical on the CPU and the GPU.

Every generated value is a pure function of (stream key, element counter), so
any slice of any tensor can be regenerated on its own, in any order, and the
GPU fill kernel in ``workloads/csrc/synth_fill.hip`` writes exactly the same
bits as the NumPy code below.

Generator
    SplitMix64 (G. Steele, D. Lea, C. Flood, "Fast splittable pseudorandom
    number generators", OOPSLA 2014) run in counter mode: element ``i`` of the
    stream with key ``k`` is ``mix64(k + (i + 1) * GAMMA)``, where ``mix64`` is
    the published 64-bit finaliser (xor-shift 30, multiply, xor-shift 27,
    multiply, xor-shift 31) and GAMMA is the golden-ratio increment.

Approximately normal values
    The 64 output bits are split into four 16-bit uniforms whose centred sum
    (Irwin-Hall, n=4) is scaled to the requested standard deviation.  All of it
    is integer arithmetic up to one correctly rounded fp64 multiply and one
    correctly rounded fp64->fp32 conversion, so both sides agree bit for bit.
    The tails are bounded at about +-3.46 sigma and the kurtosis is 2.7 instead
    of 3; for random weights and activations that is immaterial.

bf16
    Round-to-nearest-even of the fp32 value, kept as raw uint16 bits.

This module holds no arithmetic of the method itself: it only draws numbers.
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB

# Irwin-Hall(4) over 16-bit uniforms: mean 4 * 32767.5, variance (65536^2-1)/3.
IH_CENTER = 131070
IH_STD = float(np.sqrt((65536.0 ** 2 - 1.0) / 3.0))

# Stable numeric tags naming each synthetic tensor family.
TAGS = {
    "x": 1,
    "router": 2,
    "bias": 3,
    "routed": 4,
    "shared": 5,
    "draft": 6,
    "dense": 7,
    "emb": 8,
    "lm": 9,
    "token": 10,
    "perm": 11,
    "probe": 12,
}


def _mix64_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def stream_key(*fields: int) -> int:
    """Fold integer fields (config id, redraw, tag, layer, index, ...) into a key."""
    k = 0x243F6A8885A308D3  # arbitrary non-zero start (hex digits of pi)
    for f in fields:
        k = _mix64_int((k ^ (int(f) & MASK64)) + GAMMA)
    return k


def key_for(cfg_id: int, redraw: int, tag: str, layer: int = 0, index: int = 0) -> int:
    return stream_key(cfg_id, redraw, TAGS[tag], layer, index)


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
    return z ^ (z >> np.uint64(31))


def raw_bits(key: int, start: int, n: int) -> np.ndarray:
    """uint64 outputs for counters start .. start+n-1 of stream ``key``."""
    ctr = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + ctr * np.uint64(GAMMA)
        return _mix64(z)


def normal_f32_ref(key: int, n: int, std: float, start: int = 0) -> np.ndarray:
    """n approximately N(0, std^2) fp32 values from stream ``key`` (NumPy definition)."""
    out = np.empty(n, dtype=np.float32)
    chunk = 1 << 22
    scale = float(std) / IH_STD
    m16 = np.uint64(0xFFFF)
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        u = raw_bits(key, start + c0, c1 - c0)
        s = ((u & m16) + ((u >> np.uint64(16)) & m16) + ((u >> np.uint64(32)) & m16)
             + (u >> np.uint64(48))).astype(np.int64) - IH_CENTER
        out[c0:c1] = (s.astype(np.float64) * scale).astype(np.float32)
    return out


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as raw uint16 bits (no NaNs here)."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((b >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    with np.errstate(over="ignore"):
        return ((b + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16_ref(key: int, n: int, std: float, start: int = 0) -> np.ndarray:
    """bf16 bits of normal_f32_ref (NumPy definition)."""
    return f32_to_bf16_bits(normal_f32_ref(key, n, std, start))


# ---- fast path: the same streams from a small C library, run on several threads

_CLIB = None
_THREADS = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))


def _clib():
    global _CLIB
    if _CLIB is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdesynth_cpu.so")
        if not os.path.exists(path):
            _CLIB = False
        else:
            lib = ctypes.CDLL(path)
            for name in ("synth_normal_f32", "synth_normal_bf16"):
                fn = getattr(lib, name)
                fn.restype = None
                fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                               ctypes.c_double]
            _CLIB = lib
    return _CLIB


def _fill_c(fn, out: np.ndarray, key: int, std: float, start: int):
    n = out.size
    scale = float(std) / IH_STD
    esz = out.itemsize
    base = out.ctypes.data
    chunk = 1 << 20
    spans = [(c0, min(n, c0 + chunk)) for c0 in range(0, n, chunk)]
    if len(spans) <= 1:
        fn(base, n, key, start, scale)
        return out
    with ThreadPoolExecutor(max_workers=_THREADS) as ex:
        list(ex.map(lambda sp: fn(base + sp[0] * esz, sp[1] - sp[0], key, start + sp[0], scale), spans))
    return out


def normal_f32(key: int, n: int, std: float, start: int = 0) -> np.ndarray:
    """n approximately N(0, std^2) fp32 values from stream ``key``."""
    lib = _clib()
    if not lib:
        return normal_f32_ref(key, n, std, start)
    return _fill_c(lib.synth_normal_f32, np.empty(n, dtype=np.float32), key, std, start)


def normal_bf16(key: int, n: int, std: float, start: int = 0) -> np.ndarray:
    """n approximately N(0, std^2) values, rounded to bf16, as uint16 bits."""
    lib = _clib()
    if not lib:
        return normal_bf16_ref(key, n, std, start)
    return _fill_c(lib.synth_normal_bf16, np.empty(n, dtype=np.uint16), key, std, start)


def bytes_u8(key: int, n: int, start_word: int = 0) -> np.ndarray:
    """n raw bytes: the little-endian bytes of outputs start_word, start_word+1, ..."""
    return raw_bits(key, start_word, (n + 7) // 8).view(np.uint8)[:n].copy()


# Q4_0 scales: fp16 2^-8 * (1 + m / 1024) with m 10 random bits (exponent field
# 7), so that d * (q - 8) over uniform 4-bit codes has a spread like the other
# synthetic weights (about 0.027).
Q4_SCALE_EXP = 7


def q4_scale_bits(key: int, n: int, start: int = 0) -> np.ndarray:
    """n fp16 bit patterns of positive Q4_0 block scales."""
    m = (raw_bits(key, start, n) & np.uint64(0x3FF)).astype(np.uint16)
    return (np.uint16(Q4_SCALE_EXP << 10) | m).astype(np.uint16)


def uniform_int(key: int, n: int, high: int, start: int = 0) -> np.ndarray:
    """n integers in [0, high) (modulo reduction; the bias is < 2^-40 for our ranges)."""
    return (raw_bits(key, start, n) % np.uint64(high)).astype(np.int64)


def uniform_f64(key: int, n: int, start: int = 0) -> np.ndarray:
    """n doubles in [0, 1) from the top 53 bits."""
    return (raw_bits(key, start, n) >> np.uint64(11)).astype(np.float64) * (1.0 / (1 << 53))
