"""Rounding helpers used by the oracle (test infrastructure only).

bf16 values travel as uint16 bit patterns.  fp16 metadata uses directed rounding from fp64 so that the
quantization grid [z, z + (2^b - 1) s] always covers the group's [min, max] (the paper fixes
min/max-derived scale and offset, Appendix E "Quantization Setting", but not their rounding).
Zero results are stored as +0, so the sign of a zero never depends on the order of a min/max.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_to_f32(b).astype(np.float64)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even (finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


F16_MAX = 65504.0


def f16_down(x: np.ndarray) -> np.ndarray:
    """Largest finite binary16 value <= x (x fp64), saturating at -65504; returned as float16."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore"):
        h = x.astype(np.float16)                   # single rounding fp64 -> fp16, nearest-even
        over = h.astype(np.float64) > x
        h = np.where(over, np.nextafter(h, np.float16(-np.inf)), h)
    # +inf (x > 65504) was nudged down to 65504 above; -inf (x < -65504) saturates here;
    # a zero result is stored as +0 (adding +0 turns -0 into +0)
    h = np.clip(h, np.float16(-F16_MAX), np.float16(F16_MAX)).astype(np.float16)
    return (h + np.float16(0.0)).astype(np.float16)


def f16_up(x: np.ndarray) -> np.ndarray:
    """Smallest finite binary16 value >= x (x fp64), saturating at +65504; returned as float16."""
    return ((-f16_down(-np.asarray(x, dtype=np.float64))) + np.float16(0.0)).astype(np.float16)
