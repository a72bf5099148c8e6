"""Stored-value decoding and rounding, written from the IEEE-754 / bfloat16 bit layouts.

Test infrastructure only (see the package docstring).

The oracle works on the exact values the library sees: fp32, bf16 or fp16 bit patterns,
decoded exactly to fp64.  ``round_f32_to_bf16`` / ``round_f32_to_f16`` give the bits an
fp32 -> storage conversion with round-to-nearest-even must produce; they define the
expected slab contents after an upsert of fp32 rows.
"""
from __future__ import annotations

import numpy as np


def decode(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Bit patterns (uint32 for f32, uint16 for bf16 / f16) -> exact fp64 values."""
    bits = np.asarray(bits)
    if dtype == "f32":
        return bits.astype(np.uint32).view(np.float32).astype(np.float64)
    if dtype == "bf16":
        # bfloat16 is the upper half of an fp32 word.
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return bits.astype(np.uint16).view(np.float16).astype(np.float64)
    raise ValueError(dtype)


def round_f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits with round-to-nearest, ties to even; NaN stays NaN (quiet)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lower = u & 0xFFFF
    upper = u >> 16
    # Round up when the dropped half is above the midpoint, or exactly at it with an odd upper half.
    up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & 1) == 1))
    r = (upper + up.astype(np.uint64)) & 0xFFFF
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r = np.where(nan, (upper | 0x40) & 0xFFFF, r)
    return r.astype(np.uint16)


def round_f32_to_f16(x: np.ndarray) -> np.ndarray:
    """fp32 -> fp16 bits with round-to-nearest-even (numpy's IEEE half conversion)."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)
