"""TEST INFRASTRUCTURE: the parity rule between a GPU result and the oracle.

Tolerances (fixed for this path): indices, sizes, grid_thw and cu_seqlens
must be bit-exact; float32 pixel values within 2e-5 absolute of the
unrounded double-precision oracle value y; bfloat16 values pass when their
ordered-integer distance to round-to-nearest-even(y) is at most one unit in
the last place, or when |gpu - y| <= 2e-5.  The absolute floor is needed
because a bfloat16 ulp near zero (|y| below about 2^-9) is smaller than the
float32 accumulation error of the resampling sums.
"""
from __future__ import annotations

import numpy as np

F32_ATOL = 2e-5
BF16_ULPS = 1


def bf16_bits_rne(y: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bfloat16 bit patterns of double values (via float32)."""
    f = np.asarray(y, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return u.astype(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(
        np.float64)


def _ordered(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.int64)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def check_f32(gpu: np.ndarray, ref: np.ndarray) -> dict:
    g = np.asarray(gpu, dtype=np.float64)
    err = np.abs(g - ref)
    bad = ~(err <= F32_ATOL)          # NaN counts as bad
    return dict(ok=not bad.any(), n_bad=int(bad.sum()), max_err=float(np.nanmax(err)) if err.size else 0.0,
                n=int(err.size))


def check_bf16(gpu_bits: np.ndarray, ref: np.ndarray) -> dict:
    g = bf16_to_f64(gpu_bits)
    err = np.abs(g - ref)
    ulps = np.abs(_ordered(gpu_bits) - _ordered(bf16_bits_rne(ref)))
    good = (ulps <= BF16_ULPS) | (err <= F32_ATOL)
    good &= np.isfinite(g)
    return dict(ok=bool(good.all()), n_bad=int((~good).sum()), max_ulps=int(ulps.max()) if ulps.size else 0,
                max_err=float(np.nanmax(err)) if err.size else 0.0, n=int(err.size))
