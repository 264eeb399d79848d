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
    """Round-to-nearest-even bfloat16 bit patterns of double values, rounded
    once, straight from the double (no float32 step, which could round a
    value onto a bfloat16 tie first).  bfloat16 keeps 8 significant bits and
    float32's exponent range; values below the smallest normal (2^-126) round
    on the subnormal grid of 2^-133.  Finite inputs only."""
    y = np.asarray(y, dtype=np.float64)
    m, e = np.frexp(y)                          # y = m * 2^e, 0.5 <= |m| < 1 (m = 0 for y = 0)
    e = np.maximum(e, -125)                     # the smallest normal 2^-126 has e = -125
    q = np.rint(np.ldexp(y, 8 - e))             # significand on the 8-bit grid, ties to even (exact)
    v = np.ldexp(q, e - 8).astype(np.float32)   # a bfloat16 value: exact in float32
    return (v.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


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
    beyond_floor = ~(err <= F32_ATOL)
    good = (ulps <= BF16_ULPS) | ~beyond_floor
    good &= np.isfinite(g)
    # max_ulps: the largest ulp distance where the absolute floor does not apply
    return dict(ok=bool(good.all()), n_bad=int((~good).sum()),
                max_ulps=int(ulps[beyond_floor].max()) if beyond_floor.any() else 0,
                max_err=float(np.nanmax(err)) if err.size else 0.0, n=int(err.size))


def merge(results) -> dict:
    """One result from the results of several parts of an output (the parts
    are checked separately, e.g. one frame pair at a time)."""
    results = list(results)
    out = dict(ok=all(r["ok"] for r in results), n_bad=sum(r["n_bad"] for r in results),
               max_err=max((r["max_err"] for r in results), default=0.0),
               n=sum(r["n"] for r in results))
    if any("max_ulps" in r for r in results):
        out["max_ulps"] = max((r.get("max_ulps", 0) for r in results), default=0)
    return out
