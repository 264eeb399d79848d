"""CPU pins of the parity rule (oracle/compare.py): bfloat16 rounding of the
oracle's double values and the tolerance checks built on it.

The rounding must be one round-to-nearest-even step from the double to the
bfloat16 grid (8 significant bits).  Rounding through float32 first can land
a value exactly on a bfloat16 tie and then round it the wrong way; these
tests plant such values.  The reference below is exact rational arithmetic
over the neighbouring bfloat16 values, independent of the code under test.
"""
from fractions import Fraction

import numpy as np

from oracle import compare


def _bf16_float(bits: int) -> np.float32:
    return np.array([bits << 16], np.uint32).view(np.float32)[0]


def _bf16_value(bits: int) -> Fraction:
    return Fraction(float(_bf16_float(bits)))


def _nearest_even_exact(v: float) -> int:
    """The bfloat16 bit pattern nearest to v, ties to the even pattern, by
    exact comparison with the candidates around v's float32 truncation."""
    top = int(np.array([v], np.float32).view(np.uint32)[0]) >> 16
    best = None
    for c in (top - 1, top, top + 1):
        c &= 0xFFFF
        if not np.isfinite(float(_bf16_float(c))):
            continue
        d = abs(_bf16_value(c) - Fraction(v))
        key = (d, c & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_rounds_once_from_the_double():
    # 1 + 2^-8 is the tie between 1 and 1 + 2^-7; a value just above it must
    # round up, although its float32 rounding is the tie itself (which then
    # rounds to even, down)
    y = np.array([1 + 2**-8 + 2**-30, -(1 + 2**-8 + 2**-30), 1 + 2**-8, 1 + 3 * 2**-8, 1 + 3 * 2**-8 - 2**-40])
    assert compare.bf16_bits_rne(y).tolist() == [0x3F81, 0xBF81, 0x3F80, 0x3F82, 0x3F81]
    via_f32 = (y.astype(np.float32).view(np.uint32).astype(np.uint64) + 0x7FFF
               + ((y.astype(np.float32).view(np.uint32).astype(np.uint64) >> 16) & 1)) >> 16
    assert via_f32[0] == 0x3F80   # the double rounding the rule avoids


def test_matches_exact_rational_rounding():
    rng = np.random.default_rng(11)
    x = rng.standard_normal(3000) * 10.0 ** rng.integers(-30, 30, 3000)
    # values at and around bfloat16 midpoints, where a wrong rounding shows
    mids = []
    for bits in rng.integers(0x0080, 0x7F00, 300):
        a, b = _bf16_value(int(bits)), _bf16_value(int(bits) + 1)
        m = float((a + b) / 2)
        mids += [m, np.nextafter(m, 0.0), np.nextafter(m, np.inf), -m]
    x = np.concatenate([x, np.array(mids), [0.0, 2.0**-130, 3.0e-39, 1.0, 255 / 127]])
    got = compare.bf16_bits_rne(x)
    assert [int(g) for g in got] == [_nearest_even_exact(float(v)) for v in x]


def test_check_bf16_tolerance():
    y = np.array([1.0, 1.0, 1.0, 1e-7, -3.0])
    one_ulp = np.array([0x3F81, 0x3F7F, 0x3F80, 0x0000, 0xC040], np.uint16)
    assert compare.check_bf16(one_ulp, y)["ok"]
    two_ulp = one_ulp.copy()
    two_ulp[0] = 0x3F82
    r = compare.check_bf16(two_ulp, y)
    assert not r["ok"] and r["n_bad"] == 1 and r["max_ulps"] == 2
    # far in ulps but within the absolute floor of 2e-5: passes
    tiny = np.array([1.5e-5])
    assert compare.check_bf16(compare.bf16_bits_rne(np.array([0.0])), tiny)["ok"]
    nan = np.array([0x7FC0], np.uint16)
    assert not compare.check_bf16(nan, np.array([1.0]))["ok"]


def test_check_f32_tolerance():
    y = np.array([0.5, -1.25, 3.0])
    assert compare.check_f32(y + 1.9e-5, y)["ok"]
    assert not compare.check_f32(y + np.array([0.0, 2.1e-5, 0.0]), y)["ok"]
    assert not compare.check_f32(np.array([np.nan, -1.25, 3.0]), y)["ok"]


def test_merge_of_partial_results():
    a = compare.check_bf16(np.array([0x3F80], np.uint16), np.array([1.0]))
    b = compare.check_bf16(np.array([0x3F82], np.uint16), np.array([1.0]))
    m = compare.merge([a, b])
    assert m["n"] == 2 and m["n_bad"] == 1 and not m["ok"] and m["max_ulps"] == 2
