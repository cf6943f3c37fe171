"""Pins of the oracle's binary16 conversions and hi/lo split (Sec. 4.4,
eqs. corr-1..corr-4) against things other than itself:

* numpy's float32 -> float16 conversion (an independent library routine,
  round to nearest even) over every non-NaN FP32 bit pattern;
* numpy's float16 -> float64 decode over all 2^16 patterns;
* hand-worked examples in tests/golden/split_examples.txt;
* the reconstruction bound |x - (hi + lo 2^-11)| <= 2^-22 |x| for
  2^-14 <= |x| <= 65504, checked on every FP32 value in that range;
* exact rational rounding (tests/exact.py) on random values.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact import round_f16

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "split_examples.txt")


def _all_f32_bits(chunk_bits=25):
    n = 1 << 32
    step = 1 << chunk_bits
    base = np.arange(step, dtype=np.uint32)
    for start in range(0, n, step):
        yield base + np.uint32(start)


def _check_against_numpy(bits: np.ndarray) -> int:
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    hi, _ = oracle.split(x)
    return int(np.count_nonzero(hi != ref))


@pytest.mark.slow
@pytest.mark.skipif(not os.environ.get("EXHAUSTIVE"), reason="set EXHAUSTIVE=1 (about 7 min)")
def test_f32_to_f16_exhaustive_against_numpy():
    """Every non-NaN FP32 bit pattern: oracle hi == numpy astype(float16)."""
    assert sum(_check_against_numpy(b) for b in _all_f32_bits()) == 0


def test_f32_to_f16_structured_against_numpy():
    """Default-sized sweep that reaches every rounding decision:
    * every sign and exponent, with all 2^13 patterns of the low 13 fraction
      bits (the bits a normal binary16 result rounds away) under several
      patterns of the kept 10 bits (zero, odd, even, all-ones for the carry);
    * every fraction of every exponent whose binary16 result is subnormal or
      at the normal/subnormal boundary (FP32 exponents 2^-25 .. 2^-14)."""
    low = np.arange(1 << 13, dtype=np.uint32)
    highs = np.array([0, 1, 2, 0x155, 0x2AA, 0x3FE, 0x3FF], dtype=np.uint32) << 13
    frac = (highs[:, None] | low[None, :]).ravel()
    se = np.arange(512, dtype=np.uint32) << 23
    bad = _check_against_numpy((se[:, None] | frac[None, :]).ravel())
    every = np.arange(1 << 23, dtype=np.uint32)
    for e in range(127 - 26, 127 - 13):
        bad += _check_against_numpy(every | np.uint32(e << 23))
    assert bad == 0


def test_f16_to_f32_all_patterns():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = h.view(np.float16).astype(np.float64)
    mine = oracle.f16_bits_to_f64(h)
    finite = np.isfinite(ref)
    assert np.array_equal(mine[finite], ref[finite])
    assert np.array_equal(np.isinf(mine), np.isinf(ref))
    # the C decoder as well, on every finite pattern
    lib_vals = np.array([oracle.f16_to_f32_scalar(int(v)) for v in h[finite][::97]])
    assert np.array_equal(lib_vals, ref[finite][::97])


def _parse_golden():
    rows = []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            expr, hi, lo, _why = [p.strip() for p in line.split(";", 3)]
            val = Fraction(eval(expr, {"__builtins__": {}}))  # arithmetic on literals only
            x = np.float32(float(val))
            assert Fraction(float(x)) == val, f"{expr} is not an FP32 value"
            rows.append((expr, x, int(hi, 16), int(lo, 16)))
    return rows


def test_golden_worked_examples():
    rows = _parse_golden()
    assert len(rows) >= 10
    xs = np.array([r[1] for r in rows], dtype=np.float32)
    hi, lo = oracle.split(xs)
    for (expr, _x, h, l), gh, gl in zip(rows, hi, lo):
        assert (int(gh), int(gl)) == (h, l), f"split({expr})"


def test_reconstruction_bound_every_value_in_range():
    """For 2^-14 <= x <= 65504 (positive; the negative side follows from the
    sign test below): |x - (hi + lo 2^-11)| <= 2^-22 |x|."""
    lo_bits = int(np.array(2.0 ** -14, dtype=np.float32).view(np.uint32))
    hi_bits = int(np.array(65504.0, dtype=np.float32).view(np.uint32))
    step = 1 << 25
    worst = 0.0
    for start in range(lo_bits, hi_bits + 1, step):
        stop = min(start + step, hi_bits + 1)
        x = np.arange(start, stop, dtype=np.uint32).view(np.float32)
        h, l = oracle.split(x)
        rec = h.view(np.float16).astype(np.float64) + \
            l.view(np.float16).astype(np.float64) * 2.0 ** -11
        rel = np.abs(x.astype(np.float64) - rec) / x.astype(np.float64)
        worst = max(worst, float(rel.max()))
    assert worst <= 2.0 ** -22
    # the bound is attained to within a factor of two (not vacuous)
    assert worst > 2.0 ** -24


def test_sign_symmetry_and_subnormal_range():
    g = np.random.default_rng(11)
    x = (g.standard_normal(200000) * 2.0 ** g.integers(-40, 16, 200000)).astype(np.float32)
    x = x[np.abs(x) <= 65504]
    h1, l1 = oracle.split(x)
    h2, l2 = oracle.split(-x)
    v1 = h1.view(np.float16).astype(np.float64)
    v2 = h2.view(np.float16).astype(np.float64)
    assert np.array_equal(v1, -v2)
    assert np.array_equal(l1.view(np.float16).astype(np.float64),
                          -l2.view(np.float16).astype(np.float64))


def test_split_against_exact_rounding():
    """hi and lo against exact rational round-to-nearest-even (binary16)."""
    g = np.random.default_rng(5)
    x = (g.uniform(-1, 1, 3000) * 2.0 ** g.integers(-30, 16, 3000)).astype(np.float32)
    x = np.concatenate([x, np.float32([1 + 2 ** -11, 2 ** -24, 2 ** -14, 65504, -3e-5])])
    h, l = oracle.split(x)
    for xi, hi, li in zip(x, h, l):
        q = Fraction(float(xi))
        ref_hi = round_f16(q)
        assert Fraction(float(np.uint16(hi).view(np.float16))) == ref_hi
        ref_lo = round_f16((q - ref_hi) * 2048)
        assert Fraction(float(np.uint16(li).view(np.float16))) == ref_lo


def test_fp16_representable_values_have_zero_lo():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = h.view(np.float16)
    v = v[np.isfinite(v)].astype(np.float32)
    hi, lo = oracle.split(v)
    assert np.array_equal(hi.view(np.float16).astype(np.float32), v)
    assert np.all(lo.view(np.float16).astype(np.float32) == 0)


@pytest.mark.parametrize("x,expect_inf", [(65519.0, False), (65520.0, True), (1e30, True)])
def test_overflow_edge(x, expect_inf):
    hi, _ = oracle.split(np.float32([x]))
    assert bool(np.isinf(hi.view(np.float16)[0])) == expect_inf
