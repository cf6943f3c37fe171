"""Pins of the GEMM oracle (C = A.B, Sec. 2.2; error metric of Sec. 4.4.2;
method model of Sec. 4.4, eq. corr-5) against things other than itself:

* brute force on tiny shapes with exact rational arithmetic (Fractions);
* the plain FP32 product bit-for-bit against an exact model of the fmaf
  chain (one binary32 rounding per step, tests/exact.py);
* the method-exact model against exact rationals over an independently
  computed split (numpy's float16 conversion);
* exactness for integer inputs in binary16 range;
* the scan example of Sec. 4.1 (a^T U = prefix sums, u_ij = [i <= j]);
* the textbook bound |C32 - C64| <= gamma_k (|A||B|);
* consistency of the sampled form with the full form.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact import fmaf, round_f16


def _rand(shape, seed, scale_exp=0):
    g = np.random.default_rng(seed)
    x = g.uniform(-1, 1, shape) * 2.0 ** g.integers(-scale_exp, scale_exp + 1, shape)
    return x.astype(np.float32)


@pytest.mark.parametrize("m,n,k,seed", [(1, 1, 1, 0), (2, 3, 4, 1), (5, 4, 5, 2),
                                        (3, 5, 2, 3), (4, 4, 7, 4)])
def test_brute_force_exact_rationals(m, n, k, seed):
    A = _rand((1, m, k), seed, 10)
    B = _rand((1, k, n), seed + 100, 10)
    out = oracle.gemm(A, B)
    u53 = 2.0 ** -53
    for i in range(m):
        for j in range(n):
            exact = sum(Fraction(float(A[0, i, t])) * Fraction(float(B[0, t, j]))
                        for t in range(k))
            nrm = sum(abs(Fraction(float(A[0, i, t])) * Fraction(float(B[0, t, j])))
                      for t in range(k))
            # FP64 sum of exact products: at most (k-1) roundings of size u|partial|
            assert abs(Fraction(out["c64"][0, i, j]) - exact) <= k * u53 * nrm
            assert abs(Fraction(out["n64"][0, i, j]) - nrm) <= k * u53 * nrm
            # plain FP32: the fmaf chain, bit for bit
            c = np.float32(0)
            for t in range(k):
                c = fmaf(A[0, i, t], B[0, t, j], c)
            assert out["c32"][0, i, j].view(np.uint32) == c.view(np.uint32)


@pytest.mark.parametrize("k,seed", [(1, 7), (3, 8), (6, 9)])
def test_method_model_against_exact_split(k, seed):
    """CM = sum_k hiA hiB + (loA hiB + hiA loB) 2^-11, with hi/lo from numpy's
    float16 conversion and the sum taken exactly."""
    m, n = 3, 4
    A = _rand((1, m, k), seed, 12)
    B = _rand((1, k, n), seed + 1, 12)
    out = oracle.gemm(A, B, want=("cm",))

    def sp(x):
        h = np.float32(x).astype(np.float16)
        q = Fraction(float(x)) - Fraction(float(h))
        lo = round_f16(q * 2048)
        return Fraction(float(h)), lo

    for i in range(m):
        for j in range(n):
            s = Fraction(0)
            mag = Fraction(0)
            for t in range(k):
                ah, al = sp(A[0, i, t])
                bh, bl = sp(B[0, t, j])
                term = ah * bh + (al * bh + ah * bl) / 2048
                s += term
                mag += abs(term)
            assert abs(Fraction(out["cm"][0, i, j]) - s) <= k * 2.0 ** -53 * mag


def test_integer_inputs_exact():
    """fp16-representable integers with |partial sums| < 2^24: every oracle
    quantity is the exact integer product."""
    g = np.random.default_rng(3)
    A = g.integers(-31, 32, (2, 17, 40)).astype(np.float32)
    B = g.integers(-31, 32, (2, 40, 9)).astype(np.float32)
    out = oracle.gemm(A, B)
    ref = np.einsum("bik,bkj->bij", A.astype(np.int64), B.astype(np.int64))
    assert np.array_equal(out["c64"], ref.astype(np.float64))
    assert np.array_equal(out["c32"], ref.astype(np.float32))
    assert np.array_equal(out["cm"], ref.astype(np.float64))


def test_scan_example_prefix_sums():
    """Sec. 4.1: the row vector a times the upper-triangular all-ones U gives
    the prefix sums of a."""
    n = 37
    a = np.arange(1, n + 1, dtype=np.float32)[None, None, :] * np.float32(3)
    U = np.triu(np.ones((n, n), dtype=np.float32))[None]
    out = oracle.gemm(a, U)
    expect = np.cumsum(a[0, 0].astype(np.float64))
    assert np.array_equal(out["c64"][0, 0], expect)
    assert np.array_equal(out["c32"][0, 0], expect.astype(np.float32))
    assert np.array_equal(out["cm"][0, 0], expect)


def test_fp16_representable_inputs_model_equals_fp64():
    """With lo = 0 on both sides the model is the FP64 sum of the same exact
    products in the same order as C64."""
    g = np.random.default_rng(4)
    A = g.uniform(-2, 2, (1, 8, 50)).astype(np.float16).astype(np.float32)
    B = g.uniform(-2, 2, (1, 50, 6)).astype(np.float16).astype(np.float32)
    out = oracle.gemm(A, B)
    assert np.array_equal(out["cm"], out["c64"])


def test_fp32_textbook_bound_and_fp64_agreement():
    A = _rand((3, 20, 300), 5)
    B = _rand((3, 300, 11), 6)
    out = oracle.gemm(A, B)
    k = 300
    u = 2.0 ** -24
    gamma = k * u / (1 - k * u)
    assert np.all(np.abs(out["c32"] - out["c64"]) <= gamma * out["n64"])
    ref = np.einsum("bik,bkj->bij", A.astype(np.float64), B.astype(np.float64))
    assert np.allclose(out["c64"], ref, rtol=0, atol=1e-12)
    assert np.allclose(out["n64"], np.einsum("bik,bkj->bij", np.abs(A).astype(np.float64),
                                             np.abs(B).astype(np.float64)), rtol=1e-14, atol=0)


def test_dropped_correction_is_visible():
    """The model keeps both correction products: dropping one of them (a
    plausible mistake) moves the result by far more than FP64 rounding."""
    A = _rand((1, 4, 64), 12)
    B = _rand((1, 64, 4), 13)
    out = oracle.gemm(A, B)
    hiA = A.astype(np.float16).astype(np.float64)
    hiB = B.astype(np.float16).astype(np.float64)
    only_hi = np.einsum("bik,bkj->bij", hiA, hiB)
    # the model is much closer to C64 than hi*hi alone
    e_model = oracle.max_rel_err(out["cm"], out["c64"], out["n64"])
    e_hi = oracle.max_rel_err(only_hi, out["c64"], out["n64"])
    assert e_model < 2.0 ** -20 and e_hi > 2.0 ** -14


def test_transposed_operand_detected():
    A = _rand((1, 5, 5), 14)
    B = _rand((1, 5, 5), 15)
    out = oracle.gemm(A, B, want=("c64",))
    wrong = oracle.gemm(A, np.ascontiguousarray(B.transpose(0, 2, 1)), want=("c64",))
    assert not np.allclose(out["c64"], wrong["c64"])
    assert np.allclose(out["c64"][0], A[0].astype(np.float64) @ B[0].astype(np.float64),
                       rtol=0, atol=1e-13)


def test_sampled_dots_equal_full_gemm():
    A = _rand((2, 9, 33), 16)
    B = _rand((2, 33, 7), 17)
    full = oracle.gemm(A, B)
    idx = [(0, 0, 0), (1, 8, 6), (0, 4, 3), (1, 2, 5)]
    ar = np.stack([A[b, i, :] for b, i, _ in idx])
    bc = np.stack([B[b, :, j] for b, _, j in idx])
    s = oracle.dots(ar, bc)
    for t, (b, i, j) in enumerate(idx):
        for key in ("c64", "n64", "c32", "cm"):
            assert s[key][t] == full[key][b, i, j]


def test_k_zero_and_empty():
    A = np.zeros((1, 3, 0), np.float32)
    B = np.zeros((1, 0, 4), np.float32)
    out = oracle.gemm(A, B)
    assert np.all(out["c64"] == 0) and np.all(out["c32"] == 0)
    out = oracle.gemm(np.zeros((0, 3, 2), np.float32), np.zeros((0, 2, 4), np.float32))
    assert out["c64"].shape == (0, 3, 4)


def test_metric():
    c64 = np.array([1.0, 0.0, 2.0])
    n64 = np.array([2.0, 0.0, 4.0])
    assert oracle.max_rel_err(np.array([1.5, 0.0, 2.0]), c64, n64) == 0.25
    assert oracle.max_rel_err(np.array([1.0, 1e-30, 2.0]), c64, n64) == float("inf")
    assert oracle.max_rel_err(np.array([np.nan, 0.0, 2.0]), c64, n64) == float("inf")
