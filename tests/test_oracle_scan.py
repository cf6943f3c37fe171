"""Pins of the scan oracle (Sec. 4.1, eq. scan-mat: the inclusive scan of a
row a is a^T U with u_ij = 1 for i <= j, else 0):

* on short rows every quantity equals the GEMM oracle applied to the
  explicit U built from the rule with numpy (the matrix form of the scan);
* integer inputs give Python's exact running sums;
* a unit impulse at position k scans to a step starting at k;
* the FP32 running sum is one rounded addition per element (exact model);
* the last element is the row total (exact rational sum, rounded).
"""
from fractions import Fraction
from itertools import accumulate

import numpy as np
import pytest

import oracle
import synth


@pytest.mark.parametrize("length", [1, 17, 64, 100])
def test_matches_matrix_form(length):
    X = synth.uniform_exp((5, length), synth.rng(length), -8, 8).numpy()
    U = np.triu(np.ones((length, length), np.float32))
    g = oracle.gemm(X[None], U[None])
    sc = oracle.scan(X)
    for key in ("c64", "n64", "c32", "cm"):
        assert np.array_equal(sc[key], g[key][0]), key


def test_integer_exact():
    X = synth.integer_matrix((4, 300), synth.rng(2), -5000, 5000).numpy()
    sc = oracle.scan(X)
    for r in range(4):
        ref = list(accumulate(int(v) for v in X[r]))
        assert np.array_equal(sc["c64"][r], np.array(ref, np.float64))
        assert np.array_equal(sc["c32"][r], np.array(ref, np.float32))
        assert np.array_equal(sc["cm"][r], np.array(ref, np.float64))


def test_impulse_gives_step():
    X = np.zeros((3, 50), np.float32)
    X[0, 0] = 1.5
    X[1, 27] = -3.25
    X[2, 49] = 7.0
    sc = oracle.scan(X)
    for r, k, v in ((0, 0, 1.5), (1, 27, -3.25), (2, 49, 7.0)):
        step = np.where(np.arange(50) >= k, v, 0.0)
        assert np.array_equal(sc["c64"][r], step)
        assert np.array_equal(sc["n64"][r], np.abs(step))


def test_fp32_running_sum_model():
    X = synth.uniform((2, 40), synth.rng(3)).numpy()
    sc = oracle.scan(X)
    for r in range(2):
        s = np.float32(0.0)
        for j in range(40):
            s = np.float32(s + X[r, j])
            assert sc["c32"][r, j].view(np.uint32) == s.view(np.uint32)


def test_total_is_exact_sum():
    X = synth.uniform((3, 1000), synth.rng(4)).numpy()
    sc = oracle.scan(X)
    for r in range(3):
        exact = sum(Fraction(float(v)) for v in X[r])
        assert abs(Fraction(sc["c64"][r, -1]) - exact) <= 1000 * Fraction(2) ** -53 * 1000
