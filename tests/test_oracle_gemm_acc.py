"""Pins of the accumulate-form oracle D = op(A).op(B) + C (the
multiply-accumulate of a fragment API, Sec. 2.3.1; emulated as in Sec. 4.4):

* C = 0 reduces it to the plain GEMM oracle, quantity for quantity;
* A = 0 or k = 0 leaves D = C exactly, and N = |C|;
* integer inputs give the exact integer result in every quantity (brute
  force in Python integers, with the transposed storage forms);
* the FP32 chain starts from C and is bit-exact against exact fmaf;
* the method model adds C to the model of the product.
"""
import numpy as np
import pytest

import oracle
import synth
from exact import fmaf


def _draw(batch, m, n, k, seed):
    g = synth.rng(seed)
    A = synth.uniform((batch, m, k), g).numpy()
    B = synth.uniform((batch, k, n), g).numpy()
    C = synth.uniform((batch, m, n), g).numpy()
    return A, B, C


def test_zero_accumulator_is_gemm():
    A, B, _ = _draw(2, 9, 13, 21, 1)
    Z = np.zeros((2, 9, 13), np.float32)
    acc = oracle.gemm_acc(A, B, Z)
    ref = oracle.gemm(A, B)
    for key in ("c64", "n64", "c32", "cm"):
        assert np.array_equal(acc[key], ref[key]), key


@pytest.mark.parametrize("k", [0, 17])
def test_zero_product_returns_c(k):
    _, _, C = _draw(2, 7, 5, 1, 2)
    A = np.zeros((2, 7, k), np.float32)
    B = synth.uniform((2, k, 5), synth.rng(3)).numpy()
    out = oracle.gemm_acc(A, B, C)
    assert np.array_equal(out["c64"], C.astype(np.float64))
    assert np.array_equal(out["c32"], C)
    assert np.array_equal(out["cm"], C.astype(np.float64))
    assert np.array_equal(out["n64"], np.abs(C.astype(np.float64)))


@pytest.mark.parametrize("op_a,op_b", [("N", "N"), ("T", "N"), ("N", "T"), ("T", "T")])
def test_integer_exact_with_transposes(op_a, op_b):
    g = synth.rng(4)
    m, n, k = 6, 5, 7
    A = synth.integer_matrix((2, m, k), g, -50, 50).numpy()
    B = synth.integer_matrix((2, k, n), g, -50, 50).numpy()
    C = synth.integer_matrix((2, m, n), g, -1000, 1000).numpy()
    As = A.transpose(0, 2, 1).copy() if op_a == "T" else A
    Bs = B.transpose(0, 2, 1).copy() if op_b == "T" else B
    out = oracle.gemm_acc(As, Bs, C, op_a, op_b)
    for b in range(2):
        for i in range(m):
            for j in range(n):
                exact = int(C[b, i, j]) + sum(int(A[b, i, t]) * int(B[b, t, j]) for t in range(k))
                nexact = abs(int(C[b, i, j])) + sum(abs(int(A[b, i, t]) * int(B[b, t, j]))
                                                    for t in range(k))
                assert out["c64"][b, i, j] == exact
                assert out["c32"][b, i, j] == exact
                assert out["cm"][b, i, j] == exact
                assert out["n64"][b, i, j] == nexact


def test_fp32_chain_starts_from_c():
    A, B, C = _draw(1, 3, 4, 9, 5)
    out = oracle.gemm_acc(A, B, C)
    for i in range(3):
        for j in range(4):
            acc = C[0, i, j]
            for t in range(9):
                acc = fmaf(A[0, i, t], B[0, t, j], acc)
            assert out["c32"][0, i, j].view(np.uint32) == np.float32(acc).view(np.uint32)


def test_model_adds_c_to_product_model():
    A, B, C = _draw(2, 8, 8, 24, 6)
    acc = oracle.gemm_acc(A, B, C, want=("cm", "c64"))
    plain = oracle.gemm(A, B, want=("cm", "c64"))
    # FP64 sums: the accumulate form starts from C, so it differs from
    # C + (product sum) by rounding only
    assert np.allclose(acc["cm"], plain["cm"] + C, rtol=0, atol=2.0 ** -48)
    assert np.allclose(acc["c64"], plain["c64"] + C, rtol=0, atol=2.0 ** -48)
