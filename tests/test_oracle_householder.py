"""Pins of the Householder oracle (Sec. 4.2.1, eq. householder read as
H = I - 2 u u^T with u the given vector):

* H32 entries bit-for-bit against exact fmaf(-2 u_i, u_j, delta_ij);
* H64 entries against the correctly rounded FP64 value of delta - 2 u_i u_j;
* invariants of a reflector for unit u: H u = -u, H H = I, H = H^T;
* u = e_0 gives diag(-1, 1, ..., 1) exactly, so C is B with row 0 negated;
* the batched application equals the GEMM oracle on the explicit H.
"""
from fractions import Fraction

import numpy as np

import oracle
import synth
from exact import fmaf


def _unit_u(n, seed):
    u, _ = synth.householder_inputs(1, n, 1, seed)
    return u[0].numpy()


def test_h32_bitwise_against_exact_fma():
    u = _unit_u(64, 3)
    H = oracle.householder_h32(u)
    for i in range(0, 64, 7):
        for j in range(64):
            ref = fmaf(np.float32(-2) * u[i], u[j], np.float32(1.0 if i == j else 0.0))
            assert H[i, j].view(np.uint32) == ref.view(np.uint32)


def test_h64_correctly_rounded():
    u = _unit_u(64, 4)
    H = oracle.householder_h64(u)
    for i in range(0, 64, 5):
        for j in range(0, 64, 3):
            q = (1 if i == j else 0) - 2 * Fraction(float(u[i])) * Fraction(float(u[j]))
            assert H[i, j] == float(q)


def test_reflector_invariants():
    u = _unit_u(64, 5)
    norm2 = float(np.dot(u.astype(np.float64), u.astype(np.float64)))
    assert abs(norm2 - 1) < 2.0 ** -20
    H = oracle.householder_h64(u)
    uu = u.astype(np.float64)
    # H u = u - 2 u (u.u) = -u + 2 u (1 - u.u)
    assert np.allclose(H @ uu, -uu + 2 * uu * (1 - norm2), rtol=0, atol=1e-15)
    assert np.allclose(H @ H, np.eye(64) + 4 * (norm2 - 1) * np.outer(uu, uu),
                       rtol=0, atol=1e-14)
    assert np.array_equal(H, H.T)


def test_unit_basis_vector_flips_row():
    n = 64
    u = np.zeros((2, n), np.float32)
    u[0, 0] = 1.0
    u[1, 5] = -1.0
    g = synth.rng(9)
    B = synth.uniform((2, n, n), g).numpy()
    out = oracle.householder(u, B)
    e0 = B[0].astype(np.float64).copy()
    e0[0] *= -1
    e1 = B[1].astype(np.float64).copy()
    e1[5] *= -1
    assert np.array_equal(out["c64"][0], e0)
    assert np.array_equal(out["c64"][1], e1)
    assert np.array_equal(out["c32"][0], e0.astype(np.float32))


def test_batched_matches_gemm_oracle():
    u, B = synth.householder_inputs(3, 64, 64, 6)
    u = u.numpy()
    B = B.numpy()
    out = oracle.householder(u, B, items=[2, 0])
    for t, b in enumerate([2, 0]):
        H64 = oracle.householder_h64(u[b])
        H32 = oracle.householder_h32(u[b])
        g = oracle.gemm(H32[None], B[b][None], want=("c32", "cm"))
        assert np.array_equal(out["c32"][t], g["c32"][0])
        assert np.array_equal(out["cm"][t], g["cm"][0])
        ref = H64 @ B[b].astype(np.float64)
        assert np.allclose(out["c64"][t], ref, rtol=0, atol=1e-14)
        assert np.allclose(out["n64"][t], np.abs(H64) @ np.abs(B[b].astype(np.float64)),
                           rtol=1e-14, atol=0)
