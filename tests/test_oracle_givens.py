"""Pins of the Givens oracle (Sec. 4.3.1: G(i, j, theta) is the identity
except G_ii = G_jj = c, G_ij = -s, G_ji = s, applied as G . B):

* the explicit matrix against the definition written out with numpy;
* theta = 0 gives C = B exactly, theta = pi / 2 a signed swap of rows i, j;
* rows other than i and j are copied exactly; rows i and j equal the
  closed forms c b_i - s b_j and s b_i + c b_j (FP64 exactly, the FP32 chain
  bit-for-bit against exact fmaf);
* a rotation and its inverse compose to (c^2 + s^2) I, and column norms
  scale as c^2 + s^2 predicts;
* the batched application equals the GEMM oracle on the explicit G.
"""
import numpy as np
import pytest

import oracle
import synth
from exact import fmaf


def _inputs(batch, seed=7, n=64, ncols=64):
    c, s, B = synth.givens_inputs(batch, n, ncols, seed)
    return c.numpy(), s.numpy(), B.numpy()


@pytest.mark.parametrize("i,j", [(5, 37), (37, 5), (0, 1), (62, 63)])
def test_matrix_matches_definition(i, j):
    c, s = np.float32(0.6), np.float32(0.8)
    G = oracle.givens_matrix(64, i, j, c, s)
    ref = np.eye(64, dtype=np.float32)
    ref[i, i] = c
    ref[j, j] = c
    ref[i, j] = -s
    ref[j, i] = s
    assert np.array_equal(G, ref)
    # column i holds (c at row i, s at row j): the rotation of e_i
    assert G[i, i] == c and G[j, i] == s and G[i, j] == -s


def test_identity_and_quarter_turn():
    _, _, B = _inputs(2)
    c = np.array([1.0, 0.0], np.float32)
    s = np.array([0.0, 1.0], np.float32)
    out = oracle.givens(5, 37, c, s, B)
    assert np.array_equal(out["c64"][0], B[0].astype(np.float64))
    assert np.array_equal(out["c32"][0], B[0])
    swap = B[1].astype(np.float64).copy()
    swap[5] = -B[1][37]
    swap[37] = B[1][5]
    assert np.array_equal(out["c64"][1], swap)
    assert np.array_equal(out["c32"][1], swap.astype(np.float32))


@pytest.mark.parametrize("i,j", [(5, 37), (40, 3)])
def test_closed_form_rows(i, j):
    c, s, B = _inputs(3, seed=11)
    out = oracle.givens(i, j, c, s, B)
    for b in range(3):
        Bb = B[b]
        others = [r for r in range(64) if r not in (i, j)]
        assert np.array_equal(out["c64"][b][others], Bb[others].astype(np.float64))
        assert np.array_equal(out["c32"][b][others], Bb[others])
        cb, sb = np.float64(c[b]), np.float64(s[b])
        bi, bj = Bb[i].astype(np.float64), Bb[j].astype(np.float64)
        # FP64: both products are exact, the k-ascending sum rounds once
        assert np.array_equal(out["c64"][b][i], cb * bi - sb * bj)
        assert np.array_equal(out["c64"][b][j], sb * bi + cb * bj)
        # FP32 chain over k ascending: the first nonzero term is rounded by
        # one fmaf onto 0, the second by a second fmaf
        lo, hi = min(i, j), max(i, j)
        for col in range(0, 64, 9):
            gi = {i: c[b], j: -s[b]}
            gj = {i: s[b], j: c[b]}
            for row, g in ((i, gi), (j, gj)):
                acc = fmaf(g[lo], Bb[lo, col], np.float32(0.0))
                acc = fmaf(g[hi], Bb[hi, col], acc)
                assert out["c32"][b][row, col].view(np.uint32) == acc.view(np.uint32)


def test_inverse_and_norms():
    c, s, B = _inputs(4, seed=12)
    fwd = oracle.givens(5, 37, c, s, B, want=("c64",))["c64"]
    rho = c.astype(np.float64) ** 2 + s.astype(np.float64) ** 2
    assert np.all(np.abs(rho - 1) < 2.0 ** -22)
    for b in range(4):
        G = oracle.givens_matrix(64, 5, 37, c[b], s[b]).astype(np.float64)
        Ginv = oracle.givens_matrix(64, 5, 37, c[b], -s[b]).astype(np.float64)
        eye = np.eye(64)
        eye[5, 5] = eye[37, 37] = rho[b]
        assert np.allclose(Ginv @ G, eye, rtol=0, atol=1e-15)
        Bb = B[b].astype(np.float64)
        nb = (Bb ** 2).sum(axis=0)
        nc = (fwd[b] ** 2).sum(axis=0)
        pred = nb + (rho[b] - 1) * (Bb[5] ** 2 + Bb[37] ** 2)
        assert np.allclose(nc, pred, rtol=1e-14, atol=0)


def test_batched_matches_gemm_oracle():
    c, s, B = _inputs(3, seed=13)
    out = oracle.givens(31, 32, c, s, B, items=[2, 0])
    for t, b in enumerate([2, 0]):
        G = np.eye(64, dtype=np.float32)
        G[31, 31] = G[32, 32] = c[b]
        G[31, 32] = -s[b]
        G[32, 31] = s[b]
        g = oracle.gemm(G[None], B[b][None])
        for key in ("c64", "n64", "c32", "cm"):
            assert np.array_equal(out[key][t], g[key][0]), key


def test_ragged_columns():
    c, s, B = _inputs(2, seed=14, ncols=45)
    out = oracle.givens(0, 63, c, s, B)
    assert out["c64"].shape == (2, 64, 45)
    assert np.array_equal(out["c64"][1][7], B[1][7].astype(np.float64))
