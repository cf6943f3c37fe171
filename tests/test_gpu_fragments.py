"""GPU checks of the fragment maps through a single MFMA (the register-level
counterpart of the paper's mapping probe, Sec. 2.3.2) and of the device-side
split (Sec. 4.4, eqs. corr-1/corr-2), bit for bit.

The probe packs integer matrices into operand registers with mfmae_map,
runs one MFMA and unpacks the accumulator with the accumulator map: the
result must equal the integer product exactly.  This pins the row index of
A, the column index of B, the whole accumulator map and the agreement of
the k index between A and B (a k relabelling shared by both operands is not
observable through the product).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
from gpu_util import device, to_np

pytestmark = pytest.mark.gpu

SHAPES = {pkg.SHAPE_16x16x32: (16, 16, 32), pkg.SHAPE_32x32x16: (32, 32, 16)}


def _pack(shape, use, X):
    rows, cols = X.shape
    lanes = np.zeros((64, 8), dtype=np.float16)
    for i in range(rows):
        for j in range(cols):
            lane, elem = pkg.mfmae_map(shape, use, i, j)
            lanes[lane, elem] = X[i, j]
    return torch.from_numpy(lanes.view(np.int16)).to(device())


def _unpack(shape, D, m, n):
    out = np.zeros((m, n), dtype=np.float32)
    for i in range(m):
        for j in range(n):
            lane, elem = pkg.mfmae_map(shape, pkg.USE_ACC, i, j)
            out[i, j] = D[lane, elem]
    return out


def _probe(shape, A, B):
    m, n, _ = SHAPES[shape]
    D = pkg.mfmae_mma_probe(shape, _pack(shape, pkg.USE_A, A), _pack(shape, pkg.USE_B, B))
    return _unpack(shape, to_np(D), m, n)


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_probe_integer_product_exact(shape, seed):
    m, n, k = SHAPES[shape]
    g = np.random.default_rng(seed)
    A = g.integers(-16, 17, (m, k)).astype(np.float16)
    B = g.integers(-16, 17, (k, n)).astype(np.float16)
    got = _probe(shape, A, B)
    ref = A.astype(np.int64) @ B.astype(np.int64)
    assert np.array_equal(got, ref.astype(np.float32))


@pytest.mark.parametrize("shape", list(SHAPES))
def test_probe_selector_reads_every_position(shape):
    """D = X . S with S[kk][j] = [kk == j mod K]: D[i][j] = X[i][j mod K]
    exactly, so every A position shows up at a known accumulator position."""
    m, n, k = SHAPES[shape]
    X = (np.arange(m * k).reshape(m, k) % 2039).astype(np.float16)
    S = np.zeros((k, n), dtype=np.float16)
    for j in range(n):
        S[j % k, j] = 1
    got = _probe(shape, X, S)
    expect = np.stack([X[:, j % k] for j in range(n)], axis=1).astype(np.float32)
    assert np.array_equal(got, expect)


def test_probe_fp16_subnormal_inputs():
    """The smallest binary16 subnormal times one must come out as 2^-24:
    subnormal lo parts must not be flushed by the instruction."""
    shape = pkg.SHAPE_32x32x16
    A = np.zeros((32, 16), np.float16)
    B = np.zeros((16, 32), np.float16)
    A[3, 5] = np.float16(2.0 ** -24)
    B[5, 7] = np.float16(1.0)
    A[4, 2] = np.float16(3 * 2.0 ** -24)
    B[2, 9] = np.float16(-2.0)
    got = _probe(shape, A, B)
    assert got[3, 7] == np.float32(2.0 ** -24)
    assert got[4, 9] == np.float32(-6 * 2.0 ** -24)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_probe_accumulation_rounding(shape):
    """1 + (2^-24 + 2^-34) summed inside one instruction.  Round to nearest
    gives 1 + 2^-23, truncation gives 1.  The emulation's error bound holds
    under either; the test records which one the hardware does and requires
    it to be one of the two."""
    m, n, k = SHAPES[shape]
    A = np.zeros((m, k), np.float16)
    B = np.zeros((k, n), np.float16)
    A[0, 0], B[0, 0] = 1.0, 1.0
    A[0, 1], B[1, 0] = 2.0 ** -12, np.float16(2.0 ** -12 * (1 + 2.0 ** -10))
    got = _probe(shape, A, B)[0, 0]
    rn, rz = np.float32(1 + 2.0 ** -23), np.float32(1.0)
    print(f"shape {shape}: 1 + 2^-24 + 2^-34 -> {float(got).hex()}")
    assert got in (rn, rz)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_probe_accumulation_rounding_report(shape):
    """Several single-instruction sums whose correctly rounded values differ
    from their truncations; printed for the record, asserted only to lie
    within one ulp of the exact sum."""
    m, n, k = SHAPES[shape]
    cases = [(1.0, [2.0 ** -12 * 2.0 ** -12 * 1.5]),        # 1 + 1.5 2^-24: RN up
             (1.0, [2.0 ** -13, 2.0 ** -13, 2.0 ** -24]),    # carries out of the low bits
             (-1.0, [-(2.0 ** -24) * 1.5])]
    for head, tail in cases:
        A = np.zeros((m, k), np.float16)
        B = np.zeros((k, n), np.float16)
        A[0, 0], B[0, 0] = head, 1.0
        for t, v in enumerate(tail, start=1):
            if abs(v) >= 2.0 ** -24 * 2048:
                A[0, t], B[t, 0] = v, 1.0
            else:
                A[0, t], B[t, 0] = 2.0 ** -12, v / 2.0 ** -12
        exact = float(head) + sum(float(A[0, t]) * float(B[t, 0]) for t in range(1, len(tail) + 1))
        got = float(_probe(shape, A, B)[0, 0])
        print(f"shape {shape}: exact {exact.hex()} -> {got.hex()}")
        assert abs(got - exact) <= 2.0 ** -23 * abs(exact)


def _structured_f32():
    low = np.arange(1 << 13, dtype=np.uint32)
    highs = np.array([0, 1, 0x2AA, 0x3FF], dtype=np.uint32) << 13
    frac = (highs[:, None] | low[None, :]).ravel()
    # every sign and every exponent up to 2^15 (values beyond the fp16 range
    # are outside the split's domain)
    exps = np.concatenate([np.arange(0, 143, dtype=np.uint32),
                           np.arange(256, 256 + 143, dtype=np.uint32)])
    x = ((exps[:, None] << 23) | frac[None, :]).ravel().view(np.float32)
    every = np.arange(1 << 23, dtype=np.uint32)
    sub = np.concatenate([(every | np.uint32(e << 23)) for e in range(127 - 26, 127 - 13)])
    return np.concatenate([x, sub.view(np.float32), np.float32([65504, -65504, 0, -0.0])])


@pytest.mark.parametrize("form", [pkg.SPLIT_SCALAR, pkg.SPLIT_PAIR, pkg.SPLIT_EIGHT],
                         ids=["scalar", "pair", "eight"])
def test_device_split_bit_exact(form):
    """Every device form of the split (one value, a packed pair, a vector of
    eight: the forms the kernels use) against the oracle's split, bit for
    bit, over a structured sweep of FP32 (every exponent of the domain and
    sign, the low 13 bits exhaustively, every subnormal-hi value range)."""
    x = _structured_f32()
    # 1 extra value: the last group of 8 is cut short (split one at a time)
    x = np.concatenate([x, np.float32([1 + 2.0 ** -11])])
    hi_ref, lo_ref = oracle.split(x)
    xd = torch.from_numpy(x).to(device())
    print(f"case split form={form} count={x.size}", flush=True)
    hi, lo = pkg.sgemm_emu_split(xd, form=form)
    hi = to_np(hi).view(np.uint16)
    lo = to_np(lo).view(np.uint16)
    bad_hi = np.count_nonzero(hi != hi_ref)
    bad_lo = np.count_nonzero(lo != lo_ref)
    if bad_hi or bad_lo:
        idx = np.nonzero((hi != hi_ref) | (lo != lo_ref))[0][:5]
        detail = [(float(x[i]).hex(), hex(hi[i]), hex(hi_ref[i]), hex(lo[i]), hex(lo_ref[i]))
                  for i in idx]
        pytest.fail(f"split mismatches hi={bad_hi} lo={bad_lo}: {detail}")
