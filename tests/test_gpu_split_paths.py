"""The split as the production kernels compute it, pinned bit for bit.

Sec. 4.4 (eqs. corr-1..corr-4) defines hi = toFP16(x) and
lo = toFP16((x - toFP32(hi)) * 2^11) exactly.  A product with the identity
exposes what a kernel's split produced: for C = A . I (and C = I . B)

* the main accumulator sums hi(a) * 1 and zeros, the correction accumulator
  lo(a) * 1 + hi(a) * 0 (the identity's hi is 1 and its lo 0), all exact;
* the epilogue fma returns the FP32 rounding of hi + lo * 2^-11, which is
  exact: hi and lo * 2^-11 carry 11 significant bits each, at most 22 bits
  apart.

So every output must equal fl32(hi + lo 2^-11) of the oracle's split of the
input, bit for bit; with error correction off it must equal hi.  The inputs
mix the split's hard cases: binary16 ties in hi (the 13 dropped bits are
exactly one half) and in lo, hi and lo subnormal, the hand-worked examples
of tests/golden/split_examples.txt, zeros and the ends of the range, and
u * 2^e values.

Every kernel that splits operands loaded from memory is run: the full-tile
kernel's split flow on its three tiles (the 256 x 128 tile in both its
persistent and its plain launch form), its direct and staged flows, its
error-correction-off instances, the register-direct flow on both tiles, the
general kernel (reached through unaligned pointers), the accumulate kernel
on both MFMA shapes, the scan, and the Householder and Givens kernels with
an identity reflector / rotation.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
from gpu_util import device, to_np

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "split_examples.txt")


def _golden_values():
    vals = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        expr = line.split(";")[0].strip()
        vals.append(float(eval(expr, {"__builtins__": {}})))  # exact rationals of the file
    return np.float32(vals)


def split_probe_values(n: int, seed: int) -> np.ndarray:
    """n FP32 values in [-65504, 65504] mixing the split's hard cases (made
    from bit patterns; no arithmetic of the method)."""
    g = np.random.default_rng(seed)
    parts = []
    q = n // 6

    def with_exp(lo_exp, hi_exp, count):
        e = g.integers(lo_exp, hi_exp + 1, count).astype(np.uint32)
        return e << 23

    # hi ties: the 13 bits below binary16's 11 significant bits are 1 0...0
    frac = (g.integers(0, 1 << 10, q).astype(np.uint32) << 13) | np.uint32(0x1000)
    parts.append(((with_exp(127 - 14, 127 + 15, q)) | frac).view(np.float32))
    # lo ties: dropped bits d odd with 2^11 <= d < 2^12 (hi rounds down) or
    # 2^12 < d < 2^13 - 2^11 (hi rounds up)
    d = g.integers(1 << 10, 1 << 11, q).astype(np.uint32) * 2 + 1
    d = np.where(g.integers(0, 2, q) == 1, (1 << 13) - d, d).astype(np.uint32)
    frac = (g.integers(0, 1 << 10, q).astype(np.uint32) << 13) | d
    parts.append(((with_exp(127 - 14, 127 + 15, q)) | frac).view(np.float32))
    # hi subnormal (|x| < 2^-14) and lo subnormal
    parts.append(((with_exp(127 - 30, 127 - 15, q))
                  | g.integers(0, 1 << 23, q).astype(np.uint32)).view(np.float32))
    # u * 2^e, e in [-15, 15] (the batched 256^3 workload's distribution)
    u = (g.random(q) * 2 - 1).astype(np.float32)
    parts.append(np.ldexp(u, g.integers(-15, 16, q)).astype(np.float32))
    # any significand, exponents of the whole domain
    parts.append(((with_exp(127 - 24, 127 + 15, q))
                  | g.integers(0, 1 << 23, q).astype(np.uint32)).view(np.float32))
    rest = n - 5 * q
    fixed = np.concatenate([_golden_values(),
                            np.float32([65504, -65504, 65519, -65519, 0.0, -0.0, 1.0, -1.0,
                                        2.0 ** -24, -(2.0 ** -24), 2.0 ** -14, 2.0 ** 15])])
    parts.append(np.resize(fixed, rest))
    x = np.concatenate(parts).astype(np.float32)
    sign = np.where(g.integers(0, 2, n) == 1, np.uint32(0x80000000), np.uint32(0))
    x = (x.view(np.uint32) ^ sign).view(np.float32)
    x = x[g.permutation(n)]
    x = np.where(np.abs(x) > 65519.0, np.copysign(np.float32(65504.0), x), x)
    # -0 is left out: a sum of products that are all zero is +0 on every path
    return np.where(x == 0, np.float32(0.0), x).astype(np.float32)


def expected(x: np.ndarray, ec: bool) -> np.ndarray:
    """fl32(hi + lo 2^-11) of the oracle's split (exact), or hi with ec off.
    The kernels' sums start from +0, so a zero result is +0 (a tiny negative
    x has hi = -0)."""
    hi, lo = oracle.split(x)
    v = 0.0 + oracle.f16_bits_to_f64(hi)
    if ec:
        v = v + oracle.f16_bits_to_f64(lo) * 2.0 ** -11
    out = v.astype(np.float32)
    assert np.array_equal(out.astype(np.float64), v), "hi + lo 2^-11 not exact in FP32"
    return out


def assert_bits(C: np.ndarray, want: np.ndarray, label: str):
    C = np.asarray(C, dtype=np.float32)
    assert C.shape == want.shape, (C.shape, want.shape)
    bad = C.view(np.uint32) != want.view(np.uint32)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        detail = [(tuple(int(t) for t in i), float(want[tuple(i)]).hex(), float(C[tuple(i)]).hex())
                  for i in idx]
        pytest.fail(f"{label}: {int(bad.sum())} of {bad.size} outputs differ from the split "
                    f"(index, expected, got): {detail}")


def _eye(n):
    return torch.eye(n, dtype=torch.float32)


def _dev(t, offset=0):
    """t on the device; with offset > 0 its storage starts `offset` floats
    into a larger buffer (rows no longer 16-byte aligned)."""
    d = device()
    if offset == 0:
        return t.contiguous().to(d)
    flat = torch.zeros(t.numel() + offset, dtype=torch.float32, device=d)
    flat[offset:] = t.reshape(-1).to(d)
    return flat[offset:].view(t.shape)


P = pkg.Policy
# (label, policy, batch, m, k, n, expected kernel name or None)
GEMM_CASES = [
    ("full-128x128", P(pkg.FLOW_SPLIT, 1, pkg.TILE_128x128), 2, 256, 128, 128, "bgemm_big_kernel"),
    ("full-256x128-stream", P(pkg.FLOW_SPLIT, 1, pkg.TILE_256x128), 2, 256, 256, 128,
     "bgemm_big_stream_kernel"),
    ("full-256x128-plain", P(pkg.FLOW_SPLIT, 1, pkg.TILE_256x128), 1, 256, 2176, 2176,
     "bgemm_big_kernel"),
    ("full-128x256", P(pkg.FLOW_SPLIT, 1, pkg.TILE_128x256), 1, 128, 256, 256, "bgemm_big_kernel"),
    ("full-direct", P(pkg.FLOW_DIRECT, 1, pkg.TILE_128x128), 2, 128, 128, 128, "bgemm_big_kernel"),
    ("full-staged", P(pkg.FLOW_STAGED, 1, pkg.TILE_128x128), 2, 128, 128, 128, "bgemm_big_kernel"),
    ("reg-64x64", P(pkg.FLOW_REG, 1, pkg.TILE_64x64), 3, 100, 64, 64, "bgemm_reg_kernel"),
    ("reg-128x128", P(pkg.FLOW_REG, 1, pkg.TILE_128x128), 2, 200, 128, 128, "bgemm_reg_kernel"),
    ("general-split-64", P(pkg.FLOW_SPLIT, 1, pkg.TILE_64x64), 2, 70, 96, 96, "bgemm_emu_kernel"),
    ("general-split-128", P(pkg.FLOW_SPLIT, 1, pkg.TILE_128x128), 2, 130, 96, 96,
     "bgemm_emu_kernel"),
    ("general-direct-64", P(pkg.FLOW_DIRECT, 1, pkg.TILE_64x64), 2, 70, 96, 96,
     "bgemm_emu_kernel"),
    ("general-staged-64", P(pkg.FLOW_STAGED, 1, pkg.TILE_64x64), 2, 70, 96, 96,
     "bgemm_emu_kernel"),
    # error correction off: the output is hi itself
    ("full-128x128-noec", P(pkg.FLOW_SPLIT, 0, pkg.TILE_128x128), 2, 128, 128, 128,
     "bgemm_big_kernel"),
    ("full-128x256-noec", P(pkg.FLOW_SPLIT, 0, pkg.TILE_128x256), 1, 128, 256, 256,
     "bgemm_big_kernel"),
    ("reg-64x64-noec", P(pkg.FLOW_REG, 0, pkg.TILE_64x64), 2, 64, 64, 64, "bgemm_reg_kernel"),
    ("general-split-64-noec", P(pkg.FLOW_SPLIT, 0, pkg.TILE_64x64), 2, 70, 96, 96,
     "bgemm_emu_kernel"),
]


@pytest.mark.parametrize("case", GEMM_CASES, ids=[c[0] for c in GEMM_CASES])
@pytest.mark.parametrize("side", ["A.I", "I.B"])
def test_gemm_kernels_reproduce_the_split(case, side):
    label, policy, batch, m, k, n, kernel = case
    ec = bool(policy.ec)
    # A.I: A is batch x m x k, I is k x k (n = k).  I.B: I is m x m (k = m)
    # and B is batch x m x n; the same tiles run with the roles exchanged.
    seed = 1000 + 17 * len(label) + (0 if side == "A.I" else 1)
    general = kernel == "bgemm_emu_kernel"
    if side == "A.I":
        x = split_probe_values(batch * m * k, seed).reshape(batch, m, k)
        Ad, Bd = _dev(torch.from_numpy(x), 1 if general else 0), _dev(_eye(k))
        shape_c = (batch, m, k)
    else:
        if kernel == "bgemm_big_stream_kernel":
            m_, n_ = 256, 128      # I.B with 256 x 128 tiles: m = k = 256
        elif label == "full-256x128-plain":
            m_, n_ = 2304, 128     # k = m > 2048: the plain launch form
        elif label.startswith("full-128x256"):
            m_, n_ = 128, 256
        else:
            m_, n_ = (k, m) if not label.startswith("reg-64") else (64, 100 if ec else 64)
        x = split_probe_values(batch * m_ * n_, seed).reshape(batch, m_, n_)
        Ad, Bd = _dev(_eye(m_)), _dev(torch.from_numpy(x), 3 if general else 0)
        shape_c = (batch, m_, n_)
    C = torch.full(shape_c, float("nan"), dtype=torch.float32, device=device())
    _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, C, policy=policy)
    print(f"case split-path {label} {side} shape={tuple(shape_c)} kernel={kern}", flush=True)
    if kernel == "bgemm_big_stream_kernel" and side == "I.B":
        assert kern in ("bgemm_big_stream_kernel", "bgemm_big_kernel")
    else:
        assert kern == kernel, (label, side, kern)
    pkg.sgemm_emu_batched(Ad, Bd, C, policy=policy)
    assert_bits(to_np(C), expected(x, ec), f"{label} {side}")


@pytest.mark.parametrize("shape", [pkg.SHAPE_16x16x32, pkg.SHAPE_32x32x16], ids=["16x16x32",
                                                                               "32x32x16"])
@pytest.mark.parametrize("side", ["A.I", "I.B"])
def test_accumulate_kernel_reproduces_the_split(shape, side):
    batch, m, k = 2, 100, 72
    seed = 2000 + shape * 2 + (side == "I.B")
    if side == "A.I":
        x = split_probe_values(batch * m * k, seed).reshape(batch, m, k)
        Ad, Bd = _dev(torch.from_numpy(x)), _dev(_eye(k))
    else:
        x = split_probe_values(batch * k * m, seed).reshape(batch, k, m)
        Ad, Bd = _dev(_eye(k)), _dev(torch.from_numpy(x))
    D = torch.full(x.shape, float("nan"), dtype=torch.float32, device=device())
    print(f"case split-path gemm_acc shape={shape} {side}", flush=True)
    pkg.sgemm_emu_batched_acc(Ad, Bd, None, D, shape=shape)
    assert_bits(to_np(D), expected(x, True), f"gemm_acc {shape} {side}")


@pytest.mark.parametrize("length", [2048, 1000])
def test_scan_reproduces_the_split(length):
    """Rows with one nonzero value v: the inclusive scan is 0 before it and
    fl32(hi(v) + lo(v) 2^-11) from it on (U's entries are 0 and 1; every
    carry adds that value to zeros).  Aligned rows of whole 1024-value
    blocks take the whole-block path, 1000 the element-wise one."""
    rows = 4096
    g = np.random.default_rng(3000 + length)
    v = split_probe_values(rows, 3001 + length)
    pos = g.integers(0, length, rows)
    pos[:64] = np.arange(64) * 31 % length  # segment starts and ends among them
    X = np.zeros((rows, length), dtype=np.float32)
    X[np.arange(rows), pos] = v
    Xd = _dev(torch.from_numpy(X))
    Y = torch.full_like(Xd, float("nan"))
    print(f"case split-path scan rows={rows} len={length}", flush=True)
    pkg.sgemm_emu_scan(Xd, Y)
    want = np.where(np.arange(length)[None, :] >= pos[:, None],
                    expected(v, True)[:, None], np.float32(0)).astype(np.float32)
    assert_bits(to_np(Y), want, f"scan len {length}")


@pytest.mark.parametrize("mode", [pkg.HOUSEHOLDER_RULE, pkg.HOUSEHOLDER_LDS], ids=["rule", "lds"])
def test_householder_identity_reproduces_the_split(mode):
    """u = 0 gives H = I exactly (fmaf(-0, 0, delta) = delta), so C is the
    split of B, the B operand of the rule-built kernel."""
    batch, ncols = 64, 96
    x = split_probe_values(batch * 64 * ncols, 4000 + mode).reshape(batch, 64, ncols)
    u = torch.zeros((batch, 64), dtype=torch.float32, device=device())
    Bd = _dev(torch.from_numpy(x))
    C = torch.full_like(Bd, float("nan"))
    print(f"case split-path householder mode={mode}", flush=True)
    pkg.householder_emu_batched(u, Bd, C, mode=mode)
    assert_bits(to_np(C), expected(x, True), f"householder mode {mode}")


@pytest.mark.parametrize("mode,plane", [(pkg.GIVENS_MAP, (3, 40)), (pkg.GIVENS_EMBEDDED, (5, 37)),
                                        (pkg.GIVENS_LDS, (62, 63))],
                         ids=["map", "embedded", "lds"])
def test_givens_identity_reproduces_the_split(mode, plane):
    """c = 1, s = 0 gives G = I exactly, so C is the split of B."""
    batch, ncols = 64, 64
    x = split_probe_values(batch * 64 * ncols, 5000 + mode).reshape(batch, 64, ncols)
    c = torch.ones(batch, dtype=torch.float32, device=device())
    s = torch.zeros(batch, dtype=torch.float32, device=device())
    Bd = _dev(torch.from_numpy(x))
    C = torch.full_like(Bd, float("nan"))
    print(f"case split-path givens mode={mode} plane={plane}", flush=True)
    pkg.givens_emu_batched(plane[0], plane[1], c, s, Bd, C, mode=mode)
    assert_bits(to_np(C), expected(x, True), f"givens mode {mode}")
