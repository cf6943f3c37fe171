"""Oracle for the emulated SGEMM: plain, slow, obviously correct CPU code.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import this package.  The
product (``paper_2308_15152_amd``) never imports it and shares no code with
it; the only thing both sides use is the seeded input generator in
``synth``, which holds none of the method's arithmetic.

The arithmetic lives in ``oracle.c`` (built into ``liboracle.so`` by
``oracle/build.py``); this module only marshals numpy arrays and evaluates
the error metric.  What each function computes and the passage of the paper
it follows:

* :func:`f32_to_f16`, :func:`f16_to_f32`, :func:`split` -- the toFP16 /
  toFP32 conversions and the hi/lo split with the residual scaled by 2^11
  (Sec. 4.4, eqs. corr-1..corr-4), round-to-nearest-even from the binary16
  definition.
* :func:`gemm`, :func:`dots` -- for C = A.B: the FP64 product of the FP32
  inputs, the normaliser sum_k |a||b|, the plain FP32 product (sequential
  fmaf chain, ascending k) and the method-exact model of eq. corr-5 summed in
  FP64.
* :func:`gemm_acc` -- D = op(A).op(B) + C (op: as stored or transposed),
  the multiply-accumulate form of a fragment API (Sec. 2.3.1, Sec. 4.4): the
  same four quantities with C as the first term of every sum.
* :func:`scan` -- inclusive prefix sums of each row: a^T U with U the
  upper-triangular all-ones matrix of Sec. 4.1 (eq. scan-mat), written as
  running sums (FP64, |x|, FP32, and the split model).
* :func:`householder` -- H = I - 2 u u^T formed explicitly and applied to B
  (Sec. 4.2.1, eq. householder, read as an outer product of u).
* :func:`givens_matrix`, :func:`givens` -- the rotation G(i, j, theta) of
  Sec. 4.3.1 (identity except G_ii = G_jj = c, G_ij = -s, G_ji = s) formed
  explicitly from the FP32 c and s and applied to B.
* :func:`max_rel_err` -- the "max relative error" of Sec. 4.4.2, normalised
  per element by (|A||B|)_ij, evaluated in FP64.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB names another build of oracle.c (the sanitizer build, say)
LIB_PATH = os.environ.get("ORACLE_LIB", os.path.join(_HERE, "liboracle.so"))

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int, ctypes.c_int64
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_f32_to_f16.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_f16.restype = ctypes.c_uint16
    lib.oracle_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f32.restype = ctypes.c_float
    lib.oracle_split.argtypes = [i64, P, P, P]
    lib.oracle_split.restype = None
    lib.oracle_gemm.argtypes = [i32, i32, i32, i32, P, i64, i64, P, i64, i64,
                                P, P, P, P, i64, i64]
    lib.oracle_gemm.restype = None
    lib.oracle_gemm_acc.argtypes = [i32, i32, i32, i32, P, i64, i64, P, i64, i64,
                                     P, i64, i64, P, P, P, P, i64, i64]
    lib.oracle_gemm_acc.restype = None
    lib.oracle_scan.argtypes = [i64, i32, P, i64, P, P, P, P, i64]
    lib.oracle_scan.restype = None
    lib.oracle_dots.argtypes = [i64, i32, P, P, P, P, P, P]
    lib.oracle_dots.restype = None
    lib.oracle_householder_h32.argtypes = [i32, P, P]
    lib.oracle_householder_h32.restype = None
    lib.oracle_householder_h64.argtypes = [i32, P, P]
    lib.oracle_householder_h64.restype = None
    lib.oracle_householder.argtypes = [i32, i32, i32, P, P, i64, P, i64, i64,
                                       P, P, P, P, i64, i64]
    lib.oracle_householder.restype = None
    lib.oracle_givens_matrix.argtypes = [i32, i32, i32, ctypes.c_float, ctypes.c_float, P]
    lib.oracle_givens_matrix.restype = None
    lib.oracle_givens.argtypes = [i32, i32, i32, i32, i32, P, P, P, i64, P, i64, i64,
                                  P, P, P, P, i64, i64]
    lib.oracle_givens.restype = None
    _lib = lib
    return lib


def num_threads() -> int:
    """Threads the oracle's parallel loops use."""
    return int(_load().oracle_num_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# binary16 conversions and the split (Sec. 4.4, eqs. corr-1..corr-4)
# --------------------------------------------------------------------------

def f32_to_f16_scalar(x: float) -> int:
    """Bits of toFP16(x), round to nearest even."""
    return int(_load().oracle_f32_to_f16(float(np.float32(x))))


def f16_to_f32_scalar(h: int) -> float:
    return float(_load().oracle_f16_to_f32(int(h)))


def split(x: np.ndarray):
    """hi, lo bit patterns (uint16) of the split of every element of x.

    hi = toFP16(x); lo = toFP16((x - toFP32(hi)) * 2^11)  (Sec. 4.4)."""
    x = _f32(x)
    hi = np.empty(x.shape, dtype=np.uint16)
    lo = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_split(x.size, _ptr(x), _ptr(hi), _ptr(lo))
    return hi, lo


def f16_bits_to_f64(h: np.ndarray) -> np.ndarray:
    """Exact value of binary16 bit patterns, decoded from the definition."""
    h = np.asarray(h, dtype=np.uint16).astype(np.int64)
    sign = np.where(h & 0x8000, -1.0, 1.0)
    e = (h >> 10) & 0x1F
    f = h & 0x3FF
    mag = np.where(e == 0, np.ldexp(f.astype(np.float64), -24),
                   np.ldexp((1024 + f).astype(np.float64), (e - 25).astype(np.int32)))
    mag = np.where(e == 0x1F, np.where(f == 0, np.inf, np.nan), mag)
    return sign * mag


# --------------------------------------------------------------------------
# GEMM oracle
# --------------------------------------------------------------------------

def gemm(A: np.ndarray, B: np.ndarray, want=("c64", "n64", "c32", "cm")):
    """Oracle quantities for C = A.B over a batch.

    A: [batch, m, k] float32, B: [batch, k, n] float32 (contiguous copies are
    made).  Returns a dict with the requested keys among c64 (FP64 product),
    n64 (normaliser), c32 (plain FP32 fmaf chain) and cm (method-exact model),
    each shaped [batch, m, n]."""
    A = _f32(A)
    B = _f32(B)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    batch, m, k = A.shape
    kb, n = B.shape[1], B.shape[2]
    assert kb == k and B.shape[0] == batch
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros((batch, m, n), dtype=dt) if key in want else None
    _load().oracle_gemm(batch, m, n, k, _ptr(A), k, m * k, _ptr(B), n, k * n,
                        _ptr(out["c64"]), _ptr(out["n64"]), _ptr(out["c32"]),
                        _ptr(out["cm"]), n, m * n)
    return {key: v for key, v in out.items() if v is not None}


def gemm_acc(A: np.ndarray, B: np.ndarray, C: np.ndarray, op_a: str = "N", op_b: str = "N",
             want=("c64", "n64", "c32", "cm")):
    """Oracle quantities for D = op(A).op(B) + C over a batch.

    A is stored as [batch, m, k] (op_a "N") or [batch, k, m] (op_a "T", A is
    its transpose); B as [batch, k, n] ("N") or [batch, n, k] ("T"); C is
    [batch, m, n].  Transposed operands are copied into row-major form
    first; the arithmetic is the same as for "N"."""
    A = np.asarray(A, dtype=np.float32)
    B = np.asarray(B, dtype=np.float32)
    C = _f32(C)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    if C.ndim == 2:
        C = C[None]
    A = _f32(A.transpose(0, 2, 1) if op_a == "T" else A)
    B = _f32(B.transpose(0, 2, 1) if op_b == "T" else B)
    batch, m, k = A.shape
    n = B.shape[2]
    assert B.shape == (batch, k, n) and C.shape == (batch, m, n)
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros((batch, m, n), dtype=dt) if key in want else None
    _load().oracle_gemm_acc(batch, m, n, k, _ptr(A), k, m * k, _ptr(B), n, k * n,
                            _ptr(C), n, m * n, _ptr(out["c64"]), _ptr(out["n64"]),
                            _ptr(out["c32"]), _ptr(out["cm"]), n, m * n)
    return {key: v for key, v in out.items() if v is not None}


def scan(X: np.ndarray, want=("c64", "n64", "c32", "cm")):
    """Oracle quantities of the inclusive scan of every row of X
    ([rows, len] or [..., len]): c64 running FP64 sums, n64 running sums of
    |x|, c32 running FP32 sums, cm running sums of the split values."""
    X = _f32(X)
    shape = X.shape
    X2 = X.reshape(-1, shape[-1]) if X.ndim != 2 else X
    rows, length = X2.shape
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros((rows, length), dtype=dt) if key in want else None
    _load().oracle_scan(rows, length, _ptr(X2), length, _ptr(out["c64"]), _ptr(out["n64"]),
                        _ptr(out["c32"]), _ptr(out["cm"]), length)
    return {key: v.reshape(shape) for key, v in out.items() if v is not None}


def dots(arows: np.ndarray, bcols: np.ndarray, want=("c64", "n64", "c32", "cm")):
    """Oracle quantities for sampled outputs: arows[s] . bcols[s] (each [k])."""
    arows = _f32(arows)
    bcols = _f32(bcols)
    nsamp, k = arows.shape
    assert bcols.shape == (nsamp, k)
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros(nsamp, dtype=dt) if key in want else None
    _load().oracle_dots(nsamp, k, _ptr(arows), _ptr(bcols), _ptr(out["c64"]),
                        _ptr(out["n64"]), _ptr(out["c32"]), _ptr(out["cm"]))
    return {key: v for key, v in out.items() if v is not None}


# --------------------------------------------------------------------------
# Householder oracle (Sec. 4.2.1)
# --------------------------------------------------------------------------

def householder_h32(u: np.ndarray) -> np.ndarray:
    """H_ij = fmaf(-2 u_i, u_j, delta_ij) in FP32 (one rounding)."""
    u = _f32(u)
    n = u.shape[0]
    H = np.empty((n, n), dtype=np.float32)
    _load().oracle_householder_h32(n, _ptr(u), _ptr(H))
    return H


def householder_h64(u: np.ndarray) -> np.ndarray:
    """H_ij = delta_ij - 2 u_i u_j in FP64."""
    u = _f32(u)
    n = u.shape[0]
    H = np.empty((n, n), dtype=np.float64)
    _load().oracle_householder_h64(n, _ptr(u), _ptr(H))
    return H


def householder(u: np.ndarray, B: np.ndarray, items=None,
                want=("c64", "n64", "c32", "cm")):
    """Oracle quantities for C_b = (I - 2 u_b u_b^T) B_b.

    u: [batch, n], B: [batch, n, ncols].  ``items`` selects which batch items
    to evaluate (default: all); the outputs are [len(items), n, ncols]."""
    u = _f32(u)
    B = _f32(B)
    batch, n = u.shape
    ncols = B.shape[2]
    assert B.shape[:2] == (batch, n)
    items = np.arange(batch, dtype=np.int64) if items is None else \
        np.ascontiguousarray(items, dtype=np.int64)
    t = items.shape[0]
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros((t, n, ncols), dtype=dt) if key in want else None
    _load().oracle_householder(n, ncols, t, _ptr(items), _ptr(u), n, _ptr(B),
                               ncols, n * ncols, _ptr(out["c64"]), _ptr(out["n64"]),
                               _ptr(out["c32"]), _ptr(out["cm"]), ncols, n * ncols)
    return {key: v for key, v in out.items() if v is not None}


# --------------------------------------------------------------------------
# Givens oracle (Sec. 4.3.1)
# --------------------------------------------------------------------------

def givens_matrix(n: int, i: int, j: int, c, s) -> np.ndarray:
    """The n x n rotation G(i, j, theta) with c = cos theta, s = sin theta
    given as FP32 values: FP32, every entry one of 0, 1, c, s, -s."""
    assert 0 <= i < n and 0 <= j < n and i != j
    G = np.empty((n, n), dtype=np.float32)
    _load().oracle_givens_matrix(n, i, j, float(np.float32(c)), float(np.float32(s)), _ptr(G))
    return G


def givens(i: int, j: int, c: np.ndarray, s: np.ndarray, B: np.ndarray, items=None,
           want=("c64", "n64", "c32", "cm")):
    """Oracle quantities for C_b = G(i, j, theta_b) B_b.

    c, s: [batch] FP32; B: [batch, n, ncols].  ``items`` selects which batch
    items to evaluate (default: all); the outputs are [len(items), n, ncols]."""
    c = _f32(c).reshape(-1)
    s = _f32(s).reshape(-1)
    B = _f32(B)
    batch, n, ncols = B.shape
    assert c.shape == (batch,) and s.shape == (batch,)
    assert 0 <= i < n and 0 <= j < n and i != j
    items = np.arange(batch, dtype=np.int64) if items is None else \
        np.ascontiguousarray(items, dtype=np.int64)
    t = items.shape[0]
    out = {}
    for key, dt in (("c64", np.float64), ("n64", np.float64),
                    ("c32", np.float32), ("cm", np.float64)):
        out[key] = np.zeros((t, n, ncols), dtype=dt) if key in want else None
    _load().oracle_givens(n, i, j, ncols, t, _ptr(items), _ptr(c), _ptr(s), 1, _ptr(B),
                          ncols, n * ncols, _ptr(out["c64"]), _ptr(out["n64"]),
                          _ptr(out["c32"]), _ptr(out["cm"]), ncols, n * ncols)
    return {key: v for key, v in out.items() if v is not None}


# --------------------------------------------------------------------------
# Error metric (Sec. 4.4.2: max relative error, normalised by (|A||B|)_ij)
# --------------------------------------------------------------------------

def rel_err(C, c64, n64) -> np.ndarray:
    """Per-element |C - C64| / (|A||B|)_ij in FP64; 0 where both sides are 0.

    Where the normaliser is 0 every product in the sum is 0, so C must be
    exactly 0; a nonzero C there is reported as an infinite error."""
    C = np.asarray(C, dtype=np.float64)
    c64 = np.asarray(c64, dtype=np.float64)
    n64 = np.asarray(n64, dtype=np.float64)
    diff = np.abs(C - c64)
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.where(n64 > 0, diff / np.where(n64 > 0, n64, 1.0),
                     np.where(diff == 0, 0.0, np.inf))
    e = np.where(np.isnan(C), np.inf, e)
    return e


def max_rel_err(C, c64, n64) -> float:
    e = rel_err(C, c64, n64)
    return float(e.max()) if e.size else 0.0
