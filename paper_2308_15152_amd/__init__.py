"""Single-precision-emulating batched GEMM on MI355X (gfx950) matrix cores.

Python binding of ``libsgemm_emu.so`` (C ABI in ``include/sgemm_emu.h``).
Every function here only marshals arguments: sizes, strides and device
pointers are read off torch tensors and handed to the C entry point of the
same name, on the current torch stream.  All arithmetic runs in the HIP
kernels; there is no fallback path, and a missing library is an error.

Method (Ootomo & Yokota, HPC Asia 2023, Sec. 4.4): each FP32 operand is
split in registers into fp16 hi and lo = fp16((x - hi) * 2^11); three fp16
MFMA products hi.hi, lo.hi and hi.lo are accumulated in FP32, the two
correction products in their own accumulator, and C = main + corr * 2^-11.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

__all__ = [
    "SgemmEmuError", "lib_path", "load",
    "sgemm_emu_batched", "sgemm_emu_batched_ex", "sgemm_emu_resolve_policy",
    "sgemm_emu_batched_acc", "sgemm_emu_scan",
    "householder_emu_batched", "householder_emu_batched_ex", "givens_emu_batched",
    "sgemm_emu_split", "mfmae_num_elements", "mfmae_map", "mfmae_foreach", "mfmae_mma_probe",
    "sgemm_emu_strerror", "sgemm_emu_last_hip_error",
    "sgemm_emu_xcd_order", "sgemm_emu_tile_order", "sgemm_emu_block_order",
    "sgemm_emu_stream_probe", "sgemm_emu_mfma_probe",
    "HOUSEHOLDER_RULE", "HOUSEHOLDER_LDS", "SPLIT_SCALAR", "SPLIT_PAIR", "SPLIT_EIGHT",
    "OP_N", "OP_T", "ROW_MAJOR", "COL_MAJOR",
    "GIVENS_AUTO", "GIVENS_MAP", "GIVENS_EMBEDDED", "GIVENS_LDS",
    "Policy", "FLOW_AUTO", "FLOW_SPLIT", "FLOW_DIRECT", "FLOW_STAGED", "FLOW_REG",
    "TILE_AUTO", "TILE_64x64", "TILE_128x128", "TILE_256x128", "TILE_128x256",
    "SHAPE_16x16x32", "SHAPE_32x32x16", "USE_A", "USE_B", "USE_ACC",
    "EXPORTED_SYMBOLS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_NAME = "libsgemm_emu.so"

FLOW_AUTO, FLOW_SPLIT, FLOW_DIRECT, FLOW_STAGED, FLOW_REG = 0, 1, 2, 3, 4
TILE_AUTO, TILE_64x64, TILE_128x128, TILE_256x128, TILE_128x256 = 0, 1, 2, 3, 4
SHAPE_16x16x32, SHAPE_32x32x16 = 0, 1
USE_A, USE_B, USE_ACC = 0, 1, 2
GIVENS_AUTO, GIVENS_MAP, GIVENS_EMBEDDED, GIVENS_LDS = 0, 1, 2, 3
OP_N, OP_T = 0, 1
HOUSEHOLDER_RULE, HOUSEHOLDER_LDS = 0, 1
SPLIT_SCALAR, SPLIT_PAIR, SPLIT_EIGHT = 0, 1, 2
ROW_MAJOR, COL_MAJOR = 0, 1

# Every symbol declared in include/sgemm_emu.h.
EXPORTED_SYMBOLS = (
    "sgemm_emu_batched", "sgemm_emu_batched_ex", "sgemm_emu_resolve_policy",
    "sgemm_emu_batched_acc", "sgemm_emu_scan",
    "householder_emu_batched", "householder_emu_batched_ex", "givens_emu_batched",
    "sgemm_emu_split", "mfmae_num_elements", "mfmae_map", "mfmae_foreach", "mfmae_mma_probe",
    "sgemm_emu_strerror", "sgemm_emu_last_hip_error",
    "sgemm_emu_xcd_order", "sgemm_emu_tile_order", "sgemm_emu_block_order",
    "sgemm_emu_stream_probe", "sgemm_emu_mfma_probe",
)


class SgemmEmuError(RuntimeError):
    def __init__(self, code: int, where: str):
        msg = _strerror(code)
        if code == -7:
            msg += f" (hipError {sgemm_emu_last_hip_error()})"
        super().__init__(f"{where}: {msg} [code {code}]")
        self.code = code


class Stride(ctypes.Structure):
    _fields_ = [("a", ctypes.c_int64), ("b", ctypes.c_int64), ("c", ctypes.c_int64)]


class Stride4(ctypes.Structure):
    _fields_ = [("a", ctypes.c_int64), ("b", ctypes.c_int64), ("c", ctypes.c_int64),
                ("d", ctypes.c_int64)]


class Policy(ctypes.Structure):
    """Policy of the emulated product (flow, error correction, tile)."""
    _fields_ = [("flow", ctypes.c_int), ("ec", ctypes.c_int), ("tile", ctypes.c_int)]

    def __init__(self, flow: int = FLOW_AUTO, ec: int = 1, tile: int = TILE_AUTO):
        super().__init__(flow, ec, tile)


_lib = None
_NO_SWITCH = contextlib.nullcontext()


class _CheckedInt32(ctypes.c_int32):
    """int argument of the C ABI: a value outside the 32-bit range raises
    instead of being wrapped (ctypes alone would pass 2^32 + 8 as 8)."""

    @classmethod
    def from_param(cls, value):
        v = int(value)
        if not -(1 << 31) <= v < (1 << 31):
            raise ValueError(f"{v} does not fit the 32-bit int argument")
        return ctypes.c_int32(v)


class _CheckedInt64(ctypes.c_int64):
    """int64_t argument of the C ABI, range-checked the same way."""

    @classmethod
    def from_param(cls, value):
        v = int(value)
        if not -(1 << 63) <= v < (1 << 63):
            raise ValueError(f"{v} does not fit the 64-bit int argument")
        return ctypes.c_int64(v)


def lib_path() -> str:
    return os.environ.get("SGEMM_EMU_LIB", os.path.join(_HERE, LIB_NAME))


def load():
    """Load the shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise ImportError(
            f"{path} not found: build it first (python -c 'import __graft_entry__ as g; g.build()'"
            " or python paper_2308_15152_amd/build.py)")
    lib = ctypes.CDLL(path)
    i32, i64, P = _CheckedInt32, _CheckedInt64, ctypes.c_void_p
    ip = ctypes.POINTER(ctypes.c_int)
    sig = {
        "sgemm_emu_batched": ([i32, i32, i32, P, i32, P, i32, P, i32, i32, Stride, P], i32),
        "sgemm_emu_batched_ex": ([i32, i32, i32, P, i32, P, i32, P, i32, i32, Stride,
                                  ctypes.POINTER(Policy), P], i32),
        "sgemm_emu_resolve_policy": ([i32, i32, i32, P, i32, P, i32, P, i32, i32, Stride,
                                      ctypes.POINTER(Policy), ctypes.POINTER(Policy),
                                      ctypes.POINTER(ctypes.c_char_p)], i32),
        "sgemm_emu_batched_acc": ([i32, i32, i32, i32, i32, i32, P, i32, P, i32, P, i32, P, i32,
                                   i32, Stride4, i32, i32, P], i32),
        "sgemm_emu_scan": ([i64, i32, P, i64, P, i64, P], i32),
        "householder_emu_batched": ([i32, P, i64, P, i32, i64, i32, P, i32, i64, i32, P], i32),
        "householder_emu_batched_ex": ([i32, P, i64, P, i32, i64, i32, P, i32, i64, i32, i32, P],
                                       i32),
        "givens_emu_batched": ([i32, i32, i32, P, P, i64, P, i32, i64, i32, P, i32, i64, i32,
                                i32, P], i32),
        "sgemm_emu_split": ([i64, P, P, P, i32, P], i32),
        "mfmae_num_elements": ([i32, i32], i32),
        "mfmae_map": ([i32, i32, i32, i32, ip, ip], i32),
        "mfmae_foreach": ([i32, i32, i32, ip, ip], i32),
        "mfmae_mma_probe": ([i32, P, P, P, P], i32),
        "sgemm_emu_strerror": ([i32], ctypes.c_char_p),
        "sgemm_emu_last_hip_error": ([], i32),
        "sgemm_emu_xcd_order": ([i32, P], i32),
        "sgemm_emu_tile_order": ([i32, i32, P, P], i32),
        "sgemm_emu_block_order": ([i32, i32, P, P], i32),
        "sgemm_emu_stream_probe": ([i64, i64, P, P, P, i32, P], i32),
        "sgemm_emu_mfma_probe": ([i32, i32, i32, P, i32, P, i32, P, i32, P], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int if res is i32 else res  # plain int results
    _lib = lib
    return lib


def _strerror(code: int) -> str:
    return load().sgemm_emu_strerror(int(code)).decode()


def sgemm_emu_strerror(code: int) -> str:
    return _strerror(code)


def sgemm_emu_last_hip_error() -> int:
    return int(load().sgemm_emu_last_hip_error())


def _check(rc: int, where: str) -> None:
    if rc != 0:
        raise SgemmEmuError(rc, where)


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch

    if torch.cuda.is_available() and torch.cuda.is_initialized():
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(0)


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(0 if t is None else int(t.data_ptr()))


def _on_device(*ts):
    """Context for a launch on the tensors' device: every tensor given (None
    skipped) must be a device tensor of one device, which is made current so
    that the kernels and the current stream are that device's."""
    import torch

    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("every operand must be a device tensor")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"operands on different devices: {dev} and {t.device}")
    if dev is None or dev.index == torch.cuda.current_device():
        return _NO_SWITCH
    return torch.cuda.device(dev)


def _check_shape(t, shape, name: str) -> None:
    """An output the caller passes must have exactly the shape the call
    writes: the library writes every element of that shape and cannot see
    the allocation behind the pointer."""
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _matrix_view(t, name: str):
    """(batch, rows, cols, ld, batch_stride) of a 2-D or 3-D FP32 tensor whose
    rows are contiguous."""
    import torch

    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dim() == 2:
        rows, cols = t.shape
        if cols > 1 and t.stride(1) != 1:
            raise ValueError(f"{name} rows must be contiguous (stride 1 along the last dim)")
        return None, rows, cols, t.stride(0) if rows > 1 else max(cols, 1), 0
    if t.dim() != 3:
        raise ValueError(f"{name} must be 2-D or 3-D")
    b, rows, cols = t.shape
    if cols > 1 and t.stride(2) != 1:
        raise ValueError(f"{name} rows must be contiguous (stride 1 along the last dim)")
    ld = t.stride(1) if rows > 1 else max(cols, 1)
    return b, rows, cols, ld, t.stride(0) if b > 1 else 0


def _gemm_args(A, B, C):
    """(m, n, k, lda, ldb, ldc, batch, stride, C) of a batched product; C is
    allocated if None."""
    import torch

    ba, m, k, lda, sa = _matrix_view(A, "A")
    bb, kb, n, ldb, sb = _matrix_view(B, "B")
    if kb != k:
        raise ValueError(f"inner dimensions differ: A is {m}x{k}, B is {kb}x{n}")
    batch = ba if ba is not None else (bb if bb is not None else 1)
    if ba is not None and bb is not None and ba != bb:
        raise ValueError("batch sizes differ")
    if C is None:
        C = torch.empty((batch, m, n), dtype=torch.float32, device=A.device)
    bc, mc, nc, ldc, sc = _matrix_view(C if C.dim() == 3 else C.unsqueeze(0), "C")
    if (mc, nc) != (m, n) or (bc if bc is not None else 1) != batch:
        raise ValueError("C has the wrong shape")
    st = Stride(sa, sb, sc if batch > 1 else 0)
    return m, n, k, lda, ldb, ldc, batch, st, C


def sgemm_emu_batched(A, B, C=None, *, policy: Policy | None = None, stream=None):
    """C[t] := A[t] @ B[t] with the emulated FP32 product.

    A: [batch, m, k] or [m, k]; B: [batch, k, n] or [k, n] (a 2-D operand is
    broadcast over the batch); C: [batch, m, n] (allocated if None).  Rows of
    every operand must be contiguous; leading dimensions and batch strides are
    taken from the tensors' strides.  Runs on the current torch stream unless
    ``stream`` (a hipStream_t handle) is given.  With ``policy`` the call goes
    to sgemm_emu_batched_ex."""
    m, n, k, lda, ldb, ldc, batch, st, C = _gemm_args(A, B, C)
    lib = load()
    with _on_device(A, B, C):
        if policy is None:
            rc = lib.sgemm_emu_batched(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, batch,
                                       st, _stream(stream))
            _check(rc, "sgemm_emu_batched")
        else:
            rc = lib.sgemm_emu_batched_ex(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc,
                                          batch, st, ctypes.byref(policy), _stream(stream))
            _check(rc, "sgemm_emu_batched_ex")
    return C


def sgemm_emu_resolve_policy(A, B, C, *, policy: Policy | None = None):
    """(policy, kernel name) the library would run for this product, with
    AUTO flow and tile resolved (a host-side query; nothing is launched)."""
    m, n, k, lda, ldb, ldc, batch, st, C = _gemm_args(A, B, C)
    out = Policy()
    kern = ctypes.c_char_p()
    rc = load().sgemm_emu_resolve_policy(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc,
                                         batch, st, None if policy is None else
                                         ctypes.byref(policy), ctypes.byref(out),
                                         ctypes.byref(kern))
    _check(rc, "sgemm_emu_resolve_policy")
    return out, (kern.value or b"").decode()


def sgemm_emu_xcd_order(grid: int):
    """Task each workgroup of a grid of ``grid`` workgroups takes first (the
    kernels' XCD-aware numbering, computed on the host), as a numpy int32
    array of ``grid`` entries."""
    import numpy as np

    out = np.empty(max(int(grid), 0), dtype=np.int32)
    _check(load().sgemm_emu_xcd_order(int(grid), out.ctypes.data_as(ctypes.c_void_p)),
           "sgemm_emu_xcd_order")
    return out


def sgemm_emu_tile_order(tiles_m: int, tiles_n: int):
    """(tile row, tile column) of each task of one item, in task order (the
    kernels' grouped tile order, computed on the host): two numpy int32
    arrays of ``tiles_m * tiles_n`` entries."""
    import numpy as np

    count = max(int(tiles_m), 0) * max(int(tiles_n), 0)
    rows = np.empty(count, dtype=np.int32)
    cols = np.empty(count, dtype=np.int32)
    _check(load().sgemm_emu_tile_order(int(tiles_m), int(tiles_n),
                                       rows.ctypes.data_as(ctypes.c_void_p),
                                       cols.ctypes.data_as(ctypes.c_void_p)),
           "sgemm_emu_tile_order")
    return rows, cols


def sgemm_emu_block_order(tiles_m: int, tiles_n: int):
    """(tile row, tile column) of each task of a one-item launch on the
    128 x 256 full-tile kernel when both tile counts are multiples of 16 (the
    device-wide block order, computed on the host): two numpy int32 arrays
    of ``tiles_m * tiles_n`` entries."""
    import numpy as np

    count = max(int(tiles_m), 0) * max(int(tiles_n), 0)
    rows = np.empty(count, dtype=np.int32)
    cols = np.empty(count, dtype=np.int32)
    _check(load().sgemm_emu_block_order(int(tiles_m), int(tiles_n),
                                        rows.ctypes.data_as(ctypes.c_void_p),
                                        cols.ctypes.data_as(ctypes.c_void_p)),
           "sgemm_emu_block_order")
    return rows, cols


def sgemm_emu_stream_probe(A, B, C, *, threads: int = 256, stream=None):
    """Measurement reference: C[t] := A[t] + B[t] for every item t of
    [items, ...] contiguous float32 device tensors of one shape, one
    workgroup of ``threads`` threads per item (the read-A, read-B, write-C
    traffic of a batched product without its arithmetic)."""
    import torch

    for name, t in (("A", A), ("B", B), ("C", C)):
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 device tensor")
    if A.shape != B.shape or A.shape != C.shape or A.dim() < 1:
        raise ValueError("A, B and C must have one shape [items, ...]")
    items = A.shape[0]
    per = A.numel() // max(items, 1)
    with _on_device(A, B, C):
        rc = load().sgemm_emu_stream_probe(items, per, _ptr(A), _ptr(B), _ptr(C), int(threads),
                                           _stream(stream))
    _check(rc, "sgemm_emu_stream_probe")
    return C


def sgemm_emu_mfma_probe(A, B, k: int, C=None, *, stream=None):
    """Measurement reference: the full-tile kernel's products for an m x n x k
    product on 128 x 256 tiles, with the fragments of the first k chunk held
    in registers (no loads, split or LDS traffic in the k loop).  A: [m, >= 32]
    and B: [>= 32, n] float32 device tensors with contiguous rows (only
    A[:, :32] and B[:32, :] are read); C: [m, n] (allocated if None) receives
    (k / 32) * the emulated product A[:, :32] @ B[:32, :]."""
    import torch

    ba, m, ka, lda, _ = _matrix_view(A, "A")
    bb, kb, n, ldb, _ = _matrix_view(B, "B")
    if ba is not None or bb is not None:
        raise ValueError("A and B must be 2-D")
    if ka < 32 or kb < 32:
        raise ValueError("A needs 32 columns and B 32 rows")
    if C is None:
        C = torch.empty((m, n), dtype=torch.float32, device=A.device)
    _check_shape(C, (m, n), "C")
    _, _, _, ldc, _ = _matrix_view(C, "C")
    with _on_device(A, B, C):
        rc = load().sgemm_emu_mfma_probe(m, n, int(k), _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc,
                                         _stream(stream))
    _check(rc, "sgemm_emu_mfma_probe")
    return C


def sgemm_emu_batched_ex(A, B, C=None, *, policy: Policy, stream=None):
    return sgemm_emu_batched(A, B, C, policy=policy, stream=stream)


def sgemm_emu_batched_acc(A, B, C=None, D=None, *, op_a: int = OP_N, op_b: int = OP_N,
                          layout: int = ROW_MAJOR, shape: int = SHAPE_32x32x16, ec: int = 1,
                          stream=None):
    """D := op(A) @ op(B) + C per batch item.

    A, B, C, D are 2-D or 3-D float32 device tensors with contiguous rows,
    given in their stored form: A is [m, k] (op_a OP_N) or [k, m] (OP_T),
    B is [k, n] or [n, k]; C and D are [m, n] (layout ROW_MAJOR) or [n, m]
    (COL_MAJOR).  C may be None (zero) or D itself (in place); D is
    allocated if None."""
    import torch

    ba, ar, ac, lda, sa = _matrix_view(A, "A")
    bb, br, bc, ldb, sb = _matrix_view(B, "B")
    m, k = (ac, ar) if op_a == OP_T else (ar, ac)
    kb, n = (bc, br) if op_b == OP_T else (br, bc)
    if kb != k:
        raise ValueError(f"inner dimensions differ: {k} vs {kb}")
    batch = max(ba or 1, bb or 1)
    for name, b in (("A", ba), ("B", bb)):
        if b is not None and b != batch:
            raise ValueError(f"{name} batch {b} != {batch}")
    stored = (n, m) if layout == COL_MAJOR else (m, n)
    if D is None:
        shape_d = (batch, *stored) if (ba is not None or bb is not None) else stored
        D = torch.empty(shape_d, dtype=torch.float32, device=A.device)
    bd, dr, dc, ldd, sd = _matrix_view(D, "D")
    if (dr, dc) != stored or (bd or 1) != batch:
        raise ValueError("D has the wrong shape")
    ldc, sc = 1, 0
    if C is not None:
        bcx, cr, ccol, ldc, sc = _matrix_view(C, "C")
        if (cr, ccol) != stored or (bcx is not None and bcx != batch):
            raise ValueError("C has the wrong shape")
    st = Stride4(sa, sb, sc, sd)
    with _on_device(A, B, C, D):
        rc = load().sgemm_emu_batched_acc(int(op_a), int(op_b), int(layout), m, n, k, _ptr(A),
                                          lda, _ptr(B), ldb, _ptr(C), ldc, _ptr(D), ldd, batch,
                                          st, int(shape), int(ec), _stream(stream))
    _check(rc, "sgemm_emu_batched_acc")
    return D


def sgemm_emu_scan(X, Y=None, *, stream=None):
    """Inclusive scan of every row: Y[..., j] = sum_{i <= j} X[..., i].

    X: float32 device tensor whose last dimension is the row and whose rows
    are evenly spaced (2-D with contiguous rows, or any contiguous tensor).
    Y: same shape (allocated if None); Y may be X (in place)."""
    import torch

    if X.dtype != torch.float32 or not X.is_cuda:
        raise ValueError("X must be a float32 device tensor")
    if X.dim() == 2:
        rows, length = X.shape
        if length > 1 and X.stride(1) != 1:
            raise ValueError("X rows must be contiguous")
        ldx = X.stride(0) if rows > 1 else max(length, 1)
    else:
        if not X.is_contiguous():
            raise ValueError("X must be contiguous (or 2-D with contiguous rows)")
        length = X.shape[-1] if X.dim() else 1
        rows = X.numel() // max(length, 1)
        ldx = max(length, 1)
    if Y is None:
        Y = torch.empty(X.shape, dtype=torch.float32, device=X.device)
    if Y.shape != X.shape or Y.dtype != torch.float32 or not Y.is_cuda:
        raise ValueError("Y must be a float32 device tensor of X's shape")
    if Y.dim() == 2:
        if length > 1 and Y.stride(1) != 1:
            raise ValueError("Y rows must be contiguous")
        ldy = Y.stride(0) if rows > 1 else max(length, 1)
    else:
        if not Y.is_contiguous():
            raise ValueError("Y must be contiguous (or 2-D with contiguous rows)")
        ldy = max(length, 1)
    with _on_device(X, Y):
        rc = load().sgemm_emu_scan(rows, length, _ptr(X), ldx, _ptr(Y), ldy, _stream(stream))
    _check(rc, "sgemm_emu_scan")
    return Y


def householder_emu_batched(u, B, C=None, *, mode: int = HOUSEHOLDER_RULE, stream=None):
    """C[t] := (I - 2 u[t] u[t]^T) @ B[t]; u: [batch, 64], B: [batch, 64, ncols].
    mode: HOUSEHOLDER_RULE (reflector built in registers) or HOUSEHOLDER_LDS
    (baseline through LDS)."""
    import torch

    if u.dtype != torch.float32 or not u.is_cuda or u.dim() != 2:
        raise ValueError("u must be a [batch, n] float32 device tensor")
    batch, n = u.shape
    if n > 1 and u.stride(1) != 1:
        raise ValueError("u rows must be contiguous")
    bb, nb, ncols, ldb, sb = _matrix_view(B, "B")
    if nb != n or (bb or 1) != batch:
        raise ValueError("B must be [batch, n, ncols]")
    if C is None:
        C = torch.empty((batch, n, ncols), dtype=torch.float32, device=u.device)
    _check_shape(C, (batch, n, ncols) if C.dim() == 3 else (n, ncols), "C")
    if C.dim() == 2 and batch != 1:
        raise ValueError("a 2-D C holds one item")
    _, _, _, ldc, sc = _matrix_view(C, "C")
    su = u.stride(0) if batch > 1 else 0
    with _on_device(u, B, C):
        rc = load().householder_emu_batched_ex(n, _ptr(u), su, _ptr(B), ldb, sb, ncols, _ptr(C),
                                               ldc, sc, batch, int(mode), _stream(stream))
    _check(rc, "householder_emu_batched_ex")
    return C


def householder_emu_batched_ex(u, B, C=None, *, mode: int, stream=None):
    return householder_emu_batched(u, B, C, mode=mode, stream=stream)


def givens_emu_batched(i, j, c, s, B, C=None, *, mode: int = GIVENS_AUTO, stream=None):
    """C[t] := G(i, j, theta_t) @ B[t] with c[t] = cos theta_t, s[t] = sin theta_t;
    c, s: [batch] float32, B: [batch, n, ncols]."""
    import torch

    for name, v in (("c", c), ("s", s)):
        if v.dtype != torch.float32 or not v.is_cuda or v.dim() != 1:
            raise ValueError(f"{name} must be a [batch] float32 device tensor")
    if c.shape != s.shape or c.stride() != s.stride():
        raise ValueError("c and s must have the same shape and stride")
    batch = c.shape[0]
    bb, n, ncols, ldb, sb = _matrix_view(B, "B")
    if (bb or 1) != batch:
        raise ValueError("B must be [batch, n, ncols]")
    if C is None:
        C = torch.empty((batch, n, ncols), dtype=torch.float32, device=B.device)
    _check_shape(C, (batch, n, ncols) if C.dim() == 3 else (n, ncols), "C")
    if C.dim() == 2 and batch != 1:
        raise ValueError("a 2-D C holds one item")
    _, _, _, ldc, sc = _matrix_view(C, "C")
    scs = c.stride(0) if batch > 1 else 0
    with _on_device(c, s, B, C):
        rc = load().givens_emu_batched(n, int(i), int(j), _ptr(c), _ptr(s), scs, _ptr(B), ldb,
                                       sb, ncols, _ptr(C), ldc, sc, batch, int(mode),
                                       _stream(stream))
    _check(rc, "givens_emu_batched")
    return C


def sgemm_emu_split(x, *, form: int = SPLIT_SCALAR, stream=None):
    """Elementwise split on the device: (hi, lo) binary16 bit patterns as int16
    tensors of x's shape (x: contiguous float32 device tensor).  ``form``
    picks the device function: SPLIT_SCALAR, SPLIT_PAIR or SPLIT_EIGHT."""
    import torch

    if x.dtype != torch.float32 or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous float32 device tensor")
    hi = torch.empty(x.shape, dtype=torch.int16, device=x.device)
    lo = torch.empty(x.shape, dtype=torch.int16, device=x.device)
    with _on_device(x, hi, lo):
        rc = load().sgemm_emu_split(x.numel(), _ptr(x), _ptr(hi), _ptr(lo), int(form),
                                    _stream(stream))
    _check(rc, "sgemm_emu_split")
    return hi, lo


def mfmae_num_elements(shape: int, use: int) -> int:
    rc = int(load().mfmae_num_elements(shape, use))
    _check(min(rc, 0), "mfmae_num_elements")
    return rc


def mfmae_map(shape: int, use: int, i: int, j: int):
    """(lane, element) holding matrix position (i, j)."""
    lane, elem = ctypes.c_int(), ctypes.c_int()
    _check(load().mfmae_map(shape, use, i, j, ctypes.byref(lane), ctypes.byref(elem)), "mfmae_map")
    return lane.value, elem.value


def mfmae_foreach(shape: int, use: int, lane: int):
    """[(i, j) for each element of `lane`]."""
    n = mfmae_num_elements(shape, use)
    ii = (ctypes.c_int * n)()
    jj = (ctypes.c_int * n)()
    _check(load().mfmae_foreach(shape, use, lane, ii, jj), "mfmae_foreach")
    return list(zip(list(ii), list(jj)))


def mfmae_mma_probe(shape: int, a_lanes, b_lanes, *, stream=None):
    """One MFMA on operands given lane by lane: a_lanes, b_lanes are [64, 8]
    int16 device tensors of binary16 bit patterns; returns the [64, n] FP32
    accumulator (n = 4 or 16) with the accumulator starting at zero."""
    import torch

    n = mfmae_num_elements(shape, USE_ACC)
    for name, t in (("a_lanes", a_lanes), ("b_lanes", b_lanes)):
        if t.dtype != torch.int16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous int16 device tensor")
        _check_shape(t, (64, 8), name)
    d = torch.empty((64, n), dtype=torch.float32, device=a_lanes.device)
    with _on_device(a_lanes, b_lanes, d):
        rc = load().mfmae_mma_probe(shape, _ptr(a_lanes), _ptr(b_lanes), _ptr(d),
                                    _stream(stream))
    _check(rc, "mfmae_mma_probe")
    return d
