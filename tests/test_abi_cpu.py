"""Host-side checks of the C ABI (no GPU needed).

* the library loads and exports every function include/sgemm_emu.h declares;
* every invalid argument is rejected with its documented code before any HIP
  call (the fake device pointers below are never dereferenced);
* empty problems are successful no-ops;
* the fragment maps are bijections and map/foreach are mutually inverse.
"""
import ctypes
import os
import pathlib
import re
import subprocess

import pytest

import paper_2308_15152_amd as pkg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sgemm_emu.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declarations_match_binding():
    assert _declared_functions() == sorted(pkg.EXPORTED_SYMBOLS)


def test_binding_defines_every_public_name():
    for name in pkg.__all__:
        assert hasattr(pkg, name), name
    for name in pkg.EXPORTED_SYMBOLS:
        assert callable(getattr(pkg, name, None)), name


def test_library_exports_every_declared_symbol():
    lib = pkg.load()
    for name in _declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", pkg.lib_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in _declared_functions():
        assert name in exported, name


# fake, well separated device addresses: validation must reject or no-op
# before anything would touch them
PA, PB, PC = 0x10000000, 0x20000000, 0x30000000
S = pkg.Stride


def gemm(m, n, k, A=PA, lda=None, B=PB, ldb=None, C=PC, ldc=None, batch=1, st=(0, 0, 0),
         policy=None):
    lib = pkg.load()
    lda = k if lda is None else lda
    ldb = n if ldb is None else ldb
    ldc = n if ldc is None else ldc
    args = (m, n, k, ctypes.c_void_p(A), max(lda, 0), ctypes.c_void_p(B), max(ldb, 0),
            ctypes.c_void_p(C), max(ldc, 0), batch, S(*st))
    if policy is None:
        return lib.sgemm_emu_batched(*args, ctypes.c_void_p(0))
    return lib.sgemm_emu_batched_ex(*args, ctypes.byref(policy), ctypes.c_void_p(0))


@pytest.mark.parametrize("dims", [(-1, 4, 4), (4, -1, 4), (4, 4, -1)])
def test_negative_dims(dims):
    assert gemm(*dims) == -1


def test_negative_batch():
    assert gemm(4, 4, 4, batch=-2) == -1


def test_leading_dimensions():
    assert gemm(4, 8, 16, lda=15) == -2
    assert gemm(4, 8, 16, ldb=7) == -2
    assert gemm(4, 8, 16, ldc=7) == -2
    assert gemm(4, 8, 0, lda=0) == -2  # lda >= max(1, k)


def test_null_pointers():
    assert gemm(4, 4, 4, C=0) == -3
    assert gemm(4, 4, 4, A=0) == -3
    assert gemm(4, 4, 4, B=0) == -3


def test_strides():
    assert gemm(4, 4, 4, batch=2, st=(-16, 16, 16)) == -4
    assert gemm(4, 4, 4, batch=2, st=(16, 16, 15)) == -4  # C items would overlap
    # spans that run past the end of the address space (computed without wrapping)
    assert gemm(4, 4, 4, batch=2, st=(16, 16, 1 << 62)) == -4
    assert gemm(4, 4, 4, batch=2, st=(1 << 62, 16, 16)) == -4
    assert gemm(4, 4, 4, batch=1 << 30, st=(16, 1 << 34, 16)) == -4


def test_aliasing():
    assert gemm(4, 4, 4, C=PA) == -5
    assert gemm(4, 4, 4, C=PB + 8) == -5
    # the last C item reaches into B
    assert gemm(4, 4, 4, C=PB - 3 * 16 * 4, batch=4, st=(16, 16, 16)) == -5


def test_policy_values():
    assert gemm(4, 4, 4, policy=pkg.Policy(flow=7)) == -8
    assert gemm(4, 4, 4, policy=pkg.Policy(ec=2)) == -8
    assert gemm(4, 4, 4, policy=pkg.Policy(tile=9)) == -8
    # LDS of the staged flow does not fit the largest tile
    assert gemm(4, 4, 4, policy=pkg.Policy(flow=pkg.FLOW_STAGED, tile=pkg.TILE_256x128)) == -8
    # the register-direct flow has no 256x128 tile and needs 16-byte A rows
    # and, with 64-wide waves, column pairs
    reg = pkg.FLOW_REG
    assert gemm(4, 4, 4, policy=pkg.Policy(flow=reg, tile=pkg.TILE_256x128)) == -8
    assert gemm(4, 4, 6, policy=pkg.Policy(flow=reg, tile=pkg.TILE_64x64)) == -8
    assert gemm(4, 4, 4, A=PA + 4, policy=pkg.Policy(flow=reg, tile=pkg.TILE_64x64)) == -8
    assert gemm(4, 5, 4, policy=pkg.Policy(flow=reg, tile=pkg.TILE_128x128)) == -8
    assert gemm(4, 4, 4, B=PB + 4, policy=pkg.Policy(flow=reg, tile=pkg.TILE_128x128)) == -8
    assert gemm(4, 4, 4, lda=1 << 23, policy=pkg.Policy(flow=reg, tile=pkg.TILE_64x64)) == -8


def _resolve(m, n, k, batch=1, st=(0, 0, 0), policy=None, A=PA, B=PB, C=PC):
    lib = pkg.load()
    out = pkg.Policy()
    kern = ctypes.c_char_p()
    rc = lib.sgemm_emu_resolve_policy(m, n, k, ctypes.c_void_p(A), k, ctypes.c_void_p(B), n,
                                      ctypes.c_void_p(C), n, batch, S(*st),
                                      None if policy is None else ctypes.byref(policy),
                                      ctypes.byref(out), ctypes.byref(kern))
    _resolve.kernel = (kern.value or b"").decode()
    return rc, (out.flow, out.ec, out.tile)


def test_resolve_policy():
    """The automatic choice: the pipelined full-tile kernel whenever a tile
    fits (128 x 256 for large products, else 256 x 128, else 128 x 128), the
    register-direct flow for other small products (32 x 32 waves up to
    64 x 64), the general LDS split flow otherwise; explicit policies pass
    through; the same validation as the launching entry point."""
    s128 = 128 * 128
    assert _resolve(128, 128, 128, 4096, (s128, s128, s128)) == (0, (pkg.FLOW_SPLIT, 1,
                                                                       pkg.TILE_128x128))
    assert _resolve.kernel == "bgemm_big_kernel"
    s256 = 256 * 256
    assert _resolve(256, 256, 256, 1024, (s256, s256, s256)) == (0, (pkg.FLOW_SPLIT, 1,
                                                                     pkg.TILE_256x128))
    # 256 x 128 tiles with k <= 2048 run the persistent stream form
    assert _resolve.kernel == "bgemm_big_stream_kernel"
    assert _resolve(256, 256, 4096, 4, (256 * 4096, 4096 * 256, s256)) == (
        0, (pkg.FLOW_SPLIT, 1, pkg.TILE_256x128))
    assert _resolve.kernel == "bgemm_big_kernel"
    assert _resolve(8192, 8192, 8192) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))
    assert _resolve.kernel == "bgemm_big_kernel"
    # the batched experiment of Sec. 4.4.2: 128x256 from k = 1024 on
    s1m = 1024 * 1024
    apart = dict(A=1 << 40, B=2 << 40, C=3 << 40)  # gigabytes apart: no overlap
    assert _resolve(1024, 1024, 512, 256, (1024 * 512, 512 * 1024, s1m),
                    **apart) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_256x128))
    assert _resolve(1024, 1024, 1024, 256, (s1m, s1m, s1m),
                    **apart) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))
    assert _resolve(64, 64, 64, 16, (4096, 4096, 4096)) == (0, (pkg.FLOW_REG, 1,
                                                                 pkg.TILE_64x64))
    assert _resolve.kernel == "bgemm_reg_kernel"
    # ragged small products: register-direct 128x128
    assert _resolve(130, 132, 100, 8, (130 * 100, 100 * 132, 130 * 132)) == (
        0, (pkg.FLOW_REG, 1, pkg.TILE_128x128))
    # large and ragged: whole tiles of the interior on the full-tile kernel,
    # the edge strips on the register-flow kernel
    assert _resolve(8192 - 64, 8192, 8192) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))
    assert _resolve.kernel == "bgemm_big_kernel+bgemm_reg_kernel"
    assert _resolve(8000, 8000, 8008) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))  # k tail 8
    assert _resolve.kernel == "bgemm_big_kernel+bgemm_reg_kernel"
    assert _resolve(4100, 4300, 2060) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))
    assert _resolve.kernel == "bgemm_big_kernel+bgemm_reg_kernel"
    assert _resolve(6000, 6000, 960) == (0, (pkg.FLOW_SPLIT, 1, pkg.TILE_256x128))
    assert _resolve.kernel == "bgemm_big_kernel+bgemm_reg_kernel"
    # ragged products below 2^35 multiply-adds, or whose whole tiles cover
    # less than 95% of C: the register-direct flow
    for shape in ((2000, 2000, 32), (2100, 2300, 1000), (1100, 1100, 512), (3000, 3000, 3000),
                  (1100, 9000, 4000), (3300, 3500, 3000), (2300, 2200, 7000), (2700, 2700, 4740)):
        assert _resolve(*shape) == (0, (pkg.FLOW_REG, 1, pkg.TILE_128x128)), shape
        assert _resolve.kernel == "bgemm_reg_kernel"
    # B rows without 8-byte vectors (n odd): 64 x 64 register tiles below
    # 2^35 multiply-adds, the general kernel above
    assert _resolve(1100, 1101, 512) == (0, (pkg.FLOW_REG, 1, pkg.TILE_64x64))
    assert _resolve.kernel == "bgemm_reg_kernel"
    assert _resolve(4000, 4001, 4000)[1][0] == pkg.FLOW_SPLIT
    assert _resolve.kernel == "bgemm_emu_kernel"
    # unaligned rows (k not a multiple of 4): the general LDS kernel
    assert _resolve(4000, 4000, 4001)[1][0] == pkg.FLOW_SPLIT
    assert _resolve.kernel == "bgemm_emu_kernel"
    # k not a multiple of 4: no 16-byte A rows, so the LDS flow
    assert _resolve(128, 128, 130)[1][0] == pkg.FLOW_SPLIT
    assert _resolve.kernel == "bgemm_emu_kernel"
    # full tiles whose chunk byte offsets would reach 2^31: A rows 2^22
    # floats apart (128 rows x 2^24 bytes), B rows 2^24 floats apart (fake
    # operands 1 TiB apart, so that the spans do not overlap)
    big = 1 << 22
    pol = pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_128x128)
    lib = pkg.load()
    out = pkg.Policy()
    kern = ctypes.c_char_p()

    def far(lda, ldb):
        rc = lib.sgemm_emu_resolve_policy(256, 256, 256, ctypes.c_void_p(1 << 40), lda,
                                          ctypes.c_void_p(2 << 40), ldb, ctypes.c_void_p(3 << 40),
                                          256, 1, S(0, 0, 0), ctypes.byref(pol),
                                          ctypes.byref(out), ctypes.byref(kern))
        assert rc == 0, rc
        return kern.value.decode()

    assert far(big, 256) == "bgemm_emu_kernel"
    assert far(256, 1 << 24) == "bgemm_emu_kernel"
    assert far(big - 256, (1 << 24) - 256) == "bgemm_big_kernel"
    # the paper's flows on full 128 x 128 tiles run in the full-tile kernel
    for flow in (pkg.FLOW_DIRECT, pkg.FLOW_STAGED):
        assert _resolve(8192, 8192, 8192, policy=pkg.Policy(flow, 1, pkg.TILE_128x128)) == (
            0, (flow, 1, pkg.TILE_128x128))
        assert _resolve.kernel == "bgemm_big_kernel"
    pol = pkg.Policy(pkg.FLOW_DIRECT, 0, pkg.TILE_64x64)
    assert _resolve(128, 128, 128, policy=pol) == (0, (pkg.FLOW_DIRECT, 0, pkg.TILE_64x64))
    # the 128x256 tile exists only for full tiles of the split flow
    assert _resolve(128, 256, 64, policy=pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_128x256))[0] == 0
    assert _resolve(128, 200, 64, policy=pkg.Policy(pkg.FLOW_SPLIT, 1,
                                                    pkg.TILE_128x256))[0] == -8
    assert _resolve(128, 256, 64, policy=pkg.Policy(pkg.FLOW_DIRECT, 1,
                                                    pkg.TILE_128x256))[0] == -8
    # without error correction the full-tile kernel runs on its 128 x 128 and
    # 128 x 256 tiles (split flow); other tiles and flows take the general kernel
    assert _resolve(256, 256, 256, policy=pkg.Policy(pkg.FLOW_SPLIT, 0,
                                                     pkg.TILE_256x128))[0] == 0
    assert _resolve.kernel == "bgemm_emu_kernel"
    for tile in (pkg.TILE_128x128, pkg.TILE_128x256):
        assert _resolve(256, 256, 256, policy=pkg.Policy(pkg.FLOW_SPLIT, 0, tile)) == (
            0, (pkg.FLOW_SPLIT, 0, tile))
        assert _resolve.kernel == "bgemm_big_kernel"
    assert _resolve(256, 256, 256, policy=pkg.Policy(pkg.FLOW_DIRECT, 0, pkg.TILE_128x128))[0] == 0
    assert _resolve.kernel == "bgemm_emu_kernel"
    # AUTO tile without error correction: 128 x 256 for long k over much output, else 128 x 128
    assert _resolve(8192, 8192, 8192, policy=pkg.Policy(pkg.FLOW_AUTO, 0, pkg.TILE_AUTO)) == (
        0, (pkg.FLOW_SPLIT, 0, pkg.TILE_128x256))
    assert _resolve.kernel == "bgemm_big_kernel"
    assert _resolve(128, 128, 128, 4096, st=(128 * 128,) * 3,
                    policy=pkg.Policy(pkg.FLOW_AUTO, 0, pkg.TILE_AUTO)) == (
        0, (pkg.FLOW_SPLIT, 0, pkg.TILE_128x128))
    assert _resolve(-1, 4, 4)[0] == -1
    # a named flow with AUTO tile takes a tile that flow is built for (256^3 x
    # 1024 would pick 256x128 by shape, which REG and STAGED do not have)
    s256 = 256 * 256
    auto_cases = [
        ((256, 256, 256, 1024, (s256,) * 3), pkg.FLOW_REG, pkg.TILE_128x128, "bgemm_reg_kernel"),
        ((256, 256, 256, 1024, (s256,) * 3), pkg.FLOW_STAGED, pkg.TILE_128x128,
         "bgemm_big_kernel"),
        ((256, 256, 256, 1024, (s256,) * 3), pkg.FLOW_DIRECT, pkg.TILE_128x128,
         "bgemm_big_kernel"),
        ((300, 260, 96, 1024, (300 * 96, 96 * 260, 300 * 260)), pkg.FLOW_REG, pkg.TILE_128x128,
         "bgemm_reg_kernel"),
        ((300, 260, 96, 1024, (300 * 96, 96 * 260, 300 * 260)), pkg.FLOW_STAGED,
         pkg.TILE_128x128, "bgemm_emu_kernel"),
        ((64, 64, 64, 16, (4096,) * 3), pkg.FLOW_REG, pkg.TILE_64x64, "bgemm_reg_kernel"),
        ((64, 64, 64, 16, (4096,) * 3), pkg.FLOW_STAGED, pkg.TILE_64x64, "bgemm_emu_kernel"),
        # B rows without 16-byte vectors (n odd): REG falls back to 64x64
        ((1100, 1101, 512, 1, (0, 0, 0)), pkg.FLOW_REG, pkg.TILE_64x64, "bgemm_reg_kernel"),
    ]
    for (m, n, k, batch, st), flow, tile, kernel in auto_cases:
        assert _resolve(m, n, k, batch, st, policy=pkg.Policy(flow, 1, pkg.TILE_AUTO),
                        **apart) == (0, (flow, 1, tile)), (m, n, k, flow)
        assert _resolve.kernel == kernel, (m, n, k, flow, _resolve.kernel)
    lib = pkg.load()
    assert lib.sgemm_emu_resolve_policy(4, 4, 4, ctypes.c_void_p(PA), 4, ctypes.c_void_p(PB), 4,
                                        ctypes.c_void_p(PC), 4, 1, S(0, 0, 0), None,
                                        None, None) == -3


def test_empty_problems_are_noops():
    assert gemm(0, 4, 4) == 0
    assert gemm(4, 0, 4, ldb=1, ldc=1) == 0
    assert gemm(4, 4, 4, batch=0) == 0
    assert gemm(0, 4, 4, A=0, B=0, C=0) == 0


def test_householder_validation():
    lib = pkg.load()
    P = ctypes.c_void_p

    def hh(n=64, u=PA, su=64, B=PB, ldb=64, sb=4096, ncols=64, C=PC, ldc=64, sc=4096, batch=2):
        return lib.householder_emu_batched(n, P(u), su, P(B), ldb, sb, ncols, P(C), ldc, sc,
                                           batch, P(0))

    assert hh(n=-1) == -1
    assert hh(ncols=-1) == -1
    assert hh(ldb=63) == -2
    assert hh(n=32) == -6
    assert hh(u=0) == -3
    assert hh(sb=-1) == -4
    assert hh(sc=100) == -4
    assert hh(su=1 << 62) == -4
    assert hh(sc=1 << 62) == -4
    assert hh(C=PB) == -5
    assert hh(C=PA + 4) == -5
    assert hh(batch=0) == 0
    assert hh(ncols=0) == 0
    for mode in (-1, 2):
        assert lib.householder_emu_batched_ex(64, P(PA), 64, P(PB), 64, 4096, 64, P(PC), 64,
                                              4096, 2, mode, P(0)) == -8
    assert lib.householder_emu_batched_ex(64, P(0), 64, P(PB), 64, 4096, 64, P(PC), 64, 4096,
                                          2, 1, P(0)) == -3


def test_givens_validation():
    lib = pkg.load()
    P = ctypes.c_void_p
    PS = PA + 0x100000

    def gv(n=64, i=5, j=37, c=PA, s=PS, scs=1, B=PB, ldb=64, sb=4096, ncols=64, C=PC, ldc=64,
           sc=4096, batch=2, mode=0):
        return lib.givens_emu_batched(n, i, j, P(c), P(s), scs, P(B), ldb, sb, ncols, P(C), ldc,
                                      sc, batch, mode, P(0))

    assert gv(n=-1) == -1
    assert gv(ncols=-1) == -1
    assert gv(batch=-1) == -1
    assert gv(i=64) == -1
    assert gv(j=-1) == -1
    assert gv(i=7, j=7) == -1
    assert gv(mode=4) == -8
    assert gv(mode=-1) == -8
    assert gv(ldb=63) == -2
    assert gv(ldc=10) == -2
    assert gv(n=32, i=1, j=2) == -6
    assert gv(ldb=1 << 27, sb=1 << 33) == -6
    # (3, 60) has no compile-time instance: EMBEDDED refuses it, AUTO and the
    # other modes accept it (checked up to the first pointer test)
    assert gv(i=3, j=60, mode=2) == -6
    assert gv(i=3, j=60, mode=0, c=0) == -3
    assert gv(i=3, j=60, mode=1, c=0) == -3
    assert gv(i=37, j=5, mode=2, c=0) == -3
    assert gv(s=0) == -3
    assert gv(B=0) == -3
    assert gv(C=0) == -3
    assert gv(scs=-1) == -4
    assert gv(sb=-1) == -4
    assert gv(sc=100) == -4
    assert gv(scs=1 << 62) == -4
    assert gv(sb=1 << 62) == -4
    assert gv(C=PB) == -5
    assert gv(C=PA - 4) == -5
    assert gv(C=PS - 64 * 64 * 4 + 8) == -5
    assert gv(batch=0) == 0
    assert gv(ncols=0) == 0
    assert gv(n=0) == 0


def test_batched_acc_validation():
    """Every call here ends in an error before anything is launched: the
    cases that pass one check carry a negative stride, which is rejected
    after the dimension, ld and pointer checks."""
    lib = pkg.load()
    P = ctypes.c_void_p
    PD = PC + 0x1000000
    BAD = (-1, 0, 0, 64 * 48)  # rejected with -4 after every earlier check

    def acc(op_a=0, op_b=0, lay=0, m=64, n=48, k=32, A=PA, lda=32, B=PB, ldb=48, C=PC, ldc=48,
            D=PD, ldd=48, batch=2, st=BAD, shape=1, ec=1):
        return lib.sgemm_emu_batched_acc(op_a, op_b, lay, m, n, k, P(A), lda, P(B), ldb, P(C),
                                         ldc, P(D), ldd, batch, pkg.Stride4(*st), shape, ec,
                                         P(0))

    assert acc() == -4
    for bad in (dict(op_a=2), dict(op_b=-1), dict(lay=2), dict(shape=2), dict(ec=2)):
        assert acc(**bad) == -8, bad
    assert acc(m=-1) == -1
    assert acc(k=-1) == -1
    assert acc(batch=-1) == -1
    assert acc(lda=31) == -2
    assert acc(op_a=1, lda=32) == -2          # A stored k x m needs lda >= m
    assert acc(op_a=1, lda=64) == -4
    assert acc(ldb=47) == -2
    assert acc(op_b=1, ldb=32) == -4          # B stored n x k: ldb >= k
    assert acc(op_b=1, ldb=31) == -2
    assert acc(ldd=47) == -2
    assert acc(ldc=47) == -2
    assert acc(C=0, ldc=1) == -4              # no C: its ld is not checked
    assert acc(lay=1) == -2                   # stored n x m: ld >= m
    assert acc(lay=1, ldc=64, ldd=64) == -4
    assert acc(m=0) == 0
    assert acc(batch=0) == 0
    assert acc(m=1 << 30, lda=1 << 30) == -6
    assert acc(k=1 << 30, lda=1 << 30) == -6
    assert acc(D=0) == -3
    assert acc(A=0) == -3
    assert acc(B=0) == -3
    assert acc(A=0, B=0, k=0) == -4           # k = 0 reads neither
    ok = (64 * 32, 32 * 48, 64 * 48, 64 * 48)
    assert acc(st=(0, 0, 0, 100)) == -4       # D items overlap
    assert acc(st=(1 << 62, 0, 0, 64 * 48)) == -4  # A's span past the address space
    assert acc(st=(0, 0, 1 << 62, 64 * 48)) == -4
    assert acc(st=(0, 0, 0, 1 << 62)) == -4
    assert acc(st=ok, D=PB + 4) == -5
    assert acc(st=ok, D=PA) == -5
    assert acc(st=ok, D=PC + 8) == -5         # partial overlap with C
    assert acc(st=ok, C=PD, D=PD, ldc=64, ldd=48) == -5


def test_scan_validation():
    lib = pkg.load()
    P = ctypes.c_void_p

    def sc(rows=100, length=200, X=PA, ldx=200, Y=PB, ldy=200):
        return lib.sgemm_emu_scan(rows, length, P(X), ldx, P(Y), ldy, P(0))

    assert sc(rows=-1) == -1
    assert sc(length=-1) == -1
    assert sc(ldx=199) == -2
    assert sc(ldy=0) == -2
    assert sc(rows=0) == 0
    assert sc(length=0) == 0
    # rows x ld past the end of the address space (computed without wrapping)
    assert sc(rows=1 << 40, ldx=1 << 30) == -2
    assert sc(rows=2, ldy=1 << 62) == -2
    assert sc(X=0) == -3
    assert sc(Y=0) == -3
    assert sc(Y=PA + 4) == -5
    assert sc(Y=PA, ldy=256, ldx=200) == -5


def test_split_validation():
    lib = pkg.load()
    P = ctypes.c_void_p
    for form in (pkg.SPLIT_SCALAR, pkg.SPLIT_PAIR, pkg.SPLIT_EIGHT):
        assert lib.sgemm_emu_split(-1, P(PA), P(PB), P(PC), form, P(0)) == -1
        assert lib.sgemm_emu_split(0, P(0), P(0), P(0), form, P(0)) == 0
        assert lib.sgemm_emu_split(16, P(0), P(PB), P(PC), form, P(0)) == -3
        assert lib.sgemm_emu_split(16, P(PA), P(PA + 8), P(PC), form, P(0)) == -5
        assert lib.sgemm_emu_split(1 << 62, P(PA), P(PB), P(PC), form, P(0)) == -1
    assert lib.sgemm_emu_split(16, P(PA), P(PB), P(PC), 3, P(0)) == -8
    assert lib.sgemm_emu_split(16, P(PA), P(PB), P(PC), -1, P(0)) == -8


def test_binding_refuses_values_outside_the_argument_range():
    """ctypes on its own wraps an int argument modulo 2^32 (a leading
    dimension of 2^32 + 8 would reach the library as 8); the binding's
    argument types refuse such values before any call."""
    lib = pkg.load()
    S = pkg.Stride
    for bad in (1 << 31, (1 << 32) + 8, -(1 << 31) - 1):
        with pytest.raises(ctypes.ArgumentError):
            lib.sgemm_emu_batched(4, 4, 4, None, bad, None, 4, None, 4, 1, S(0, 0, 0), None)
        with pytest.raises(ctypes.ArgumentError):
            lib.mfmae_num_elements(bad, 0)
    with pytest.raises(ctypes.ArgumentError):
        lib.sgemm_emu_scan(1 << 63, 4, None, 4, None, 4, None)
    # the edges of the range pass through to the library's own validation
    assert lib.sgemm_emu_batched(4, 4, 4, None, (1 << 31) - 1, None, 4, None, 4, 1, S(0, 0, 0),
                                 None) == -3
    assert lib.sgemm_emu_batched(-(1 << 31), 4, 4, None, 4, None, 4, None, 4, 1, S(0, 0, 0),
                                 None) == -1
    assert lib.sgemm_emu_scan((1 << 63) - 1, 4, None, 4, None, 4, None) != 0
    assert isinstance(lib.mfmae_num_elements(1, 0), int)


def test_strerror_covers_codes():
    for code in range(-8, 1):
        assert "unknown" not in pkg.sgemm_emu_strerror(code)
    assert "unknown" in pkg.sgemm_emu_strerror(-99)


# --------------------------------------------------------------------------
# fragment maps
# --------------------------------------------------------------------------
DIMS = {  # (shape, use) -> (rows, cols, elements per lane)
    (pkg.SHAPE_16x16x32, pkg.USE_A): (16, 32, 8),
    (pkg.SHAPE_16x16x32, pkg.USE_B): (32, 16, 8),
    (pkg.SHAPE_16x16x32, pkg.USE_ACC): (16, 16, 4),
    (pkg.SHAPE_32x32x16, pkg.USE_A): (32, 16, 8),
    (pkg.SHAPE_32x32x16, pkg.USE_B): (16, 32, 8),
    (pkg.SHAPE_32x32x16, pkg.USE_ACC): (32, 32, 16),
}


@pytest.mark.parametrize("shape,use", list(DIMS))
def test_map_is_bijection_and_inverse_of_foreach(shape, use):
    rows, cols, ne = DIMS[(shape, use)]
    assert pkg.mfmae_num_elements(shape, use) == ne
    seen = {}
    for i in range(rows):
        for j in range(cols):
            lane, elem = pkg.mfmae_map(shape, use, i, j)
            assert 0 <= lane < 64 and 0 <= elem < ne
            assert (lane, elem) not in seen
            seen[(lane, elem)] = (i, j)
    assert len(seen) == 64 * ne
    for lane in range(64):
        for elem, (i, j) in enumerate(pkg.mfmae_foreach(shape, use, lane)):
            assert seen[(lane, elem)] == (i, j)


def test_map_structure():
    """Row of A and column of B/C are a function of the lane alone (one
    element per lane per row), and the 8 elements of an A/B lane are 8
    consecutive k; C's 32x32 layout interleaves 4-row groups of the two
    half-waves."""
    for shape, m in ((pkg.SHAPE_16x16x32, 16), (pkg.SHAPE_32x32x16, 32)):
        for lane in range(64):
            a = pkg.mfmae_foreach(shape, pkg.USE_A, lane)
            assert len({i for i, _ in a}) == 1 and a[0][0] == lane % m
            ks = [j for _, j in a]
            assert ks == list(range(ks[0], ks[0] + 8)) and ks[0] % 8 == 0
            b = pkg.mfmae_foreach(shape, pkg.USE_B, lane)
            assert len({j for _, j in b}) == 1 and b[0][1] == lane % m
            assert [i for i, _ in b] == ks  # the same k set as A on this lane
    acc = pkg.mfmae_foreach(pkg.SHAPE_32x32x16, pkg.USE_ACC, 33)
    assert [i for i, _ in acc] == [4, 5, 6, 7, 12, 13, 14, 15, 20, 21, 22, 23, 28, 29, 30, 31]
    assert {j for _, j in acc} == {1}


def test_map_rejects_out_of_range():
    lib = pkg.load()
    lane, elem = ctypes.c_int(), ctypes.c_int()
    assert lib.mfmae_map(0, 0, 16, 0, ctypes.byref(lane), ctypes.byref(elem)) == -1
    assert lib.mfmae_map(1, 0, 0, 16, ctypes.byref(lane), ctypes.byref(elem)) == -1
    assert lib.mfmae_map(2, 0, 0, 0, ctypes.byref(lane), ctypes.byref(elem)) == -6
    assert lib.mfmae_map(0, 3, 0, 0, ctypes.byref(lane), ctypes.byref(elem)) == -6
    assert lib.mfmae_num_elements(0, 5) == -6
    ii = (ctypes.c_int * 16)()
    assert lib.mfmae_foreach(0, 0, 64, ii, ii) == -1


def test_header_constants_match_binding():
    """Every value constant of the C header (policy flows and tiles, operand
    layouts, modes, MFMA shapes and uses) has the same value in the Python
    binding, under the header's name without its prefix; error codes match
    the library's own strerror table."""
    text = pathlib.Path(pkg.__file__).resolve().parents[1].joinpath(
        "include", "sgemm_emu.h").read_text()
    consts = {m.group(1): int(m.group(2)) for m in re.finditer(
        r"^#define\s+((?:SGEMM_EMU|MFMAE)_\w+)\s+\(?(-?\d+)\)?", text, flags=re.M)}
    assert len(consts) >= 30
    for name, value in consts.items():
        short = re.sub(r"^(SGEMM_EMU|MFMAE)_", "", name)
        if short == "OK" or short.startswith("ERR_"):
            assert value <= 0
            continue
        assert getattr(pkg, short) == value, name
    codes = sorted(v for k, v in consts.items() if k.startswith("SGEMM_EMU_ERR_"))
    assert codes == list(range(-8, 0))
    for code in codes:
        assert "unknown" not in pkg.sgemm_emu_strerror(code)


def test_mfma_probe_validation():
    lib = pkg.load()
    P = ctypes.c_void_p
    a, b, c = P(1 << 40), P(2 << 40), P(3 << 40)

    def mp(m=256, n=512, k=64, A=a, lda=64, B=b, ldb=512, C=c, ldc=512):
        return lib.sgemm_emu_mfma_probe(m, n, k, A, lda, B, ldb, C, ldc, P(0))

    assert mp(m=-128) == -1 and mp(k=-32) == -1
    assert mp(m=0, A=P(0), B=P(0), C=P(0)) == 0 and mp(n=0) == 0
    for bad in (dict(m=200), dict(n=384), dict(k=48), dict(k=0)):
        assert mp(**bad) == -6, bad
    assert mp(lda=31) == -2 and mp(ldb=511) == -2 and mp(ldc=500) == -2
    assert mp(A=P(0)) == -3 and mp(C=P(0)) == -3
    assert mp(C=P((1 << 40) + 1024)) == -5      # C over A's rows
    assert mp(m=1 << 30, n=1 << 30) == -1       # more tiles than one launch counts


def test_stream_probe_validation():
    lib = pkg.load()
    P = ctypes.c_void_p
    n = 1 << 14
    far = [P(1 << 40), P(2 << 40), P(3 << 40)]
    assert lib.sgemm_emu_stream_probe(-1, n, *far, 256, P(0)) == -1
    assert lib.sgemm_emu_stream_probe(4, -4, *far, 256, P(0)) == -1
    assert lib.sgemm_emu_stream_probe(0, n, P(0), P(0), P(0), 256, P(0)) == 0
    assert lib.sgemm_emu_stream_probe(4, n, P(0), far[1], far[2], 256, P(0)) == -3
    for threads in (0, 128, 2048):
        assert lib.sgemm_emu_stream_probe(4, n, *far, threads, P(0)) == -6
    assert lib.sgemm_emu_stream_probe(4, 6, *far, 256, P(0)) == -6          # not whole vectors
    assert lib.sgemm_emu_stream_probe(4, 1 << 31, *far, 256, P(0)) == -6    # item too long
    assert lib.sgemm_emu_stream_probe(4, n, P((1 << 40) + 4), far[1], far[2], 256, P(0)) == -6
    assert lib.sgemm_emu_stream_probe(1 << 40, 1 << 30, *far, 256, P(0)) == -1  # span wraps
    # C overlapping A
    assert lib.sgemm_emu_stream_probe(4, n, far[0], far[1], P((1 << 40) + 4 * n), 256,
                                      P(0)) == -5
