"""Parity of the batched emulated SGEMM (Sec. 4.4) against the oracle, through
the C ABI on the GPU.

* every policy (split flow, direct flow, staged flow, register-direct flow;
  error correction on and off; every tile) on shapes that span several
  tiles and ragged tails, and every k-loop path of the register-direct
  flow;
* edge cases: k = 0, empty problems, a single element, broadcast operands
  (zero batch stride), padded leading dimensions, leading dimensions at and
  just past the full-tile kernel's offset limit, unaligned pointers (the
  scalar-load path);
* exactness on integer inputs in binary16 range;
* the error-correction-off control must be visibly worse (the correction
  terms are live);
* determinism (no atomics, no split-k);
* the full-size workloads in the launch configuration the benchmark times:
  every output written (NaN beforehand, finite after) and 4096 or more
  outputs spread over every item held to the parity bar.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
import synth
from gpu_util import (assert_periodic, device, gate, gate_applies, gate_repeated, gemm_sampled,
                      nan_output, periodic_batch, to_np)

pytestmark = pytest.mark.gpu

POLICIES = [
    pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_64x64),
    pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_128x128),
    pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_256x128),
    pkg.Policy(pkg.FLOW_DIRECT, 1, pkg.TILE_64x64),
    pkg.Policy(pkg.FLOW_DIRECT, 1, pkg.TILE_128x128),
    pkg.Policy(pkg.FLOW_DIRECT, 1, pkg.TILE_256x128),
    pkg.Policy(pkg.FLOW_STAGED, 1, pkg.TILE_64x64),
    pkg.Policy(pkg.FLOW_STAGED, 1, pkg.TILE_128x128),
    pkg.Policy(pkg.FLOW_REG, 1, pkg.TILE_64x64),
    pkg.Policy(pkg.FLOW_REG, 1, pkg.TILE_128x128),
]


def _pid(p):
    return f"flow{p.flow}-ec{p.ec}-tile{p.tile}"


def _reg_supported(policy, k, n):
    """The register-direct flow needs 16-byte A rows (k a multiple of 4 for a
    packed operand) and, for its 64-wide waves, column pairs (n even)."""
    if policy is None or policy.flow != pkg.FLOW_REG:
        return True
    return k % 4 == 0 and (policy.tile == pkg.TILE_64x64 or n % 2 == 0)


def _run(A, B, policy=None, C=None):
    dev = device()
    Ad = A.to(dev) if A.device.type == "cpu" else A
    Bd = B.to(dev) if B.device.type == "cpu" else B
    return to_np(pkg.sgemm_emu_batched(Ad, Bd, C, policy=policy))


SHAPES = [  # batch, m, n, k
    (2, 64, 64, 64),
    (3, 130, 77, 65),
    (1, 257, 129, 96),
    (2, 17, 33, 300),
    (1, 1, 1, 1),
    (2, 3, 5, 7),
    (1, 300, 260, 33),
]


@pytest.mark.parametrize("policy", POLICIES, ids=_pid)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_policies_ragged_shapes(policy, shape):
    batch, m, n, k = shape
    print(f"case policy={_pid(policy)} shape={shape}", flush=True)
    A, B = synth.gemm_inputs(batch, m, n, k, seed=11 + m + n + k)
    if not _reg_supported(policy, k, n):
        with pytest.raises(pkg.SgemmEmuError) as ei:
            _run(A, B, policy)
        assert ei.value.code == -8
        return
    C = _run(A, B, policy)
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(C, ref, k, f"{_pid(policy)} {shape}", max_gate=gate_applies(ref))


# Shapes for the register-direct flow: every k-loop path of its register
# ring (k < 16 D, exactly D steps, steady state, 1 .. D - 1 extra steps, a
# partial last step), ragged m and n, a wave tile entirely outside C.
REG_SHAPES = [  # batch, m, n, k
    (2, 64, 64, 64),
    (3, 130, 66, 100),
    (1, 257, 130, 208),
    (2, 17, 34, 300),
    (1, 70, 96, 36),
    (2, 33, 64, 4),
    (1, 96, 128, 112),
    (2, 128, 128, 80),
    (1, 192, 256, 192),
    (2, 40, 200, 48),
    (1, 160, 98, 144),
]


@pytest.mark.parametrize("tile", [pkg.TILE_64x64, pkg.TILE_128x128])
@pytest.mark.parametrize("shape", REG_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_register_direct_flow_shapes(tile, shape):
    batch, m, n, k = shape
    policy = pkg.Policy(pkg.FLOW_REG, 1, tile)
    print(f"case policy={_pid(policy)} shape={shape}", flush=True)
    A, B = synth.gemm_inputs(batch, m, n, k, seed=31 + m + n + k)
    C = _run(A, B, policy)
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(C, ref, k, f"{_pid(policy)} {shape}", max_gate=gate_applies(ref))


# Shapes for the pipelined full-tile kernels (split flow): per tile, one,
# two, three and five k chunks (every path of the two-stage loop), several
# tiles and items, padded leading dimensions.
BIG_SHAPES = {  # tile: [(batch, m, n, k, pad)]
    2: [(1, 128, 128, 32, 0), (2, 256, 256, 64, 0), (1, 384, 128, 96, 4),
        (3, 128, 256, 160, 8)],
    3: [(1, 256, 128, 32, 0), (2, 256, 256, 64, 0), (1, 512, 384, 96, 0),
        (3, 256, 128, 160, 4), (1, 768, 256, 320, 8)],
    4: [(1, 128, 256, 32, 0), (2, 256, 512, 64, 0), (1, 384, 256, 96, 4),
        (2, 128, 256, 160, 8)],
}
# the 128 x 128 tile also runs the paper's direct and staged data flows
BIG_CASES = [(f, t, sh) for t, shapes in BIG_SHAPES.items()
             for f in ([pkg.FLOW_SPLIT, pkg.FLOW_DIRECT, pkg.FLOW_STAGED] if t == 2
                       else [pkg.FLOW_SPLIT])
             for sh in shapes]


@pytest.mark.parametrize("flow,tile,shape", BIG_CASES,
                         ids=lambda v: str(v) if isinstance(v, int) else "x".join(map(str, v)))
def test_full_tile_kernel_shapes(flow, tile, shape):
    batch, m, n, k, pad = shape
    dev = device()
    policy = pkg.Policy(flow, 1, tile)
    print(f"case full-tile flow={flow} tile={tile} shape={shape}", flush=True)
    A, B = synth.gemm_inputs(batch, m, n, k, seed=51 + m + n + k)
    Ab = torch.zeros((batch, m, k + pad), device=dev)
    Bb = torch.zeros((batch, k, n + pad), device=dev)
    Ab[:, :, :k] = A.to(dev)
    Bb[:, :, :n] = B.to(dev)
    Ad, Bd = Ab[:, :, :k], Bb[:, :, :n]
    Cd = torch.empty((batch, m, n), device=dev)
    _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, Cd, policy=policy)
    assert kern in ("bgemm_big_kernel", "bgemm_big_stream_kernel")
    pkg.sgemm_emu_batched(Ad, Bd, Cd, policy=policy)
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(to_np(Cd), ref, k, f"full-tile {tile} {shape}")


@pytest.mark.parametrize("shape", [(2048, 4096, 64), (4096, 4096, 32), (2048, 8192, 32)],
                         ids=lambda s: "x".join(map(str, s)))
def test_full_tile_kernel_in_device_blocks(shape):
    """One product on the 128 x 256 tile whose tile grid is a multiple of
    16 x 16: the kernel takes its tiles in device-wide 16 x 16 blocks (one,
    two and four blocks here, down the columns and across). Every output,
    prefilled with NaN, against the oracle."""
    m, n, k = shape
    dev = device()
    policy = pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_128x256)
    print(f"case device blocks {shape}", flush=True)
    A, B = synth.gemm_inputs(1, m, n, k, seed=71 + m // 1024 + n // 1024)
    Ad, Bd = A.to(dev), B.to(dev)
    Cd = torch.full((1, m, n), float("nan"), device=dev)
    _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, Cd, policy=policy)
    assert kern == "bgemm_big_kernel"
    pkg.sgemm_emu_batched(Ad, Bd, Cd, policy=policy)
    C = to_np(Cd)
    assert np.isfinite(C).all()
    gate(C, oracle.gemm(A.numpy(), B.numpy()), k, f"device blocks {shape}")


LIMIT_CASES = [(pkg.FLOW_SPLIT, pkg.TILE_128x128, 128, 128),
               (pkg.FLOW_SPLIT, pkg.TILE_256x128, 256, 128),
               (pkg.FLOW_SPLIT, pkg.TILE_128x256, 128, 256),
               (pkg.FLOW_DIRECT, pkg.TILE_128x128, 128, 128),
               (pkg.FLOW_STAGED, pkg.TILE_128x128, 128, 128)]


@pytest.mark.parametrize("flow,tile,bm,bn", LIMIT_CASES,
                         ids=["split-128x128", "split-256x128", "split-128x256", "direct-128x128",
                              "staged-128x128"])
def test_full_tile_kernel_at_its_offset_limit(flow, tile, bm, bn):
    """The largest leading dimensions the full-tile kernel takes (a chunk's
    byte offsets just below 2^31: A rows about 2^29 / bm floats apart, B rows
    about 2^24; operands of 2-4 GB) and one step past that on A and on B,
    where the general kernel takes over: all three agree with the oracle.
    Two chunks, so that the chunk descriptors move along A and B too."""
    dev = device()
    m, n, k = bm, bn, 64

    def lda_max(rows):  # largest multiple of 4 with (rows lda + 32) 4 < 2^31
        return ((2**29 - 32 - 1) // rows) // 4 * 4

    def ldb_max(cols):  # largest multiple of 4 with (32 ldb + cols) 4 < 2^31
        return ((2**29 - cols - 1) // 32) // 4 * 4

    A, B = synth.gemm_inputs(1, m, n, k, seed=71 + bm + bn + flow)
    ref = oracle.gemm(A.numpy(), B.numpy())
    policy = pkg.Policy(flow, 1, tile)
    # the general kernel has no 128 x 256 tile: past the limit that case
    # names 128 x 128, whose limit on ldb is higher
    past_policy, past_bn = policy, bn
    if tile == pkg.TILE_128x256:
        past_policy, past_bn = pkg.Policy(flow, 1, pkg.TILE_128x128), 128
    for lda, ldb, pol, full in [(lda_max(bm), ldb_max(bn), policy, True),
                                (lda_max(bm) + 4, n, past_policy, False),
                                (k, ldb_max(past_bn) + 4, past_policy, False)]:
        print(f"case offset limit flow={flow} tile={tile} lda={lda} ldb={ldb}", flush=True)
        Ab = torch.empty((1, m, lda), device=dev)
        Bb = torch.empty((1, k, ldb), device=dev)
        Ab[:, :, :k] = A.to(dev)
        Bb[:, :, :n] = B.to(dev)
        Ad, Bd = Ab[:, :, :k], Bb[:, :, :n]
        Cd = nan_output((1, m, n))
        _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, Cd, policy=pol)
        if full:
            assert kern in ("bgemm_big_kernel", "bgemm_big_stream_kernel"), kern
        else:
            assert kern == "bgemm_emu_kernel", kern
        pkg.sgemm_emu_batched(Ad, Bd, Cd, policy=pol)
        gate(to_np(Cd), ref, k, f"offset limit {tile} lda={lda} ldb={ldb}")
        del Ab, Bb, Ad, Bd, Cd
        torch.cuda.empty_cache()


@pytest.mark.parametrize("batch,k", [(600, 96), (513, 32), (300, 160)])
def test_full_tile_stream_many_tasks(batch, k):
    """More 256 x 128 tiles than workgroups on the GPU: the persistent form
    walks several tasks per workgroup as one stream of k chunks (odd and
    even chunk counts, one chunk per task); sampled items are compared."""
    m, n = 256, 128
    policy = pkg.Policy(pkg.FLOW_SPLIT, 1, pkg.TILE_256x128)
    print(f"case full-tile stream batch={batch} k={k}", flush=True)
    A, B = synth.gemm_inputs(batch, m, n, k, seed=61 + batch + k)
    C = _run(A, B, policy)
    items = sorted(set([0, 1, batch // 2, batch - 2, batch - 1] + list(range(3, batch, 37))))
    ref = oracle.gemm(A[items].numpy(), B[items].numpy())
    gate(C[items], ref, k, f"stream batch={batch} k={k}")


@pytest.mark.parametrize("tile", [2, 3, 4])
def test_full_tile_kernel_integer_exact(tile):
    g = synth.rng(9)
    A = synth.integer_matrix((2, 256, 96), g, -8, 8)
    B = synth.integer_matrix((2, 96, 256), g, -8, 8)
    C = _run(A, B, pkg.Policy(pkg.FLOW_SPLIT, 1, tile))
    ref = np.einsum("bik,bkj->bij", A.numpy().astype(np.int64), B.numpy().astype(np.int64))
    assert np.array_equal(C, ref.astype(np.float32))


def test_register_direct_flow_b_pairs():
    """B 8-byte but not 16-byte aligned: the 128x128 tile falls back from
    4-wide to 2-wide B loads (waves of 64 x 64)."""
    dev = device()
    A, B = synth.gemm_inputs(2, 96, 132, 72, seed=43)
    flat = torch.zeros(B.numel() + 2, device=dev)
    flat[2:] = B.reshape(-1).to(dev)
    Bd = flat[2:].view(2, 72, 132)
    C = to_np(pkg.sgemm_emu_batched(A.to(dev), Bd, policy=pkg.Policy(pkg.FLOW_REG, 1,
                                                                      pkg.TILE_128x128)))
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(C, ref, 72, "reg B pairs")


def test_register_direct_flow_odd_columns_32_wide():
    """32x32 waves load single columns, so an odd n is fine there."""
    policy = pkg.Policy(pkg.FLOW_REG, 1, pkg.TILE_64x64)
    A, B = synth.gemm_inputs(2, 75, 77, 68, seed=41)
    C = _run(A, B, policy)
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(C, ref, 68, "reg odd n")


@pytest.mark.parametrize("policy", POLICIES, ids=_pid)
def test_integer_inputs_exact(policy):
    g = synth.rng(7)
    A = synth.integer_matrix((2, 96, 160), g, -8, 8)
    B = synth.integer_matrix((2, 160, 72), g, -8, 8)
    C = _run(A, B, policy)
    ref = np.einsum("bik,bkj->bij", A.numpy().astype(np.int64), B.numpy().astype(np.int64))
    assert np.array_equal(C, ref.astype(np.float32))


@pytest.mark.parametrize("flow", [pkg.FLOW_SPLIT, pkg.FLOW_DIRECT, pkg.FLOW_STAGED, pkg.FLOW_REG])
def test_error_correction_is_live(flow):
    """Without the two correction products the error is at the fp16 level
    (about 2^-11 relative); with them it is at the FP32 level."""
    A, B = synth.gemm_inputs(2, 128, 128, 128, seed=3)
    ref = oracle.gemm(A.numpy(), B.numpy(), want=("c64", "n64", "c32"))
    on = _run(A, B, pkg.Policy(flow, 1, pkg.TILE_128x128))
    off = _run(A, B, pkg.Policy(flow, 0, pkg.TILE_128x128))
    e_on = oracle.max_rel_err(on, ref["c64"], ref["n64"])
    e_off = oracle.max_rel_err(off, ref["c64"], ref["n64"])
    print(f"flow {flow}: ec on {e_on:.3e}, ec off {e_off:.3e}")
    assert e_off > 2.0 ** -16
    assert e_on < 2.0 ** -20
    # ec off computes exactly the product of the hi parts
    hiA = A.numpy().astype(np.float16).astype(np.float64)
    hiB = B.numpy().astype(np.float16).astype(np.float64)
    hh = np.einsum("bik,bkj->bij", hiA, hiB)
    assert np.all(np.abs(off - hh) <= 130 * 2.0 ** -23 * ref["n64"])


def test_k_zero_stores_zeros():
    dev = device()
    A = torch.zeros((2, 8, 0), device=dev)
    B = torch.zeros((2, 0, 5), device=dev)
    C = torch.full((2, 8, 5), 7.0, device=dev)
    pkg.sgemm_emu_batched(A, B, C)
    assert np.all(to_np(C) == 0)


def test_empty_batch_and_rows_leave_output_untouched():
    """m = 0 and batch = 0 are no-ops: the output buffer they point into is
    not written."""
    dev = device()
    C = torch.full((2, 4, 4), 3.0, device=dev)
    A = torch.ones((2, 4, 4), device=dev)
    B = torch.ones((2, 4, 4), device=dev)
    pkg.sgemm_emu_batched(A[:, :0, :], B, C[:, :0, :])
    pkg.sgemm_emu_batched(A[:0], B[:0], C[:0])
    assert np.all(to_np(C) == 3.0)


def test_broadcast_operand():
    """A 2-D B is shared by every item (batch stride 0)."""
    A, B = synth.gemm_inputs(4, 70, 90, 50, seed=21)
    B0 = B[0]
    C = _run(A, B0)
    ref = oracle.gemm(A.numpy(), np.broadcast_to(B0.numpy(), (4, 50, 90)))
    gate(C, ref, 50, "broadcast B")


def test_padded_leading_dimensions_and_strides():
    """Operands that are views into larger buffers: lda > k, ldb > n,
    ldc > n and batch strides larger than the matrices."""
    dev = device()
    A_big, B_big = synth.gemm_inputs(3, 100, 140, 120, seed=23)
    A = A_big[:, :90, :70].to(dev)
    B = B_big[:, :70, :110].to(dev)
    C_big = torch.full((3, 96, 128), -5.0, device=dev)
    C = C_big[:, :90, :110]
    pkg.sgemm_emu_batched(A, B, C)
    out = to_np(C_big)
    ref = oracle.gemm(A.cpu().numpy(), B.cpu().numpy())
    gate(out[:, :90, :110], ref, 70, "padded")
    assert np.all(out[:, 90:, :] == -5.0) and np.all(out[:, :, 110:] == -5.0)


def test_unaligned_pointers_take_scalar_path():
    dev = device()
    A, B = synth.gemm_inputs(2, 65, 66, 67, seed=25)
    flatA = torch.zeros(A.numel() + 1, device=dev)
    flatB = torch.zeros(B.numel() + 3, device=dev)
    flatA[1:] = A.reshape(-1).to(dev)
    flatB[3:] = B.reshape(-1).to(dev)
    Ad = flatA[1:].view(2, 65, 67)
    Bd = flatB[3:].view(2, 67, 66)
    C = to_np(pkg.sgemm_emu_batched(Ad, Bd))
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(C, ref, 67, "unaligned")


def test_deterministic():
    A, B = synth.gemm_inputs(8, 128, 128, 128, seed=27)
    c1 = _run(A, B)
    c2 = _run(A, B)
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


# ---------------------------------------------------------------------------
# Full-size workloads, in the configuration the benchmark times (automatic
# policy): the output starts as NaN and must be finite everywhere after the
# call; the values are compared with the oracle on samples spread over every
# item (4096 or more).
# ---------------------------------------------------------------------------

def _full_gemm_sampled(name, count=8192, max_gate=True):
    w = synth.WORKLOADS[name]
    print(f"case workload={name} batch={w.batch} m={w.m} n={w.n} k={w.k}", flush=True)
    A, B = synth.workload_inputs(w)
    dev = device()
    Ad, Bd = A.to(dev), B.to(dev)
    C = nan_output((w.batch, w.m, w.n))
    _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, C)
    pkg.sgemm_emu_batched(Ad, Bd, C)
    e = gemm_sampled(C, A, B, count, seed=w.seed, label=f"{name} [{kern}]", max_gate=max_gate)
    print(f"{name} [{kern}]: err {e[0]:.3e} fp32 {e[1]:.3e}")
    return e


def test_workload_gemm_64_full():
    w = synth.WORKLOADS["gemm_64"]
    A, B = synth.workload_inputs(w)
    C = _run(A, B)
    assert np.isfinite(C).all()
    gate(C, oracle.gemm(A.numpy(), B.numpy()), w.k, "gemm_64")


def test_workload_gemm_128_sampled():
    _full_gemm_sampled("gemm_128", count=16384)


def test_workload_gemm_256e_sampled():
    _full_gemm_sampled("gemm_256e", count=8192)


def test_workload_gemm_8192_sampled():
    _full_gemm_sampled("gemm_8192", count=8192)


@pytest.mark.parametrize("k", [128, 256, 4096])
def test_workload_paper_sweep_sampled(k):
    """The batched experiment of Sec. 4.4.2 (256 products of 1024 x k .
    k x 1024) at the sweep's ends and at k = 256, in the configuration the
    sweep times: k = 128 and 256 run the 256 x 128 tile in its persistent
    form, k = 4096 the 128 x 256 tile."""
    _full_gemm_sampled(f"paper_k{k}", count=8192)
    torch.cuda.empty_cache()


# Large ragged products: interior of whole tiles on the full-tile kernel, a
# k tail added in place, edge strips on the register-flow kernel.
TILED_SHAPES = [(1, 4100, 4300, 2060),   # 128 x 256 interior, k tail of 12, both strips
                (2, 2600, 2600, 2560),   # whole k chunks, batch of 2
                (1, 6000, 6000, 960),    # 256 x 128 interior
                (1, 4096, 4200, 2048),   # right strip only
                (1, 4200, 4096, 2048)]   # bottom strip only
# Ragged products on the register-direct flow (below 2^35 multiply-adds or
# without a nearly full interior): many tiles and long k; n odd takes the
# 64 x 64 tiles.
REG_SHAPES = [(1, 2100, 2300, 1000), (2, 1500, 1800, 1024), (3, 1200, 1300, 1000),
              (1, 3300, 3500, 3000), (1, 1100, 1101, 512)]


def _seams(m, n, bm, bn, seed):
    mi, ni = m - m % bm, n - n % bn
    g = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, bm - 1, bm, mi - 1, min(mi, m - 1), m - 1],
                                     g.integers(0, m, 10)]))
    cols = np.unique(np.concatenate([[0, bn - 1, bn, ni - 1, min(ni, n - 1), n - 1],
                                     g.integers(0, n, 10)]))
    rr, cc = np.meshgrid(rows, cols, indexing="ij")
    return rr.ravel(), cc.ravel()


def _check_sampled(shape, expect_kernel, label):
    batch, m, n, k = shape
    print(f"case {label} {shape}", flush=True)
    dev = device()
    A, B = synth.gemm_inputs(batch, m, n, k, seed=71 + m + k)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.full((batch, m, n), float("nan"), device=dev)
    pol, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, C)
    assert kern == expect_kernel, kern
    pkg.sgemm_emu_batched(Ad, Bd, C)
    bm = 256 if pol.tile == pkg.TILE_256x128 else 64 if pol.tile == pkg.TILE_64x64 else 128
    bn = 256 if pol.tile == pkg.TILE_128x256 else 64 if pol.tile == pkg.TILE_64x64 else 128
    rr, cc = _seams(m, n, bm, bn, m + n + k)
    for b in range(batch):
        Cb = C[b].cpu().numpy()
        assert np.isfinite(Cb).all()
        An, Bn = A[b].numpy(), B[b].numpy()
        ref = oracle.dots(An[rr], np.ascontiguousarray(Bn[:, cc].T))
        gate(Cb[rr, cc], ref, k, f"{label} {shape} item {b}")


@pytest.mark.parametrize("shape", TILED_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_tiled_ragged_large(shape):
    _check_sampled(shape, "bgemm_big_kernel+bgemm_reg_kernel", "tiled")


@pytest.mark.parametrize("shape", REG_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_register_flow_ragged_large(shape):
    _check_sampled(shape, "bgemm_reg_kernel", "register flow")


def test_register_flow_batch_past_one_launch():
    """A batch of small products larger than one launch holds: the 64 x 64
    register-flow tile is one 256-thread workgroup per item, so a launch
    takes at most 2^31 / 256 - 1 = 8,388,607 items and this batch needs two.
    A pool of P items (k with a tail after two full steps) is checked against
    the oracle and repeated across the batch; every item must equal its pool
    item bitwise."""
    P, m, n, k = 1021, 2, 3, 36
    per_launch = (1 << 31) // 256 - 1
    batch = per_launch + 2 * P + 7
    print(f"case register flow batch={batch} m={m} n={n} k={k}", flush=True)
    dev = device()
    A, B = synth.gemm_inputs(P, m, n, k, seed=97)
    Ad = periodic_batch(A.to(dev), batch)
    Bd = periodic_batch(B.to(dev), batch)
    C = torch.full((batch, m, n), float("nan"), device=dev)
    pol, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, C)
    assert kern == "bgemm_reg_kernel" and pol.tile == pkg.TILE_64x64, (pol, kern)
    pkg.sgemm_emu_batched(Ad, Bd, C)
    ref = oracle.gemm(A.numpy(), B.numpy())
    gate(to_np(C[:P]), ref, k, "register flow pool")
    gate_repeated(C, ref, P, [per_launch - 1, per_launch, per_launch + 1, batch - 1], k,
                  "register flow, launch boundary")
    assert_periodic(C, P, "register flow batch")


@pytest.mark.parametrize("tile", [pkg.TILE_128x128, pkg.TILE_128x256])
def test_full_tile_kernel_without_error_correction(tile):
    """The full-tile kernel with error correction off (the measurement
    variant of the hi.hi product alone) runs on both of its tiles: its result
    is the product of the operands' hi parts up to FP32 accumulation, and its
    error against the FP64 product is at the fp16 level."""
    A, B = synth.gemm_inputs(2, 256, 512, 192, seed=23)
    dev = device()
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.full((2, 256, 512), float("nan"), device=dev)
    pol = pkg.Policy(pkg.FLOW_SPLIT, 0, tile)
    _, kern = pkg.sgemm_emu_resolve_policy(Ad, Bd, C, policy=pol)
    assert kern == "bgemm_big_kernel"
    pkg.sgemm_emu_batched(Ad, Bd, C, policy=pol)
    off = to_np(C)
    ref = oracle.gemm(A.numpy(), B.numpy(), want=("c64", "n64"))
    hiA = A.numpy().astype(np.float16).astype(np.float64)
    hiB = B.numpy().astype(np.float16).astype(np.float64)
    hh = np.einsum("bik,bkj->bij", hiA, hiB)
    assert np.all(np.abs(off - hh) <= (192 + 2) * 2.0 ** -23 * ref["n64"])
    assert oracle.max_rel_err(off, ref["c64"], ref["n64"]) > 2.0 ** -16


def _random_shapes(n, seed):
    g = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        out.append((int(g.integers(1, 4)), int(g.integers(1, 300)), int(g.integers(1, 300)),
                    int(g.integers(1, 400))))
    return out


RANDOM_SHAPES = _random_shapes(12, 2024)


@pytest.mark.parametrize("shape", RANDOM_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_random_shapes_every_policy(shape):
    """Seeded random ragged shapes (batch 1-3, m and n 1-299, k 1-399) on the
    automatic policy and every explicit policy that accepts them."""
    batch, m, n, k = shape
    print(f"case random {shape}", flush=True)
    A, B = synth.gemm_inputs(batch, m, n, k, seed=7 * m + 3 * n + k)
    ref = oracle.gemm(A.numpy(), B.numpy())
    for policy in [None] + POLICIES:
        if not _reg_supported(policy, k, n):
            continue
        if policy is not None and policy.tile == pkg.TILE_128x256:
            continue
        C = _run(A, B, policy)
        gate(C, ref, k, f"{shape} {_pid(policy) if policy else 'auto'}",
             max_gate=gate_applies(ref))
