"""Parity of D = op(A).op(B) + C computed by the kernel written with the
fragment interface (mfmae/wmma_tcec.hpp: load_matrix_sync, mma_sync,
store_matrix_sync; Sec. 2.3.1 and Sec. 4.4), against the accumulate-form
oracle:

* every combination of instruction shape, operand transposes and C/D
  layout, on ragged sizes (partial tiles in m, n and k) and on full tiles
  (the 16-byte access path);
* in-place accumulation (C is D), no C, k = 0, broadcast operands and
  unaligned bases (the element-wise path);
* integer inputs give the exact result;
* the error-correction policy: off computes the hi.hi product (plus C) and
  is at the fp16 error level, on is at the FP32 level.

The bar is that of the GEMM tests (gpu_util.gate) with k the depth of the
product; C enters the normaliser as |C|.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
import synth
from gpu_util import (assert_all_finite, assert_periodic, device, gate, gate_applies,
                      gate_repeated, nan_output, periodic_batch, spread_items, to_np)

pytestmark = pytest.mark.gpu

SHAPES = {"s16": pkg.SHAPE_16x16x32, "s32": pkg.SHAPE_32x32x16}


def _store(X, op):
    """Stored form of X ([batch, r, c]): itself or its transpose."""
    return X if op == pkg.OP_N else X.transpose(1, 2).contiguous()


def _run(A, B, C, op_a, op_b, layout, shape, ec=1, inplace=False, offset=0):
    """Run with operands in stored form built from the logical A (m x k),
    B (k x n), C (m x n); returns D in logical (m x n) form."""
    dev = device()
    As = _store(A, op_a).to(dev)
    Bs = _store(B, op_b).to(dev)
    Cs = None if C is None else _store(C, pkg.OP_T if layout == pkg.COL_MAJOR else pkg.OP_N)
    if offset:
        # unaligned bases: views one element into a larger buffer
        def shift(t):
            flat = torch.zeros(t.numel() + offset, device=dev)
            flat[offset:] = t.reshape(-1).to(dev)
            return flat[offset:].view(t.shape)
        As, Bs = shift(As), shift(Bs)
        if Cs is not None:
            Cs = shift(Cs)
    elif Cs is not None:
        Cs = Cs.to(dev)
    if inplace:
        D = pkg.sgemm_emu_batched_acc(As, Bs, Cs, Cs, op_a=op_a, op_b=op_b, layout=layout,
                                      shape=shape, ec=ec)
    else:
        D = pkg.sgemm_emu_batched_acc(As, Bs, Cs, op_a=op_a, op_b=op_b, layout=layout,
                                      shape=shape, ec=ec)
    D = to_np(D)
    return D.transpose(0, 2, 1) if layout == pkg.COL_MAJOR else D


def _draw(batch, m, n, k, seed):
    g = synth.rng(seed)
    return (synth.uniform((batch, m, k), g), synth.uniform((batch, k, n), g),
            synth.uniform((batch, m, n), g))


COMBOS = [(s, oa, ob, lay) for s in SHAPES for oa in (pkg.OP_N, pkg.OP_T)
          for ob in (pkg.OP_N, pkg.OP_T) for lay in (pkg.ROW_MAJOR, pkg.COL_MAJOR)]


def _cid(c):
    s, oa, ob, lay = c
    return f"{s}-{'NT'[oa]}{'NT'[ob]}-{'rc'[lay]}"


@pytest.mark.parametrize("combo", COMBOS, ids=_cid)
def test_ragged_all_layouts(combo):
    s, oa, ob, lay = combo
    print(f"case acc ragged {_cid(combo)}", flush=True)
    A, B, C = _draw(3, 75, 77, 68, seed=81)
    D = _run(A, B, C, oa, ob, lay, SHAPES[s])
    ref = oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy())
    gate(D, ref, 68, f"acc ragged {_cid(combo)}")


@pytest.mark.parametrize("combo", COMBOS, ids=_cid)
def test_full_tiles_all_layouts(combo):
    s, oa, ob, lay = combo
    print(f"case acc full {_cid(combo)}", flush=True)
    A, B, C = _draw(4, 128, 64, 96, seed=82)
    D = _run(A, B, C, oa, ob, lay, SHAPES[s])
    ref = oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy())
    gate(D, ref, 96, f"acc full {_cid(combo)}")


@pytest.mark.parametrize("s", list(SHAPES))
def test_in_place_and_no_c(s):
    A, B, C = _draw(2, 64, 96, 80, seed=83)
    D = _run(A, B, C, pkg.OP_N, pkg.OP_N, pkg.ROW_MAJOR, SHAPES[s], inplace=True)
    gate(D, oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy()), 80, "acc in place")
    D0 = _run(A, B, None, pkg.OP_T, pkg.OP_N, pkg.ROW_MAJOR, SHAPES[s])
    gate(D0, oracle.gemm(A.numpy(), B.numpy()), 80, "acc no C")


def test_k_zero_copies_c():
    dev = device()
    C = synth.uniform((2, 33, 20), synth.rng(84)).to(dev)
    A = torch.zeros((2, 33, 0), device=dev)
    B = torch.zeros((2, 0, 20), device=dev)
    D = to_np(pkg.sgemm_emu_batched_acc(A, B, C))
    assert np.array_equal(D, to_np(C))
    D0 = to_np(pkg.sgemm_emu_batched_acc(A, B, None))
    assert np.all(D0 == 0)


@pytest.mark.parametrize("offset", [1, 2])
def test_unaligned_bases(offset):
    A, B, C = _draw(2, 64, 64, 64, seed=85)
    for lay in (pkg.ROW_MAJOR, pkg.COL_MAJOR):
        D = _run(A, B, C, pkg.OP_N, pkg.OP_T, lay, pkg.SHAPE_32x32x16, offset=offset)
        gate(D, oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy()), 64, f"acc offset {offset}")


def test_broadcast_b():
    dev = device()
    A, B, C = _draw(3, 40, 50, 36, seed=86)
    B0 = B[:1].expand(3, -1, -1).contiguous()
    D = to_np(pkg.sgemm_emu_batched_acc(A.to(dev), B[0].to(dev), C.to(dev)))
    gate(D, oracle.gemm_acc(A.numpy(), B0.numpy(), C.numpy()), 36, "acc broadcast B")


@pytest.mark.parametrize("combo", [c for c in COMBOS if c[3] == pkg.ROW_MAJOR], ids=_cid)
def test_integer_exact(combo):
    s, oa, ob, lay = combo
    g = synth.rng(87)
    A = synth.integer_matrix((2, 70, 90), g, -8, 8)
    B = synth.integer_matrix((2, 90, 40), g, -8, 8)
    C = synth.integer_matrix((2, 70, 40), g, -1000, 1000)
    D = _run(A, B, C, oa, ob, lay, SHAPES[s])
    exact = (np.einsum("bik,bkj->bij", A.numpy().astype(np.int64), B.numpy().astype(np.int64))
             + C.numpy().astype(np.int64))
    assert np.array_equal(D, exact.astype(np.float32))


@pytest.mark.parametrize("s", list(SHAPES))
def test_error_correction_policy(s):
    A, B, C = _draw(2, 96, 96, 128, seed=88)
    ref = oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy(), want=("c64", "n64", "c32"))
    on = _run(A, B, C, pkg.OP_N, pkg.OP_N, pkg.ROW_MAJOR, SHAPES[s], ec=1)
    off = _run(A, B, C, pkg.OP_N, pkg.OP_N, pkg.ROW_MAJOR, SHAPES[s], ec=0)
    e_on = oracle.max_rel_err(on, ref["c64"], ref["n64"])
    e_off = oracle.max_rel_err(off, ref["c64"], ref["n64"])
    print(f"acc {s}: ec on {e_on:.3e}, ec off {e_off:.3e}")
    assert e_off > 2.0 ** -16
    assert e_on < 2.0 ** -20
    hiA = A.numpy().astype(np.float16).astype(np.float64)
    hiB = B.numpy().astype(np.float16).astype(np.float64)
    hh = np.einsum("bik,bkj->bij", hiA, hiB) + C.numpy().astype(np.float64)
    assert np.all(np.abs(off - hh) <= 130 * 2.0 ** -23 * ref["n64"])


def test_batch_past_one_launch():
    """A batch larger than one launch holds: each wave takes one item of at
    most 64 x 64, four waves a workgroup, so a launch takes at most
    (2^31 / 256 - 1) * 4 = 33,554,428 items and this batch needs two.  A pool
    of P items (k with a tail after one full step) is checked against the
    oracle and repeated across the batch; every item of D must equal its pool
    item bitwise."""
    P, m, n, k = 1021, 2, 3, 20
    per_launch = ((1 << 31) // 256 - 1) * 4
    batch = per_launch + 2 * P + 7
    print(f"case acc batch={batch} m={m} n={n} k={k}", flush=True)
    dev = device()
    A, B, C = _draw(P, m, n, k, seed=89)
    Ad = periodic_batch(A.to(dev), batch)
    Bd = periodic_batch(B.to(dev), batch)
    Cd = periodic_batch(C.to(dev), batch)
    D = torch.full((batch, m, n), float("nan"), device=dev)
    pkg.sgemm_emu_batched_acc(Ad, Bd, Cd, D)
    ref = oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy())
    gate(to_np(D[:P]), ref, k, "acc pool")
    gate_repeated(D, ref, P, [per_launch - 1, per_launch, per_launch + 1, batch - 1], k,
                  "acc, launch boundary")
    assert_periodic(D, P, "acc batch")


def _random_shapes(n, seed):
    g = np.random.default_rng(seed)
    return [(int(g.integers(1, 4)), int(g.integers(1, 200)), int(g.integers(1, 200)),
             int(g.integers(0, 300))) for _ in range(n)]


@pytest.mark.parametrize("shape", _random_shapes(8, 4048), ids=lambda s: "x".join(map(str, s)))
def test_random_shapes_all_layouts(shape):
    """Seeded random ragged shapes (k = 0 included in the range) under every
    combination of instruction shape, transposes and C/D layout."""
    batch, m, n, k = shape
    print(f"case acc random {shape}", flush=True)
    A, B, C = _draw(batch, m, n, k, seed=11 * m + n + 3 * k)
    ref = oracle.gemm_acc(A.numpy(), B.numpy(), C.numpy())
    for combo in COMBOS:
        s, oa, ob, lay = combo
        D = _run(A, B, C, oa, ob, lay, SHAPES[s])
        gate(D, ref, max(k, 1), f"acc random {shape} {_cid(combo)}",
             max_gate=gate_applies(ref))


def test_workload_gemm_acc_128_sampled():
    """The full workload (4096 items of D = A^T B + C, 128^3) in the launch
    configuration the benchmark times: every output written (NaN
    beforehand, finite after) and 64 whole items spread over the batch held
    to the bar."""
    w = synth.WORKLOADS["gemm_acc_128"]
    print(f"case workload=gemm_acc_128 batch={w.batch}", flush=True)
    At, B, C = synth.workload_inputs(w)
    dev = device()
    D = nan_output((w.batch, w.m, w.n))
    pkg.sgemm_emu_batched_acc(At.to(dev), B.to(dev), C.to(dev), D, op_a=pkg.OP_T)
    assert_all_finite(D, "gemm_acc_128")
    items = spread_items(w.batch, 64)
    ref = oracle.gemm_acc(At[items].numpy(), B[items].numpy(), C[items].numpy(), "T", "N")
    got = to_np(D[torch.from_numpy(items).to(dev)])
    e = gate(got, ref, w.k, "gemm_acc_128")
    print(f"gemm_acc_128: err {e[0]:.3e} fp32 {e[1]:.3e}")
