"""Parity of the batched Householder application C = (I - 2 u u^T) B with the
reflector built in registers (Sec. 4.2.1) in emulated FP32 (Sec. 4.4).

* the reflector entries the kernel forms are fmaf(-2 u_i, u_j, delta_ij):
  with B = I every output is hi(h) + lo(h) 2^-11 rounded once, which the
  oracle computes from its own split of H32 (this pins h and the split up
  to pairs (hi, lo) that reconstruct the same value); a constructed binary16
  tie pins the split of the FP32 entry itself;
* the accuracy gate against the FP64 product and the plain FP32 product;
* u = +-e_i flips one row of B exactly up to the split of B;
* ragged column counts and padded leading dimensions;
* the full-size workload on sampled items;
* the baseline that forms H in LDS (the comparison of Sec. 4.2.1) places
  the same entries: bit-identical to the register-built reflector.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
import synth
from gpu_util import (assert_all_finite, assert_periodic, device, gate, gate_repeated, nan_output,
                      periodic_batch, spread_items, to_np)

pytestmark = pytest.mark.gpu


def _run(u, B, C=None, mode=pkg.HOUSEHOLDER_RULE):
    dev = device()
    return to_np(pkg.householder_emu_batched(u.to(dev), B.to(dev), C, mode=mode))


def test_reflector_entries_bit_exact():
    u, _ = synth.householder_inputs(6, 64, 64, seed=31)
    eye = torch.eye(64).expand(6, 64, 64).contiguous()
    C = _run(u, eye)
    for b in range(6):
        H32 = oracle.householder_h32(u[b].numpy())
        hi, lo = oracle.split(H32)
        rec = (hi.view(np.float16).astype(np.float32) +
               lo.view(np.float16).astype(np.float32) * np.float32(2.0 ** -11))
        assert np.array_equal(C[b].view(np.uint32), rec.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("ncols", [64, 1, 33, 100, 130])
def test_parity_column_counts(ncols):
    print(f"case householder ncols={ncols}", flush=True)
    u, B = synth.householder_inputs(9, 64, ncols, seed=32 + ncols)
    C = _run(u, B)
    ref = oracle.householder(u.numpy(), B.numpy())
    gate(C, ref, 64, f"householder ncols={ncols}")


def test_basis_vector_flips_row():
    n = 64
    u = torch.zeros((3, n))
    u[0, 0] = 1.0
    u[1, 17] = -1.0
    u[2, 63] = 1.0
    B = synth.integer_matrix((3, n, n), synth.rng(5), -100, 100)
    C = _run(u, B)
    expect = B.numpy().copy()
    expect[0, 0] *= -1
    expect[1, 17] *= -1
    expect[2, 63] *= -1
    assert np.array_equal(C, expect)


def test_padded_leading_dimensions():
    dev = device()
    u, B = synth.householder_inputs(4, 64, 80, seed=41)
    Bd = B.to(dev)[:, :, :70]
    C_big = torch.full((4, 64, 96), 9.0, device=dev)
    pkg.householder_emu_batched(u.to(dev), Bd, C_big[:, :, :70])
    out = to_np(C_big)
    ref = oracle.householder(u.numpy(), np.ascontiguousarray(B.numpy()[:, :, :70]))
    gate(out[:, :, :70], ref, 64, "householder padded")
    assert np.all(out[:, :, 70:] == 9.0)


@pytest.mark.parametrize("mode", [pkg.HOUSEHOLDER_RULE, pkg.HOUSEHOLDER_LDS], ids=["rule", "lds"])
def test_workload_householder_sampled(mode):
    """The full workload in the launch configuration the benchmark times:
    every output written (NaN beforehand, finite after) and 512 whole items
    spread over the batch (2M outputs) held to the parity bar."""
    w = synth.WORKLOADS["householder_64"]
    print(f"case workload=householder_64 mode={mode} batch={w.batch}", flush=True)
    u, B = synth.workload_inputs(w)
    C = nan_output((w.batch, w.m, w.n))
    pkg.householder_emu_batched(u.to(device()), B.to(device()), C, mode=mode)
    assert_all_finite(C, "householder_64")
    items = spread_items(w.batch, 512)
    ref = oracle.householder(u.numpy(), B.numpy(), items=items)
    got = to_np(C[torch.from_numpy(items).to(C.device)])
    e = gate(got, ref, 64, f"householder_64 mode {mode}")
    print(f"householder_64 mode {mode}: err {e[0]:.3e} fp32 {e[1]:.3e}")
    del C
    torch.cuda.empty_cache()


@pytest.mark.parametrize("ncols", [64, 33, 130])
def test_lds_baseline_bit_identical(ncols):
    u, B = synth.householder_inputs(7, 64, ncols, seed=51 + ncols)
    reg = _run(u, B)
    lds = _run(u, B, mode=pkg.HOUSEHOLDER_LDS)
    assert np.array_equal(reg.view(np.uint32), lds.view(np.uint32))
    gate(lds, oracle.householder(u.numpy(), B.numpy()), 64, f"householder lds ncols={ncols}")


def test_lds_baseline_reflector_entries():
    u, _ = synth.householder_inputs(4, 64, 64, seed=52)
    eye = torch.eye(64).expand(4, 64, 64).contiguous()
    C = _run(u, eye, mode=pkg.HOUSEHOLDER_LDS)
    for b in range(4):
        hi, lo = oracle.split(oracle.householder_h32(u[b].numpy()))
        rec = (hi.view(np.float16).astype(np.float32) +
               lo.view(np.float16).astype(np.float32) * np.float32(2.0 ** -11))
        assert np.array_equal(C[b].view(np.uint32), rec.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("mode", [pkg.HOUSEHOLDER_RULE, pkg.HOUSEHOLDER_LDS])
def test_reflector_split_of_a_binary16_tie(mode):
    """h_01 = fl32(-2 u_0 u_1) = 1 + 2^-11 is a binary16 tie while the exact
    product lies just above it: the split of the FP32 entry takes hi = 1
    (ties to even), lo = 1; rounding the exact product to binary16 in one
    step (a fused multiply-add with a binary16 result) would give hi = 1 +
    2^-10, lo = -1, which reconstructs the same value.  With B rows
    (2^-22, 2 - 2^-10) the two splits give different sums: row 0 of C must
    equal the method model rounded to FP32."""
    u = torch.zeros((1, 64))
    u[0, 0] = -0.5 * (1 + 2.0 ** -23)
    u[0, 1] = 1 + 4095 * 2.0 ** -23
    B = torch.zeros((1, 64, 64))
    B[0, 0, :] = 2.0 ** -22
    B[0, 1, :] = 2 - 2.0 ** -10
    h01 = oracle.householder_h32(u[0].numpy())[0, 1]
    hi, lo = oracle.split(np.array([h01], np.float32))
    assert h01 == np.float32(1 + 2.0 ** -11)
    assert hi.view(np.float16)[0] == 1.0 and lo.view(np.float16)[0] == 1.0
    C = _run(u, B, mode=mode)
    cm = oracle.householder(u.numpy(), B.numpy(), want=("cm",))["cm"]
    assert np.array_equal(C[0, 0].view(np.uint32), cm[0, 0].astype(np.float32).view(np.uint32))


def test_batch_past_one_launch():
    """A batch larger than one launch holds: each wave takes one item (up to
    64 columns), four waves a workgroup, so a launch takes at most
    (2^31 / 256 - 1) * 4 = 33,554,428 items and this batch needs two.  A pool
    of P items is checked against the oracle and repeated across the batch;
    every item must equal its pool item bitwise."""
    P, ncols = 1021, 2
    per_launch = ((1 << 31) // 256 - 1) * 4
    batch = per_launch + 2 * P + 7
    print(f"case householder batch={batch} ncols={ncols}", flush=True)
    dev = device()
    u, B = synth.householder_inputs(P, 64, ncols, seed=43)
    ud = periodic_batch(u.to(dev), batch)
    Bd = periodic_batch(B.to(dev), batch)
    C = torch.full((batch, 64, ncols), float("nan"), device=dev)
    pkg.householder_emu_batched(ud, Bd, C)
    ref = oracle.householder(u.numpy(), B.numpy())
    gate(to_np(C[:P]), ref, 64, "householder pool")
    gate_repeated(C, ref, P, [per_launch - 1, per_launch, per_launch + 1, batch - 1], 64,
                  "householder, launch boundary")
    assert_periodic(C, P, "householder batch")
    del ud, Bd, C
    torch.cuda.empty_cache()
