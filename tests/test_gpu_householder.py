"""Parity of the batched Householder application C = (I - 2 u u^T) B with the
reflector built in registers (Sec. 4.2.1) in emulated FP32 (Sec. 4.4).

* the reflector entries the kernel forms are fmaf(-2 u_i, u_j, delta_ij),
  bit for bit: with B = I every output is hi(h) + lo(h) 2^-11 rounded once,
  which the oracle computes from its own split of H32;
* the accuracy gate against the FP64 product and the plain FP32 product;
* u = +-e_i flips one row of B exactly up to the split of B;
* ragged column counts and padded leading dimensions;
* the full-size workload on sampled items.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
import synth
from gpu_util import device, gate, to_np

pytestmark = pytest.mark.gpu


def _run(u, B, C=None):
    dev = device()
    return to_np(pkg.householder_emu_batched(u.to(dev), B.to(dev), C))


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


def test_workload_householder_sampled():
    w = synth.WORKLOADS["householder_64"]
    print(f"case workload=householder_64 batch={w.batch}", flush=True)
    u, B = synth.workload_inputs(w)
    C = _run(u, B)
    items = [0, 1, 4095, 131072, w.batch - 1]
    ref = oracle.householder(u.numpy(), B.numpy(), items=items)
    e = gate(C[items], ref, 64, "householder_64")
    print(f"householder_64: err {e[0]:.3e} fp32 {e[1]:.3e}")
