"""Parity of the batched inclusive scan computed as x^T U with the
upper-triangular all-ones U built from its rule by foreach_ij (Sec. 4.1,
eq. scan-mat), in emulated FP32 (Sec. 4.4), against the scan oracle.

* row counts around the 8-row share of a wave (1, 7, 8, 9, 100) and
  lengths around the 1024-value block and the 32-value segment (1, 31, 33,
  1000, 1024, 1025, 3072), on both the whole-block path (lengths that are
  multiples of 1024, aligned rows) and the element-wise path;
* integer inputs give the exact running sums; a unit impulse gives a step;
* in place, padded row strides, unaligned bases (the element-wise path);
* the full-size workload on sampled rows.

Tolerance: an output sums at most 32 split values inside its segment
(accumulated by the matrix instruction), then takes one fused combine of
the two accumulators, the segment offset from a five-level scan of segment
totals and one addition of it, and one carry addition per earlier block of
the row: at most 32 + 9 + len / 1024 roundings of partial sums bounded by
N.  The element-wise bounds of the GEMM tests (gpu_util.gate) are applied
with k = min(len, 64) + 2 ceil(len / 64), which is at least that count.
|Y - YM| <= (k + 2) 2^-23 N and |Y - Y64| <= (k + 8) 2^-23 N, N the running
sum of |x|.  The ratio gate against the plain FP32 running sum is not
applied: on short prefixes that sum is exact by construction.
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


def _k_eff(length):
    return min(length, 64) + 2 * ((length + 63) // 64)


@pytest.mark.parametrize("rows", [1, 7, 8, 9, 100])
@pytest.mark.parametrize("length", [1, 31, 33, 1000, 1024, 1025, 3072])
def test_parity_shapes(rows, length):
    print(f"case scan rows={rows} len={length}", flush=True)
    X = synth.uniform((rows, length), synth.rng(rows * 7 + length))
    Y = to_np(pkg.sgemm_emu_scan(X.to(device())))
    ref = oracle.scan(X.numpy())
    gate(Y, ref, _k_eff(length), f"scan {rows}x{length}", max_gate=False)


@pytest.mark.parametrize("length", [3000, 4096])
def test_integer_exact_and_in_place(length):
    X = synth.integer_matrix((70, length), synth.rng(5), -1000, 1000)
    Xd = X.to(device())
    pkg.sgemm_emu_scan(Xd, Xd)
    exact = np.cumsum(X.numpy().astype(np.int64), axis=1)
    assert np.array_equal(to_np(Xd), exact.astype(np.float32))


@pytest.mark.parametrize("length", [300, 2048])
def test_impulse_gives_step(length):
    X = torch.zeros((40, length))
    X[3, 0] = 2.5
    X[39, length - 1] = -1.0
    X[17, 64] = 3.0
    X[20, min(1023, length - 2)] = 0.75
    Y = to_np(pkg.sgemm_emu_scan(X.to(device())))
    expect = np.cumsum(X.numpy().astype(np.float64), axis=1).astype(np.float32)
    assert np.array_equal(Y, expect)


@pytest.mark.parametrize("offset", [0, 1])
@pytest.mark.parametrize("length,pitch", [(130, 136), (1024, 1040)])
def test_padded_and_unaligned(offset, length, pitch):
    dev = device()
    X = synth.uniform((45, length), synth.rng(6))
    buf = torch.zeros(45 * pitch + offset, device=dev)
    Xv = buf[offset:].view(45, pitch)[:, :length]
    Xv.copy_(X.to(dev))
    Ybuf = torch.full((45, pitch + 4), 5.0, device=dev)
    pkg.sgemm_emu_scan(Xv, Ybuf[:, :length])
    out = to_np(Ybuf)
    gate(out[:, :length], oracle.scan(X.numpy()), _k_eff(length), "scan padded",
         max_gate=False)
    assert np.all(out[:, length:] == 5.0)


def test_unaligned_output_only():
    """X aligned, Y one element off 16-byte alignment: the 16-byte stores of
    the whole-block path must not be used."""
    dev = device()
    X = synth.uniform((9, 2048), synth.rng(7)).to(dev)
    ybuf = torch.full((9 * 2048 + 1,), 5.0, device=dev)
    Y = ybuf[1:].view(9, 2048)
    pkg.sgemm_emu_scan(X, Y)
    out = to_np(ybuf)
    assert out[0] == 5.0
    gate(out[1:].reshape(9, 2048), oracle.scan(to_np(X)), _k_eff(2048), "scan unaligned Y",
         max_gate=False)


def test_workload_scan_sampled():
    """The full workload: every output written (NaN beforehand, finite
    after) and 4096 whole rows spread over the batch held to the bar."""
    w = synth.WORKLOADS["scan_2048"]
    print(f"case workload=scan_2048 rows={w.batch} len={w.n}", flush=True)
    (X,) = synth.workload_inputs(w)
    Y = nan_output((w.batch, w.n))
    pkg.sgemm_emu_scan(X.to(device()), Y)
    assert_all_finite(Y, "scan_2048")
    rows = spread_items(w.batch, 4096)
    Ys = to_np(Y[torch.from_numpy(rows).to(Y.device)])
    ref = oracle.scan(X[rows].numpy())
    e = gate(Ys, ref, _k_eff(w.n), "scan_2048", max_gate=False)
    print(f"scan_2048: err {e[0]:.3e} fp32 running sum {e[1]:.3e}")


def test_rows_past_one_launch():
    """More rows than one launch holds: a wave scans 8 rows, four waves a
    workgroup, so a launch takes at most (2^31 / 256 - 1) * 32 = 268,435,424
    rows and this scan needs two.  A pool of P rows is checked against the
    oracle and repeated down the rows; every output row must equal its pool
    row bitwise."""
    P, length = 1021, 5
    per_launch = ((1 << 31) // 256 - 1) * 32
    rows = per_launch + 2 * P + 7
    print(f"case scan rows={rows} len={length}", flush=True)
    X = synth.uniform((P, length), synth.rng(99))
    Xd = periodic_batch(X.to(device()), rows)
    Y = torch.full((rows, length), float("nan"), device=device())
    pkg.sgemm_emu_scan(Xd, Y)
    ref = oracle.scan(X.numpy())
    gate(to_np(Y[:P]), ref, _k_eff(length), "scan pool", max_gate=False)
    gate_repeated(Y, ref, P, [per_launch - 1, per_launch, per_launch + 1, rows - 1],
                  _k_eff(length), "scan, launch boundary")
    assert_periodic(Y, P, "scan rows")
    del Xd, Y
    torch.cuda.empty_cache()
