"""Shared helpers of the GPU parity tests.

Parity bar for the emulated product (floating point, several correct results
are possible because the matrix instruction's internal summation order is
not specified):

* the accuracy gate: with C64 the FP64 product of the FP32 inputs, N the
  normaliser (|A||B|)_ij and C32 the plain FP32 product,
      max_ij |C - C64| / N  <=  2 * max_ij |C32 - C64| / N   and  <= k * 2^-23;
* element by element against the method-exact model CM (eq. corr-5 with the
  split taken exactly, summed in FP64): every FP32 addition on the device
  path moves the result by at most one ulp of a partial sum bounded by N
  (for round-to-nearest half an ulp; one ulp also covers truncation), so
      |C - CM|_ij <= (k + 2) * 2^-23 * N_ij;
* element by element against the FP64 product: the split represents each
  operand to within 2^-22 of its magnitude and the dropped lo.lo term is at
  most 2^-22 |a||b|, so each product is off by at most about 3 * 2^-22 |a||b|
  before accumulation, and
      |C - C64|_ij <= (k + 8) * 2^-23 * N_ij.

The two max-error gates compare statistics of rounding errors.  With a
handful of terms the plain FP32 chain can be exact by chance (k = 1 is one
correctly rounded product), so the ratio says nothing there; the gates are
applied to every workload and to every shape with k >= 32 and at least 256
outputs, and the element-wise bounds to every shape.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle


def device():
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    return torch.device("cuda:0")


def gate_applies(k, outputs) -> bool:
    return k >= 32 and outputs >= 256


def gate(C, ref, k, label="", max_gate=True):
    """Assert the element-wise bounds and (if ``max_gate``) the accuracy gate;
    return the errors for reporting."""
    C = np.asarray(C, dtype=np.float32)
    assert np.isfinite(C).all(), f"{label}: non-finite output"
    e_emu = oracle.max_rel_err(C, ref["c64"], ref["n64"])
    e_32 = oracle.max_rel_err(ref["c32"], ref["c64"], ref["n64"])
    if max_gate:
        assert e_emu <= 2 * e_32, f"{label}: err {e_emu:.3e} > 2 x fp32 err {e_32:.3e}"
        assert e_emu <= max(k, 1) * 2.0 ** -23, f"{label}: err {e_emu:.3e} > k 2^-23"
    dev64 = np.abs(C.astype(np.float64) - ref["c64"])
    bad = dev64 > (k + 8) * 2.0 ** -23 * ref["n64"]
    assert not bad.any(), f"{label}: {int(bad.sum())} elements beyond (k+8) 2^-23 N"
    if "cm" in ref:
        dev = np.abs(C.astype(np.float64) - ref["cm"])
        bound = (k + 2) * 2.0 ** -23 * ref["n64"]
        bad = dev > bound
        assert not bad.any(), (f"{label}: {int(bad.sum())} elements off the method model, "
                               f"worst {float((dev / np.maximum(ref['n64'], 1e-300)).max()):.3e}")
    return e_emu, e_32


def to_np(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


# ---------------------------------------------------------------------------
# Batches past one launch.  The launchers split a batch into pieces below
# 2^31 work-items; to cross that boundary with the memory of one device, a
# pool of P items checked against the oracle is repeated across the batch
# (item t holds pool item t mod P), and every output item is compared bit for
# bit with the pool item it repeats: an item the kernel left unwritten (the
# output starts as NaN), wrote twice or computed from another item's operands
# breaks the period.
# ---------------------------------------------------------------------------

def periodic_batch(pool: torch.Tensor, batch: int) -> torch.Tensor:
    """[batch, ...] on the pool's device: item t is pool[t % P]."""
    P = pool.shape[0]
    reps = (batch + P - 1) // P
    return pool.repeat(reps, *([1] * (pool.dim() - 1)))[:batch]


def assert_periodic(C: torch.Tensor, P: int, label: str = "", slab_items: int = 1 << 22):
    """Every item of C equals item t mod P, bitwise (compared on the device
    in slabs of whole periods)."""
    flat = C.reshape(C.shape[0], -1).view(torch.int32)
    head = flat[:P]
    per = max(1, slab_items // P) * P
    for t0 in range(0, flat.shape[0], per):
        s = flat[t0:t0 + per]
        q, r = divmod(s.shape[0], P)
        if q:
            body = s[:q * P].view(q, P, -1)
            bad = (body != head.unsqueeze(0)).any(dim=2)
            if bool(bad.any()):
                first = int(bad.flatten().nonzero()[0])
                raise AssertionError(f"{label}: item {t0 + first} differs from pool item "
                                     f"{first % P}")
        if r:
            if not torch.equal(s[q * P:], head[:r]):
                raise AssertionError(f"{label}: an item in [{t0 + q * P}, {t0 + s.shape[0]}) "
                                     f"differs from its pool item")


def gate_repeated(C: torch.Tensor, ref: dict, P: int, items, k: int, label: str = ""):
    """Element-wise bounds for chosen items of a periodic batch against the
    oracle's results for the pool items they repeat (item t holds pool item
    t mod P): the items on both sides of a launch boundary, say."""
    items = sorted(set(int(t) for t in items))
    got = to_np(C[items])
    sub = {key: np.asarray(v)[[t % P for t in items]] for key, v in ref.items()}
    return gate(got, sub, k, label, max_gate=False)
