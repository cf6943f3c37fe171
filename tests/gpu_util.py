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

When the ratio gate applies.  The device's error splits into the method's
own error and its accumulation error:

    |C - C64| / N  <=  |CM - C64| / N  +  |C - CM| / N.

The first term is a property of the inputs alone: each product carries the
split's representation error and the dropped lo.lo term, at most about
3 * 2^-22 |a||b|, whatever the arithmetic; the oracle evaluates it exactly
(CM is summed in FP64).  The second term comes from the FP32 roundings of the
device's sums, of the same kind and number as the plain FP32 chain's.  So the
ratio gate is a requirement any correct implementation can meet only where
the method's own error leaves room for the accumulation's: it is applied
wherever max |CM - C64| / N <= max |C32 - C64| / N (the method's own error
takes at most half of the 2x budget).  With one product (k = 1) the FP32
result is one correctly rounded product, at most 2^-24 |a||b| off, against
the split's 3 * 2^-22: no implementation of the method meets the ratio
there, and the condition leaves it out.  Every configured workload meets the
condition by a wide margin; the element-wise bounds apply to every shape.
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


def gate_applies(ref) -> bool:
    """True where the ratio gate can be required of a correct implementation:
    the method-exact model's own error is at most the plain FP32 error."""
    e_m = oracle.max_rel_err(ref["cm"], ref["c64"], ref["n64"])
    e_32 = oracle.max_rel_err(ref["c32"], ref["c64"], ref["n64"])
    return e_m <= e_32


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


# ---------------------------------------------------------------------------
# Full-size workloads.  The output starts as NaN and must be finite
# everywhere after the call (a tile or item the kernel skipped stays NaN);
# the values are compared with the oracle on samples spread over every item
# of the batch.
# ---------------------------------------------------------------------------

def nan_output(shape) -> torch.Tensor:
    return torch.full(shape, float("nan"), dtype=torch.float32, device=device())


def assert_all_finite(C: torch.Tensor, label: str = ""):
    """Every output element written (checked on the device)."""
    bad = int((~torch.isfinite(C)).sum())
    assert bad == 0, f"{label}: {bad} of {C.numel()} outputs not written or not finite"


def spread_items(batch: int, count: int) -> np.ndarray:
    """`count` item indices covering the batch evenly, first and last
    included (every item when count >= batch)."""
    if count >= batch:
        return np.arange(count, dtype=np.int64) % batch
    return np.unique(np.linspace(0, batch - 1, count).round().astype(np.int64))


def spread_samples(batch: int, m: int, n: int, count: int, seed: int):
    """(item, row, col) of `count` output elements spread over every item:
    items evenly over the batch, rows and columns at random, and the four
    corners of the first and last item."""
    g = np.random.default_rng(seed)
    items = np.sort(spread_items(batch, count))
    items = np.resize(items, count)
    rows = g.integers(0, m, count)
    cols = g.integers(0, n, count)
    corner = [(0, 0, 0), (0, m - 1, n - 1), (batch - 1, 0, n - 1), (batch - 1, m - 1, 0)]
    for t, (b, r, c) in enumerate(corner):
        items[t], rows[t], cols[t] = b, r, c
    return items, rows, cols


def gemm_sampled(C: torch.Tensor, A: torch.Tensor, B: torch.Tensor, count: int, seed: int,
                 label: str = "", max_gate: bool = True):
    """C (device, [batch, m, n]) = A B (host [batch, m, k], [batch, k, n]):
    whole output finite, and `count` elements spread over every item held to
    the parity bar against the oracle's dot products."""
    assert_all_finite(C, label)
    batch, m, n = C.shape
    k = A.shape[-1]
    items, rows, cols = spread_samples(batch, m, n, count, seed)
    An, Bn = A.numpy(), B.numpy()
    arows = An[items, rows, :]
    bcols = Bn[items, :, cols]
    ref = oracle.dots(arows, bcols)
    it = torch.from_numpy(items).to(C.device)
    got = to_np(C[it, torch.from_numpy(rows).to(C.device), torch.from_numpy(cols).to(C.device)])
    return gate(got, ref, k, f"{label} ({count} sampled outputs over {batch} items)",
                max_gate=max_gate)
