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
      |C - CM|_ij <= (k + 2) * 2^-23 * N_ij.
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


def gate(C, ref, k, label=""):
    """Assert the accuracy gate and the element-wise model bound; return the
    errors for reporting."""
    C = np.asarray(C, dtype=np.float32)
    assert np.isfinite(C).all(), f"{label}: non-finite output"
    e_emu = oracle.max_rel_err(C, ref["c64"], ref["n64"])
    e_32 = oracle.max_rel_err(ref["c32"], ref["c64"], ref["n64"])
    assert e_emu <= 2 * e_32, f"{label}: err {e_emu:.3e} > 2 x fp32 err {e_32:.3e}"
    assert e_emu <= max(k, 1) * 2.0 ** -23, f"{label}: err {e_emu:.3e} > k 2^-23"
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
