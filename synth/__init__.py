"""Seeded synthetic inputs for the emulated-SGEMM workloads.

This module is shared by the tests, the benchmark and the smoke check; it
draws random numbers and nothing else (none of the method's arithmetic lives
here).  The paper's batched SGEMM benchmark (Sec. 4.4.2) and Householder
benchmark (Sec. 4.2.1) use random matrices whose distribution it does not
state; the workloads below fix one.

Every generator draws on a CPU ``torch.Generator`` seeded with the workload's
seed, in a fixed order, so the device path and the oracle see identical bits.

Workloads (row-major, contiguous, FP32):

* ``gemm_64``    batch 16,     64 x 64 x 64,   entries uniform(-1, 1),     seed 1
* ``gemm_128``   batch 4096,   128 x 128 x 128, entries uniform(-1, 1),    seed 2
* ``gemm_256e``  batch 1024,   256 x 256 x 256, entries u * 2^e, u uniform(-1, 1),
  e integer uniform in [-15, 15] per entry,                                seed 3
* ``gemm_8192``  batch 1,      8192 x 8192 x 8192, entries uniform(-1, 1), seed 4
* ``householder_64``  batch 262144, u in R^64 standard normal then divided by
  its FP32 2-norm, B 64 x 64 uniform(-1, 1),                               seed 5
* ``paper_k<K>``  batch 256, 1024 x 1024 x K for K in PAPER_SWEEP_K,
  entries uniform(-1, 1),                                                  seed 6
* ``gemm_acc_128``  batch 4096, D = A^T B + C with A stored k x m (128 x 128),
  B 128 x 128, C 128 x 128, entries uniform(-1, 1), drawn A, B, C,         seed 8
* ``scan_2048``  131072 rows of 2048 values uniform(-1, 1) (batch = rows,
  n = the row length), inclusive scan of every row,                        seed 9
* ``givens_64``  batch 262144, rotation plane (i, j) = (5, 37) of n = 64,
  theta uniform in [0, 2 pi) per item with c, s = cos, sin theta evaluated
  in FP64 and rounded to FP32, B 64 x 64 uniform(-1, 1),                   seed 7

uniform(-1, 1) is drawn as ``2 * torch.rand - 1`` in FP32, which is exact and
lies on a 2^-23 grid.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str        # "gemm", "gemm_acc", "householder", "givens" or "scan"
    batch: int
    m: int
    n: int
    k: int
    dist: str        # "uniform" or "uniform_exp"
    seed: int
    plane: tuple = (0, 1)   # rotation plane (i, j) of a Givens workload

    @property
    def flops(self) -> float:
        """Emulated flops counted as 2 m n k per item (Sec. 4.4.2); for the
        Householder and Givens workloads the left matrix is formed
        explicitly as a fragment, so the same dense count applies with
        m = k = 64.  A scan counts one addition per element."""
        if self.kind == "scan":
            return float(self.batch * self.n)
        return 2.0 * self.m * self.n * self.k * self.batch

    @property
    def algorithmic_bytes(self) -> int:
        """Bytes the product must move at least once: read A (or u, or c
        and s) and B, write C, all FP32."""
        if self.kind == "householder":
            per = 4 * (self.m + self.k * self.n + self.m * self.n)
        elif self.kind == "givens":
            per = 4 * (2 + self.k * self.n + self.m * self.n)
        elif self.kind == "scan":
            per = 8 * self.n  # read the row, write its scan
        elif self.kind == "gemm_acc":
            # read A, B and C, write D
            per = 4 * (self.m * self.k + self.k * self.n + 2 * self.m * self.n)
        else:
            per = 4 * (self.m * self.k + self.k * self.n + self.m * self.n)
        return per * self.batch


WORKLOADS = {
    "gemm_64": Workload("gemm_64", "gemm", 16, 64, 64, 64, "uniform", 1),
    "gemm_128": Workload("gemm_128", "gemm", 4096, 128, 128, 128, "uniform", 2),
    "gemm_256e": Workload("gemm_256e", "gemm", 1024, 256, 256, 256, "uniform_exp", 3),
    "gemm_8192": Workload("gemm_8192", "gemm", 1, 8192, 8192, 8192, "uniform", 4),
    "householder_64": Workload("householder_64", "householder", 262144, 64, 64, 64,
                               "householder", 5),
}

# The batched SGEMM experiment of Sec. 4.4.2: 256 products of
# (1024 x k) . (k x 1024), swept over k (the k values are only in the
# paper's missing figure; these span its range of shapes).
PAPER_SWEEP_K = (128, 256, 512, 1024, 2048, 4096)
for _k in PAPER_SWEEP_K:
    WORKLOADS[f"paper_k{_k}"] = Workload(f"paper_k{_k}", "gemm", 256, 1024, 1024, _k,
                                         "uniform", 6)


WORKLOADS["scan_2048"] = Workload("scan_2048", "scan", 131072, 1, 2048, 1, "uniform", 9)
WORKLOADS["gemm_acc_128"] = Workload("gemm_acc_128", "gemm_acc", 4096, 128, 128, 128, "uniform", 8)
WORKLOADS["givens_64"] = Workload("givens_64", "givens", 262144, 64, 64, 64, "givens", 7,
                                  (5, 37))


def _gen(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def uniform(shape, g: torch.Generator) -> torch.Tensor:
    """uniform(-1, 1) on the 2^-23 grid, FP32 (exact: 2r - 1 for r in [0,1))."""
    return torch.rand(shape, generator=g, dtype=torch.float32) * 2.0 - 1.0


def uniform_exp(shape, g: torch.Generator, emin: int = -15, emax: int = 15) -> torch.Tensor:
    """u * 2^e with u uniform(-1, 1) and e integer uniform in [emin, emax]
    (torch.ldexp by an integer power of two is exact here)."""
    u = uniform(shape, g)
    e = torch.randint(emin, emax + 1, shape, generator=g, dtype=torch.int32)
    return torch.ldexp(u, e.to(torch.float32))


def gemm_inputs(batch: int, m: int, n: int, k: int, seed: int,
                dist: str = "uniform"):
    """A [batch, m, k] then B [batch, k, n], drawn in that order."""
    g = _gen(seed)
    draw = uniform if dist == "uniform" else uniform_exp
    A = draw((batch, m, k), g)
    B = draw((batch, k, n), g)
    return A, B


def householder_inputs(batch: int, n: int, ncols: int, seed: int):
    """u [batch, n] (standard normal, divided by its FP32 2-norm), then
    B [batch, n, ncols] uniform(-1, 1), drawn in that order."""
    g = _gen(seed)
    u = torch.randn((batch, n), generator=g, dtype=torch.float32)
    u = u / torch.linalg.vector_norm(u, dim=1, keepdim=True)
    B = uniform((batch, n, ncols), g)
    return u, B


def gemm_acc_inputs(batch: int, m: int, n: int, k: int, seed: int):
    """For D = A^T B + C: A stored as [batch, k, m], then B [batch, k, n],
    then C [batch, m, n], all uniform(-1, 1), drawn in that order."""
    g = _gen(seed)
    At = uniform((batch, k, m), g)
    B = uniform((batch, k, n), g)
    C = uniform((batch, m, n), g)
    return At, B, C


def givens_inputs(batch: int, n: int, ncols: int, seed: int):
    """c [batch], s [batch] (theta uniform in [0, 2 pi), cos and sin in FP64
    rounded to FP32), then B [batch, n, ncols] uniform(-1, 1), drawn in that
    order."""
    g = _gen(seed)
    theta = torch.rand((batch,), generator=g, dtype=torch.float64) * (2.0 * torch.pi)
    c = torch.cos(theta).to(torch.float32)
    s = torch.sin(theta).to(torch.float32)
    B = uniform((batch, n, ncols), g)
    return c, s, B


def workload_inputs(w: Workload, batch: int | None = None):
    """Inputs of a named workload; ``batch`` may shrink the batch (the first
    items are then a prefix of what a smaller draw would give only for the
    same batch size, so parity cases always regenerate at their own size)."""
    b = w.batch if batch is None else batch
    if w.kind == "householder":
        return householder_inputs(b, w.m, w.n, w.seed)
    if w.kind == "givens":
        return givens_inputs(b, w.m, w.n, w.seed)
    if w.kind == "gemm_acc":
        return gemm_acc_inputs(b, w.m, w.n, w.k, w.seed)
    if w.kind == "scan":
        return (uniform((b, w.n), _gen(w.seed)),)
    return gemm_inputs(b, w.m, w.n, w.k, w.seed, w.dist)


def integer_matrix(shape, g: torch.Generator, lo: int, hi: int) -> torch.Tensor:
    """Integer-valued FP32 entries uniform in [lo, hi]."""
    return torch.randint(lo, hi + 1, shape, generator=g, dtype=torch.int32).to(torch.float32)


def rng(seed: int) -> torch.Generator:
    return _gen(seed)
