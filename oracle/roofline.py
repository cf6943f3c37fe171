"""The paper's roofline model of shared-memory traffic for Tensor-Core matrix
multiplication, written out from its formulas.

TEST INFRASTRUCTURE ONLY (same rule as the rest of ``oracle``): it pins the
performance model the method is argued from; the product path never uses it.

* :func:`mma_ai`, :func:`mma_regs` -- a register-blocked (n, n, n) product
  on Tensor Cores with FP16 A, B and FP32 C, D held in shared memory: its
  arithmetic intensity against shared memory (Sec. 3, eq. simple-mma-ai)
  and the 32-bit registers per thread its fragments need when every element
  is held by one lane only (eq. simple-mma-reg).  The printed right-hand side
  of eq. simple-mma-ai, n/5, is not what its middle expression evaluates to:
  2n^3 / (2n^2 * 2 + 2n^2 * 4) = n/6; the expression is taken as written.
* :func:`emu_smem_bytes`, :func:`emu_ai`, :func:`emu_peak` -- the SGEMM
  emulation with error correction (Sec. 4.4, theoretical performance
  analysis): three products per emulated one, so the compute roof is the
  FP16 Tensor-Core peak over 3.  Two data flows (Fig. 6): with the fragment
  API alone each FP32 element of A and B is read from shared memory, written
  back as hi and lo (FP16 each) and both are read again (12 bytes per
  element); with fragments built straight from the FP32 values only the
  4-byte read remains.
* :func:`emu_regs` -- registers per thread for the fragments of the
  error-corrected product: A, dA, B, dB as FP16 and C, dC as FP32.
"""

FP16 = 2
FP32 = 4

# bytes of shared-memory traffic per element of A and B, per data flow
FLOW_BYTES = {
    "staged": FP32 + 2 * FP16 + 2 * FP16,  # read FP32, write hi and lo, read both
    "direct": FP32,                        # read FP32, split in registers
}


def mma_ai(n: float) -> float:
    """Flops per shared-memory byte of one (n, n, n) block: A, B in FP16 and
    C, D in FP32 moved once each (eq. simple-mma-ai, middle expression)."""
    return 2 * n ** 3 / ((n * n + n * n) * FP16 + (n * n + n * n) * FP32)


def mma_regs(n: float, warp: int = 32) -> float:
    """32-bit registers per thread for A, B (two FP16 per register) and C
    (FP32) fragments of an (n, n, n) block spread over one warp
    (eq. simple-mma-reg)."""
    return ((n * n + n * n) / 2 + n * n) / warp


def emu_smem_bytes(n: float, flow: str) -> float:
    """Shared-memory bytes of one (n, n, n) block of the emulated product:
    n^2 elements of A and n^2 of B, each costing FLOW_BYTES[flow]."""
    return (n * n + n * n) * FLOW_BYTES[flow]


def emu_ai(n: float, flow: str) -> float:
    """Emulated flops (2 n^3 per block, one product's worth) per byte."""
    return 2 * n ** 3 / emu_smem_bytes(n, flow)


def emu_peak(n: float, flow: str, smem_gbps: float, tc_fp16_tflops: float) -> float:
    """Roofline bound in TFLOP/s: the smaller of AI x shared-memory bandwidth
    and a third of the FP16 Tensor-Core peak."""
    return min(emu_ai(n, flow) * smem_gbps / 1000.0, tc_fp16_tflops / 3.0)


def emu_regs(n: float, warp: int = 32) -> float:
    """Fragment registers per thread of the error-corrected (n, n, n) block:
    A, dA, B, dB (FP16, two per register) and C, dC (FP32)."""
    return (4 * n * n / 2 + 2 * n * n) / warp
