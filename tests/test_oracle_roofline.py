"""Pins of the oracle's roofline model (oracle.roofline) to the paper.

* the values the paper prints for the A100 (tests/golden/roofline_a100.txt):
  registers at n = 64 (256) and for the error-corrected (32, 32, 32) block
  (128), and the emulation's bounds at register blocking 32 with the fragment
  API alone (52.0 TFLOP/s, shared-memory bound) and with fragments built from
  FP32 data (104.0 TFLOP/s, a third of the FP16 Tensor-Core peak); a wrong
  byte count per element, a missing factor of 3 or a wrong register packing
  moves one of them;
* the closed forms: the middle expression of eq. simple-mma-ai is n/6 (the
  paper prints n/5), eq. simple-mma-reg is n^2/16, the staged and direct
  emulation intensities are n/12 and n/4, so the direct flow has 3x the
  intensity of the staged one at every n.
"""
import pathlib

import pytest

from oracle import roofline

GOLDEN = pathlib.Path(__file__).parent / "golden" / "roofline_a100.txt"


def _golden():
    vals = {}
    for line in GOLDEN.read_text().splitlines():
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = line.split()
            vals[k] = float(v)
    return vals


def test_paper_values_a100():
    g = _golden()
    assert roofline.mma_regs(64) == g["mma_regs_n64"]
    assert roofline.emu_regs(32) == g["emu_regs_n32"]
    staged = roofline.emu_peak(32, "staged", g["smem_gbps"], g["tc_fp16_tflops"])
    direct = roofline.emu_peak(32, "direct", g["smem_gbps"], g["tc_fp16_tflops"])
    assert round(staged, 1) == g["emu_peak_staged_n32"]
    assert round(direct, 1) == g["emu_peak_direct_n32"]
    # the direct flow at n = 32 is compute-bound: its shared-memory bound is higher
    assert roofline.emu_ai(32, "direct") * g["smem_gbps"] / 1000 > g["tc_fp16_tflops"] / 3


@pytest.mark.parametrize("n", [8, 16, 32, 48, 64, 128])
def test_closed_forms(n):
    assert roofline.mma_ai(n) == pytest.approx(n / 6, rel=1e-15)
    assert roofline.mma_ai(n) != pytest.approx(n / 5)
    assert roofline.mma_regs(n) == pytest.approx(n * n / 16, rel=1e-15)
    assert roofline.emu_ai(n, "staged") == pytest.approx(n / 12, rel=1e-15)
    assert roofline.emu_ai(n, "direct") == pytest.approx(n / 4, rel=1e-15)
    assert roofline.emu_ai(n, "direct") == pytest.approx(3 * roofline.emu_ai(n, "staged"))
    assert roofline.emu_regs(n) == pytest.approx(n * n / 8, rel=1e-15)


def test_byte_counts_by_hand():
    # one (2, 2, 2) block: 4 elements of A and 4 of B; 16 flops
    assert roofline.emu_smem_bytes(2, "direct") == 8 * 4
    assert roofline.emu_smem_bytes(2, "staged") == 8 * (4 + 2 + 2 + 2 + 2)
    assert roofline.emu_ai(2, "direct") == 16 / 32
