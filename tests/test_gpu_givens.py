"""Parity of the batched Givens rotation C = G(i, j, theta) B with G built in
registers through the element map (Sec. 4.3.1), in emulated FP32 (Sec. 4.4),
for the three ways of building G: map with (i, j) as kernel arguments, map
with (i, j) fixed at compile time, and G stored in LDS.

* the entries the kernel places are G's, bit for bit: with B = I every
  output is one product g . 1, i.e. hi(g) + lo(g) 2^-11 rounded once, which
  the oracle computes from its own split of G; a misplaced, transposed or
  sign-flipped entry fails this;
* the three modes feed identical operands to identical instructions, so
  their outputs agree bit for bit;
* theta = pi / 2 on integer B is an exact signed swap of rows i and j;
* the element-wise bounds against the FP64 product and the method model,
  ragged column counts, padded leading dimensions, and the full-size
  workload on sampled items.

Tolerance: every output is a sum with at most two nonzero terms (rows other
than i and j have one), so the element-wise bounds of the GEMM tests apply
with k = 2: |C - C64| <= 10 2^-23 N and |C - CM| <= 4 2^-23 N.  The
"at most twice the FP32 error" gate is not applied: the plain FP32 product
of this matrix is exact on every row but i and j, while the split of B
alone moves an entry by up to 2^-22 of its size.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2308_15152_amd as pkg
import synth
from gpu_util import assert_all_finite, device, gate, nan_output, spread_items, to_np

pytestmark = pytest.mark.gpu

MODES = {"map": pkg.GIVENS_MAP, "embedded": pkg.GIVENS_EMBEDDED, "lds": pkg.GIVENS_LDS}
EMBEDDED_PLANES = [(5, 37), (37, 5), (0, 1), (31, 32), (62, 63)]
OTHER_PLANES = [(3, 60), (16, 17), (47, 15), (32, 31), (63, 0)]
K_EFF = 2


def _run(i, j, c, s, B, C=None, mode=pkg.GIVENS_AUTO):
    dev = device()
    return to_np(pkg.givens_emu_batched(i, j, c.to(dev), s.to(dev), B.to(dev), C, mode=mode))


def _cases():
    out = []
    for name in MODES:
        planes = EMBEDDED_PLANES if name == "embedded" else EMBEDDED_PLANES + OTHER_PLANES
        out += [(name, p) for p in planes]
    return out


@pytest.mark.parametrize("mode,plane", _cases())
def test_rotation_entries_bit_exact(mode, plane):
    i, j = plane
    print(f"case givens entries mode={mode} plane={plane}", flush=True)
    c, s, _ = synth.givens_inputs(5, 64, 1, seed=40 + i + 64 * j)
    eye = torch.eye(64).expand(5, 64, 64).contiguous()
    C = _run(i, j, c, s, eye, mode=MODES[mode])
    for b in range(5):
        G = oracle.givens_matrix(64, i, j, c[b].item(), s[b].item())
        hi, lo = oracle.split(G)
        rec = (hi.view(np.float16).astype(np.float32) +
               lo.view(np.float16).astype(np.float32) * np.float32(2.0 ** -11))
        assert np.array_equal(C[b].view(np.uint32), rec.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("ncols", [64, 1, 33, 100, 130])
def test_modes_agree_and_parity(ncols):
    print(f"case givens ncols={ncols}", flush=True)
    i, j = 5, 37
    c, s, B = synth.givens_inputs(9, 64, ncols, seed=50 + ncols)
    outs = {name: _run(i, j, c, s, B, mode=m) for name, m in MODES.items()}
    for name in ("embedded", "lds"):
        assert np.array_equal(outs[name].view(np.uint32), outs["map"].view(np.uint32)), name
    ref = oracle.givens(i, j, c.numpy(), s.numpy(), B.numpy())
    gate(outs["map"], ref, K_EFF, f"givens ncols={ncols}", max_gate=False)


@pytest.mark.parametrize("mode", list(MODES))
def test_runtime_plane_parity(mode):
    i, j = (31, 32) if mode == "embedded" else (47, 15)
    c, s, B = synth.givens_inputs(7, 64, 64, seed=61)
    C = _run(i, j, c, s, B, mode=MODES[mode])
    ref = oracle.givens(i, j, c.numpy(), s.numpy(), B.numpy())
    gate(C, ref, K_EFF, f"givens {mode} plane=({i},{j})", max_gate=False)


@pytest.mark.parametrize("mode", list(MODES))
def test_quarter_turn_integer_exact(mode):
    i, j = 62, 63
    B = synth.integer_matrix((3, 64, 64), synth.rng(8), -1000, 1000)
    c = torch.zeros(3)
    s = torch.ones(3)
    C = _run(i, j, c, s, B, mode=MODES[mode])
    expect = B.numpy().copy()
    expect[:, i] = -B.numpy()[:, j]
    expect[:, j] = B.numpy()[:, i]
    assert np.array_equal(C, expect)


def test_padded_leading_dimensions_and_strided_angles():
    dev = device()
    c, s, B = synth.givens_inputs(4, 64, 80, seed=71)
    cs = torch.stack([c, s], dim=1).to(dev)  # c and s interleaved: stride 2
    Bd = B.to(dev)[:, :, :70]
    C_big = torch.full((4, 64, 96), 9.0, device=dev)
    pkg.givens_emu_batched(0, 1, cs[:, 0], cs[:, 1], Bd, C_big[:, :, :70])
    out = to_np(C_big)
    ref = oracle.givens(0, 1, c.numpy(), s.numpy(), np.ascontiguousarray(B.numpy()[:, :, :70]))
    gate(out[:, :, :70], ref, K_EFF, "givens padded", max_gate=False)
    assert np.all(out[:, :, 70:] == 9.0)


@pytest.mark.parametrize("mode", list(MODES))
def test_workload_givens_sampled(mode):
    """The full workload: every output written (NaN beforehand, finite
    after) and 512 whole items spread over the batch held to the bar."""
    w = synth.WORKLOADS["givens_64"]
    i, j = w.plane
    print(f"case workload=givens_64 mode={mode} batch={w.batch}", flush=True)
    c, s, B = synth.workload_inputs(w)
    C = nan_output((w.batch, w.m, w.n))
    pkg.givens_emu_batched(i, j, c.to(device()), s.to(device()), B.to(device()), C,
                           mode=MODES[mode])
    assert_all_finite(C, f"givens_64 {mode}")
    items = spread_items(w.batch, 512)
    ref = oracle.givens(i, j, c.numpy(), s.numpy(), B.numpy(), items=items)
    got = to_np(C[torch.from_numpy(items).to(C.device)])
    e = gate(got, ref, K_EFF, f"givens_64 {mode}", max_gate=False)
    print(f"givens_64 {mode}: err {e[0]:.3e} fp32 {e[1]:.3e}")
    del C
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", list(MODES))
def test_broadcast_angle_single_item_and_column_groups(mode):
    """One (c, s) for every item (stride 0), a single item, and 200 columns
    (four column groups, the last partial, odd pairing off)."""
    dev = device()
    i, j = (62, 63) if mode == "embedded" else (9, 50)
    c, s, B = synth.givens_inputs(4, 64, 200, seed=91)
    cb = c[:1].to(dev).expand(4)
    sb = s[:1].to(dev).expand(4)
    C = to_np(pkg.givens_emu_batched(i, j, cb, sb, B.to(dev), mode=MODES[mode]))
    c4 = np.full(4, c[0].item(), np.float32)
    s4 = np.full(4, s[0].item(), np.float32)
    gate(C, oracle.givens(i, j, c4, s4, B.numpy()), K_EFF, f"givens broadcast {mode}",
         max_gate=False)
    one = to_np(pkg.givens_emu_batched(i, j, c[:1].to(dev), s[:1].to(dev), B[:1, :, :199]
                                       .contiguous().to(dev), mode=MODES[mode]))
    gate(one, oracle.givens(i, j, c[:1].numpy(), s[:1].numpy(),
                            np.ascontiguousarray(B[:1, :, :199].numpy())), K_EFF,
         f"givens single {mode}", max_gate=False)
