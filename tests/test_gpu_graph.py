"""The library's calls inside a HIP graph (torch.cuda.CUDAGraph): they are
plain kernel launches on the caller's stream that allocate nothing and
record no memset, so a captured call replays as the same kernels.  Each
graph is replayed several times with the program's own eager work and
synchronizations between the replays (the output refilled with NaN by a
fill kernel, an eager call of the same product into another buffer), and
every replay must equal the eager result bit for bit (the kernels are
deterministic)."""
import numpy as np
import pytest
import torch

import paper_2308_15152_amd as pkg
import synth
from gpu_util import device, to_np

pytestmark = pytest.mark.gpu

# register-direct 64 x 64, full-tile 128 x 128, full-tile 256 x 128 (persistent
# stream form), register-direct 128 x 128 on a ragged product
SHAPES = [(16, 64, 64, 64), (8, 128, 128, 128), (2, 256, 256, 128), (3, 100, 90, 70)]


def _capture(fn):
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    return g


def _bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_gemm_graph_replays_match_eager(shape):
    dev = device()
    A, B = synth.gemm_inputs(*shape, seed=500 + shape[1])
    Ad, Bd = A.to(dev), B.to(dev)
    eager = to_np(pkg.sgemm_emu_batched(Ad, Bd))
    C = torch.full(eager.shape, float("nan"), device=dev)
    g = _capture(lambda: pkg.sgemm_emu_batched(Ad, Bd, C))
    for _ in range(3):
        C.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_bits(to_np(C)), _bits(eager))
        other = to_np(pkg.sgemm_emu_batched(Ad, Bd))
        assert np.array_equal(_bits(other), _bits(eager))


def test_scan_and_householder_graph_replays_match_eager():
    dev = device()
    X = synth.uniform((300, 2048), synth.rng(510)).to(dev)
    u, B = synth.householder_inputs(40, 64, 64, seed=511)
    ud, Bd = u.to(dev), B.to(dev)
    y_eager = to_np(pkg.sgemm_emu_scan(X))
    h_eager = to_np(pkg.householder_emu_batched(ud, Bd))
    Y = torch.full(X.shape, float("nan"), device=dev)
    H = torch.full((40, 64, 64), float("nan"), device=dev)

    def step():
        pkg.sgemm_emu_scan(X, Y)
        pkg.householder_emu_batched(ud, Bd, H)

    g = _capture(step)
    for _ in range(3):
        Y.fill_(float("nan"))
        H.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_bits(to_np(Y)), _bits(y_eager))
        assert np.array_equal(_bits(to_np(H)), _bits(h_eager))
        assert np.array_equal(_bits(to_np(pkg.sgemm_emu_scan(X))), _bits(y_eager))
