"""The Python binding's own checks, on device tensors: an output the caller
passes must have the shape the call writes (the library cannot see the
allocation behind a pointer), probe operands must be [64, 8] int16, and
every operand must be a device tensor.  Each rejected call raises before
anything is launched, and the output is left untouched."""
import pytest
import torch

import paper_2308_15152_amd as pkg
from gpu_util import device

pytestmark = pytest.mark.gpu


def test_householder_rejects_wrong_output_shape():
    dev = device()
    u = torch.nn.functional.normalize(torch.randn(3, 64, device=dev), dim=1)
    B = torch.rand(3, 64, 10, device=dev)
    for shape in [(3, 64, 9), (2, 64, 10), (3, 63, 10), (64, 10)]:
        C = torch.full(shape, 5.0, device=dev)
        with pytest.raises(ValueError):
            pkg.householder_emu_batched(u, B, C)
        assert bool((C == 5.0).all())
    C = torch.empty(3, 64, 10, device=dev)
    pkg.householder_emu_batched(u, B, C)  # the right shape still runs
    torch.cuda.synchronize()


def test_givens_rejects_wrong_output_shape():
    dev = device()
    c = torch.full((4,), 0.6, device=dev)
    s = torch.full((4,), 0.8, device=dev)
    B = torch.rand(4, 64, 8, device=dev)
    for shape in [(4, 64, 7), (3, 64, 8), (64, 8)]:
        C = torch.full(shape, 5.0, device=dev)
        with pytest.raises(ValueError):
            pkg.givens_emu_batched(5, 37, c, s, B, C)
        assert bool((C == 5.0).all())


def test_probe_rejects_bad_operands():
    dev = device()
    ok = torch.zeros(64, 8, dtype=torch.int16, device=dev)
    for bad in [torch.zeros(64, 4, dtype=torch.int16, device=dev),
                torch.zeros(32, 8, dtype=torch.int16, device=dev),
                torch.zeros(64, 8, dtype=torch.float16, device=dev),
                torch.zeros(8, 64, dtype=torch.int16, device=dev).t()]:
        with pytest.raises(ValueError):
            pkg.mfmae_mma_probe(pkg.SHAPE_32x32x16, bad, ok)
        with pytest.raises(ValueError):
            pkg.mfmae_mma_probe(pkg.SHAPE_32x32x16, ok, bad)


def test_operands_must_be_device_tensors():
    dev = device()
    A = torch.rand(2, 8, 8, device=dev)
    with pytest.raises((ValueError, TypeError)):
        pkg.sgemm_emu_batched(A, torch.rand(2, 8, 8))
    with pytest.raises(ValueError):
        pkg.sgemm_emu_scan(torch.rand(4, 8))


def test_calls_from_several_threads():
    """The library's calls are thread-safe: four host threads, each on its own
    stream (default priority), run products concurrently (the binding's
    foreign calls release the interpreter lock) through three different
    kernels; every result equals the same product run alone, bit for bit
    (the kernels are deterministic)."""
    import threading

    import numpy as np

    import synth
    from gpu_util import to_np

    dev = device()
    shapes = [(64, 128, 128, 128), (2, 96, 80, 72), (3, 256, 256, 64), (5, 64, 64, 64)]
    inputs = [tuple(t.to(dev) for t in synth.gemm_inputs(*s, seed=300 + i))
              for i, s in enumerate(shapes)]
    alone = [to_np(pkg.sgemm_emu_batched(A, B)) for A, B in inputs]
    results = [[None] * 10 for _ in shapes]
    errors = []

    def work(i):
        try:
            A, B = inputs[i]
            s = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(s):
                for r in range(10):
                    results[i][r] = pkg.sgemm_emu_batched(A, B)
            s.synchronize()
        except Exception as e:  # reported below, in the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(shapes))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    for i in range(len(shapes)):
        for r in range(10):
            got = to_np(results[i][r])
            assert np.array_equal(got.view(np.uint32), alone[i].view(np.uint32)), (i, r)


@pytest.mark.parametrize("threads", [256, 512, 1024])
def test_stream_probe_computes_the_sum(threads):
    """The measurement reference moves A, B and C and adds: C = A + B exactly."""
    dev = device()
    g = torch.Generator().manual_seed(threads)
    A = torch.rand((37, 64, 68), generator=g).to(dev)
    B = torch.rand((37, 64, 68), generator=g).to(dev)
    C = torch.full_like(A, float("nan"))
    pkg.sgemm_emu_stream_probe(A, B, C, threads=threads)
    assert torch.equal(C, A + B)


def test_mfma_probe_computes_the_repeated_chunk_product():
    """The products-only reference runs the full-tile kernel's products on
    the first k chunk's fragments k / 32 times.  With small integers (hi
    exact, lo zero) its output is exactly (k / 32) A[:, :32] @ B[:32, :];
    the columns of A and rows of B it must not read hold NaN, and every
    output is written.  With uniform inputs the correction products are
    live: the error stays at the emulation's level (dropping lo would leave
    errors near 2^-11 of the magnitudes)."""
    dev = device()
    g = torch.Generator().manual_seed(5)
    m, n, k = 256, 512, 128
    A = torch.full((m, 48), float("nan"))
    B = torch.full((40, n), float("nan"))
    A[:, :32] = torch.randint(-4, 5, (m, 32), generator=g).float()
    B[:32, :] = torch.randint(-4, 5, (32, n), generator=g).float()
    C = torch.full((m, n), float("nan"), device=dev)
    pkg.sgemm_emu_mfma_probe(A.to(dev), B.to(dev), k, C)
    want = (k // 32) * (A[:, :32].double() @ B[:32, :].double())
    assert torch.equal(C.cpu().double(), want)

    A = torch.rand((m, 32), generator=g) * 2 - 1
    B = torch.rand((32, n), generator=g) * 2 - 1
    C = pkg.sgemm_emu_mfma_probe(A.to(dev), B.to(dev), k)
    exact = (k // 32) * (A.double() @ B.double())
    norm = (k // 32) * (A.double().abs() @ B.double().abs())
    err = ((C.cpu().double() - exact).abs() / norm).max().item()
    assert err < 64 * 2.0**-23, err

