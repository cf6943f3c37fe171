"""Host checks of the helpers behind the GPU tests of batches past one
launch: the periodic check accepts a correctly repeated batch and rejects an
unwritten item, an item shifted by one position, and a corrupted item in the
partial last period."""
import pytest
import torch

from gpu_util import assert_periodic, periodic_batch


def _batch(P=7, batch=59):
    pool = torch.arange(P * 6, dtype=torch.float32).view(P, 2, 3)
    return pool, periodic_batch(pool, batch).clone()


def test_repeats_pool():
    pool, C = _batch()
    assert C.shape == (59, 2, 3)
    for t in range(59):
        assert torch.equal(C[t], pool[t % 7])
    assert_periodic(C, 7, slab_items=10)


@pytest.mark.parametrize("t", [7, 30, 48, 57])
def test_rejects_unwritten_item(t):
    _, C = _batch()
    C[t] = float("nan")
    with pytest.raises(AssertionError):
        assert_periodic(C, 7, slab_items=10)


def test_rejects_shifted_items():
    _, C = _batch()
    C[21:28] = torch.roll(C[21:28], 1, dims=0)
    with pytest.raises(AssertionError):
        assert_periodic(C, 7, slab_items=14)


def test_rejects_corrupted_tail():
    _, C = _batch()
    C[-1, 1, 2] += 1
    with pytest.raises(AssertionError):
        assert_periodic(C, 7)
