"""The GEMM kernels' work distribution, checked exactly on the host (no GPU).

The kernels compute which task a workgroup takes (the XCD-aware numbering)
and which output tile a task is (groups of 8 tile rows) with functions that
the library also runs on the host (``sgemm_emu_xcd_order``,
``sgemm_emu_tile_order``).  Every output tile is computed exactly once only
if both are bijections; this is index work, so it is checked exactly, for
every grid size up to 4096 workgroups and every tile grid up to 64 x 64
(which includes every remainder of the 8-row grouping).
"""
import ctypes

import numpy as np
import pytest

import paper_2308_15152_amd as pkg


def test_xcd_order_is_a_bijection_for_every_grid():
    for G in range(1, 4097):
        t = pkg.sgemm_emu_xcd_order(G)
        assert np.array_equal(np.sort(t), np.arange(G)), G


def test_xcd_order_gives_each_xcd_one_contiguous_range():
    """Workgroup b runs on XCD b mod 8: the tasks of one XCD form one
    contiguous range, the ranges follow the XCD order, and within an XCD the
    tasks follow the dispatch order; XCDs below G mod 8 hold one task more."""
    for G in list(range(1, 300)) + [512, 1000, 2047, 2048, 4095, 4096]:
        t = pkg.sgemm_emu_xcd_order(G)
        b = np.arange(G)
        start = 0
        for x in range(8):
            mine = t[b % 8 == x]
            size = G // 8 + (1 if x < G % 8 else 0)
            assert len(mine) == size
            assert np.array_equal(mine, np.arange(start, start + size)), (G, x)
            start += size


def test_xcd_order_hand_values():
    # G = 16: XCD x holds tasks 2x, 2x + 1; workgroup b = 8i + x takes 2x + i
    assert pkg.sgemm_emu_xcd_order(16).tolist() == [0, 2, 4, 6, 8, 10, 12, 14,
                                                    1, 3, 5, 7, 9, 11, 13, 15]
    # G = 10: XCDs 0 and 1 hold two tasks each, the others one
    assert pkg.sgemm_emu_xcd_order(10).tolist() == [0, 2, 4, 5, 6, 7, 8, 9, 1, 3]
    assert pkg.sgemm_emu_xcd_order(1).tolist() == [0]


def test_persistent_walk_covers_every_task_once():
    """The persistent kernels: workgroup b of G walks xcd(b), xcd(b) + G, ...
    below ntasks; every task is taken exactly once."""
    for G in (1, 7, 8, 13, 256, 512, 1000):
        start = pkg.sgemm_emu_xcd_order(G)
        for ntasks in (1, G - 1, G, G + 1, 3 * G + 5, 4096):
            if ntasks < 1:
                continue
            seen = np.zeros(ntasks, dtype=np.int64)
            for t0 in start:
                seen[np.arange(t0, ntasks, G)] += 1
            assert (seen == 1).all(), (G, ntasks)


def test_tile_order_is_a_bijection_for_every_grid():
    for tm in range(1, 65):
        for tn in range(1, 65):
            r, c = pkg.sgemm_emu_tile_order(tm, tn)
            assert r.min() >= 0 and r.max() < tm and c.min() >= 0 and c.max() < tn
            flat = r.astype(np.int64) * tn + c
            assert np.array_equal(np.sort(flat), np.arange(tm * tn)), (tm, tn)


def test_tile_order_groups_of_eight_rows():
    """Tasks come in groups of 8 tile rows (the last group holds the rest),
    column by column inside a group, rows ascending inside a column."""
    for tm, tn in [(64, 32), (17, 5), (8, 3), (7, 9), (1, 4), (13, 1), (64, 64)]:
        r, c = pkg.sgemm_emu_tile_order(tm, tn)
        t = 0
        for first in range(0, tm, 8):
            gm = min(8, tm - first)
            for col in range(tn):
                for row in range(first, first + gm):
                    assert (r[t], c[t]) == (row, col), (tm, tn, t)
                    t += 1
        assert t == tm * tn


def test_block_order_is_a_bijection():
    for tm in range(16, 129, 16):
        for tn in range(16, 129, 16):
            r, c = pkg.sgemm_emu_block_order(tm, tn)
            assert r.min() >= 0 and r.max() < tm and c.min() >= 0 and c.max() < tn
            flat = r.astype(np.int64) * tn + c
            assert np.array_equal(np.sort(flat), np.arange(tm * tn)), (tm, tn)


def test_block_order_runs_one_block_of_tiles_at_a_time():
    """With one workgroup per task dispatched round-robin over the 8 XCDs,
    the 256 workgroups b in [256 w, 256 w + 256) (32 per XCD, one per CU)
    take the tiles of one 16 x 16 block, blocks down the columns first, and
    each XCD an 8 x 4 part of it: rows 8 (x mod 2) .. + 8, columns
    4 (x div 2) .. + 4 of the block."""
    for tm, tn in [(64, 32), (16, 16), (32, 48), (128, 16)]:
        G = tm * tn
        task = pkg.sgemm_emu_xcd_order(G)
        r, c = pkg.sgemm_emu_block_order(tm, tn)
        for w in range(G // 256):
            bm, bn = w % (tm // 16), w // (tm // 16)
            b = np.arange(256 * w, 256 * w + 256)
            rows, cols = r[task[b]], c[task[b]]
            assert set(zip(rows.tolist(), cols.tolist())) == {
                (16 * bm + i, 16 * bn + j) for i in range(16) for j in range(16)}, (tm, tn, w)
            x = b % 8
            assert ((rows - 16 * bm) // 8 == x % 2).all()
            assert ((cols - 16 * bn) // 4 == x // 2).all()


def test_block_order_only_for_grids_of_whole_blocks():
    lib = pkg.load()
    buf = (ctypes.c_int * 4)()
    for tm, tn in [(64, 33), (8, 16), (16, 8), (0, 16), (24, 32)]:
        assert lib.sgemm_emu_block_order(tm, tn, buf, buf) == -1, (tm, tn)
    assert lib.sgemm_emu_block_order(16, 16, None, buf) == -3


def test_task_to_item_and_tile_covers_a_launch():
    """A launch of `items` items: task // tiles is the item and the grouped
    order of task % tiles the tile; with the XCD numbering over a grid of one
    workgroup per task, every (item, tile) is computed once."""
    for items, tm, tn in [(3, 5, 7), (1, 64, 32), (4096, 1, 1), (16, 2, 2)]:
        tiles = tm * tn
        G = items * tiles
        task = pkg.sgemm_emu_xcd_order(G)
        r, c = pkg.sgemm_emu_tile_order(tm, tn)
        item = task // tiles
        within = task % tiles
        key = (item.astype(np.int64) * tm + r[within]) * tn + c[within]
        assert np.array_equal(np.sort(key), np.arange(G))


def test_work_maps_reject_bad_arguments():
    lib = pkg.load()
    buf = (ctypes.c_int * 4)()
    assert lib.sgemm_emu_xcd_order(0, buf) == -1
    assert lib.sgemm_emu_xcd_order(4, None) == -3
    assert lib.sgemm_emu_tile_order(0, 3, buf, buf) == -1
    assert lib.sgemm_emu_tile_order(3, -1, buf, buf) == -1
    assert lib.sgemm_emu_tile_order(1 << 16, 1 << 16, buf, buf) == -1
    assert lib.sgemm_emu_tile_order(2, 2, None, buf) == -3
    with pytest.raises(pkg.SgemmEmuError):
        pkg.sgemm_emu_xcd_order(0)
