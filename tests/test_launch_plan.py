"""The host's launch decisions for a call (no GPU): from per-segment counts
only, the work queue's capacity, the tile kernel's grid, and whether the
finalize pass may have work.  The finalize pass forms the tag of every
segment with more than one queue entry; leaving it out when a one-tile
segment's tile is cut would leave that segment without a tag, so it must be
launched whenever the expansion kernel's cut can reach a one-tile segment."""
import ctypes
import subprocess

import numpy as np
import pytest

from paper_2608_25431_amd import gift

THREADS, ROWS = 1024, 128
PIECE_ROWS = ROWS // 4


class QueuePlan(ctypes.Structure):
    _fields_ = [("cap", ctypes.c_uint64), ("grid", ctypes.c_uint32), ("finalize", ctypes.c_bool)]


@pytest.fixture(scope="module")
def plan_queue():
    if not __import__("os").path.exists(gift.LIB_PATH):
        from paper_2608_25431_amd import build
        build.build()
    lib = gift.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", gift.LIB_PATH], capture_output=True, text=True).stdout
    names = [l.split()[-1] for l in out.splitlines() if l.strip()]
    fn = getattr(lib, next(n for n in names if n.startswith("_ZN4gift10plan_queue")))
    fn.argtypes = [ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32]
    fn.restype = QueuePlan
    return fn


def can_cut_one_tile(n_tiles, rows_all, one_rows_max, cus):
    """Whether the expansion kernel's rule can cut the tile of a one-tile
    segment with one_rows_max rows: with fewer tiles than CUs it cuts tiles
    of more than ceil(rows_all / cus) rows (none when that is a whole tile or
    more); otherwise only tiles of more than PIECE_ROWS rows."""
    if n_tiles < cus:
        p = -(-rows_all // cus)
        return p < ROWS and one_rows_max > p
    return one_rows_max > PIECE_ROWS


@pytest.mark.parametrize("cus", [256, 64, 7, 1])
def test_plan_covers_the_kernel_rule(plan_queue, cus):
    r = np.random.default_rng(cus)
    for _ in range(400):
        n_one = int(r.integers(0, 40))
        n_multi = int(r.integers(0, 3)) if r.random() < 0.5 else 0
        one_rows = r.integers(1, ROWS + 1, n_one)
        multi_tiles = r.integers(2, 12, n_multi)
        multi_first = r.integers(1, ROWS + 1, n_multi)
        n_tiles = n_one + int(multi_tiles.sum())
        rows_all = int(one_rows.sum()) + int(((multi_tiles - 1) * ROWS + multi_first).sum())
        one_max = int(one_rows.max()) if n_one else 0
        q = plan_queue(n_tiles, rows_all, n_multi, one_max, cus)
        if n_tiles == 0:
            assert (q.cap, q.grid, q.finalize) == (0, 0, False)
            continue
        assert q.cap == n_tiles + (ROWS // PIECE_ROWS - 1) * cus
        assert 1 <= q.grid <= cus
        # enough workgroups for every entry up to one per CU
        assert q.grid >= min(cus, n_tiles)
        need = n_multi > 0 or can_cut_one_tile(n_tiles, rows_all, one_max, cus)
        assert q.finalize == need


def test_examples(plan_queue):
    # one 1.5 MiB segment on 256 CUs: cut into one-row pieces, tag from the finalize pass
    q = plan_queue(1, 96, 0, 96, 256)
    assert q.finalize and q.grid == 96
    # 256 short one-tile segments: nothing to cut, no finalize pass
    q = plan_queue(256, 256 * 4, 0, 4, 256)
    assert not q.finalize and q.grid == 256
    # more one-tile segments than CUs, longer than a quarter tile: the tail cut can reach them
    q = plan_queue(300, 300 * 96, 0, 96, 256)
    assert q.finalize and q.grid == 256
