"""The work queue the segment-table expansion kernel builds on the device,
called through the library's internal test hook on random segment tables.

What the GCM kernels rely on: tile_base is the exclusive scan of each
segment's tiles and the small list names the small segments in order; every
tile's rows that hold blocks are covered exactly once by its entries; a tile
that is cut has no whole-tile entry (a whole tile stores its GHASH partial,
pieces XOR theirs into it); entries come longest first and the queue is
padded with empty entries up to its capacity; the tiles cut are the ones the
rule names (with fewer tiles than CUs every tile longer than ceil(rows /
CUs); otherwise up to one per CU, the largest longer than a quarter tile);
a one-tile segment whose tile is cut is marked cut (its tag comes from the
finalize pass)."""
import ctypes
import subprocess

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from paper_2608_25431_amd import gift  # noqa: E402

# compile-time constants of the library (gift_internal.hpp)
THREADS, ROWS = 1024, 128
TILE_BLOCKS = THREADS * ROWS
PIECE_ROWS = ROWS // 4
SMALL_MAX_BLOCKS = 64
SEG_SMALL, SEG_ONE_TILE = 2, 4
NO_TILE = 0xFFFFFFFF

SEGDESC = np.dtype([("byte_off", "<u8"), ("len", "<u8"), ("row_begin", "<u8"), ("row_count", "<u8"),
                    ("iv", "<u4", 3), ("user", "<u4"), ("nblocks", "<u4"), ("flags", "<u4"), ("chunk0", "<u8")])
TILEENT = np.dtype([("g", "<u4"), ("s", "<u4"), ("trow", "<u4"), ("user", "<u4")])
assert SEGDESC.itemsize == 64 and TILEENT.itemsize == 16


@pytest.fixture(scope="module")
def expand():
    lib = gift.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", gift.LIB_PATH], capture_output=True, text=True).stdout
    names = [l.split()[-1] for l in out.splitlines() if l.strip()]
    fn = getattr(lib, next(n for n in names if n.startswith("_ZN4gift15expand_for_test")))
    P, U32 = ctypes.c_void_p, ctypes.c_uint32
    fn.argtypes = [P, U32, U32, P, P, P, P, U32, ctypes.POINTER(U32)]
    fn.restype = ctypes.c_int
    return fn


def descs_of(nblocks, rng):
    d = np.zeros(len(nblocks), SEGDESC)
    d["nblocks"] = nblocks
    d["user"] = rng.integers(0, 1000, len(nblocks))
    small = d["nblocks"] <= SMALL_MAX_BLOCKS
    one = ~small & (d["nblocks"] <= TILE_BLOCKS)
    d["flags"] = 1 | np.where(small, SEG_SMALL, 0) | np.where(one, SEG_ONE_TILE, 0)
    return d


def tile_rows(m, t):
    # rows of tile t that hold blocks: tiles end at the segment's end
    missing = (t + 1) * TILE_BLOCKS - m
    return ROWS if missing <= 0 else ROWS - missing // THREADS


def plan(expand, d, cus):
    """Runs the expansion kernel; returns the tile count, the flags before,
    the segments left with more than one entry, the piece rows, which tiles
    are cut, the entries, tile_base and the small list.  d's one-tile flag is
    cleared where the kernel marks the segment cut."""
    n = len(d)
    n_tiles = int(sum(-(-int(m) // TILE_BLOCKS) for m, f in zip(d["nblocks"], d["flags"]) if not f & SEG_SMALL))
    flags0 = d["flags"].copy()
    cap = n_tiles + (ROWS // PIECE_ROWS - 1) * cus
    seg_cut = np.full(n, 0xEEEEEEEE, np.uint32)
    tile_base = np.full(n + 1, 0xEEEEEEEE, np.uint32)
    small = np.full(n, 0xEEEEEEEE, np.uint32)
    order = np.zeros(max(cap, 1), TILEENT)
    n_ents = ctypes.c_uint32(0)
    assert expand(d.ctypes.data, n, cus, seg_cut.ctypes.data, tile_base.ctypes.data, small.ctypes.data,
                  order.ctypes.data, cap, ctypes.byref(n_ents)) == 0
    ne = n_ents.value
    assert ne <= cap
    assert (order[ne:cap]["g"] == NO_TILE).all(), "the queue is padded with empty entries"
    assert set(np.unique(seg_cut)) <= {0, 1}
    # a one-tile segment whose tile is cut takes the multi-entry path
    d["flags"] = np.where(seg_cut == 1, d["flags"] & ~np.uint32(SEG_ONE_TILE), d["flags"])
    ents = order[:ne]
    r0, r1 = (ents["trow"] >> 16) & 0xFF, ents["trow"] >> 24
    whole = (r0 == 0) & (r1 == ROWS)
    cut = np.zeros(max(n_tiles, 1), np.uint8)
    cut[ents["g"][~whole]] = 1
    piece = int((r1 - r0)[~whole].max()) if (~whole).any() else 0
    n_multi = sum(1 for i in range(n) if not d["flags"][i] & (SEG_SMALL | SEG_ONE_TILE))
    return n_tiles, flags0, n_multi, piece, cut[:n_tiles], ents, tile_base, small


def check(d, cus, n_tiles, flags0, n_multi, piece, cut, ents, tile_base_dev, small_dev):
    segs = [i for i in range(len(d)) if not flags0[i] & SEG_SMALL]
    tile_base, rows, g = {}, [], 0
    exp_tb = []
    for i in range(len(d)):
        exp_tb.append(g)
        if i not in set(segs):
            continue
        tile_base[i] = g
        nt = -(-int(d["nblocks"][i]) // TILE_BLOCKS)
        rows += [tile_rows(int(d["nblocks"][i]), t) for t in range(nt)]
        g += nt
    assert g == n_tiles
    assert tile_base_dev.tolist() == exp_tb + [n_tiles], "tile_base: exclusive scan of tiles per segment"
    small_segs = [i for i in range(len(d)) if flags0[i] & SEG_SMALL]
    assert small_dev[:len(small_segs)].tolist() == small_segs, "the small segments, in table order"
    rows = np.array(rows, np.int64)
    assert set(np.unique(cut)) <= {0, 1}
    cut = cut.astype(bool)
    # which tiles are cut, into pieces of how many rows
    if n_tiles == 0:
        assert piece == 0
    elif n_tiles < cus:
        fine = -(-int(rows.sum()) // cus)
        assert (cut == (rows > fine)).all()
        assert piece == (fine if cut.any() else 0)
    else:
        assert piece == (PIECE_ROWS if cut.any() else 0)
        assert cut.sum() <= cus and (rows[cut] > PIECE_ROWS).all()
        longer = rows > PIECE_ROWS
        if cut.sum() < cus:
            assert (cut == longer).all(), "every tile longer than a piece is cut"
        if cut.any() and (longer & ~cut).any():
            assert rows[cut].min() >= rows[longer & ~cut].max(), "the largest tiles are cut"
    t_of = ents["trow"] & 0xFFFF
    r0, r1 = (ents["trow"] >> 16) & 0xFF, ents["trow"] >> 24
    assert (r0 < r1).all() and (r1 <= ROWS).all()
    run = []
    covered = {}
    for k in range(len(ents)):
        s, t = int(ents["s"][k]), int(t_of[k])
        assert s in tile_base and ents["user"][k] == d["user"][s]
        assert ents["g"][k] == tile_base[s] + t
        lo = ROWS - tile_rows(int(d["nblocks"][s]), t)
        a, b = max(int(r0[k]), lo), int(r1[k])
        assert a < b, "an entry runs no row"
        run.append(b - a)
        covered.setdefault(int(ents["g"][k]), []).append((a, b, int(r0[k]), int(r1[k]), lo))
    assert run == sorted(run, reverse=True), "longest entries first"
    # whole uncut tiles (the bulk of a long call) come in tile order, and so
    # do the whole pieces of cut tiles, each tile's from its end down
    gk = [int(ents["g"][k]) for k in range(len(ents)) if run[k] == ROWS]
    assert gk == sorted(gk), "whole tiles in tile order"
    if piece:
        whole = [(int(ents["g"][k]), -int(r1[k])) for k in range(len(ents))
                 if run[k] == piece and cut[int(ents["g"][k])] and int(r1[k]) - int(r0[k]) == piece]
        assert whole == sorted(whole), "whole pieces in tile order"
    assert len(covered) == n_tiles
    for gg, parts in covered.items():
        parts.sort()
        lo = parts[0][4]
        assert parts[0][0] == lo and parts[-1][1] == ROWS
        for x, y in zip(parts, parts[1:]):
            assert x[1] == y[0], "rows covered exactly once"
        if cut[gg]:
            assert len(parts) > 1
            assert all(not (p[2] == 0 and p[3] == ROWS) for p in parts), "a cut tile has no whole-tile entry"
            assert all((ROWS - p[3]) % piece == 0 and p[3] - p[2] <= piece for p in parts), "pieces end-aligned"
        else:
            assert len(parts) == 1 and parts[0][2:4] == (0, ROWS)
    # cut marks: exactly the one-tile segments whose tile was cut
    for i in segs:
        had = bool(flags0[i] & SEG_ONE_TILE)
        assert bool(d["flags"][i] & SEG_ONE_TILE) == (had and not cut[tile_base[i]])


REGIMES = {
    "tiny": lambda r, n: r.integers(1, 7000, n),
    "one_tile": lambda r, n: r.integers(65, TILE_BLOCKS + 1, n),
    "mixed": lambda r, n: np.concatenate([r.integers(1, 200, n // 3), r.integers(65, TILE_BLOCKS + 1, n // 3),
                                          r.integers(TILE_BLOCKS, 9 * TILE_BLOCKS, n - 2 * (n // 3))]),
    "multi": lambda r, n: r.integers(TILE_BLOCKS // 2, 40 * TILE_BLOCKS, n),
    "whole_tiles": lambda r, n: TILE_BLOCKS * r.integers(1, 6, n),
}


@pytest.mark.parametrize("regime", sorted(REGIMES))
@pytest.mark.parametrize("cus", [256, 64, 7, 1])
def test_queue_covers_every_row_once_longest_first(expand, regime, cus):
    rng = np.random.default_rng(1000 * sorted(REGIMES).index(regime) + cus)
    for n in (1, 2, 5, 33, 200, 3000):
        d = descs_of(REGIMES[regime](rng, n), rng)
        res = plan(expand, d, cus)
        check(d, cus, *res)


def test_single_small_tile_is_cut_across_the_device(expand):
    # a 1.5 MiB segment (96 tile rows) on 256 CUs: 96 one-row pieces
    d = descs_of(np.array([96 * THREADS]), np.random.default_rng(1))
    n_tiles, flags0, n_multi, piece, cut, ents, _, _ = plan(expand, d, 256)
    assert (n_tiles, piece, len(ents), n_multi) == (1, 1, 96, 1)
    assert not d["flags"][0] & SEG_ONE_TILE


def test_full_device_queue_of_short_tiles_is_not_cut(expand):
    # as many short tiles as CUs: nothing to cut, one-tile segments keep their path
    d = descs_of(np.full(256, 3 * THREADS + 5), np.random.default_rng(2))
    n_tiles, flags0, n_multi, piece, cut, ents, _, _ = plan(expand, d, 256)
    assert piece == 0 and len(ents) == 256 and n_multi == 0
    assert (d["flags"] & SEG_ONE_TILE).all()


def test_one_tile_segments_past_the_cu_count_share_the_tail(expand):
    # 300 one-tile segments of 96 rows on 256 CUs: 256 of them are cut into
    # three pieces, so no CU runs two whole tiles while others idle
    d = descs_of(np.full(300, 96 * THREADS), np.random.default_rng(3))
    n_tiles, flags0, n_multi, piece, cut, ents, _, _ = plan(expand, d, 256)
    assert (piece, int(cut.sum()), len(ents), n_multi) == (PIECE_ROWS, 256, 44 + 3 * 256, 256)
