"""Parity of the HIP library (through its C ABI) with the CPU oracle.

Small and ragged cases, decode_batch at full size, the GCM length limit and
the paged calls compare every output byte, tag and verdict with the oracle;
the full-size llama3_8b_kv ciphertext is also checked by OpenSSL.  The other
large workloads are compared with the oracle in test_gpu_fullsize.py.  The
tolerance is zero everywhere: all of this is integer work.
"""
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import oracle  # noqa: E402
from gpu_helpers import (DEV, dev_u32, dev_u8, expected_block, host, open_, oracle_segments, seal,  # noqa: E402
                         status_of)
from paper_2608_25431_amd import gift  # noqa: E402
from paper_2608_25431_amd import workloads as W  # noqa: E402

rng = np.random.default_rng(4242)


def keyset(n):
    return rng.integers(0, 256, (n, 32), dtype=np.uint8), rng.integers(0, 256, (n, 12), dtype=np.uint8)


@pytest.fixture(scope="module")
def kt3():
    keys, nb = keyset(3)
    kt = gift.KeyTable(keys)
    yield keys, nb, kt
    kt.destroy()


def full_compare(keys, nb, kt, data, n_rows, rb, table, labels=None, in_place=False):
    """Seal + open on the GPU vs the oracle, every byte."""
    st, o_out, o_tags, o_ver = oracle.seal(data, n_rows, rb, table, keys, nb, labels=labels)
    assert st == 0
    d = dev_u8(data)
    lab = None if labels is None else dev_u32(labels)
    out, tags, ver = seal(d, n_rows, rb, table, kt, nb, labels_dev=lab, out=d if in_place else None)
    n = len(table)
    assert host(out).tobytes() == o_out.tobytes()
    assert host(tags)[:16 * n].tobytes() == o_tags.tobytes()
    assert host(ver)[:n].tolist() == o_ver.tolist()
    st, o_back, o_ver2 = oracle.open_(o_out, n_rows, rb, table, keys, nb, o_tags, labels=labels)
    back, ver2 = open_(out, n_rows, rb, table, kt, nb, tags, labels_dev=lab)
    assert host(back).tobytes() == o_back.tobytes()
    assert host(ver2)[:n].tolist() == o_ver2.tolist()
    return out, tags


def test_key_table_lifecycle():
    keys, _ = keyset(5)
    kt = gift.KeyTable(keys)
    assert kt.users == 5
    kt.destroy()
    assert status_of(gift.KeyTable, np.zeros(0, np.uint8), 0) == gift.E_INVALID


def test_tiny_config_every_byte():
    w = W.tiny()
    t = w.tensors[0]
    kt = gift.KeyTable(w.keys)
    data = t.generate("cpu").numpy()
    _, tags = full_compare(w.keys, w.nonce_base, kt, data, t.n_rows, t.row_bytes, t.segs)
    kt.destroy()
    # and the stored oracle tags (tests/golden/seeded_outputs.txt)
    golden = {}
    for line in open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "seeded_outputs.txt")):
        if line.startswith("tiny.tag"):
            k, v = line.split()
            golden[int(k[len("tiny.tag"):])] = v
    h = host(tags)
    assert [bytes(h[16 * i:16 * i + 16]).hex() for i in range(len(t.segs))] == [golden[i] for i in range(len(t.segs))]


def segmentations(n_rows):
    import itertools
    for choice in itertools.product((0, 1, 2), repeat=n_rows):
        segs, cur = [], None
        for r, c in enumerate(choice):
            if c == 0:
                cur = None
            elif c == 1 or cur is None:
                segs.append([r, 1])
                cur = segs[-1]
            else:
                cur[1] += 1
        yield [tuple(s) for s in segs]


@pytest.mark.parametrize("row_bytes", [4, 12, 16, 20, 48])
def test_brute_force_tiny_tensors(kt3, row_bytes):
    keys, nb, kt = kt3
    for n_rows in (1, 2, 3):
        data = rng.integers(0, 256, n_rows * row_bytes, dtype=np.uint8)
        for segs in segmentations(n_rows):
            table = [(b, c, i % 3, 1000 * n_rows + 10 * b + i) for i, (b, c) in enumerate(segs)]
            full_compare(keys, nb, kt, data, n_rows, row_bytes, table)
            full_compare(keys, nb, kt, data, n_rows, row_bytes, table, in_place=True)


@pytest.mark.parametrize("row_bytes,rows", [
    (16384, [1, 63, 64, 65, 129, 130, 200]),   # aligned; 2 MiB tiles: 128 rows = 1 tile
    (1000, [1, 17, 2100, 3, 4200]),            # unaligned starts, multi-tile
    (65536 + 16, [33, 1, 70]),                 # aligned, tiles end mid-row
    (48, [1, 2, 21, 22, 23, 44000]),           # small segments next to a 2 MiB one
    (16, [63, 64, 65, 1, 1024, 1025]),         # the small-segment limit (64 blocks) exactly, and one row of a tile
    (1, [1023, 1024, 1025, 1, 15, 17]),        # byte lengths around 64 blocks and around one block
])
def test_ragged_multi_tile_every_byte(kt3, row_bytes, rows):
    keys, nb, kt = kt3
    # segments with gaps of one row between them
    table, r = [], 1
    for i, n in enumerate(rows):
        table.append((r, n, i % 3, 7 + i))
        r += n + 1
    n_rows = r
    data = rng.integers(0, 256, n_rows * row_bytes, dtype=np.uint8)
    full_compare(keys, nb, kt, data, n_rows, row_bytes, table)


def test_five_tile_segment_every_byte(kt3):
    keys, nb, kt = kt3
    rb = 4096
    n = 2560 + 7  # 10 MiB + 28 KiB: 5 full tiles and a ragged first tile
    data = rng.integers(0, 256, n * rb, dtype=np.uint8)
    full_compare(keys, nb, kt, data, n, rb, [(0, n, 1, 99)])


def test_owner_labels_fused_and_standalone(kt3):
    keys, nb, kt = kt3
    rb, n_rows = 4096, 700
    table = [(0, 10, 0, 1), (10, 600, 1, 1), (610, 80, 2, 1), (690, 10, 0, 2)]
    lab = np.zeros(n_rows, np.uint32)
    for b, c, u, _ in table:
        lab[b:b + c] = u
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    full_compare(keys, nb, kt, data, n_rows, rb, table, labels=lab)
    for row, v in ((5, 2), (300, gift.LABEL_PARAM), (650, gift.LABEL_UNOWNED), (695, 1)):
        l2 = lab.copy()
        l2[row] = v
        full_compare(keys, nb, kt, data, n_rows, rb, table, labels=l2)
        ver = torch.full((4,), -1, dtype=torch.int32, device=DEV)
        gift.check_owner(table, dev_u32(l2), n_rows, ver)
        st, o = oracle.check_owner(table, l2, n_rows)
        assert host(ver).tolist() == o.tolist()


def test_propagated_labels_drive_the_fused_check(kt3):
    # host ownership tracking of a hidden-state tensor through AddBias and
    # AddResidual, then a seal whose segments the framework claims: segments
    # that disagree with the propagated labels are rejected on the device
    keys, nb, kt = kt3
    rows, cols = 96, 2048  # bf16: 4096-byte rows
    rb = 2 * cols
    x = torch.empty(rows * rb, dtype=torch.uint8, device=DEV)
    res = torch.empty_like(x)
    y = torch.empty_like(x)
    bias = torch.empty(rb, dtype=torch.uint8, device=DEV)
    o = gift.Ownership()
    for t in (x, res, y):
        o.register(t, (rows, cols), 2)
    o.register(bias, (cols,), 2, odims=())
    o.set(bias, 0, 1, gift.LABEL_PARAM)
    for t in (x, res):
        o.set(t, 0, 40, 0)
        o.set(t, 40, 50, 1)
        o.set(t, 90, 6, 2)
    assert o.add_bias(x, x, bias, rows, cols, 2) == gift.OK
    assert o.add_residual(y, x, res, rows, cols, 2) == gift.OK
    o.set(res, 45, 1, 2)  # one row of the residual now holds user 2's data
    assert o.add_residual(y, x, res, rows, cols, 2) == gift.E_REJECTED  # nothing changes
    labels = o.labels(y)
    data = rng.integers(0, 256, rows * rb, dtype=np.uint8)
    honest = [(0, 40, 0, 7), (40, 50, 1, 7), (90, 6, 2, 7)]
    forged = [(0, 41, 0, 8), (41, 49, 1, 8), (90, 6, 1, 9)]  # claims a user-1 row and user 2's rows
    for table in (honest, forged):
        full_compare(keys, nb, kt, data, rows, rb, table, labels=labels)
    _, _, ver = seal(dev_u8(data), rows, rb, forged, kt, nb, labels_dev=dev_u32(labels))
    assert host(ver)[:3].tolist() == [gift.SEG_OWNER_MIXED, gift.SEG_OK, gift.SEG_OWNER_MIXED]
    o.destroy()


def test_validation_status_matches_oracle(kt3):
    keys, nb, kt = kt3
    n_rows, rb = 6, 16
    d = dev_u8(np.zeros(n_rows * rb, np.uint8))
    cases = [
        [(0, 0, 0, 0)], [(0, 1, 0, 0, 1)], [(0, 1, gift.LABEL_PARAM, 0)], [(0, 1, gift.LABEL_UNOWNED, 0)],
        [(5, 2, 0, 0)], [(7, 1, 0, 0)], [(0, 1, 3, 0)], [(0, 2, 0, 0), (1, 2, 1, 0)],
        [(0, 1, 0, 5), (3, 1, 0, 5)], [(0, 1, 0, 5), (3, 1, 1, 5)], [(0, 0, 0, 0), (9, 1, 0, 0)],
        [(9, 1, 0, 0), (0, 0, 0, 0)], [], [(0, 6, 2, 1)],
    ]
    for table in cases:
        st_o = oracle.seal(np.zeros(n_rows * rb, np.uint8), n_rows, rb, table, keys, nb)[0]
        st_g = status_of(seal, d, n_rows, rb, table, kt, nb)
        assert st_g == st_o, table
    # partial overlap of out and data is rejected; exact aliasing is fine
    big = dev_u8(np.zeros(2 * n_rows * rb, np.uint8))
    tags = torch.zeros(16, dtype=torch.uint8, device=DEV)
    s = status_of(gift.seal, big[:n_rows * rb], n_rows, rb, [(0, 1, 0, 0)], kt, nb, big[16:16 + n_rows * rb], tags)
    assert s == gift.E_INVALID
    assert status_of(gift.seal, big, n_rows, rb, [(0, 1, 0, 0)], kt, nb, big, tags) == 0
    # open needs verdicts
    assert status_of(gift.open, big, n_rows, rb, [(0, 1, 0, 0)], kt, nb, big, tags, None) == gift.E_INVALID


def random_table(r, n_rows, n_users):
    """A small segment table that is valid or breaks one rule at random."""
    n = int(r.integers(0, 7))
    table, used = [], set()
    for _ in range(n):
        rb_ = int(r.integers(0, n_rows))
        rc = int(r.integers(1, n_rows - rb_ + 1))
        table.append([rb_, rc, int(r.integers(0, n_users)), int(r.integers(0, 4)), 0])
    if table and r.random() < 0.6:  # one defect
        i = int(r.integers(0, len(table)))
        kind = int(r.integers(0, 7))
        if kind == 0:
            table[i][1] = 0                                       # empty
        elif kind == 1:
            table[i][4] = 1                                       # reserved != 0
        elif kind == 2:
            table[i][2] = int(r.choice([gift.LABEL_PARAM, gift.LABEL_UNOWNED]))
        elif kind == 3:
            table[i][2] = n_users + int(r.integers(0, 3))         # user beyond the key set
        elif kind == 4:
            table[i][0] = n_rows + int(r.integers(0, 3))          # rows beyond the tensor
        elif kind == 5:
            table[i][1] = n_rows + 1 - table[i][0] + int(r.integers(0, 3))
        else:
            j = int(r.integers(0, len(table)))                    # a (user, iv_seq) twin
            table[i][2], table[i][3] = table[j][2], table[j][3]
    return [tuple(t) for t in table]


def test_random_tables_status_and_output_match_oracle(kt3):
    # overlapping rows, gaps, defects of every kind: the status is the
    # oracle's, and when the call is valid so is every byte of the result
    keys, nb, kt = kt3
    r = np.random.default_rng(77)
    n_ok = 0
    for case in range(300):
        n_rows, rb = int(r.integers(1, 9)), int(r.choice([4, 16, 20, 48]))
        table = random_table(r, n_rows, 3)
        data = r.integers(0, 256, n_rows * rb, dtype=np.uint8)
        st_o, o_out, o_tags, o_ver = oracle.seal(data, n_rows, rb, table, keys, nb)
        d = dev_u8(data)
        st_g = status_of(seal, d, n_rows, rb, table, kt, nb)
        assert st_g == st_o, (case, table)
        if st_o == 0:
            n_ok += 1
            out, tags, _ = seal(d, n_rows, rb, table, kt, nb)
            assert host(out).tobytes() == o_out.tobytes(), (case, table)
            assert host(tags)[:16 * len(table)].tobytes() == o_tags.tobytes(), (case, table)
    assert n_ok > 50


def test_random_multi_tile_tables_with_labels_and_tamper(kt3):
    # Segments of one to three 2 MiB tiles next to gaps and shorter ones:
    # every whole tile of a longer segment is cut into pieces at the tail of
    # the work queue (there are fewer than one per CU), one-tile segments get
    # their tags in the tile kernel.  Fused owner check with one relabelled
    # row, then open after one ciphertext bit and one tag bit are flipped:
    # every byte, tag and verdict equals the oracle's.
    keys, nb, kt = kt3
    r = np.random.default_rng(2024)
    for case in range(5):
        rb = int(r.choice([65536, 65536 + 48, 40000]))
        seg_rows = [int(x) for x in r.choice([1, 5, 32, 33, 47, 64, 65, 90], size=int(r.integers(3, 6)))]
        table, row, seq = [], 0, 1000 * case
        for k, n in enumerate(seg_rows):
            row += int(r.integers(0, 3))  # gap rows
            table.append((row, n, int(r.integers(0, 3)), seq + k))
            row += n
        n_rows = row + int(r.integers(0, 2))
        data = r.integers(0, 256, n_rows * rb, dtype=np.uint8)
        labels = np.full(n_rows, 0xFFFFFFFF, np.uint32)
        for (b, n, u, _) in table:
            labels[b:b + n] = u
        mixed = int(r.integers(0, len(table)))
        b, n, u, _ = table[mixed]
        labels[b + int(r.integers(0, n))] = (u + 1) % 3
        st, o_out, o_tags, o_ver = oracle.seal(data, n_rows, rb, table, keys, nb, labels=labels)
        assert st == 0
        d, lab = dev_u8(data), dev_u32(labels)
        out, tags, ver = seal(d, n_rows, rb, table, kt, nb, labels_dev=lab)
        n = len(table)
        assert host(ver)[:n].tolist() == o_ver.tolist(), (case, table)
        assert host(out).tobytes() == o_out.tobytes(), (case, table)
        assert host(tags)[:16 * n].tobytes() == o_tags.tobytes(), (case, table)
        # open without labels after flipping one ciphertext bit and one tag bit
        ok = [i for i in range(n) if i != mixed]
        ct_np, tg_np = o_out.copy().reshape(-1), o_tags.copy().reshape(-1)
        i_ct = ok[int(r.integers(0, len(ok)))]
        b, nr, _, _ = table[i_ct]
        ct_np[b * rb + int(r.integers(0, nr * rb))] ^= np.uint8(1 << int(r.integers(0, 8)))
        i_tg = ok[int(r.integers(0, len(ok)))]
        tg_np[16 * i_tg + int(r.integers(0, 16))] ^= np.uint8(1 << int(r.integers(0, 8)))
        st, o_back, o_ver2 = oracle.open_(ct_np, n_rows, rb, table, keys, nb, tg_np)
        assert st == 0
        back, ver2 = open_(dev_u8(ct_np), n_rows, rb, table, kt, nb, dev_u8(tg_np))
        assert host(ver2)[:n].tolist() == o_ver2.tolist(), (case, table)
        assert host(back).tobytes() == o_back.tobytes(), (case, table)


def test_one_tile_segments_cut_at_the_queue_tail(kt3):
    # More one-tile segments than CUs, most longer than a 32-row piece: the
    # largest tiles (up to one per CU) are cut into pieces at the tail of the
    # work queue, their segments lose the one-tile path and get their tags and
    # open verdicts from the finalize pass, next to uncut ones (short
    # segments, and long ones beyond the CU count).  Fused owner check with
    # two relabelled rows, then open with one ciphertext bit and one tag bit
    # flipped; the references are per-segment oracle GCM messages.
    keys, nb, kt = kt3
    r = np.random.default_rng(77)
    rb = 16384  # one tile row per tensor row
    seg_rows = [int(x) for x in r.integers(33, 41, 260)] + [int(x) for x in r.integers(1, 5, 40)]
    r.shuffle(seg_rows)
    table, row = [], 0
    for k, n in enumerate(seg_rows):
        table.append((row, n, k % 3, 5000 + k))
        row += n
    n_rows = row + 2  # two uncovered rows at the end
    n = len(table)
    data = r.integers(0, 256, n_rows * rb, dtype=np.uint8)
    labels = np.full(n_rows, 0xFFFFFFFF, np.uint32)
    for (b, nr, u, _) in table:
        labels[b:b + nr] = u
    mixed = [int(x) for x in r.choice(n, 2, replace=False)]
    for i in mixed:
        b, nr, u, _ = table[i]
        labels[b + int(r.integers(0, nr))] = (u + 1) % 3
    segs = gift.as_segments(table)
    ref = oracle_segments(keys, nb, segs, rb, lambda i: data[table[i][0] * rb:(table[i][0] + table[i][1]) * rb].tobytes())
    exp_out = np.zeros(n_rows * rb, np.uint8)
    exp_tags = np.zeros(16 * n, np.uint8)
    for i, (b, nr, _, _) in enumerate(table):
        if i not in mixed:
            exp_out[b * rb:(b + nr) * rb] = np.frombuffer(ref[i][0], np.uint8)
            exp_tags[16 * i:16 * i + 16] = np.frombuffer(ref[i][1], np.uint8)
    out, tags, ver = seal(dev_u8(data), n_rows, rb, table, kt, nb, labels_dev=dev_u32(labels))
    exp_ver = [gift.SEG_OWNER_MIXED if i in mixed else gift.SEG_OK for i in range(n)]
    assert host(ver)[:n].tolist() == exp_ver
    assert host(tags)[:16 * n].tobytes() == exp_tags.tobytes()
    assert host(out).tobytes() == exp_out.tobytes()
    # open, without labels, the sealed tensor with one ciphertext and one tag bit flipped
    ok = [i for i in range(n) if i not in mixed and seg_rows[i] > 32]
    i_ct, i_tg = [int(x) for x in r.choice(ok, 2, replace=False)]
    ct = exp_out.copy()
    b, nr, _, _ = table[i_ct]
    ct[b * rb + int(r.integers(0, nr * rb))] ^= np.uint8(1 << int(r.integers(0, 8)))
    tg = exp_tags.copy()
    tg[16 * i_tg + int(r.integers(0, 16))] ^= np.uint8(1 << int(r.integers(0, 8)))
    back, ver2 = open_(dev_u8(ct), n_rows, rb, table, kt, nb, dev_u8(tg))
    bad = set(mixed) | {i_ct, i_tg}  # the mixed segments' zero tags do not verify either
    assert host(ver2)[:n].tolist() == [gift.SEG_AUTH_FAIL if i in bad else gift.SEG_OK for i in range(n)]
    exp_back = np.zeros(n_rows * rb, np.uint8)
    for i, (b, nr, _, _) in enumerate(table):
        if i not in bad:
            exp_back[b * rb:(b + nr) * rb] = data[b * rb:(b + nr) * rb]
    assert host(back).tobytes() == exp_back.tobytes()


def test_one_tile_open_tamper_without_finalize(kt3):
    # At least one tile per CU, none longer than a 32-row piece: no tile is
    # cut, every segment is an uncut one-tile segment, and the call has no
    # finalize pass (the launch plan says so).  Open with ciphertext bits
    # flipped in three segments and tag bits in three others: the tile
    # kernel zeroes each failed tile itself (no later zeroing pass runs).
    # Whole-block rows and rows with a ragged, unaligned last block, out of
    # place and in place; every byte and verdict equals the oracle's open of
    # the tampered copy.
    import ctypes
    import subprocess
    keys, nb, kt = kt3
    lib = gift.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", gift.LIB_PATH], capture_output=True, text=True).stdout
    names = [l.split()[-1] for l in out.splitlines() if l.strip()]

    class QueuePlan(ctypes.Structure):
        _fields_ = [("cap", ctypes.c_uint64), ("grid", ctypes.c_uint32), ("finalize", ctypes.c_bool)]
    plan = getattr(lib, next(n for n in names if n.startswith("_ZN4gift10plan_queue")))
    plan.argtypes = [ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32]
    plan.restype = QueuePlan
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    r = np.random.default_rng(31)
    for rb in (16384, 16408):
        seg_rows = [int(x) for x in r.integers(1, 5, cus + 44)]
        table, row = [], 0
        for k, nr in enumerate(seg_rows):
            row += int(r.integers(0, 2))  # gap rows
            table.append((row, nr, k % 3, 7000 + k))
            row += nr
        n_rows, n = row, len(table)
        tile_rows = [-(-(-(-nr * rb // 16)) // 1024) for nr in seg_rows]
        assert not plan(n, sum(tile_rows), 0, max(tile_rows), cus).finalize
        data = r.integers(0, 256, n_rows * rb, dtype=np.uint8)
        st, ct_np, tg_np, _ = oracle.seal(data, n_rows, rb, table, keys, nb)
        assert st == 0
        ct_np, tg_np = ct_np.copy().reshape(-1), tg_np.copy().reshape(-1)
        picks = [int(x) for x in r.choice(n, 6, replace=False)]
        for i in picks[:3]:
            b, nr, _, _ = table[i]
            ct_np[b * rb + int(r.integers(0, nr * rb))] ^= np.uint8(1 << int(r.integers(0, 8)))
        for i in picks[3:]:
            tg_np[16 * i + int(r.integers(0, 16))] ^= np.uint8(1 << int(r.integers(0, 8)))
        st, o_back, o_ver = oracle.open_(ct_np, n_rows, rb, table, keys, nb, tg_np)
        assert st == 0
        assert sorted(i for i in range(n) if o_ver[i] != gift.SEG_OK) == sorted(picks)
        back, ver = open_(dev_u8(ct_np), n_rows, rb, table, kt, nb, dev_u8(tg_np))
        assert host(ver)[:n].tolist() == o_ver.tolist(), rb
        assert host(back).tobytes() == o_back.tobytes(), rb
        # in place: the failed tiles are zeroed over their own ciphertext
        buf = dev_u8(ct_np)
        back, ver = open_(buf, n_rows, rb, table, kt, nb, dev_u8(tg_np), out=buf)
        assert host(ver)[:n].tolist() == o_ver.tolist(), rb
        assert host(buf).tobytes() == o_back.tobytes(), rb


def test_in_place_rejection_and_tamper(kt3):
    # out == data with the owner check fused: a rejected segment is zeroed in
    # place and every other byte is sealed in place, for each kind of
    # segment -- small (one wave), one-tile (tag at the tile end), one-tile
    # cut into pieces at the queue tail (tag from the finalize pass) and
    # multi-tile with cut tiles; the call has more tiles than CUs, so the
    # largest tiles are cut at the tail of the work queue.  Then an in-place
    # open with one ciphertext bit and one tag bit flipped.  Every byte, tag
    # and verdict is compared with the oracle run in place on a host copy.
    keys, nb, kt = kt3
    r = np.random.default_rng(606)
    rb = 256
    kinds = ([("small", int(x)) for x in r.integers(1, 5, 6)] +
             [("one", int(x)) for x in r.integers(18, 25, 250)] +
             [("cut_one", int(x)) for x in r.integers(5200, 8100, 3)] +
             [("multi", int(x)) for x in r.integers(16500, 24000, 3)])
    order = r.permutation(len(kinds))
    kinds = [kinds[i] for i in order]
    table, row = [], 0
    for k, (_, n) in enumerate(kinds):
        row += int(r.random() < 0.02)  # a few uncovered rows
        table.append((row, n, int(r.integers(0, 3)), 9000 + k))
        row += n
    n_rows = row + 1
    n = len(table)
    labels = np.full(n_rows, 0xFFFFFFFF, np.uint32)
    for (b, nr, u, _) in table:
        labels[b:b + nr] = u
    mixed = []
    for kind in ("small", "one", "cut_one", "multi"):
        i = next(j for j in range(n) if kinds[j][0] == kind and j not in mixed)
        b, nr, u, _ = table[i]
        labels[b + int(r.integers(0, nr))] = (u + 1) % 3
        mixed.append(i)
    data = r.integers(0, 256, n_rows * rb, dtype=np.uint8)
    buf = data.copy()
    st, _, o_tags, o_ver = oracle.seal(buf, n_rows, rb, table, keys, nb, labels=labels, out=buf)
    assert st == 0 and sorted(np.flatnonzero(o_ver).tolist()) == sorted(mixed)
    d, lab = dev_u8(data), dev_u32(labels)
    out, tags, ver = seal(d, n_rows, rb, table, kt, nb, labels_dev=lab, out=d)
    assert out.data_ptr() == d.data_ptr()
    assert host(ver)[:n].tolist() == o_ver.tolist()
    assert host(tags)[:16 * n].tobytes() == o_tags.tobytes()
    assert host(d).tobytes() == buf.tobytes()
    # flip one ciphertext bit of a sealed multi-tile segment and one tag bit
    # of a sealed cut one-tile segment, on both sides
    i_ct = next(j for j in range(n) if kinds[j][0] == "multi" and j not in mixed)
    i_tg = next(j for j in range(n) if kinds[j][0] == "cut_one" and j not in mixed)
    b, nr, _, _ = table[i_ct]
    pos, bit = b * rb + int(r.integers(0, nr * rb)), int(r.integers(0, 8))
    buf[pos] ^= np.uint8(1 << bit)
    d[pos] ^= (1 << bit)
    tpos, tbit = 16 * i_tg + int(r.integers(0, 16)), int(r.integers(0, 8))
    tg = o_tags.reshape(-1).copy()
    tg[tpos] ^= np.uint8(1 << tbit)
    tags[tpos] ^= (1 << tbit)
    st, _, o_ver2 = oracle.open_(buf, n_rows, rb, table, keys, nb, tg, labels=labels, out=buf)
    assert st == 0
    _, ver2 = open_(d, n_rows, rb, table, kt, nb, tags, labels_dev=lab, out=d)
    assert host(ver2)[:n].tolist() == o_ver2.tolist()
    assert o_ver2[i_ct] == gift.SEG_AUTH_FAIL and o_ver2[i_tg] == gift.SEG_AUTH_FAIL
    assert host(d).tobytes() == buf.tobytes()
    # everything that verified is back to the plaintext
    for i, (b, nr, _, _) in enumerate(table):
        if o_ver2[i] == gift.SEG_OK:
            assert buf[b * rb:(b + nr) * rb].tobytes() == data[b * rb:(b + nr) * rb].tobytes(), i


def test_wrong_key_table_fails_every_segment(kt3):
    keys, nb, kt = kt3
    keys2, _ = keyset(3)
    kt2 = gift.KeyTable(keys2)
    n_rows, rb = 300, 8192
    data = dev_u8(rng.integers(0, 256, n_rows * rb, dtype=np.uint8))
    table = [(0, 1, 0, 1), (1, 200, 1, 1), (201, 99, 2, 1)]
    ct, tags, _ = seal(data, n_rows, rb, table, kt, nb)
    back, ver = open_(ct, n_rows, rb, table, kt2, nb, tags)
    assert host(ver)[:3].tolist() == [gift.SEG_AUTH_FAIL] * 3
    assert not host(back).any()
    kt2.destroy()


def test_non_default_stream(kt3):
    keys, nb, kt = kt3
    n_rows, rb = 200, 16384
    data_np = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    table = [(0, 150, 0, 3), (150, 50, 1, 3)]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        d = dev_u8(data_np)
        out, tags, _ = seal(d, n_rows, rb, table, kt, nb)
    s.synchronize()
    st, o_out, o_tags, _ = oracle.seal(data_np, n_rows, rb, table, keys, nb)
    assert host(out).tobytes() == o_out.tobytes() and host(tags)[:32].tobytes() == o_tags.tobytes()


def test_two_threads_on_two_streams_share_a_key_table(kt3):
    # calls from several host threads, each on its own stream, share one key
    # table and the library's per-device staging ring
    import threading
    keys, nb, kt = kt3
    n_rows, rb = 96, 65536  # 6 MiB per tensor: multi-tile segments
    cases = []
    for i in range(2):
        cases.append((rng.integers(0, 256, n_rows * rb, dtype=np.uint8),
                      [(0, 40, i, 100 + i), (40, 56, 2, 200 + i)]))
    results, errors = [None, None], []

    def work(i):
        try:
            data_np, table = cases[i]
            s = torch.cuda.Stream()
            outs = []
            with torch.cuda.stream(s):
                for _ in range(4):
                    d = dev_u8(data_np)
                    out, tags, _ = seal(d, n_rows, rb, table, kt, nb)
                    back, ver = open_(out, n_rows, rb, table, kt, nb, tags)
                    outs.append((out, tags, back, ver))
            s.synchronize()
            results[i] = [(o.cpu().numpy(), tg.cpu().numpy(), b.cpu().numpy(), v.cpu().numpy())
                          for o, tg, b, v in outs]
        except Exception as e:  # surfaced in the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i, (data_np, table) in enumerate(cases):
        st, o_out, o_tags, _ = oracle.seal(data_np, n_rows, rb, table, keys, nb)
        assert st == 0
        for out, tags, back, ver in results[i]:
            assert out.tobytes() == o_out.tobytes()
            assert tags[:32].tobytes() == o_tags.tobytes()
            assert back.tobytes() == data_np.tobytes()
            assert ver[:2].tolist() == [gift.SEG_OK, gift.SEG_OK]


def test_a_call_does_not_wait_for_another_streams_call(kt3):
    # A call's staging event also marks its scratch buffer's last use, and the
    # staging ring hands a completed event out again, here to a call on
    # stream B queued behind a long busy wait.  The next call on stream A must
    # not wait for stream B through that event.
    import time
    keys, nb, kt = kt3
    n_rows, rb = 16, 8192
    table = [(0, 8, 0, 900), (8, 8, 1, 901)]
    data_np = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    d = dev_u8(data_np)
    outs = [torch.empty_like(d) for _ in range(3)]
    tags = [torch.zeros(32, dtype=torch.uint8, device=DEV) for _ in range(3)]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    # size a bounded busy wait of about 0.3 s on this GPU
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    torch.cuda._sleep(10 ** 7)
    torch.cuda.synchronize()
    per_cycle = (time.perf_counter() - t0) / 1e7
    if per_cycle <= 0:
        pytest.skip("torch.cuda._sleep does not wait on this build")
    cycles = int(min(0.3 / per_cycle, 5e10))
    gift.seal(d, n_rows, rb, table, kt, nb, outs[0], tags[0], stream=sa)
    torch.cuda.synchronize()  # A's call is done: its staging event goes back to the ring's pool
    with torch.cuda.stream(sb):
        torch.cuda._sleep(cycles)
    gift.seal(d, n_rows, rb, table, kt, nb, outs[1], tags[1], stream=sb)  # takes that event, behind the wait
    t0 = time.perf_counter()
    gift.seal(d, n_rows, rb, table, kt, nb, outs[2], tags[2], stream=sa)
    sa.synchronize()
    dt = time.perf_counter() - t0
    b_busy = not sb.query()
    torch.cuda.synchronize()
    assert b_busy, "stream B finished before the check could see it"
    assert dt < 0.1, f"the call on stream A waited {dt:.3f} s for stream B"
    st, o_out, o_tags, _ = oracle.seal(data_np, n_rows, rb, table, keys, nb)
    assert st == 0
    for o, t in zip(outs, tags):
        assert host(o).tobytes() == o_out.tobytes() and host(t).tobytes() == o_tags.tobytes()


def test_scratch_reuse_across_streams_threads_and_sizes(kt3):
    # the library keeps each stream's device scratch between calls: more
    # streams than it caches (buffers change hands), two host threads on one
    # stream, and growing then shrinking tables on one stream
    import threading
    keys, nb, kt = kt3
    cases = []
    for i in range(24):
        n_segs = [1, 3, 40, 700][i % 4]
        rb = 64 if n_segs > 3 else 4096 + 48 * i
        n_rows = n_segs * (2 if rb == 64 else 5)
        data_np = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
        per = n_rows // n_segs
        table = [(k * per, per, (k + i) % 3, 1000 * i + k) for k in range(n_segs)]
        st, o_out, o_tags, _ = oracle.seal(data_np, n_rows, rb, table, keys, nb)
        assert st == 0
        cases.append((data_np, n_rows, rb, table, o_out, o_tags))

    def check(i, out, tags, back, ver):
        data_np, n_rows, rb, table, o_out, o_tags = cases[i]
        n = len(table)
        assert host(out).tobytes() == o_out.tobytes(), i
        assert host(tags)[:16 * n].tobytes() == o_tags.tobytes(), i
        assert host(back).tobytes() == data_np.tobytes(), i
        assert (host(ver)[:n] == gift.SEG_OK).all(), i

    def run(i, stream):
        data_np, n_rows, rb, table, _, _ = cases[i]
        with torch.cuda.stream(stream):
            d = dev_u8(data_np)
            out, tags, _ = seal(d, n_rows, rb, table, kt, nb)
            back, ver = open_(out, n_rows, rb, table, kt, nb, tags)
        return out, tags, back, ver

    streams = [torch.cuda.Stream() for _ in range(20)]
    res = [run(i, streams[i % 20]) for i in range(24)]
    torch.cuda.synchronize()
    for i, r in enumerate(res):
        check(i, *r)

    shared = torch.cuda.Stream()
    got, errors = {}, []

    def work(t):
        try:
            for i in range(t, 24, 2):
                got[i] = run(i, shared)
        except Exception as e:  # surfaced in the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for i, r in got.items():
        check(i, *r)
    assert len(got) == 24


def test_scratch_reuse_when_one_handle_names_several_streams(kt3):
    # a stream destroyed while the library's work on it is in flight hands its
    # handle to the next stream created, and hipStreamPerThread is one handle
    # for a different stream in each thread: each must get scratch of its own
    import ctypes
    import threading
    hip = ctypes.CDLL("libamdhip64.so")
    keys, nb, kt = kt3

    def case(n_segs, rows_per_seg, rb, user0, seq0):
        n_rows = n_segs * rows_per_seg
        data_np = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
        table = [(k * rows_per_seg, rows_per_seg, (user0 + k) % 3, seq0 + k) for k in range(n_segs)]
        return data_np, n_rows, rb, table

    def buffers(c):
        data_np, n_rows, rb, table = c
        n = len(table)
        return (dev_u8(data_np), torch.empty(n_rows * rb, dtype=torch.uint8, device=DEV),
                torch.zeros(n * 16, dtype=torch.uint8, device=DEV))

    def check(c, out, tags):
        # segments tile the rows in order, so the output is their concatenation
        data_np, n_rows, rb, table = c
        segs = gift.as_segments(table)
        per = int(segs[0]["row_count"]) * rb
        ref = oracle_segments(keys, nb, segs, rb, lambda i: data_np[i * per:(i + 1) * per].tobytes())
        assert host(out).tobytes() == b"".join(ct for ct, _ in ref)
        assert host(tags).tobytes() == b"".join(tag for _, tag in ref)

    big = case(32, 128, 65536, 0, 50000)     # 256 MiB, still running when the next call is enqueued
    small = case(40, 2, 64, 1, 60000)
    bufs_big, bufs_small = buffers(big), buffers(small)
    torch.cuda.synchronize()
    sa, sb = ctypes.c_void_p(), ctypes.c_void_p()
    assert hip.hipStreamCreate(ctypes.byref(sa)) == 0
    gift.seal(bufs_big[0], big[1], big[2], big[3], kt, nb, bufs_big[1], bufs_big[2], stream=sa.value)
    assert hip.hipStreamDestroy(sa) == 0
    assert hip.hipStreamCreate(ctypes.byref(sb)) == 0
    gift.seal(bufs_small[0], small[1], small[2], small[3], kt, nb, bufs_small[1], bufs_small[2], stream=sb.value)
    assert hip.hipStreamSynchronize(sb) == 0
    torch.cuda.synchronize()
    assert hip.hipStreamDestroy(sb) == 0
    check(big, bufs_big[1], bufs_big[2])
    check(small, bufs_small[1], bufs_small[2])

    per_thread = 2  # hipStreamPerThread
    cases = [[case(n, r, rb, t, 70000 + 1000 * t + 100 * i)
              for i, (n, r, rb) in enumerate([(8, 64, 8192), (40, 2, 64), (3, 20, 4096), (700, 2, 64)])]
             for t in range(2)]
    bufs = [[buffers(c) for c in cs] for cs in cases]
    torch.cuda.synchronize()
    errors = []

    def work(t):
        try:
            for c, (d, out, tags) in zip(cases[t], bufs[t]):
                gift.seal(d, c[1], c[2], c[3], kt, nb, out, tags, stream=per_thread)
            assert hip.hipStreamSynchronize(ctypes.c_void_p(per_thread)) == 0
        except Exception as e:  # surfaced in the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for t in range(2):
        for c, (d, out, tags) in zip(cases[t], bufs[t]):
            check(c, out, tags)


def test_llama3_8b_kv_every_segment_verifies_in_openssl():
    # Every ciphertext byte and every tag at full size, checked by an
    # independent GCM implementation (OpenSSL, which also pins the oracle):
    # it must accept each segment's tag and decrypt to the plaintext.  The
    # work queue here splits 256 of the 4,321 tiles into pieces, inside
    # segments whose other tiles stay whole.
    import openssl_ref
    if not openssl_ref.available():
        pytest.skip("libcrypto not found")
    from concurrent.futures import ThreadPoolExecutor
    w = W.llama3_8b_kv()
    t = w.tensors[0]
    kt = gift.KeyTable(w.keys)
    d = t.generate(DEV)
    ct, tags, ver = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base)
    assert (host(ver) == 0).all()
    ct_h, pt_h, tg = host(ct), host(d), host(tags).reshape(-1, 16)
    del ct, d
    kt.destroy()

    def verifies(i):
        s = t.segs[i]
        off, ln = t.seg_bytes(i)
        u = int(s["user"])
        iv = oracle.segment_iv(w.nonce_base[u].tobytes(), int(s["iv_seq"]))
        p = openssl_ref.gcm_decrypt(w.keys[u].tobytes(), iv, ct_h[off:off + ln], tg[i].tobytes())
        return p is not None and p == pt_h[off:off + ln].tobytes()

    with ThreadPoolExecutor(8) as ex:
        ok = list(ex.map(verifies, range(len(t.segs))))
    assert all(ok), [i for i, o in enumerate(ok) if not o]


def test_decode_batch_full_size():
    w = W.decode_batch()
    kt = gift.KeyTable(w.keys)
    for t in w.tensors:
        data = t.generate("cpu").numpy()
        d = dev_u8(data)
        ct, tags, ver = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base)
        res = oracle_segments(w.keys, w.nonce_base, t.segs, t.row_bytes,
                              lambda i: data[slice(*(lambda o, l: (o, o + l))(*t.seg_bytes(i)))].tobytes())
        got = host(ct)
        gt = host(tags).reshape(-1, 16)
        for i in range(len(t.segs)):
            off, ln = t.seg_bytes(i)
            assert got[off:off + ln].tobytes() == res[i][0], (t.name, i)
            assert gt[i].tobytes() == res[i][1], (t.name, i)
        back, ver2 = open_(ct, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base, tags)
        assert (host(ver2) == 0).all() and torch.equal(back, d)
    kt.destroy()


# --------------------------------------------------------------------------
# limits
# --------------------------------------------------------------------------
def test_segment_at_the_gcm_length_limit():
    """One segment of exactly 2^32 - 2 blocks (64 GiB - 32 B): the last block
    uses counter 2^32 - 1.  2^31 - 1 is prime, so the segment is 2 rows of
    16 * (2^31 - 1) bytes."""
    keys, nb = keyset(1)
    kt = gift.KeyTable(keys)
    rb = 16 * ((1 << 31) - 1)
    n_rows = 2
    total = n_rows * rb
    d = torch.empty(total, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    chunk = 1 << 30
    for o in range(0, total, chunk):
        n = min(chunk, total - o)
        d[o:o + n] = torch.randint(0, 256, (n,), dtype=torch.uint8, device=DEV, generator=g)
    ref = d.clone()
    table = [(0, 2, 0, 123)]
    tags = torch.zeros(16, dtype=torch.uint8, device=DEV)
    ver = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    gift.seal(d, n_rows, rb, table, kt, nb, d, tags, verdicts=ver)
    seg = oracle.as_segments(table)[0]
    nblk = (1 << 32) - 2
    picks = [0, 1, 2, 4095, 65535, 65536, 1 << 20, (1 << 31) - 2, (1 << 31) - 1, nblk - 65537, nblk - 3, nblk - 2,
             nblk - 1] + [int(x) for x in rng.integers(0, nblk, 48)]
    idx = torch.tensor([16 * j + k for j in picks for k in range(16)], dtype=torch.int64, device=DEV)
    plain = host(ref[idx])
    got = host(d[idx])
    for n, j in enumerate(picks):
        exp = expected_block(keys, nb, seg, j, plain[16 * n:16 * n + 16].tobytes())
        assert got[16 * n:16 * n + 16].tobytes() == exp, j
    gift.open(d, n_rows, rb, table, kt, nb, d, tags, ver)
    assert host(ver)[0] == gift.SEG_OK
    assert torch.equal(d, ref)
    # a single flipped bit anywhere in the 64 GiB ciphertext fails the segment
    gift.seal(d, n_rows, rb, table, kt, nb, d, tags, verdicts=ver)
    d[total - 1] ^= 0x80
    gift.open(d, n_rows, rb, table, kt, nb, d, tags, ver)
    assert host(ver)[0] == gift.SEG_AUTH_FAIL
    assert not d[total - (1 << 20):].any().item() and not d[:1 << 20].any().item()
    del d, ref
    torch.cuda.empty_cache()
    kt.destroy()


def test_one_block_over_the_limit_is_rejected(kt3):
    keys, nb, kt = kt3
    small = dev_u8(np.zeros(64, np.uint8))
    tags = torch.zeros(16, dtype=torch.uint8, device=DEV)
    # 2^32 - 1 blocks: never touched, rejected on the host.  The library
    # trusts the declared tensor size, so only calls that the host rejects may
    # describe more bytes than the buffer holds; raw addresses keep the
    # binding's own size check out of the way of the C ABI's.
    p, tp = small.data_ptr(), tags.data_ptr()
    s = status_of(gift.seal, p, 1, 16 * ((1 << 32) - 1), [(0, 1, 0, 0)], kt, nb, p, tp)
    assert s == gift.E_TOO_LARGE
    s = status_of(gift.seal, p, 3, 16 * ((1 << 31) - 1), [(0, 3, 0, 0)], kt, nb, p, tp)
    assert s == gift.E_TOO_LARGE
    with pytest.raises(ValueError, match="data: 64 bytes"):
        gift.seal(small, 1, 16 * ((1 << 32) - 1), [(0, 1, 0, 0)], kt, nb, small, tags)


def test_many_segments_and_users():
    """70,000 segments (descriptors larger than half the pinned ring) over
    5,000 users, mixing one-block, small and tiled segments."""
    n_users = 5000
    keys = rng.integers(0, 256, (n_users, 32), dtype=np.uint8)
    nb = rng.integers(0, 256, (n_users, 12), dtype=np.uint8)
    kt = gift.KeyTable(keys)
    rb = 48
    sizes = rng.integers(1, 4, 70000)
    sizes[::997] = 3000  # a few 144 KB segments -> tiled path with a ragged tile
    table, r = [], 0
    for i, n in enumerate(sizes):
        table.append((r, int(n), int(rng.integers(0, n_users)), i))
        r += int(n) + (i % 3 == 0)
    n_rows = r
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    st, o_out, o_tags, _ = oracle.seal(data, n_rows, rb, table, keys, nb)
    d = dev_u8(data)
    out, tags, ver = seal(d, n_rows, rb, table, kt, nb)
    assert host(out).tobytes() == o_out.tobytes()
    assert host(tags)[:16 * len(table)].tobytes() == o_tags.tobytes()
    back, ver2 = open_(out, n_rows, rb, table, kt, nb, tags)
    assert (host(ver2) == 0).all()
    covered = np.zeros(n_rows, bool)
    for b, c, _, _ in table:
        covered[b:b + c] = True
    exp = data.reshape(n_rows, rb).copy()
    exp[~covered] = 0
    assert host(back).tobytes() == exp.tobytes()
    kt.destroy()


# --------------------------------------------------------------------------
# per-token encryption (GIFT Sec. 4.5)
# --------------------------------------------------------------------------
def dev_u64(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint64).view(np.int64).copy()).to(DEV)


def host_u64(t):
    return host(t).view(np.uint64)


def token_case(keys, kt, segs, tok, non, eos):
    n = tok.size
    st, o_blocks = oracle.token_encrypt(segs, tok, non, keys, eos)
    assert st == 0
    out = torch.full((max(n, 1) * 16,), 0x5A, dtype=torch.uint8, device=DEV)
    gift.token_encrypt(segs, dev_u64(tok), dev_u64(non), n, kt, eos, out)
    assert host(out)[:16 * n].tobytes() == o_blocks.tobytes()
    st, o_tok, o_non = oracle.token_decrypt(segs, o_blocks, keys, eos)
    t_out = torch.full((max(n, 1),), 77, dtype=torch.int64, device=DEV)
    n_out = torch.full((max(n, 1),), 77, dtype=torch.int64, device=DEV)
    gift.token_decrypt(segs, out, n, kt, eos, t_out, n_out)
    assert (host_u64(t_out)[:n] == o_tok).all() and (host_u64(n_out)[:n] == o_non).all()


def test_token_encryption_matches_oracle():
    w = W.decode_batch()
    t = w.tensors[1]  # int32 token buffer with the decode batch's ownership
    kt = gift.KeyTable(w.keys)
    tok = t.generate("cpu").numpy().view(np.int32).astype(np.uint64)
    eos = 128001
    tok[::97] = eos
    non = W.u64s(w.seed, "token_nonce", tok.size)
    token_case(w.keys, kt, t.segs, tok, non, eos)
    # gaps, EOS everywhere, a single token, a user appearing twice, no segments
    token_case(w.keys, kt, [(1, 3, 5, 0), (7, 2, 5, 1)], tok[:12], non[:12], eos)
    token_case(w.keys, kt, [(0, 12, 3, 0)], np.full(12, eos, np.uint64), non[:12], eos)
    token_case(w.keys, kt, [(0, 1, 1023, 0)], tok[:1], non[:1], eos)
    token_case(w.keys, kt, [], tok[:5], non[:5], eos)
    # 100k tokens of one user (many rows per workgroup)
    big = W.u64s(1, "big_tok", 100000) % np.uint64(128256)
    token_case(w.keys, kt, [(0, 100000, 7, 0)], big, W.u64s(1, "big_non", 100000), eos)
    # 64-token chunks that end inside, at and just past a segment, a table out
    # of row order, gaps between segments
    token_case(w.keys, kt, [(300, 65, 4, 0), (0, 64, 2, 0), (64, 63, 3, 0), (130, 1, 5, 0), (131, 128, 6, 0),
                            (500, 200, 2, 1)], big[:800], W.u64s(2, "chunk_non", 800), eos)
    # segment counts around the 64-way chunk search's steps (one, two and three
    # rounds), segments of 1-130 tokens (one to three chunks each)
    r = np.random.default_rng(64)
    for n_seg in (63, 64, 65, 4097):
        rows = r.integers(1, 131, n_seg)
        starts = np.concatenate([[0], np.cumsum(rows)[:-1]])
        segs = [(int(b), int(c), int(u), 0) for b, c, u in zip(starts, rows, r.integers(0, 1024, n_seg))]
        n_tok = int(rows.sum())
        token_case(w.keys, kt, segs, W.u64s(3, "search_tok", n_tok) % np.uint64(128256),
                   W.u64s(3, "search_non", n_tok), eos)
    # validation agrees with the oracle
    dt, dn = dev_u64(tok[:8]), dev_u64(non[:8])
    out = torch.zeros(128, dtype=torch.uint8, device=DEV)
    for segs in ([(0, 0, 0, 0)], [(7, 2, 0, 0)], [(0, 2, 1024, 0)], [(0, 2, 0, 0), (1, 2, 1, 0)],
                 [(0, 2, 0, 7), (2, 2, 0, 7)]):
        st_o = oracle.token_encrypt(segs, tok[:8], non[:8], w.keys, eos)[0]
        assert status_of(gift.token_encrypt, segs, dt, dn, 8, kt, eos, out) == st_o, segs
    kt.destroy()


# --------------------------------------------------------------------------
# paged KV: seal from / open into a paged cache through block tables
# --------------------------------------------------------------------------
def paged_geom(layout, layers, parts, blocks, chunk):
    if layout == "lbp":
        ps, bs, ls = chunk, parts * chunk, blocks * parts * chunk
    else:
        bs, ps, ls = chunk, blocks * chunk, parts * blocks * chunk
    return oracle.PagedKV(layers * ls, ls, bs, ps, chunk, layers, parts, blocks)


def dev_kv(g, cache_dev):
    return gift.paged_kv(cache_dev, g.cache_bytes, g.layer_stride, g.block_stride, g.part_stride, g.chunk_bytes,
                         g.n_layers, g.n_parts, g.n_blocks)


def gather_blocks(cache, g, bids):
    """The bytes of the given blocks, every layer and part, from a host copy."""
    out = []
    for b in bids:
        for l in range(g.n_layers):
            for p in range(g.n_parts):
                o = l * g.layer_stride + int(b) * g.block_stride + p * g.part_stride
                out.append(cache[o:o + g.chunk_bytes].tobytes())
    return b"".join(out)


def paged_case(keys, nb, kt, g, reqs, moved=None, labels=None, tamper=None, want_cache=False):
    cache = rng.integers(0, 256, g.cache_bytes, dtype=np.uint8)
    st, o_sealed, o_tags, o_ver = oracle.seal_paged(cache, g, reqs, keys, nb, labels=labels)
    assert st == 0
    c_dev = dev_u8(cache)
    kv = dev_kv(g, c_dev)
    n = len(reqs)
    total = o_sealed.size
    sealed = torch.full((max(total, 16),), 0x5A, dtype=torch.uint8, device=DEV)
    tags = torch.zeros(16 * n, dtype=torch.uint8, device=DEV)
    ver = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    lab = None if labels is None else dev_u32(labels)
    gift.seal_paged(kv, reqs, kt, nb, sealed, tags, block_labels=lab, verdicts=ver)
    assert host(sealed)[:total].tobytes() == o_sealed.tobytes()
    assert host(tags).tobytes() == o_tags.tobytes()
    assert host(ver).tolist() == o_ver.tolist()
    assert torch.equal(c_dev, dev_u8(cache))  # the source cache is untouched
    if tamper is not None:
        o_sealed = o_sealed.copy()
        o_sealed[tamper] ^= 1
        sealed[tamper] ^= 1
    dst = moved if moved is not None else reqs
    st, o_after, o_ver2 = oracle.open_paged(cache, g, dst, keys, nb, o_sealed, o_tags, labels=labels)
    ver2 = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    gift.open_paged(kv, dst, kt, nb, sealed, tags, ver2, block_labels=lab)
    assert host(ver2).tolist() == o_ver2.tolist()
    after = host(c_dev)
    assert after.tobytes() == o_after.tobytes()
    if want_cache:
        return o_ver, o_ver2, cache, after
    return o_ver, o_ver2


def random_tables(n_blocks, sizes, n_users, rng_):
    perm = rng_.permutation(n_blocks)
    reqs, p = [], 0
    for i, k in enumerate(sizes):
        reqs.append((perm[p:p + k].astype(np.uint32), int(rng_.integers(0, n_users)), 100 + i))
        p += k
    return reqs, perm[p:]


@pytest.mark.parametrize("layout,layers,parts,blocks,chunk,sizes", [
    ("lbp", 4, 1, 40, 65536, [4, 1, 3, 6, 2, 5]),      # K+V in one 64 KiB chunk per layer
    ("lpb", 3, 2, 64, 32768, [3, 3, 1, 8, 2]),         # K and V planes apart
    ("lbp", 5, 2, 300, 256, [20, 1, 37, 64, 5, 90]),   # rows span many chunks
    ("lpb", 2, 1, 5000, 16, [1000, 1, 2047, 900]),     # one block per chunk
])
def test_paged_seal_open_every_byte(kt3, layout, layers, parts, blocks, chunk, sizes):
    keys, nb, kt = kt3
    g = paged_geom(layout, layers, parts, blocks, chunk)
    r_ = np.random.default_rng(blocks)
    reqs, spare = random_tables(blocks, sizes, 3, r_)
    ver, ver2 = paged_case(keys, nb, kt, g, reqs)
    assert (ver == 0).all() and (ver2 == 0).all()
    # swap-in: the same sealed data opened into other (spare + shuffled) blocks
    pool = r_.permutation(np.concatenate([np.concatenate([b for b, _, _ in reqs]), spare]))
    moved, p = [], 0
    for b, u, q in reqs:
        moved.append((pool[p:p + len(b)].astype(np.uint32), u, q))
        p += len(b)
    paged_case(keys, nb, kt, g, reqs, moved=moved)


def test_paged_manipulated_table_and_tamper(kt3):
    keys, nb, kt = kt3
    g = paged_geom("lbp", 3, 2, 50, 4096)
    r_ = np.random.default_rng(11)
    reqs, _ = random_tables(50, [5, 4, 6, 3], 3, r_)
    labels = np.full(50, gift.LABEL_UNOWNED, np.uint32)
    for b, u, _ in reqs:
        labels[b] = u
    ver, ver2 = paged_case(keys, nb, kt, g, reqs, labels=labels)
    assert (ver == 0).all() and (ver2 == 0).all()
    # request 1's table now also names request 0's block (different owner)
    other = reqs[0][1] if reqs[0][1] != reqs[1][1] else None
    evil = list(reqs)
    if other is None:
        labels[reqs[0][0][0]] = (reqs[1][1] + 1) % 3
    evil[1] = (np.concatenate([reqs[1][0], reqs[0][0][:1]]), reqs[1][1], reqs[1][2])
    evil[0] = (reqs[0][0][1:], reqs[0][1], reqs[0][2])
    ver, ver2, before, after = paged_case(keys, nb, kt, g, evil, labels=labels, want_cache=True)
    assert ver[1] == gift.SEG_OWNER_MIXED and ver2[1] == gift.SEG_OWNER_MIXED
    # the rejected open wrote nothing: the foreign block named by the
    # manipulated table, and the request's own blocks, keep their contents
    for b in evil[1][0]:
        assert gather_blocks(after, g, [b]) == gather_blocks(before, g, [b]), f"block {b}" 
    # a flipped ciphertext bit in request 2 fails it and zeroes its blocks
    per = g.n_layers * g.n_parts * g.chunk_bytes
    off = per * (len(reqs[0][0]) + len(reqs[1][0])) + 77
    ver, ver2 = paged_case(keys, nb, kt, g, reqs, tamper=off)
    assert ver2.tolist() == [0, 0, gift.SEG_AUTH_FAIL, 0]


def test_paged_validation_matches_oracle(kt3):
    keys, nb, kt = kt3
    g = paged_geom("lbp", 3, 2, 10, 64)
    cache = np.zeros(g.cache_bytes, np.uint8)
    c_dev = dev_u8(cache)
    out = torch.zeros(1 << 16, dtype=torch.uint8, device=DEV)
    tags = torch.zeros(64, dtype=torch.uint8, device=DEV)
    geoms = [g, paged_geom("lbp", 3, 2, 10, 48),
             oracle.PagedKV(g.cache_bytes, g.layer_stride, 32, g.part_stride, 64, 3, 2, 10),
             oracle.PagedKV(g.cache_bytes // 2, g.layer_stride, g.block_stride, g.part_stride, 64, 3, 2, 10)]
    tables = [[([1], 0, 0)], [([], 0, 0)], [([10], 0, 0)], [([1], 3, 0)], [([1, 2], 0, 0), ([2], 1, 0)],
              [([1], 0, 4), ([2], 0, 4)], [([1], gift.LABEL_PARAM, 0)]]
    for gg in geoms:
        for reqs in tables:
            st_o = oracle.seal_paged(cache, gg, reqs, keys, nb)[0]
            st_g = status_of(gift.seal_paged, dev_kv(gg, c_dev), reqs, kt, nb, out, tags)
            assert st_g == st_o, (gg.chunk_bytes, gg.block_stride, gg.cache_bytes, reqs)
    # the export buffer may not overlap the cache
    assert status_of(gift.seal_paged, dev_kv(g, c_dev), [([1], 0, 0)], kt, nb, c_dev[64:], tags) == gift.E_INVALID


def test_paged_full_size_equals_contiguous_seal():
    """The llama3_8b_kv tensor scattered into a vLLM-style per-layer cache
    ([layer][block][64 KiB], 5% spare blocks, random placement): sealing
    through the block tables reproduces the contiguous seal exactly, and
    opening into fresh blocks restores every chunk."""
    w = W.llama3_8b_kv()
    t = w.tensors[0]
    kt = gift.KeyTable(w.keys)
    L, C = 32, t.row_bytes
    nblk_req = [int(s["row_count"]) // L for s in t.segs]
    B = sum(nblk_req)
    NB = B + B // 20
    d = t.generate(DEV)
    ct, tags, _ = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base)
    r_ = np.random.default_rng(3)
    perm = r_.permutation(NB)[:B]
    cache = torch.zeros(L * NB * C, dtype=torch.uint8, device=DEV)
    cv = cache.view(L, NB, C)
    pidx = torch.from_numpy(perm).to(DEV)
    cv[:, pidx, :] = d.view(B, L, C).transpose(0, 1)
    reqs, p = [], 0
    for i, k in enumerate(nblk_req):
        s = t.segs[i]
        reqs.append((perm[p:p + k].astype(np.uint32), int(s["user"]), int(s["iv_seq"])))
        p += k
    kv = gift.paged_kv(cache, cache.numel(), NB * C, C, 0, C, L, 1, NB)
    sealed = torch.empty_like(d)
    ptags = torch.zeros_like(tags)
    ver = torch.full((len(reqs),), -1, dtype=torch.int32, device=DEV)
    gift.seal_paged(kv, reqs, kt, w.nonce_base, sealed, ptags, verdicts=ver)
    assert (host(ver) == 0).all()
    assert torch.equal(sealed, ct) and torch.equal(ptags, tags)
    # open into a fresh placement
    perm2 = r_.permutation(NB)[:B]
    moved, p = [], 0
    for (b, u, q), k in zip(reqs, nblk_req):
        moved.append((perm2[p:p + k].astype(np.uint32), u, q))
        p += k
    cache.zero_()
    gift.open_paged(kv, moved, kt, w.nonce_base, sealed, ptags, ver)
    assert (host(ver) == 0).all()
    assert torch.equal(cv[:, torch.from_numpy(perm2).to(DEV), :], d.view(B, L, C).transpose(0, 1))
    kt.destroy()
