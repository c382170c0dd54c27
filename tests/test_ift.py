"""Host-side ownership records, IFT rules and launch-order checking of
libgift.so (include/gift_ift.h) against the element-level and history-graph
oracle (oracle/ift.py).  No GPU: these entry points make no HIP call."""
import os

import numpy as np
import pytest

from oracle import ift
from paper_2608_25431_amd import gift

P, X = gift.LABEL_PARAM, gift.LABEL_UNOWNED


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(gift.LIB_PATH):
        from paper_2608_25431_amd import build
        build.build()


# fake device addresses: records are keyed by address, nothing is dereferenced
def addrs(n, stride=1 << 24):
    return [0x7F0000000000 + i * stride for i in range(n)]


# --- ownership records (Sec. 4.1-4.2) --------------------------------------
def test_batched_records_one_per_row():
    # Sec. 4.1 Insight 1: a [B, H] hidden-state matrix needs B records, not B*H
    o = gift.Ownership()
    (a,) = addrs(1)
    o.register(a, (32, 4096), 2, odims=(0,))
    assert o.units(a) == 32
    assert list(o.labels(a)) == [X] * 32


def test_kv_tensor_block_slice_ownership():
    # Sec. 4.1 Insight 3 / 4.2: a 5-D paged KV tensor C with odim (0, 1, 3);
    # the slice C[1, 2, :, 0:8, :] is eight units, contiguous in flat order
    o = gift.Ownership()
    (c,) = addrs(1)
    shape = (3, 4, 2, 16, 64)  # (layer, block, k/v, head, dim) for example
    o.register(c, shape, 2, odims=(0, 1, 3))
    assert o.units(c) == 3 * 4 * 16
    f0 = o.flat_index(c, (1, 2, 0))
    assert f0 == (1 * 4 + 2) * 16
    o.set(c, f0, 8, 7)
    lab = o.labels(c).reshape(3, 4, 16)
    assert (lab[1, 2, :8] == 7).all() and (lab[1, 2, 8:] == X).all()
    assert (lab[0] == X).all() and (lab[2] == X).all() and (lab[1, [0, 1, 3]] == X).all()
    assert o.get(c, f0 + 7) == 7 and o.get(c, f0 + 8) == X
    with pytest.raises(gift.GiftError) as e:
        o.flat_index(c, (1, 4, 0))
    assert e.value.status == gift.E_RANGE


def test_records_without_odim_have_one_unit():
    o = gift.Ownership()
    (w,) = addrs(1)
    o.register(w, (64, 64), 2, odims=())
    assert o.units(w) == 1 and o.flat_index(w, ()) == 0


def test_register_rejections():
    o = gift.Ownership()
    a, b = addrs(2, stride=4096)
    o.register(a, (16, 128), 2)  # exactly 4096 bytes
    o.register(b, (1,), 1)  # adjacent, not overlapping
    with pytest.raises(gift.GiftError) as e:
        o.register(a + 4094, (2,), 2)
    assert e.value.status == gift.E_OVERLAP
    for bad in [((0, 4), 2, (0,)), ((4,), 0, (0,)), ((4,), 2, (1,)), ((2,) * 9, 1, (0,))]:
        with pytest.raises(gift.GiftError) as e:
            o.register(a + (1 << 30), *bad)
        assert e.value.status == gift.E_INVALID
    with pytest.raises(gift.GiftError) as e:
        o.set(a, 10, 7, 1)
    assert e.value.status == gift.E_RANGE


def test_release_clears_records():
    # Sec. 4.2: records are cleared when the tensor is released
    o = gift.Ownership()
    (a,) = addrs(1)
    o.register(a, (4, 8), 4)
    o.set(a, 0, 4, 3)
    o.release(a)
    with pytest.raises(gift.GiftError):
        o.labels(a)
    o.register(a, (4, 8), 4)
    assert list(o.labels(a)) == [X] * 4


# --- the 2B+1 operation count (Sec. 4.1 Insight 2) --------------------------
@pytest.mark.parametrize("B", [1, 7, 64, 1000])
def test_add_bias_costs_two_b_plus_one_record_operations(B):
    # check the bias is parameter-owned (1), read B input row records (B),
    # write B output row records (B)
    H = 4096
    o = gift.Ownership()
    x, bias, y = addrs(3, stride=1 << 30)
    o.register(x, (B, H), 2)
    o.register(bias, (H,), 2, odims=())
    o.register(y, (B, H), 2)
    o.set(bias, 0, 1, P)
    o.set(x, 0, B, 5)
    before = o.ops
    assert o.add_bias(y, x, bias, B, H, 2) == gift.OK
    assert o.ops - before == 2 * B + 1


# --- rules versus the element-level oracle ----------------------------------
def _rand_rows(rng, n, users, p_param=0.05, p_unowned=0.03):
    r = rng.choice(users, n).astype(np.uint64)
    u = rng.random(n)
    r[u < p_param] = P
    r[(u >= p_param) & (u < p_param + p_unowned)] = X
    return r


@pytest.mark.parametrize("seed", range(40))
def test_rules_match_element_level_tracking(seed):
    rng = np.random.default_rng(1000 + seed)
    rows, cols, k = int(rng.integers(1, 7)), int(rng.integers(1, 5)), int(rng.integers(1, 5))
    users = [1, 2] if seed % 2 else [3]
    kind = ["add_residual", "add_bias", "find_max", "matmul"][seed % 4]
    o = gift.Ownership()
    t_in, t_res, t_par, t_out = addrs(4)
    in_rows = _rand_rows(rng, rows, users)
    width = k if kind == "matmul" else cols
    o.register(t_in, (rows, width), 2)
    o.set(t_in, 0, 0, 0)
    for i, v in enumerate(in_rows):
        o.set(t_in, i, 1, int(v))
    prev_out = _rand_rows(rng, rows, [9])
    if kind == "add_residual":
        res_rows = in_rows.copy() if rng.random() < 0.6 else _rand_rows(rng, rows, users)
        o.register(t_res, (rows, cols), 2)
        for i, v in enumerate(res_rows):
            o.set(t_res, i, 1, int(v))
        owners = {"in": ift.expand_rows(in_rows, cols), "res": ift.expand_rows(res_rows, cols)}
        out_shape, flow = (rows, cols), ift.flow_add_residual(rows, cols)
        o.register(t_out, (rows, cols), 2)
        call = lambda: o.add_residual(t_out, t_in, t_res, rows, cols, 2)
    elif kind in ("add_bias", "matmul"):
        pshape = (cols,) if kind == "add_bias" else (k, cols)
        # parameter operand with one owner per element (any odim is allowed)
        pown = np.full(pshape, P, np.uint64)
        if rng.random() < 0.3:
            pown[tuple(int(rng.integers(0, s)) for s in pshape)] = rng.choice([1, X])
        o.register(t_par, pshape, 2, odims=tuple(range(len(pshape))))
        for f, v in enumerate(pown.reshape(-1)):
            o.set(t_par, f, 1, int(v))
        o.register(t_out, (rows, cols), 2)
        if kind == "add_bias":
            owners = {"in": ift.expand_rows(in_rows, cols), "bias": pown}
            out_shape, flow = (rows, cols), ift.flow_add_bias(rows, cols)
            call = lambda: o.add_bias(t_out, t_in, t_par, rows, cols, 2)
        else:
            owners = {"in": ift.expand_rows(in_rows, k), "weight": pown}
            out_shape, flow = (rows, cols), ift.flow_matmul(rows, k, cols)
            call = lambda: o.matmul(t_out, t_in, t_par, rows, k, cols, 2)
    else:
        owners = {"in": ift.expand_rows(in_rows, cols)}
        out_shape, flow = (rows,), ift.flow_find_max(rows, cols)
        o.register(t_out, (rows,), 8)
        call = lambda: o.find_max(t_out, t_in, rows, cols, 2, 8)
    for i, v in enumerate(prev_out):
        o.set(t_out, i, 1, int(v))
    want_st, want = ift.propagate(out_shape, flow, owners)
    got_st = call()
    assert got_st == want_st
    if want_st == ift.OK:
        assert list(o.labels(t_out)) == list(ift.rows_of(want))
    else:
        assert list(o.labels(t_out)) == list(prev_out)  # nothing changed


def test_rule_steps_1_to_3_shapes_and_aliasing():
    o = gift.Ownership()
    a, b, c, w, bias, v = addrs(6)
    for t in (a, b, c):
        o.register(t, (4, 8), 2)
        o.set(t, 0, 4, 1)
    o.register(w, (8, 8), 2, odims=())
    o.set(w, 0, 1, P)
    o.register(bias, (8,), 2, odims=())
    o.set(bias, 0, 1, P)
    o.register(v, (4,), 4)
    R = gift.E_REJECTED
    # step 1: unknown tensor; step 2: shape or element size mismatch
    assert o.add_residual(a, b, 0x1234, 4, 8, 2) == R
    assert o.add_residual(a, b, c, 4, 4, 2) == R
    assert o.add_residual(a, b, c, 4, 8, 4) == R
    assert o.matmul(a, b, w, 4, 8, 4, 2) == R
    assert o.find_max(v, a, 4, 8, 2, 8) == R
    # step 3: in-place outputs are allowed where the kernel writes in place
    assert o.add_residual(a, a, c, 4, 8, 2) == gift.OK
    assert o.add_bias(a, a, bias, 4, 8, 2) == gift.OK
    assert o.add_residual(a, b, a, 4, 8, 2) == R
    assert o.add_residual(a, b, b, 4, 8, 2) == R
    assert o.matmul(a, a, w, 4, 8, 8, 2) == R
    assert o.matmul(a, b, w, 4, 8, 8, 2) == gift.OK
    assert o.find_max(v, a, 4, 8, 2, 4) == gift.OK
    # step 4: a weight that is not parameter-owned
    o.set(w, 0, 1, 1)
    assert o.matmul(a, b, w, 4, 8, 8, 2) == R


def test_labels_feed_the_owner_check():
    # propagated row labels are what the fused seal check consumes: the oracle
    # check accepts a segment exactly when its rows carry its user
    import oracle
    o = gift.Ownership()
    x, r, y = addrs(3)
    for t in (x, r, y):
        o.register(t, (6, 16), 2)
    for t in (x, r):
        o.set(t, 0, 2, 1)
        o.set(t, 2, 4, 2)
    assert o.add_residual(y, x, r, 6, 16, 2) == gift.OK
    labels = o.labels(y)
    segs = oracle.as_segments([(0, 2, 1, 0), (2, 4, 2, 0)])
    st, ver = oracle.check_owner(segs, labels, 6)
    assert st == oracle.OK and list(ver) == [oracle.SEG_OK, oracle.SEG_OK]
    segs = oracle.as_segments([(0, 3, 1, 0), (3, 3, 2, 0)])
    st, ver = oracle.check_owner(segs, labels, 6)
    assert st == oracle.OK and list(ver) == [oracle.SEG_OWNER_MIXED, oracle.SEG_OK]


# --- launch order versus the history-graph oracle (Sec. 4.4) -----------------
def _random_ops(rng, n_ops, n_streams=3, space=48):
    ops = []
    for _ in range(n_ops):
        u = rng.random()
        s = int(rng.integers(0, n_streams))
        if u < 0.6:
            def rr():
                out = []
                for _ in range(int(rng.integers(0, 3))):
                    a = int(rng.integers(0, space))
                    out.append((a, int(rng.integers(0, 12))))
                return out
            ops.append(("launch", s, rr(), rr()))
        elif u < 0.78:
            ops.append(("wait", s, int(rng.integers(0, n_streams)), int(rng.integers(0, 6))))
        elif u < 0.88:
            ops.append(("sync", s))
        elif u < 0.92:
            ops.append(("sync_all",))
        else:
            ops.append(("release", int(rng.integers(0, space)), int(rng.integers(0, 16))))
    return ops


@pytest.mark.parametrize("seed", range(60))
def test_race_checker_matches_history_graph(seed):
    rng = np.random.default_rng(seed)
    model, lib = ift.LaunchOrder(), gift.RaceChecker()
    for op in _random_ops(rng, 45):
        if op[0] == "launch":
            assert lib.launch(op[1], op[2], op[3]) == model.launch(op[1], op[2], op[3]), op
        elif op[0] == "wait":
            assert lib.wait(*op[1:]) == model.wait(*op[1:]), op
        elif op[0] == "sync":
            lib.sync(op[1])
            model.sync(op[1])
        elif op[0] == "sync_all":
            lib.sync_all()
            model.sync_all()
        else:
            lib.release(op[1], op[2])
            model.release(op[1], op[2])


def test_race_checker_paper_scenarios():
    MAIN, SWAP = 0, 1
    kv = [(4096, 65536)]
    c = gift.RaceChecker()
    assert c.launch(MAIN, reads=kv) == (gift.OK, 1)
    assert c.launch(SWAP, writes=kv)[0] == gift.E_RACE
    assert c.launch(SWAP, writes=[(4096 + 65536, 16)]) == (gift.OK, 1)  # a different block
    c.sync(MAIN)
    assert c.launch(SWAP, writes=kv) == (gift.OK, 2)
    # collective order: receiver between two writers, ordered by stream waits
    S1, S2, buf = 5, 6, [(1 << 40, 1 << 20)]
    _, w1 = c.launch(S1, writes=buf)
    assert c.wait(S2, S1, w1) == gift.OK
    _, r2 = c.launch(S2, reads=buf)
    assert c.launch(S1, writes=buf)[0] == gift.E_RACE
    assert c.wait(S1, S2, r2) == gift.OK
    assert c.launch(S1, writes=buf)[0] == gift.OK
    assert c.wait(S1, S2, 99) == gift.E_RANGE


def test_race_checker_large_addresses_and_many_ranges():
    c = gift.RaceChecker()
    base = (1 << 47) - (1 << 20)
    blocks = [(base + i * 4096, 4096) for i in range(256)]
    assert c.launch(0, writes=blocks)[0] == gift.OK
    assert c.launch(1, reads=[(base + 255 * 4096 + 4095, 1)])[0] == gift.E_RACE
    assert c.launch(1, reads=[(base + 256 * 4096, 1)])[0] == gift.OK
    assert c.launch(1, reads=[(base, 0)])[0] == gift.OK  # empty range
    c.release(base, 256 * 4096)
    assert c.launch(1, writes=blocks)[0] == gift.OK
