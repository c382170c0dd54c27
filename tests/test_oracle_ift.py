"""Pins of the ownership-propagation and launch-order oracle (oracle/ift.py)
against the paper's worked scenarios and against brute force."""
import itertools

import numpy as np
import pytest

from oracle import ift

P, X = ift.LABEL_PARAM, ift.LABEL_UNOWNED


# --- the declared information flow is the kernels' real data dependence -----
# Sec. 4.3 validates hand-built flow graphs against the kernel code (there by
# symbolic execution).  Here every input element is perturbed in turn and the
# output elements that change are compared with the flow's declared sources.

def _kernels(rows, cols, k, n):
    rng = np.random.default_rng(7)
    return {
        "add_residual": (lambda t: t["in"] + t["res"], {"in": (rows, cols), "res": (rows, cols)},
                         ift.flow_add_residual(rows, cols)),
        "add_bias": (lambda t: t["in"] + t["bias"][None, :], {"in": (rows, cols), "bias": (cols,)},
                     ift.flow_add_bias(rows, cols)),
        "find_max": (lambda t: np.argmax(t["in"], axis=1), {"in": (rows, cols)}, ift.flow_find_max(rows, cols)),
        "matmul": (lambda t: t["in"] @ t["weight"], {"in": (rows, k), "weight": (k, n)}, ift.flow_matmul(rows, k, n)),
    }, rng


@pytest.mark.parametrize("name", ["add_residual", "add_bias", "find_max", "matmul"])
def test_flow_matches_perturbation(name):
    kernels, rng = _kernels(3, 4, 5, 2)
    fn, shapes, flow = kernels[name]
    declared = {}
    for out_idx, srcs, params in flow:
        for s in srcs + params:
            declared.setdefault(s, set()).add(out_idx)
    base = {nm: rng.uniform(-1, 1, sh) for nm, sh in shapes.items()}
    ref = fn(base)
    observed = {}
    for nm, sh in shapes.items():
        for e in itertools.product(*map(range, sh)):
            changed = set()
            # a small change, and changes that win and lose every comparison
            for delta in (0.37, 1e6, -1e6):
                t = {k: v.copy() for k, v in base.items()}
                t[nm][e] += delta
                d = fn(t) != ref
                changed |= {tuple(int(i) for i in ix) for ix in np.argwhere(d)}
            if changed:
                observed[(nm, e)] = changed
    assert observed == declared


# --- Fig. 5 scenarios, worked by hand ---------------------------------------
U1, U2, U3 = 1, 2, 3


def _mat(row_owners, cols):
    return ift.expand_rows(row_owners, cols)


def test_add_residual_keeps_row_owners():
    st, out = ift.propagate((2, 3), ift.flow_add_residual(2, 3),
                            {"in": _mat([U1, U2], 3), "res": _mat([U1, U2], 3)})
    assert st == ift.OK and list(ift.rows_of(out)) == [U1, U2]


def test_add_residual_mixing_is_rejected():
    st, out = ift.propagate((2, 3), ift.flow_add_residual(2, 3),
                            {"in": _mat([U1, U2], 3), "res": _mat([U1, U3], 3)})
    assert st == ift.E_REJECTED and out is None


def test_add_bias_requires_parameter_bias():
    ok, out = ift.propagate((2, 3), ift.flow_add_bias(2, 3),
                            {"in": _mat([U2, U1], 3), "bias": np.full(3, P, np.uint64)})
    assert ok == ift.OK and list(ift.rows_of(out)) == [U2, U1]
    bad = np.full(3, P, np.uint64)
    bad[1] = U2  # a "bias" that holds user data
    assert ift.propagate((2, 3), ift.flow_add_bias(2, 3), {"in": _mat([U2, U2], 3), "bias": bad})[0] == ift.E_REJECTED


def test_find_max_output_row_owner():
    st, out = ift.propagate((3,), ift.flow_find_max(3, 4), {"in": _mat([U3, U1, U2], 4)})
    assert st == ift.OK and list(out) == [U3, U1, U2]


def test_find_max_rejects_a_row_with_two_owners():
    own = _mat([U1, U2], 4)
    own[1, 2] = U1  # one element of row 1 belongs to someone else
    assert ift.propagate((2,), ift.flow_find_max(2, 4), {"in": own})[0] == ift.E_REJECTED
    # element granularity: the other row alone would have been fine
    assert ift.rows_of(own) is None


def test_matmul_weight_must_be_parameter():
    w = np.full((4, 2), P, np.uint64)
    st, out = ift.propagate((2, 2), ift.flow_matmul(2, 4, 2), {"in": _mat([U1, U2], 4), "weight": w})
    assert st == ift.OK and list(ift.rows_of(out)) == [U1, U2]
    w[3, 1] = U1
    assert ift.propagate((2, 2), ift.flow_matmul(2, 4, 2), {"in": _mat([U1, U1], 4), "weight": w})[0] == ift.E_REJECTED


def test_unowned_memory_is_never_read():
    assert ift.propagate((2, 3), ift.flow_add_residual(2, 3),
                         {"in": _mat([U1, X], 3), "res": _mat([U1, X], 3)})[0] == ift.E_REJECTED
    assert ift.propagate((2, 3), ift.flow_add_bias(2, 3),
                         {"in": _mat([U1, U1], 3), "bias": np.full(3, X, np.uint64)})[0] == ift.E_REJECTED


def test_parameter_only_rows_stay_parameter_owned():
    st, out = ift.propagate((2, 3), ift.flow_add_residual(2, 3), {"in": _mat([P, U1], 3), "res": _mat([P, U1], 3)})
    assert st == ift.OK and list(ift.rows_of(out)) == [P, U1]
    assert ift.propagate((1, 3), ift.flow_add_residual(1, 3),
                         {"in": _mat([P], 3), "res": _mat([U1], 3)})[0] == ift.E_REJECTED


# --- launch order: Sec. 4.4 scenarios ---------------------------------------
MAIN, SWAP = 0, 1
KV = (0, 64)  # a KV block


def test_swap_overwriting_kv_under_attention_is_refused():
    # attention on the main stream reads user A's block; the background swap
    # stream must not overwrite it with user B's data until attention is done
    m = ift.LaunchOrder()
    assert m.launch(MAIN, reads=[KV]) == (ift.OK, 1)
    assert m.launch(SWAP, writes=[KV])[0] == ift.E_RACE
    m.sync(MAIN)
    assert m.launch(SWAP, writes=[KV]) == (ift.OK, 1)


def test_attention_reading_a_block_being_swapped_in_is_refused():
    m = ift.LaunchOrder()
    assert m.launch(SWAP, writes=[KV]) == (ift.OK, 1)
    assert m.launch(MAIN, reads=[KV])[0] == ift.E_RACE
    assert m.launch(MAIN, writes=[KV])[0] == ift.E_RACE  # write-write
    m.sync(SWAP)
    assert m.launch(MAIN, reads=[KV]) == (ift.OK, 1)


def test_same_stream_and_read_read_never_race():
    m = ift.LaunchOrder()
    assert m.launch(MAIN, writes=[KV])[0] == ift.OK
    assert m.launch(MAIN, reads=[KV], writes=[KV])[0] == ift.OK
    m.sync_all()
    assert m.launch(MAIN, reads=[KV])[0] == ift.OK
    assert m.launch(SWAP, reads=[KV])[0] == ift.OK


def test_collective_order_is_admitted_through_stream_waits():
    S1, S2 = 1, 2
    m = ift.LaunchOrder()
    _, w1 = m.launch(S1, writes=[KV])
    # the receiver reads only after the first writer finished ...
    assert m.launch(S2, reads=[KV])[0] == ift.E_RACE
    assert m.wait(S2, S1, w1) == ift.OK
    _, r2 = m.launch(S2, reads=[KV])
    assert r2 == 1
    # ... and the second writer starts only after the transfer finished
    assert m.launch(S1, writes=[KV])[0] == ift.E_RACE
    assert m.wait(S1, S2, r2) == ift.OK
    assert m.launch(S1, writes=[KV]) == (ift.OK, 2)


def test_waits_are_transitive_and_syncs_cover_what_was_waited_on():
    A, B, C = 0, 1, 2
    m = ift.LaunchOrder()
    m.launch(A, writes=[KV])
    m.wait(B, A, 1)
    m.launch(B, writes=[(100, 4)])
    m.wait(C, B, 1)
    assert m.launch(C, reads=[KV])[0] == ift.OK  # A -> B -> C
    m2 = ift.LaunchOrder()
    m2.launch(A, writes=[KV])
    m2.wait(B, A, 1)
    assert m2.launch(C, reads=[KV])[0] == ift.E_RACE
    m2.sync(B)  # B waited on A's kernel, so it has finished
    assert m2.launch(C, reads=[KV])[0] == ift.OK


def test_release_drops_history_and_waits_on_unlaunched_kernels_fail():
    m = ift.LaunchOrder()
    m.launch(MAIN, writes=[(0, 32)])
    m.release(0, 16)
    assert m.launch(SWAP, writes=[(0, 16)])[0] == ift.OK
    assert m.launch(SWAP, writes=[(16, 1)])[0] == ift.E_RACE
    assert m.wait(SWAP, MAIN, 2) == ift.E_RANGE
