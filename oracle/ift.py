"""Oracle for ownership propagation (GIFT Sec. 4.1-4.3) and for the legal
launch order of kernels on several streams (Sec. 4.4).

TEST INFRASTRUCTURE ONLY: only the test suite may import this module.  Pure
Python, no code shared with the library.  Both models are written at the
finest granularity the paper contrasts its design with, so that the library's
coarse, incremental bookkeeping is checked against a different formulation of
the same rules:

* ``propagate`` tracks ownership per element (the element-level tracking of
  Sec. 4.1, Insight 1).  Every output element collects the owners of every
  input element that the kernel's arithmetic reads to produce it (its
  information flow, Sec. 4.3 "Building IFGs"); the rule of Sec. 4.3 step 5 is
  then applied element by element: every source that is not a parameter
  operand must carry one and the same owner, which the output element takes.
  Sec. 4.2 ("Unowned memory") forbids reading memory without an owner, and
  Sec. 4.3 step 4 requires parameter operands to be parameter-owned.  A
  violation anywhere rejects the whole launch and changes nothing.

* ``LaunchOrder`` keeps the whole history of launches, stream waits and host
  synchronisations as a graph and decides, for each new launch, whether every
  earlier kernel that conflicts with it on some byte (one of the two writes
  it) has finished before it may start: the kernel is on the same stream, or
  it reaches the new launch's stream through program order and event waits,
  or a host synchronisation of a stream (or of the device) that it reaches was
  recorded after it (Sec. 4.4, "Concurrency control": a kernel launched
  before a synchronisation has completed).  Freed bytes drop out of the
  history.

Parity pins: the 2B+1 operation count of Sec. 4.1 Insight 2 is checked against
the library; these models are checked by hand-worked scenarios of Sec. 4.3
(Fig. 5 kernels) and Sec. 4.4 (the swap-versus-attention race, the collective
order) and by brute-force properties in the tests.
"""
import itertools
from collections import deque

import numpy as np

OK, E_RANGE, E_REJECTED, E_RACE = 0, -2, -8, -9
LABEL_PARAM, LABEL_UNOWNED = 0xFFFFFFFE, 0xFFFFFFFF


# ---------------------------------------------------------------------------
# element-level information flow of the four kernels of Sec. 4.3 (Fig. 5)
# ---------------------------------------------------------------------------
def flow_add_residual(rows, cols):
    """out[i,j] = in[i,j] + res[i,j]."""
    for i, j in itertools.product(range(rows), range(cols)):
        yield (i, j), [("in", (i, j)), ("res", (i, j))], []


def flow_add_bias(rows, cols):
    """out[i,j] = in[i,j] + bias[j]; bias is a parameter operand."""
    for i, j in itertools.product(range(rows), range(cols)):
        yield (i, j), [("in", (i, j))], [("bias", (j,))]


def flow_find_max(rows, cols):
    """out[i] = argmax_j in[i,j]: every element of row i is compared."""
    for i in range(rows):
        yield (i,), [("in", (i, j)) for j in range(cols)], []


def flow_matmul(rows, k, n):
    """out[i,j] = sum_t in[i,t] * weight[t,j]; weight is a parameter operand."""
    for i, j in itertools.product(range(rows), range(n)):
        yield (i, j), [("in", (i, t)) for t in range(k)], [("weight", (t, j)) for t in range(k)]


def propagate(out_shape, flow, owners):
    """Element-level rule application.

    owners: operand name -> numpy array of per-element owners.
    Returns (status, out_owner_array or None)."""
    out = np.full(out_shape, LABEL_UNOWNED, np.uint64)
    for idx, sources, params in flow:
        seen = {int(owners[name][e]) for name, e in sources}
        param_owners = {int(owners[name][e]) for name, e in params}
        if LABEL_UNOWNED in seen or LABEL_UNOWNED in param_owners:
            return E_REJECTED, None  # a read of unowned memory
        if param_owners - {LABEL_PARAM}:
            return E_REJECTED, None  # a parameter operand that is not a parameter
        if len(seen) != 1:
            return E_REJECTED, None  # sources of one output element mix owners
        out[idx] = seen.pop()
    return OK, out


def expand_rows(row_owner, cols):
    """Per-element owners of a matrix whose rows carry row_owner."""
    return np.repeat(np.asarray(row_owner, np.uint64)[:, None], cols, axis=1)


def rows_of(elem_owner):
    """Row owners of an element-owner matrix (None if a row is not uniform)."""
    e = np.asarray(elem_owner)
    if e.ndim == 1:
        return e.copy()
    if not (e == e[:, :1]).all():
        return None
    return e[:, 0].copy()


# ---------------------------------------------------------------------------
# legal launch order (Sec. 4.4)
# ---------------------------------------------------------------------------
class LaunchOrder:
    """History graph of launches, waits and synchronisations over byte sets."""

    def __init__(self):
        self.nodes = []  # dicts: kind in {"launch", "wait", "sync", "sync_all", "release"}
        self.issued = {}

    # -- graph helpers ------------------------------------------------------
    def _kernel_pos(self, stream, seq):
        n = 0
        for p, nd in enumerate(self.nodes):
            if nd["kind"] == "launch" and nd["stream"] == stream:
                n += 1
                if n == seq:
                    return p
        raise KeyError((stream, seq))

    def _successors(self, p):
        nd = self.nodes[p]
        out = []
        # program order: the next launch or wait on the same stream
        for q in range(p + 1, len(self.nodes)):
            if self.nodes[q]["kind"] in ("launch", "wait") and self.nodes[q]["stream"] == nd["stream"]:
                out.append(q)
                break
        # event waits on this kernel and anything after it on its stream are
        # covered by program order followed by the wait edge of a later kernel
        if nd["kind"] == "launch":
            for q in range(p + 1, len(self.nodes)):
                w = self.nodes[q]
                if w["kind"] == "wait" and w["pos"] == p:
                    out.append(q)
        return out

    def _reach(self, p, before):
        """Positions < before reachable from p (p included)."""
        seen, todo = {p}, deque([p])
        while todo:
            x = todo.popleft()
            for y in self._successors(x):
                if y < before and y not in seen:
                    seen.add(y)
                    todo.append(y)
        return seen

    def _finished_before(self, p, stream, now):
        """Does kernel node p finish before a launch on `stream` at position now?"""
        reach = self._reach(p, now)
        if any(self.nodes[q]["stream"] == stream for q in reach if self.nodes[q]["kind"] in ("launch", "wait")):
            return True  # same stream, or the stream waited on it (transitively)
        for q in range(p + 1, now):
            s = self.nodes[q]
            if s["kind"] == "sync_all":
                return True
            if s["kind"] == "sync" and any(self.nodes[r]["stream"] == s["stream"] and r < q for r in reach
                                            if self.nodes[r]["kind"] in ("launch", "wait")):
                return True
        return False

    def _live(self, p, nbytes, now):
        """Bytes of node p not freed between p and now."""
        live = set(nbytes)
        for q in range(p + 1, now):
            if self.nodes[q]["kind"] == "release":
                live -= self.nodes[q]["bytes"]
        return live

    # -- operations ---------------------------------------------------------
    @staticmethod
    def _bytes(ranges):
        b = set()
        for a, n in ranges:
            b.update(range(a, a + n))
        return b

    def launch(self, stream, reads=(), writes=()):
        now = len(self.nodes)
        r, w = self._bytes(reads), self._bytes(writes)
        for p, x in enumerate(self.nodes):
            if x["kind"] != "launch":
                continue
            conflict = (self._live(p, x["writes"], now) & (r | w)) | (self._live(p, x["reads"], now) & w)
            if conflict and not self._finished_before(p, stream, now):
                return E_RACE, 0
        seq = self.issued.get(stream, 0) + 1
        self.issued[stream] = seq
        self.nodes.append({"kind": "launch", "stream": stream, "seq": seq, "reads": r, "writes": w})
        return OK, seq

    def wait(self, stream, on_stream, seq):
        if seq > self.issued.get(on_stream, 0):
            return E_RANGE
        if seq == 0 or on_stream == stream:
            return OK
        self.nodes.append({"kind": "wait", "stream": stream, "pos": self._kernel_pos(on_stream, seq)})
        return OK

    def sync(self, stream):
        self.nodes.append({"kind": "sync", "stream": stream})

    def sync_all(self):
        self.nodes.append({"kind": "sync_all", "stream": None})

    def release(self, addr, nbytes):
        self.nodes.append({"kind": "release", "stream": None, "bytes": set(range(addr, addr + nbytes))})
