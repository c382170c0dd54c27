"""Helpers shared by the GPU tests: device buffers, library calls, and
oracle references computed segment by segment on a thread pool."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
from paper_2608_25431_amd import gift

DEV = "cuda"
# worker threads for the oracle: the cores this process may run on, at most
# the 16-core share of one GPU on the test hosts
CORES = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 4)
THREADS = max(1, min(16, CORES))


def dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint8).reshape(-1).copy()).to(DEV)


def dev_u32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint32).view(np.int32).copy()).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def seal(data_dev, n_rows, row_bytes, segs, kt, nb, labels_dev=None, out=None, want_verdicts=True):
    n = len(segs)
    out = torch.empty_like(data_dev) if out is None else out
    tags = torch.zeros(max(n, 1) * 16, dtype=torch.uint8, device=DEV)
    ver = torch.full((max(n, 1),), -99, dtype=torch.int32, device=DEV) if want_verdicts else None
    gift.seal(data_dev, n_rows, row_bytes, segs, kt, nb, out, tags, row_labels=labels_dev, verdicts=ver)
    return out, tags, ver


def open_(data_dev, n_rows, row_bytes, segs, kt, nb, tags, labels_dev=None, out=None):
    n = len(segs)
    out = torch.empty_like(data_dev) if out is None else out
    ver = torch.full((max(n, 1),), -99, dtype=torch.int32, device=DEV)
    gift.open(data_dev, n_rows, row_bytes, segs, kt, nb, out, tags, ver, row_labels=labels_dev)
    return out, ver


def status_of(fn, *a, **k):
    try:
        fn(*a, **k)
        return 0
    except gift.GiftError as e:
        return e.status


def oracle_segments(keys, nb, segs, row_bytes, seg_plain):
    """Per-segment oracle GCM in parallel: seg_plain(i) -> plaintext bytes.
    Returns a list of (ciphertext, tag)."""
    def one(i):
        s = segs[i]
        u = int(s["user"])
        iv = oracle.segment_iv(nb[u].tobytes(), int(s["iv_seq"]))
        return oracle.gcm_encrypt(keys[u].tobytes(), iv, seg_plain(i))
    with ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(one, range(len(segs))))


def expected_block(keys, nb, seg, j, plain16):
    """Ciphertext of block j of a segment, from the oracle's GCTR alone."""
    u = int(seg["user"])
    iv = oracle.segment_iv(nb[u].tobytes(), int(seg["iv_seq"]))
    icb = iv + (2 + j).to_bytes(4, "big")
    return oracle.gctr(keys[u].tobytes(), icb, plain16)
