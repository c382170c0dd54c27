"""Pins of the oracle's paged-KV semantics (GIFT Sec. 4.2 KV blocks, Sec. 4.5
block tables, Sec. 2.2 manipulated block tables) -- no GPU.

The sealed stream of a request must equal OpenSSL's GCM over its chunks
gathered here with numpy (block table order, then layer, then part); open
must scatter the plaintext into the (possibly different) destination blocks;
a block labelled with another owner must reject the request.
"""
import numpy as np
import pytest

import oracle
import openssl_ref

pytestmark = pytest.mark.skipif(not openssl_ref.available(), reason="libcrypto not available")

rng = np.random.default_rng(5)


def geom(layers=3, parts=2, blocks=10, chunk=64, layout="lbp"):
    if layout == "lbp":   # [layer][block][part][chunk]
        ps, bs, ls = chunk, parts * chunk, blocks * parts * chunk
    else:                 # [layer][part][block][chunk] (K and V planes apart)
        bs, ps, ls = chunk, blocks * chunk, parts * blocks * chunk
    return oracle.PagedKV(layers * ls if layout == "lbp" else layers * ls, ls, bs, ps, chunk, layers, parts, blocks)


def gather_np(cache, g, bids):
    out = []
    for b in bids:
        for l in range(g.n_layers):
            for p in range(g.n_parts):
                o = l * g.layer_stride + b * g.block_stride + p * g.part_stride
                out.append(cache[o:o + g.chunk_bytes])
    return np.concatenate(out)


def setup(g, n_users=3):
    keys = rng.integers(0, 256, (n_users, 32), dtype=np.uint8)
    nb = rng.integers(0, 256, (n_users, 12), dtype=np.uint8)
    cache = rng.integers(0, 256, g.cache_bytes, dtype=np.uint8)
    return keys, nb, cache


def iv_of(nb, q):
    iv = bytearray(nb)
    for k in range(8):
        iv[11 - k] ^= (q >> (8 * k)) & 0xFF
    return bytes(iv)


@pytest.mark.parametrize("layout", ["lbp", "lpb"])
def test_sealed_streams_match_openssl(layout):
    g = geom(layout=layout)
    keys, nb, cache = setup(g)
    reqs = [([3, 1, 7], 0, 5), ([0], 2, 5), ([9, 8, 2, 4], 1, 6)]
    st, out, tags, ver = oracle.seal_paged(cache, g, reqs, keys, nb)
    assert st == 0 and (ver == 0).all()
    off = 0
    for i, (bids, u, q) in enumerate(reqs):
        msg = gather_np(cache, g, bids).tobytes()
        ct, tag = openssl_ref.gcm_encrypt(keys[u].tobytes(), iv_of(nb[u].tobytes(), q), msg)
        assert out[off:off + len(msg)].tobytes() == ct and tags[i].tobytes() == tag
        off += len(msg)


def test_open_scatters_into_new_blocks():
    g = geom()
    keys, nb, cache = setup(g)
    reqs = [([3, 1], 0, 1), ([5], 1, 1)]
    _, sealed, tags, _ = oracle.seal_paged(cache, g, reqs, keys, nb)
    moved = [([6, 0], 0, 1), ([9], 1, 1)]  # swap-in to other blocks
    st, after, ver = oracle.open_paged(np.zeros_like(cache), g, moved, keys, nb, sealed, tags)
    assert st == 0 and (ver == 0).all()
    for (src, _, _), (dst, _, _) in zip(reqs, moved):
        assert gather_np(after, g, dst).tobytes() == gather_np(cache, g, src).tobytes()
    untouched = set(range(10)) - {6, 0, 9}
    for b in untouched:
        assert not gather_np(after, g, [b]).any()


def test_manipulated_block_table_is_rejected_by_labels():
    g = geom()
    keys, nb, cache = setup(g)
    labels = np.array([0, 0, 1, 1, 2, 2, 0, 1, 2, 0], np.uint32)
    honest = [([0, 1, 6], 0, 1), ([2, 3], 1, 1)]
    st, out, tags, ver = oracle.seal_paged(cache, g, honest, keys, nb, labels=labels)
    assert (ver == 0).all()
    # user 1's table points at user 0's block 9 (confused deputy)
    evil = [([0, 1, 6], 0, 2), ([2, 9], 1, 2)]
    st, out, tags, ver = oracle.seal_paged(cache, g, evil, keys, nb, labels=labels)
    assert ver.tolist() == [0, oracle.SEG_OWNER_MIXED]
    per = g.n_layers * g.n_parts * g.chunk_bytes
    assert not out[3 * per:].any() and not tags[1].any()
    # the parameter label is never a user's
    l2 = labels.copy()
    l2[1] = oracle.LABEL_PARAM
    assert oracle.seal_paged(cache, g, honest, keys, nb, labels=l2)[3].tolist() == [oracle.SEG_OWNER_MIXED, 0]


def test_open_with_a_manipulated_table_writes_nothing():
    # user 1's table on open names user 0's resident block 9: the request is
    # rejected before anything runs, so block 9 (and user 1's own blocks)
    # keep their contents; only the honest request is opened
    g = geom()
    keys, nb, cache = setup(g)
    labels = np.array([0, 0, 1, 1, 2, 2, 0, 1, 2, 0], np.uint32)
    honest = [([0, 1, 6], 0, 1), ([2, 3], 1, 1)]
    _, sealed, tags, _ = oracle.seal_paged(cache, g, honest, keys, nb, labels=labels)
    resident = np.random.default_rng(3).integers(0, 256, cache.size, dtype=np.uint8)
    evil = [([0, 1, 6], 0, 1), ([2, 9], 1, 1)]
    st, after, ver = oracle.open_paged(resident, g, evil, keys, nb, sealed, tags, labels=labels)
    assert st == 0 and ver.tolist() == [0, oracle.SEG_OWNER_MIXED]
    for b in (2, 3, 9):
        assert gather_np(after, g, [b]).tobytes() == gather_np(resident, g, [b]).tobytes()
    assert gather_np(after, g, [0, 1, 6]).tobytes() == gather_np(cache, g, [0, 1, 6]).tobytes()


def test_tampered_request_fails_and_its_blocks_are_zeroed():
    g = geom()
    keys, nb, cache = setup(g)
    reqs = [([3, 1], 0, 1), ([5, 7], 1, 1)]
    _, sealed, tags, _ = oracle.seal_paged(cache, g, reqs, keys, nb)
    s2 = sealed.copy()
    s2[-1] ^= 1
    st, after, ver = oracle.open_paged(cache, g, reqs, keys, nb, s2, tags)
    assert ver.tolist() == [0, oracle.SEG_AUTH_FAIL]
    assert not gather_np(after, g, [5, 7]).any()
    assert gather_np(after, g, [3, 1]).tobytes() == gather_np(cache, g, [3, 1]).tobytes()


def test_validation_codes():
    g = geom()
    keys, nb, cache = setup(g)

    def code(reqs, gg=g):
        return oracle.seal_paged(cache, gg, reqs, keys, nb)[0]

    assert code([([1], 0, 0)]) == 0
    bad = geom(chunk=48)  # not a power of two
    assert code([([1], 0, 0)], bad) == oracle.E_INVALID
    ov = oracle.PagedKV(g.cache_bytes, g.layer_stride, 32, g.part_stride, 64, 3, 2, 10)  # blocks overlap
    assert code([([1], 0, 0)], ov) == oracle.E_INVALID
    assert code([([], 0, 0)]) == oracle.E_INVALID
    assert code([([10], 0, 0)]) == oracle.E_RANGE
    assert code([([1], 3, 0)]) == oracle.E_RANGE
    small = oracle.PagedKV(g.cache_bytes // 2, g.layer_stride, g.block_stride, g.part_stride, 64, 3, 2, 10)
    assert code([([1], 0, 0)], small) == oracle.E_RANGE
    assert code([([1, 2], 0, 0), ([2], 1, 0)]) == oracle.E_OVERLAP
    assert code([([1], 0, 4), ([2], 0, 4)]) == oracle.E_NONCE_REUSE
