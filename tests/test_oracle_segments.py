"""Segment semantics of the oracle (no GPU), checked against independent
per-segment GCM (OpenSSL) and the invariants the GIFT paper states:
  - Sec. 3 (steps 3, 5-6): each owner's data is sealed under that owner's key;
    manipulated ownership metadata (wrong user, wrong iv_seq, moved data)
    yields only a decryption failure;
  - Sec. 4.2: ownership per contiguous segment; memory without an ownership
    record is never released (zero);
  - Sec. 4.3, rule step 5: a segment whose rows carry another owner, the
    parameter label or no label is rejected.
"""
import itertools

import numpy as np
import pytest

import oracle
import openssl_ref

pytestmark = pytest.mark.skipif(not openssl_ref.available(), reason="libcrypto not available")

rng = np.random.default_rng(77)


def setup(n_users):
    keys = rng.integers(0, 256, (n_users, 32), dtype=np.uint8)
    nb = rng.integers(0, 256, (n_users, 12), dtype=np.uint8)
    return keys, nb


def segmentations(n_rows):
    """All ways to cover 0..n_rows with segments and gaps (each row: start a
    new segment, continue the current one, or be uncovered)."""
    for choice in itertools.product((0, 1, 2), repeat=n_rows):
        segs, cur = [], None
        ok = True
        for r, c in enumerate(choice):
            if c == 0:
                cur = None
            elif c == 1 or cur is None:
                segs.append([r, 1])
                cur = segs[-1]
            else:
                cur[1] += 1
        if ok:
            yield [tuple(s) for s in segs]


def iv_of(nb, seq):
    iv = bytearray(nb)
    for k in range(8):
        iv[11 - k] ^= (seq >> (8 * k)) & 0xFF
    return bytes(iv)


def test_segment_iv_derivation():
    nb = bytes(range(12))
    assert oracle.segment_iv(nb, 0) == nb
    assert oracle.segment_iv(nb, 0x0102030405060708) == iv_of(nb, 0x0102030405060708)
    assert oracle.segment_iv(nb, 1)[:4] == nb[:4]


@pytest.mark.parametrize("row_bytes", [4, 12, 16, 20, 48])
@pytest.mark.parametrize("n_rows", [1, 2, 3])
def test_brute_force_tiny_tensors_against_openssl(row_bytes, n_rows):
    keys, nb = setup(3)
    data = rng.integers(0, 256, n_rows * row_bytes, dtype=np.uint8)
    for segs in segmentations(n_rows):
        table = [(b, c, i % 3, 100 + i) for i, (b, c) in enumerate(segs)]
        st, out, tags, ver = oracle.seal(data, n_rows, row_bytes, table, keys, nb)
        assert st == oracle.OK
        covered = np.zeros(n_rows, bool)
        for i, (b, c, u, q) in enumerate(table):
            lo, hi = b * row_bytes, (b + c) * row_bytes
            ct, tag = openssl_ref.gcm_encrypt(keys[u].tobytes(), iv_of(nb[u].tobytes(), q), data[lo:hi].tobytes())
            assert out[lo:hi].tobytes() == ct
            assert tags[i].tobytes() == tag
            assert ver[i] == oracle.SEG_OK
            covered[b:b + c] = True
        for r in range(n_rows):
            if not covered[r]:
                assert not out[r * row_bytes:(r + 1) * row_bytes].any()
        st, back, ver = oracle.open_(out, n_rows, row_bytes, table, keys, nb, tags)
        assert st == oracle.OK and (ver == oracle.SEG_OK).all()
        for b, c, _, _ in table:
            assert back[b * row_bytes:(b + c) * row_bytes].tobytes() == data[b * row_bytes:(b + c) * row_bytes].tobytes()


def test_segment_order_does_not_matter():
    keys, nb = setup(4)
    n_rows, rb = 10, 24
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    table = [(0, 3, 0, 5), (3, 1, 1, 6), (5, 4, 2, 7), (9, 1, 3, 8)]
    st, out, tags, _ = oracle.seal(data, n_rows, rb, table, keys, nb)
    perm = [2, 0, 3, 1]
    st2, out2, tags2, _ = oracle.seal(data, n_rows, rb, [table[i] for i in perm], keys, nb)
    assert st == st2 == 0
    assert out.tobytes() == out2.tobytes()
    for j, i in enumerate(perm):
        assert tags2[j].tobytes() == tags[i].tobytes()


def test_in_place_equals_out_of_place():
    keys, nb = setup(2)
    n_rows, rb = 6, 40
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    table = [(0, 2, 0, 1), (3, 3, 1, 2)]
    _, out, tags, _ = oracle.seal(data, n_rows, rb, table, keys, nb)
    buf = data.copy()
    st, out2, tags2, _ = oracle.seal(buf, n_rows, rb, table, keys, nb, out=buf)
    assert st == 0 and buf.tobytes() == out.tobytes() and tags2.tobytes() == tags.tobytes()


def test_manipulated_metadata_yields_decryption_failure():
    keys, nb = setup(3)
    n_rows, rb = 8, 32
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    table = [(0, 3, 0, 1), (3, 3, 1, 1), (6, 2, 2, 4)]
    _, ct, tags, _ = oracle.seal(data, n_rows, rb, table, keys, nb)
    # wrong user on segment 0
    bad = [(0, 3, 1, 9)] + table[1:]
    st, out, ver = oracle.open_(ct, n_rows, rb, bad, keys, nb, tags)
    assert st == 0 and ver.tolist() == [oracle.SEG_AUTH_FAIL, 0, 0] and not out[:3 * rb].any()
    # wrong iv_seq on segment 2
    bad = table[:2] + [(6, 2, 2, 5)]
    st, out, ver = oracle.open_(ct, n_rows, rb, bad, keys, nb, tags)
    assert ver.tolist() == [0, 0, oracle.SEG_AUTH_FAIL] and not out[6 * rb:].any()
    # tags swapped between two segments
    t2 = tags.copy()
    t2[[0, 1]] = t2[[1, 0]]
    st, out, ver = oracle.open_(ct, n_rows, rb, table, keys, nb, t2)
    assert ver.tolist() == [oracle.SEG_AUTH_FAIL, oracle.SEG_AUTH_FAIL, 0]
    # ciphertext of segment 1 moved onto segment 0's rows (confused deputy)
    ct2 = ct.copy()
    ct2[:3 * rb] = ct[3 * rb:6 * rb]
    st, out, ver = oracle.open_(ct2, n_rows, rb, table, keys, nb, tags)
    assert ver.tolist() == [oracle.SEG_AUTH_FAIL, 0, 0]
    # the released bytes of verified segments are exactly the plaintext
    assert out[3 * rb:].tobytes() == data[3 * rb:].tobytes()


def test_owner_labels_reject_mixed_param_and_unowned_rows():
    keys, nb = setup(3)
    n_rows, rb = 9, 16
    data = rng.integers(0, 256, n_rows * rb, dtype=np.uint8)
    table = [(0, 3, 0, 1), (3, 3, 1, 1), (6, 3, 2, 1)]
    lab = np.array([0, 0, 0, 1, 1, 1, 2, 2, 2], np.uint32)
    st, out, tags, ver = oracle.seal(data, n_rows, rb, table, keys, nb, labels=lab)
    assert ver.tolist() == [0, 0, 0]
    for bad_label, row in ((2, 1), (oracle.LABEL_PARAM, 4), (oracle.LABEL_UNOWNED, 8)):
        l2 = lab.copy()
        l2[row] = bad_label
        st, out, tags, ver = oracle.seal(data, n_rows, rb, table, keys, nb, labels=l2)
        seg = row // 3
        assert ver[seg] == oracle.SEG_OWNER_MIXED
        assert not out[seg * 3 * rb:(seg + 1) * 3 * rb].any() and not tags[seg].any()
        others = [i for i in range(3) if i != seg]
        assert all(ver[i] == 0 for i in others)
        st, v2 = oracle.check_owner(table, l2, n_rows)
        assert st == 0 and v2.tolist() == ver.tolist()


def test_validation_codes():
    keys, nb = setup(2)
    d = np.zeros(4 * 8, np.uint8)

    def code(table, n_rows=4, rb=8):
        return oracle.seal(np.zeros(n_rows * rb, np.uint8), n_rows, rb, table, keys, nb)[0]

    assert code([(0, 0, 0, 0)]) == oracle.E_INVALID
    assert code([(0, 1, 0, 0, 1)]) == oracle.E_INVALID  # reserved != 0
    assert code([(0, 1, oracle.LABEL_PARAM, 0)]) == oracle.E_INVALID
    assert code([(3, 2, 0, 0)]) == oracle.E_RANGE
    assert code([(0, 1, 2, 0)]) == oracle.E_RANGE
    assert code([(0, 2, 0, 0), (1, 2, 1, 0)]) == oracle.E_OVERLAP
    assert code([(0, 1, 0, 7), (2, 1, 0, 7)]) == oracle.E_NONCE_REUSE
    assert code([(0, 1, 0, 7), (2, 1, 1, 7)]) == oracle.OK
    # (2^32 - 2) * 16 bytes is the limit
    big_rows = ((1 << 32) - 2) * 16 // 64 + 1
    assert oracle.seal(d, 4, 8, [(0, 1, 0, 0)], keys, nb)[0] == 0
    st = oracle.lib().oracle_seal(None, big_rows, 64, oracle.as_segments([(0, big_rows, 0, 0)]).ctypes.data, 1,
                                  None, keys.ctypes.data, 2, nb.ctypes.data, None, np.zeros(16, np.uint8).ctypes.data,
                                  None)
    assert st == oracle.E_INVALID  # null data is caught first
    # precedence: an earlier segment's INVALID wins over a later RANGE
    assert code([(0, 0, 0, 0), (9, 1, 0, 0)]) == oracle.E_INVALID
    assert code([(9, 1, 0, 0), (0, 0, 0, 0)]) == oracle.E_RANGE


def test_empty_table_zeroes_everything():
    keys, nb = setup(1)
    data = rng.integers(1, 256, 5 * 8, dtype=np.uint8)
    st, out, tags, ver = oracle.seal(data, 5, 8, [], keys, nb)
    assert st == 0 and not out.any()
