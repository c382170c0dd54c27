"""gift_seal_noalloc (the seal on the device's fixed workspace) against
gift_seal through the C ABI: two calls in a row, the second with a smaller
input, each bit-exact with the allocating entry point and with the oracle;
and the size limit, rejected before anything is enqueued."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import oracle  # noqa: E402
from gpu_helpers import DEV, dev_u32, dev_u8, host  # noqa: E402
from paper_2608_25431_amd import gift  # noqa: E402

RB = 1024  # one row is 64 blocks: one-row segments take the small-segment path


def make_case(r, rows_list, users, seq0):
    table, row = [], 0
    for k, n in enumerate(rows_list):
        row += int(r.random() < 0.2)  # some uncovered rows
        table.append((row, n, int(r.integers(0, users)), seq0 + k))
        row += n
    n_rows = row + 1
    labels = np.full(n_rows, gift.LABEL_UNOWNED, np.uint32)
    for (b, n, u, _) in table:
        labels[b:b + n] = u
    i = int(r.integers(0, len(table)))  # one mixed segment
    b, n, u, _ = table[i]
    labels[b + int(r.integers(0, n))] = (u + 1) % users
    data = r.integers(0, 256, n_rows * RB, dtype=np.uint8)
    return table, n_rows, labels, data


def seal_both(kt, keys, nb, table, n_rows, labels, data, verdicts):
    """The same call through gift_seal and gift_seal_noalloc; outputs of both,
    and the oracle's."""
    n = len(table)
    d, lab = dev_u8(data), dev_u32(labels)
    res = []
    for fn in (gift.seal, gift.seal_noalloc):
        out = torch.full_like(d, 0x5A)
        tags = torch.full((16 * n,), 0xA5, dtype=torch.uint8, device=DEV)
        ver = torch.full((n,), -7, dtype=torch.int32, device=DEV) if verdicts else None
        fn(d, n_rows, RB, table, kt, nb, out, tags, row_labels=lab, verdicts=ver)
        res.append((host(out), host(tags), None if ver is None else host(ver)))
    st, o_out, o_tags, o_ver = oracle.seal(data, n_rows, RB, table, keys, nb, labels=labels)
    assert st == 0
    return res, (o_out, o_tags.reshape(-1), o_ver)


def test_noalloc_matches_seal_on_two_calls_the_second_smaller():
    r = np.random.default_rng(31)
    keys = r.integers(0, 256, (4, 32), dtype=np.uint8)
    nb = r.integers(0, 256, (4, 12), dtype=np.uint8)
    kt = gift.KeyTable(keys)
    # call 1: small, one-tile and multi-tile segments, 38 tiles: fewer tiles
    # than CUs, so every tile is cut into pieces that XOR into zeroed partials
    big = [1, 1, 1] + [int(x) for x in r.integers(100, 2000, 10)] + [int(x) for x in r.integers(2100, 9000, 7)]
    r.shuffle(big)
    # call 2: fewer and shorter segments on the same workspace
    small = [1] + [int(x) for x in r.integers(50, 900, 4)] + [int(x) for x in r.integers(2100, 3000, 2)]
    for k, (rows, verdicts) in enumerate([(big, True), (small, False)]):
        table, n_rows, labels, data = make_case(r, rows, 4, 100 * k)
        (a, b), (o_out, o_tags, o_ver) = seal_both(kt, keys, nb, table, n_rows, labels, data, verdicts)
        n = len(table)
        assert b[0].tobytes() == a[0].tobytes(), f"call {k}: ciphertext differs from gift_seal"
        assert b[1].tobytes() == a[1].tobytes(), f"call {k}: tags differ from gift_seal"
        assert b[0].tobytes() == o_out.tobytes(), f"call {k}: ciphertext differs from the oracle"
        assert b[1].tobytes() == o_tags.tobytes(), f"call {k}: tags differ from the oracle"
        if verdicts:
            assert b[2].tolist() == a[2].tolist() == o_ver.tolist()
        assert int((o_ver != 0).sum()) == 1
        assert n == len(rows)
    kt.destroy()


def test_noalloc_rejects_a_call_beyond_the_workspace():
    # 150,000 one-row segments need 9.6 MB of descriptors alone: more than
    # the workspace; the call fails before enqueuing anything
    r = np.random.default_rng(32)
    keys = r.integers(0, 256, (1, 32), dtype=np.uint8)
    nb = r.integers(0, 256, (1, 12), dtype=np.uint8)
    kt = gift.KeyTable(keys)
    n = 150_000
    rb = 16
    segs = np.zeros(n, gift.SEGMENT_DTYPE)
    segs["row_begin"] = np.arange(n)
    segs["row_count"] = 1
    segs["iv_seq"] = np.arange(n)
    d = torch.zeros(n * rb, dtype=torch.uint8, device=DEV)
    out = torch.full_like(d, 0x5A)
    tags = torch.full((16 * n,), 0xA5, dtype=torch.uint8, device=DEV)
    with pytest.raises(gift.GiftError) as ei:
        gift.seal_noalloc(d, n, rb, segs, kt, nb, out, tags)
    assert ei.value.status == gift.E_NOMEM
    torch.cuda.synchronize()
    assert (out == 0x5A).all().item() and (tags == 0xA5).all().item()
    # the allocating entry point takes the same call
    gift.seal(d, n, rb, segs, kt, nb, out, tags)
    torch.cuda.synchronize()
    assert not (tags == 0xA5).all().item()
    kt.destroy()
