"""Parity with the oracle at the full sizes of the large workloads, in the
launch configuration the benchmark times (tolerance zero: integer work).

- llama3_8b_kv (9.06 GB, 64 segments), sealed with the owner check fused:
  every ciphertext byte and tag against the oracle's seal of each segment;
  then every byte and verdict of the open against the oracle's open of the
  same ciphertext.
- tamper (18.4 GB, 128 segments): every ciphertext byte and tag of the seal
  against the oracle; the standalone owner check against the oracle's; the
  fused seal (mixed segments zeroed with zero tags, the others equal to the
  verified unfused seal); then the open of the tampered buffer (one flipped
  ciphertext bit, one flipped tag bit) against the oracle's open of the same
  tampered host copy, every byte and verdict.
- llama3_70b_kv (50.5 GB, 32 segments), sealed in place with the owner check
  fused: the eight shortest segments (25% of the segments) whole against the
  oracle's seal -- every byte and the tag; every byte of the other 24 against
  the oracle's GCTR (SP 800-38D Algorithm 3) over 64 MiB pieces, each from its
  own initial counter block, with the plaintext regenerated from the seed per
  piece, and their tags from the oracle's GHASH of each ciphertext piece (GHASH
  is linear: a segment's hash is the sum of its pieces' hashes, each times H
  to the number of blocks after the piece, the length block last) and the
  oracle's E_K(J0); then the in-place open back to the plaintext, every byte.

The oracle runs segment by segment on a thread pool, longest jobs first; each
segment goes through the oracle's own segmented entry points over a
one-segment table (its rows renumbered from 0), so the IV derivation and the
owner check are the oracle's too.
"""
import time
from concurrent.futures import FIRST_COMPLETED, ThreadPoolExecutor, wait

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import oracle  # noqa: E402
from gpu_helpers import DEV, THREADS, dev_u32, host, open_, seal  # noqa: E402
from paper_2608_25431_amd import gift  # noqa: E402
from paper_2608_25431_amd import workloads as W  # noqa: E402

PIECE = 64 << 20  # bytes per oracle GCTR job on the in-place workload


_capsys = None


@pytest.fixture(autouse=True)
def _progress_uncaptured(capsys):
    """Progress lines go to the real stdout even when pytest captures the
    tests' output (-q without -s), so a long comparison never falls silent."""
    global _capsys
    _capsys = capsys
    yield
    _capsys = None


def log(msg):
    if _capsys is not None:
        with _capsys.disabled():
            print(f"[fullsize] {msg}", flush=True)
    else:
        print(f"[fullsize] {msg}", flush=True)


def table1(t, i):
    """Segment i as a one-segment table over its own rows."""
    s = t.segs[i:i + 1].copy()
    s["row_begin"] = 0
    return s


def seg_labels(t, labels, i):
    if labels is None:
        return None
    b, n = int(t.segs[i]["row_begin"]), int(t.segs[i]["row_count"])
    return labels[b:b + n]


def first_diff(a, b):
    d = np.flatnonzero(np.asarray(a) != np.asarray(b))
    return int(d[0]) if d.size else None


def run_longest_first(jobs, fn, every_s=30.0):
    """fn(job) for every job on THREADS threads, the largest first (job[0] is
    its size); returns the failures fn reports.  Prints progress every
    every_s seconds."""
    jobs = sorted(jobs, key=lambda j: -j[0])
    total = sum(j[0] for j in jobs)
    res, done, t0, last = [], 0, time.perf_counter(), time.perf_counter()
    with ThreadPoolExecutor(THREADS) as ex:
        futs = {ex.submit(fn, j): j for j in jobs}
        pending = set(futs)
        while pending:
            finished, pending = wait(pending, timeout=every_s, return_when=FIRST_COMPLETED)
            for f in finished:
                res.append(f.result())
                done += futs[f][0]
            if time.perf_counter() - last >= every_s:
                last = time.perf_counter()
                log(f"  {done / 1e9:.2f} of {total / 1e9:.2f} GB checked after {last - t0:.0f} s")
    return [r for r in res if r]


def oracle_seal_compare(w, t, pt_h, ct_h, tags_h, ver_h, labels=None):
    """Seal of every segment by the oracle against the library's output."""
    rb = t.row_bytes

    def one(job):
        _, i = job
        off, ln = t.seg_bytes(i)
        st, o_ct, o_tag, o_ver = oracle.seal(pt_h[off:off + ln], ln // rb, rb, table1(t, i), w.keys, w.nonce_base,
                                             labels=seg_labels(t, labels, i))
        if st != 0:
            return f"segment {i}: oracle status {st}"
        if not np.array_equal(o_ct, ct_h[off:off + ln]):
            return f"segment {i}: ciphertext differs at byte {first_diff(o_ct, ct_h[off:off + ln])}"
        if o_tag.tobytes() != tags_h[i].tobytes():
            return f"segment {i}: tag differs"
        if int(o_ver[0]) != int(ver_h[i]):
            return f"segment {i}: verdict {int(ver_h[i])}, oracle {int(o_ver[0])}"
        return None

    return run_longest_first([(t.seg_bytes(i)[1], i) for i in range(len(t.segs))], one)


def oracle_open_compare(w, t, ct_h, tags_h, back_h, ver_h, labels=None):
    """Open of every segment by the oracle against the library's output."""
    rb = t.row_bytes

    def one(job):
        _, i = job
        off, ln = t.seg_bytes(i)
        st, o_back, o_ver = oracle.open_(ct_h[off:off + ln], ln // rb, rb, table1(t, i), w.keys, w.nonce_base,
                                         tags_h[i], labels=seg_labels(t, labels, i))
        if st != 0:
            return f"segment {i}: oracle status {st}"
        if int(o_ver[0]) != int(ver_h[i]):
            return f"segment {i}: verdict {int(ver_h[i])}, oracle {int(o_ver[0])}"
        if not np.array_equal(o_back, back_h[off:off + ln]):
            return f"segment {i}: open output differs at byte {first_diff(o_back, back_h[off:off + ln])}"
        return None

    return run_longest_first([(t.seg_bytes(i)[1], i) for i in range(len(t.segs))], one)


def gf_pow(h, e):
    """h^e in GF(2^128) by square and multiply over the oracle's multiply."""
    r, b = (0x80).to_bytes(1, "big") + bytes(15), h  # the field's 1 is the bit string 10...0
    while e:
        if e & 1:
            r = oracle.gf128_mul(r, b)
        e >>= 1
        if e:
            b = oracle.gf128_mul(b, b)
    return r


def covered_exactly(t):
    """The workloads' segments tile their tensor with no gap."""
    ends = [int(s["row_begin"] + s["row_count"]) for s in t.segs]
    begins = [int(s["row_begin"]) for s in t.segs]
    return begins[0] == 0 and begins[1:] == ends[:-1] and ends[-1] == t.n_rows


def test_llama3_8b_kv_every_byte_against_oracle():
    w = W.llama3_8b_kv()
    t = w.tensors[0]
    assert covered_exactly(t)
    labels = np.full(t.n_rows, gift.LABEL_UNOWNED, np.uint32)
    for s in t.segs:
        labels[int(s["row_begin"]):int(s["row_begin"] + s["row_count"])] = s["user"]
    kt = gift.KeyTable(w.keys)
    d = t.generate(DEV)
    lab = dev_u32(labels)
    ct, tags, ver = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base, labels_dev=lab)
    back, ver2 = open_(ct, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base, tags, labels_dev=lab)
    n = len(t.segs)
    pt_h, ct_h, back_h = host(d), host(ct), host(back)
    tags_h, ver_h, ver2_h = host(tags).reshape(-1, 16)[:n], host(ver)[:n], host(ver2)[:n]
    del d, ct, back
    kt.destroy()
    torch.cuda.empty_cache()
    t0 = time.perf_counter()
    bad = oracle_seal_compare(w, t, pt_h, ct_h, tags_h, ver_h, labels)
    log(f"llama3_8b_kv seal: {n} segments, {t.nbytes / 1e9:.2f} GB against the oracle on {THREADS} threads "
        f"in {time.perf_counter() - t0:.0f} s")
    assert not bad, bad
    assert (ver_h == gift.SEG_OK).all()
    t0 = time.perf_counter()
    bad = oracle_open_compare(w, t, ct_h, tags_h, back_h, ver2_h, labels)
    log(f"llama3_8b_kv open: against the oracle in {time.perf_counter() - t0:.0f} s")
    assert not bad, bad
    assert np.array_equal(back_h, pt_h)


def test_tamper_every_byte_against_oracle():
    w = W.tamper()
    t = w.tensors[0]
    assert covered_exactly(t)
    n = len(t.segs)
    kt = gift.KeyTable(w.keys)
    d = t.generate(DEV)
    ct, tags, ver = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base)
    # standalone owner check and the fused seal, both against the oracle
    lab = dev_u32(t.labels)
    cv = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    gift.check_owner(t.segs, lab, t.n_rows, cv)
    st, o_cv = oracle.check_owner(t.segs, t.labels, t.n_rows)
    assert st == 0 and host(cv).tolist() == o_cv.tolist()
    mixed = sorted(i for (_, i, _, _) in w.mixed)
    assert np.flatnonzero(o_cv).tolist() == mixed
    ct2, tags2, ver2 = seal(d, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base, labels_dev=lab)
    ver2_h, tags2_h = host(ver2)[:n], host(tags2).reshape(-1, 16)[:n]
    tags1_h = host(tags).reshape(-1, 16)[:n]
    for i in range(n):
        off, ln = t.seg_bytes(i)
        if i in mixed:
            # the oracle's fused seal of a mixed segment
            sub = seg_labels(t, t.labels, i)
            st, o_ct, o_tag, o_ver = oracle.seal(np.zeros(ln, np.uint8), ln // t.row_bytes, t.row_bytes, table1(t, i),
                                                 w.keys, w.nonce_base, labels=sub)
            assert st == 0 and int(o_ver[0]) == gift.SEG_OWNER_MIXED and not o_ct.any() and not o_tag.any()
            assert int(ver2_h[i]) == gift.SEG_OWNER_MIXED and not tags2_h[i].any(), i
            assert not ct2[off:off + ln].any().item(), i
        else:
            # equal to the unfused seal, which is compared with the oracle below
            assert int(ver2_h[i]) == gift.SEG_OK and tags2_h[i].tobytes() == tags1_h[i].tobytes(), i
            assert torch.equal(ct2[off:off + ln], ct[off:off + ln]), i
    del ct2
    # tamper the sealed buffer on the device and the same bits on a host copy
    pt_h, ct_h, tags_h, ver_h = host(d), host(ct), tags1_h.copy(), host(ver)[:n]
    del d
    t0 = time.perf_counter()
    bad = oracle_seal_compare(w, t, pt_h, ct_h, tags_h, ver_h)
    log(f"tamper seal: {n} segments, {t.nbytes / 1e9:.2f} GB against the oracle in {time.perf_counter() - t0:.0f} s")
    assert not bad, bad
    del pt_h
    flipped = set()
    for (_, i, kind, off, bit) in w.tamper:
        if kind == "ct":
            ct[off] ^= (1 << bit)
            ct_h[off] ^= np.uint8(1 << bit)
        else:
            tags[16 * i + off] ^= (1 << bit)
            tags_h[i, off] ^= np.uint8(1 << bit)
        flipped.add(i)
    assert host(tags).reshape(-1, 16)[:n].tobytes() == tags_h.tobytes()
    back, ver3 = open_(ct, t.n_rows, t.row_bytes, t.segs, kt, w.nonce_base, tags)
    back_h, ver3_h = host(back), host(ver3)[:n]
    del back, ct
    kt.destroy()
    torch.cuda.empty_cache()
    t0 = time.perf_counter()
    bad = oracle_open_compare(w, t, ct_h, tags_h, back_h, ver3_h)
    log(f"tamper open: against the oracle's open of the tampered copy in {time.perf_counter() - t0:.0f} s")
    assert not bad, bad
    assert np.flatnonzero(ver3_h).tolist() == sorted(flipped)
    assert all(int(ver3_h[i]) == gift.SEG_AUTH_FAIL for i in flipped)


def test_llama3_70b_kv_in_place_against_oracle():
    w = W.llama3_70b_kv()
    t = w.tensors[0]
    assert covered_exactly(t)
    n = len(t.segs)
    rb = t.row_bytes
    kt = gift.KeyTable(w.keys)
    d = t.generate(DEV)
    lab = dev_u32(t.labels)
    _, tags, ver = seal(d, t.n_rows, rb, t.segs, kt, w.nonce_base, labels_dev=lab, out=d)
    tags_h, ver_h = host(tags).reshape(-1, 16)[:n], host(ver)[:n]
    assert (ver_h == gift.SEG_OK).all()
    whole = sorted(range(n), key=lambda i: (t.seg_bytes(i)[1], i))[:8]
    jobs = [(t.seg_bytes(i)[1], "whole", i, 0) for i in whole]
    for i in range(n):
        if i in whole:
            continue
        _, ln = t.seg_bytes(i)
        jobs += [(min(PIECE, ln - o), "gctr", i, o) for o in range(0, ln, PIECE)]

    hashes = {}  # (segment, piece offset) -> oracle GHASH of the ciphertext piece

    def one(job):
        ln, kind, i, o = job
        off, _ = t.seg_bytes(i)
        pt = t.generate(DEV, off + o, ln).cpu().numpy()
        got = d[off + o:off + o + ln].cpu().numpy()
        s = t.segs[i]
        u = int(s["user"])
        if kind == "whole":
            st, o_ct, o_tag, o_ver = oracle.seal(pt, ln // rb, rb, table1(t, i), w.keys, w.nonce_base,
                                                 labels=seg_labels(t, t.labels, i))
            if st != 0 or int(o_ver[0]) != gift.SEG_OK:
                return f"segment {i}: oracle status {st}, verdict {int(o_ver[0])}"
            if o_tag.tobytes() != tags_h[i].tobytes():
                return f"segment {i}: tag differs"
            exp = o_ct
        else:
            iv = oracle.segment_iv(w.nonce_base[u].tobytes(), int(s["iv_seq"]))
            icb = iv + (2 + o // 16).to_bytes(4, "big")
            exp = np.frombuffer(oracle.gctr(w.keys[u].tobytes(), icb, pt), np.uint8)
            hashes[(i, o)] = oracle.ghash(h_of[u], got)
        if not np.array_equal(exp, got):
            return f"segment {i} ({kind}) at +{o}: ciphertext differs at byte {first_diff(exp, got)}"
        return None

    h_of = {u: oracle.aes_encrypt_block(w.keys[u].tobytes(), bytes(16)) for u in set(int(x) for x in t.segs["user"])}
    t0 = time.perf_counter()
    bad = run_longest_first(jobs, one)
    whole_bytes = sum(t.seg_bytes(i)[1] for i in whole)
    log(f"llama3_70b_kv: {len(whole)} whole segments ({whole_bytes / 1e9:.2f} GB, tags too) and "
        f"{(t.nbytes - whole_bytes) / 1e9:.2f} GB in {PIECE >> 20} MiB GCTR + GHASH pieces against the oracle "
        f"in {time.perf_counter() - t0:.0f} s")
    assert not bad, bad
    # tags of the segments checked in pieces: S = sum over pieces of
    # GHASH(piece) * H^(blocks after the piece, the length block included),
    # plus L * H for the length block L; tag = E_K(J0) xor S
    for i in range(n):
        if i in whole:
            continue
        s = t.segs[i]
        u = int(s["user"])
        _, ln = t.seg_bytes(i)
        assert ln % 16 == 0
        m = ln // 16 + 1  # blocks hashed, the length block last
        acc = bytes(16)
        for o in range(0, ln, PIECE):
            b = (o + min(PIECE, ln - o)) // 16
            acc = bytes(x ^ y for x, y in zip(acc, oracle.gf128_mul(hashes[(i, o)], gf_pow(h_of[u], m - b))))
        lblock = (0).to_bytes(8, "big") + (8 * ln).to_bytes(8, "big")
        acc = bytes(x ^ y for x, y in zip(acc, oracle.gf128_mul(lblock, h_of[u])))
        iv = oracle.segment_iv(w.nonce_base[u].tobytes(), int(s["iv_seq"]))
        ekj0 = oracle.aes_encrypt_block(w.keys[u].tobytes(), iv + (1).to_bytes(4, "big"))
        tag = bytes(x ^ y for x, y in zip(ekj0, acc))
        assert tag == tags_h[i].tobytes(), f"segment {i}: tag differs from the oracle's"
    # in-place open: back to the plaintext, regenerated piece by piece
    _, ver2 = open_(d, t.n_rows, rb, t.segs, kt, w.nonce_base, tags, labels_dev=lab, out=d)
    assert (host(ver2)[:n] == gift.SEG_OK).all()
    for o in range(0, t.nbytes, 1 << 30):
        m = min(1 << 30, t.nbytes - o)
        assert torch.equal(d[o:o + m], t.generate(DEV, o, m)), f"open output differs in [{o}, +{m})"
    del d
    kt.destroy()
    torch.cuda.empty_cache()
