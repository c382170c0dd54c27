"""CPU oracle for segmented per-user AES-256-GCM seal/open and the owner check.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It wraps the plain C
oracle (liboracle.so) with ctypes and numpy; it shares no code with the GPU
library.  See gift_oracle.h for the sources each function follows.
"""
import ctypes
import os

import numpy as np

from . import build as _build

OK, E_INVALID, E_RANGE, E_OVERLAP, E_NONCE_REUSE, E_TOO_LARGE = 0, -1, -2, -3, -4, -5
SEG_OK, SEG_AUTH_FAIL, SEG_OWNER_MIXED = 0, 1, 2
LABEL_PARAM, LABEL_UNOWNED = 0xFFFFFFFE, 0xFFFFFFFF

SEGMENT_DTYPE = np.dtype([("row_begin", "<u8"), ("row_count", "<u8"), ("user", "<u4"),
                          ("reserved", "<u4"), ("iv_seq", "<u8")])


class _Segment(ctypes.Structure):
    _fields_ = [("row_begin", ctypes.c_uint64), ("row_count", ctypes.c_uint64),
                ("user", ctypes.c_uint32), ("reserved", ctypes.c_uint32), ("iv_seq", ctypes.c_uint64)]


assert ctypes.sizeof(_Segment) == SEGMENT_DTYPE.itemsize == 32

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P = ctypes.c_void_p
        U64, U32, SZ = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_size_t
        L.oracle_aes_sbox.argtypes = [P, P]
        L.oracle_aes256_key_expansion.argtypes = [P, P]
        L.oracle_aes256_cipher.argtypes = [P, P, P]
        L.oracle_aes256_inv_cipher.argtypes = [P, P, P]
        L.oracle_gf128_mul.argtypes = [P, P, P]
        L.oracle_ghash.argtypes = [P, P, SZ, P]
        L.oracle_gctr.argtypes = [P, P, P, SZ, P]
        L.oracle_gcm_ae.argtypes = [P, P, P, SZ, P, P]
        L.oracle_gcm_ad.argtypes = [P, P, P, SZ, P, P]
        L.oracle_gcm_ad.restype = ctypes.c_int
        L.oracle_segment_iv.argtypes = [P, U64, P]
        L.oracle_seal.argtypes = [P, U64, U64, P, U32, P, P, U32, P, P, P, P]
        L.oracle_seal.restype = ctypes.c_int
        L.oracle_open.argtypes = [P, U64, U64, P, U32, P, P, U32, P, P, P, P]
        L.oracle_open.restype = ctypes.c_int
        L.oracle_check_owner.argtypes = [P, U32, P, U64, P]
        L.oracle_check_owner.restype = ctypes.c_int
        L.oracle_seal_paged.argtypes = [P, P, P, U32, P, P, U32, P, P, P, P]
        L.oracle_seal_paged.restype = ctypes.c_int
        L.oracle_open_paged.argtypes = [P, P, P, U32, P, P, U32, P, P, P, P]
        L.oracle_open_paged.restype = ctypes.c_int
        L.oracle_token_encrypt.argtypes = [P, U32, U64, P, P, P, U32, U64, P]
        L.oracle_token_encrypt.restype = ctypes.c_int
        L.oracle_token_decrypt.argtypes = [P, U32, U64, P, P, U32, U64, P, P]
        L.oracle_token_decrypt.restype = ctypes.c_int
        _lib = L
    return _lib


def _buf(a):
    return None if a is None else a.ctypes.data


def _u8(b, n=None):
    a = np.frombuffer(bytes(b), dtype=np.uint8) if not isinstance(b, np.ndarray) else np.ascontiguousarray(b, np.uint8)
    if n is not None:
        assert a.size == n, (a.size, n)
    return a


def sbox():
    s = np.zeros(256, np.uint8)
    inv = np.zeros(256, np.uint8)
    lib().oracle_aes_sbox(_buf(s), _buf(inv))
    return s, inv


def key_expansion(key):
    k = _u8(key, 32)
    w = np.zeros(240, np.uint8)
    lib().oracle_aes256_key_expansion(_buf(k), _buf(w))
    return w


def aes_encrypt_block(key, block):
    w = key_expansion(key)
    b = _u8(block, 16)
    o = np.zeros(16, np.uint8)
    lib().oracle_aes256_cipher(_buf(w), _buf(b), _buf(o))
    return o.tobytes()


def aes_decrypt_block(key, block):
    w = key_expansion(key)
    b = _u8(block, 16)
    o = np.zeros(16, np.uint8)
    lib().oracle_aes256_inv_cipher(_buf(w), _buf(b), _buf(o))
    return o.tobytes()


def gf128_mul(x, y):
    a, b = _u8(x, 16), _u8(y, 16)
    z = np.zeros(16, np.uint8)
    lib().oracle_gf128_mul(_buf(a), _buf(b), _buf(z))
    return z.tobytes()


def ghash(h, data):
    hh = _u8(h, 16)
    d = _u8(data)
    assert d.size % 16 == 0
    y = np.zeros(16, np.uint8)
    lib().oracle_ghash(_buf(hh), _buf(d) if d.size else None, d.size // 16, _buf(y))
    return y.tobytes()


def gcm_encrypt(key, iv, plaintext):
    k, v, p = _u8(key, 32), _u8(iv, 12), _u8(plaintext)
    c = np.zeros(max(p.size, 1), np.uint8)
    t = np.zeros(16, np.uint8)
    lib().oracle_gcm_ae(_buf(k), _buf(v), _buf(p) if p.size else None, p.size, _buf(c), _buf(t))
    return c[:p.size].tobytes(), t.tobytes()


def gcm_decrypt(key, iv, ciphertext, tag):
    """Returns the plaintext, or None when the tag does not verify."""
    k, v, c, t = _u8(key, 32), _u8(iv, 12), _u8(ciphertext), _u8(tag, 16)
    p = np.zeros(max(c.size, 1), np.uint8)
    ok = lib().oracle_gcm_ad(_buf(k), _buf(v), _buf(c) if c.size else None, c.size, _buf(t), _buf(p))
    return p[:c.size].tobytes() if ok else None


def segment_iv(nonce_base, iv_seq):
    nb = _u8(nonce_base, 12)
    iv = np.zeros(12, np.uint8)
    lib().oracle_segment_iv(_buf(nb), ctypes.c_uint64(iv_seq), _buf(iv))
    return iv.tobytes()


def as_segments(segs):
    """Accepts a structured array of SEGMENT_DTYPE or a list of
    (row_begin, row_count, user, iv_seq) tuples."""
    if isinstance(segs, np.ndarray) and segs.dtype == SEGMENT_DTYPE:
        return np.ascontiguousarray(segs)
    a = np.zeros(len(segs), SEGMENT_DTYPE)
    for i, s in enumerate(segs):
        a[i]["row_begin"], a[i]["row_count"], a[i]["user"], a[i]["iv_seq"] = s[0], s[1], s[2], s[3]
        if len(s) > 4:
            a[i]["reserved"] = s[4]
    return a


def seal(data, n_rows, row_bytes, segs, keys, nonce_base, labels=None, out=None):
    """Returns (status, out_bytes, tags[n,16], verdicts[n])."""
    d = np.ascontiguousarray(np.frombuffer(data, np.uint8) if isinstance(data, (bytes, bytearray)) else data,
                             np.uint8).reshape(-1)
    assert d.size == n_rows * row_bytes
    sg = as_segments(segs)
    o = np.zeros(max(d.size, 1), np.uint8) if out is None else out
    tags = np.zeros((max(len(sg), 1), 16), np.uint8)
    ver = np.full(max(len(sg), 1), -99, np.int32)
    lab = None if labels is None else np.ascontiguousarray(labels, np.uint32)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    nb = np.ascontiguousarray(nonce_base, np.uint8).reshape(-1)
    st = lib().oracle_seal(_buf(d), n_rows, row_bytes, _buf(sg), len(sg), _buf(lab), _buf(k), k.size // 32,
                           _buf(nb), _buf(o), _buf(tags), _buf(ver))
    return st, o[:d.size], tags[:len(sg)], ver[:len(sg)]


def open_(data, n_rows, row_bytes, segs, keys, nonce_base, tags, labels=None, out=None):
    """Returns (status, out_bytes, verdicts[n])."""
    d = np.ascontiguousarray(np.frombuffer(data, np.uint8) if isinstance(data, (bytes, bytearray)) else data,
                             np.uint8).reshape(-1)
    assert d.size == n_rows * row_bytes
    sg = as_segments(segs)
    o = np.zeros(max(d.size, 1), np.uint8) if out is None else out
    t = np.ascontiguousarray(tags, np.uint8).reshape(-1)
    if t.size == 0:
        t = np.zeros(16, np.uint8)
    ver = np.full(max(len(sg), 1), -99, np.int32)
    lab = None if labels is None else np.ascontiguousarray(labels, np.uint32)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    nb = np.ascontiguousarray(nonce_base, np.uint8).reshape(-1)
    st = lib().oracle_open(_buf(d), n_rows, row_bytes, _buf(sg), len(sg), _buf(lab), _buf(k), k.size // 32,
                           _buf(nb), _buf(o), _buf(t), _buf(ver))
    return st, o[:d.size], ver[:len(sg)]


def check_owner(segs, labels, n_rows):
    """Returns (status, verdicts[n])."""
    sg = as_segments(segs)
    lab = None if labels is None else np.ascontiguousarray(labels, np.uint32)
    ver = np.full(max(len(sg), 1), -99, np.int32)
    st = lib().oracle_check_owner(_buf(sg), len(sg), _buf(lab), n_rows, _buf(ver))
    return st, ver[:len(sg)]


def gctr(key, icb, data):
    """GCTR_K(ICB, X) (SP 800-38D Algorithm 3) -- lets a test check any block
    of a long message one at a time."""
    w = key_expansion(key)
    cb = _u8(icb, 16)
    x = _u8(data)
    y = np.zeros(max(x.size, 1), np.uint8)
    lib().oracle_gctr(_buf(w), _buf(cb), _buf(x) if x.size else None, x.size, _buf(y))
    return y[:x.size].tobytes()


def token_encrypt(segs, tokens, nonces, keys, eos_token):
    """GIFT Sec. 4.5 per-token encryption.  Returns (status, blocks[n, 16])."""
    sg = as_segments(segs)
    t = np.ascontiguousarray(tokens, np.uint64)
    n = np.ascontiguousarray(nonces, np.uint64)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    out = np.zeros((max(t.size, 1), 16), np.uint8)
    st = lib().oracle_token_encrypt(_buf(sg) if len(sg) else None, len(sg), t.size, _buf(t), _buf(n), _buf(k),
                                    k.size // 32, ctypes.c_uint64(eos_token), _buf(out))
    return st, out[:t.size]


def token_decrypt(segs, blocks, keys, eos_token):
    """Returns (status, tokens[n], nonces[n])."""
    sg = as_segments(segs)
    b = np.ascontiguousarray(blocks, np.uint8).reshape(-1, 16)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    nt = b.shape[0]
    tok = np.zeros(max(nt, 1), np.uint64)
    non = np.zeros(max(nt, 1), np.uint64)
    st = lib().oracle_token_decrypt(_buf(sg) if len(sg) else None, len(sg), nt, _buf(b), _buf(k), k.size // 32,
                                    ctypes.c_uint64(eos_token), _buf(tok), _buf(non))
    return st, tok[:nt], non[:nt]


class PagedKV(ctypes.Structure):
    _fields_ = [("cache_bytes", ctypes.c_uint64), ("layer_stride", ctypes.c_uint64),
                ("block_stride", ctypes.c_uint64), ("part_stride", ctypes.c_uint64),
                ("chunk_bytes", ctypes.c_uint64), ("n_layers", ctypes.c_uint32), ("n_parts", ctypes.c_uint32),
                ("n_blocks", ctypes.c_uint64)]


class _Request(ctypes.Structure):
    _fields_ = [("block_ids", ctypes.c_void_p), ("n_block_ids", ctypes.c_uint32), ("user", ctypes.c_uint32),
                ("iv_seq", ctypes.c_uint64)]


def _requests(reqs):
    """reqs: list of (block_ids, user, iv_seq); returns (ctypes array, keep-alive list)."""
    keep = [np.ascontiguousarray(b, np.uint32) for b, _, _ in reqs]
    arr = (_Request * max(len(reqs), 1))()
    for i, ((_, u, q), b) in enumerate(zip(reqs, keep)):
        arr[i] = _Request(b.ctypes.data if b.size else None, b.size, u, q)
    return arr, keep


def seal_paged(cache, geom, reqs, keys, nonce_base, labels=None):
    """cache: host uint8 array of geom.cache_bytes; geom: PagedKV; reqs: list of
    (block_ids, user, iv_seq).  Returns (status, out, tags[n,16], verdicts[n])."""
    c = np.ascontiguousarray(cache, np.uint8).reshape(-1)
    arr, keep = _requests(reqs)
    per = geom.n_layers * geom.n_parts * geom.chunk_bytes
    total = sum(per * len(b) for b in keep)
    out = np.zeros(max(total, 1), np.uint8)
    tags = np.zeros((max(len(reqs), 1), 16), np.uint8)
    ver = np.full(max(len(reqs), 1), -99, np.int32)
    lab = None if labels is None else np.ascontiguousarray(labels, np.uint32)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    nb = np.ascontiguousarray(nonce_base, np.uint8).reshape(-1)
    st = lib().oracle_seal_paged(_buf(c), ctypes.byref(geom), ctypes.addressof(arr), len(reqs), _buf(lab), _buf(k),
                                 k.size // 32, _buf(nb), _buf(out), _buf(tags), _buf(ver))
    return st, out[:total], tags[:len(reqs)], ver[:len(reqs)]


def open_paged(cache, geom, reqs, keys, nonce_base, sealed, tags, labels=None):
    """Opens into a copy of cache; returns (status, cache_after, verdicts[n])."""
    c = np.array(cache, np.uint8).reshape(-1)
    arr, keep = _requests(reqs)
    s_ = np.ascontiguousarray(sealed, np.uint8).reshape(-1)
    t = np.ascontiguousarray(tags, np.uint8).reshape(-1)
    ver = np.full(max(len(reqs), 1), -99, np.int32)
    lab = None if labels is None else np.ascontiguousarray(labels, np.uint32)
    k = np.ascontiguousarray(keys, np.uint8).reshape(-1)
    nb = np.ascontiguousarray(nonce_base, np.uint8).reshape(-1)
    st = lib().oracle_open_paged(_buf(c), ctypes.byref(geom), ctypes.addressof(arr), len(reqs), _buf(lab), _buf(k),
                                 k.size // 32, _buf(nb), _buf(s_) if s_.size else None, _buf(t) if t.size else None,
                                 _buf(ver))
    return st, c, ver[:len(reqs)]
