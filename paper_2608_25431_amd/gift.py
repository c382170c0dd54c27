"""ctypes binding of libgift.so (include/gift.h): argument marshalling only.

Every entry point has the C name without the ``gift_`` prefix.  Device
buffers may be passed as torch tensors (their ``data_ptr()`` is used) or as
raw integer device addresses; host arrays are numpy arrays or bytes.  A
non-OK status raises :class:`GiftError`.  There is no fallback: if the HIP
library is not built, importing the binding's functions raises.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgift.so")

OK, E_INVALID, E_RANGE, E_OVERLAP, E_NONCE_REUSE, E_TOO_LARGE, E_HIP, E_NOMEM = 0, -1, -2, -3, -4, -5, -6, -7
SEG_OK, SEG_AUTH_FAIL, SEG_OWNER_MIXED = 0, 1, 2
LABEL_PARAM, LABEL_UNOWNED = 0xFFFFFFFE, 0xFFFFFFFF

# Host layout of gift_segment (32 bytes).
SEGMENT_DTYPE = np.dtype([("row_begin", "<u8"), ("row_count", "<u8"), ("user", "<u4"),
                          ("reserved", "<u4"), ("iv_seq", "<u8")])


class GiftError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"gift status {status}: {message}")
        self.status = status


class _Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n_rows", ctypes.c_uint64), ("row_bytes", ctypes.c_uint64)]


class _Segment(ctypes.Structure):
    _fields_ = [("row_begin", ctypes.c_uint64), ("row_count", ctypes.c_uint64), ("user", ctypes.c_uint32),
                ("reserved", ctypes.c_uint32), ("iv_seq", ctypes.c_uint64)]


class _SegTable(ctypes.Structure):
    _fields_ = [("segs", ctypes.c_void_p), ("n_segs", ctypes.c_uint32), ("row_labels", ctypes.c_void_p),
                ("verdicts", ctypes.c_void_p)]


class _PagedKV(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("cache_bytes", ctypes.c_uint64), ("layer_stride", ctypes.c_uint64),
                ("block_stride", ctypes.c_uint64), ("part_stride", ctypes.c_uint64), ("chunk_bytes", ctypes.c_uint64),
                ("n_layers", ctypes.c_uint32), ("n_parts", ctypes.c_uint32), ("n_blocks", ctypes.c_uint64)]


class _Request(ctypes.Structure):
    _fields_ = [("block_ids", ctypes.c_void_p), ("n_block_ids", ctypes.c_uint32), ("user", ctypes.c_uint32),
                ("iv_seq", ctypes.c_uint64)]


assert ctypes.sizeof(_Segment) == SEGMENT_DTYPE.itemsize == 32

EXPORTS = ("gift_key_table_create", "gift_key_table_users", "gift_key_table_destroy", "gift_seal", "gift_open",
           "gift_check_owner", "gift_seal_paged", "gift_open_paged", "gift_token_encrypt", "gift_token_decrypt", "gift_profile_next_call",
           "gift_status_string", "gift_last_error")

_lib = None


def lib():
    """Loads libgift.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_25431_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        st = ctypes.c_int
        L.gift_key_table_create.argtypes = [P, ctypes.c_uint32, P, ctypes.POINTER(ctypes.c_void_p)]
        L.gift_key_table_create.restype = st
        L.gift_key_table_users.argtypes = [P]
        L.gift_key_table_users.restype = ctypes.c_uint32
        L.gift_key_table_destroy.argtypes = [P]
        L.gift_key_table_destroy.restype = st
        L.gift_seal.argtypes = [ctypes.POINTER(_Tensor), ctypes.POINTER(_SegTable), P, P, P, P, P]
        L.gift_seal.restype = st
        L.gift_open.argtypes = [ctypes.POINTER(_Tensor), ctypes.POINTER(_SegTable), P, P, P, P, P]
        L.gift_open.restype = st
        L.gift_check_owner.argtypes = [ctypes.POINTER(_SegTable), P, ctypes.c_uint64, P]
        L.gift_check_owner.restype = st
        L.gift_seal_paged.argtypes = [ctypes.POINTER(_PagedKV), P, ctypes.c_uint32, P, P, P, P, P, P, P]
        L.gift_seal_paged.restype = st
        L.gift_open_paged.argtypes = [ctypes.POINTER(_PagedKV), P, ctypes.c_uint32, P, P, P, P, P, P, P]
        L.gift_open_paged.restype = st
        L.gift_token_encrypt.argtypes = [ctypes.POINTER(_SegTable), P, P, ctypes.c_uint64, P, ctypes.c_uint64, P, P]
        L.gift_token_encrypt.restype = st
        L.gift_token_decrypt.argtypes = [ctypes.POINTER(_SegTable), P, ctypes.c_uint64, P, ctypes.c_uint64, P, P, P]
        L.gift_token_decrypt.restype = st
        L.gift_profile_next_call.argtypes = [P, P]
        L.gift_profile_next_call.restype = st
        L.gift_status_string.argtypes = [st]
        L.gift_status_string.restype = ctypes.c_char_p
        L.gift_last_error.argtypes = []
        L.gift_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(s):
    return lib().gift_status_string(s).decode()


def last_error():
    return lib().gift_last_error().decode()


def _check(s):
    if s != OK:
        raise GiftError(s, last_error() or status_string(s))


def _ptr(x):
    """Device/host address of a torch tensor, numpy array or int (None -> NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(stream):
    if stream is None:
        try:
            import torch
            if torch.cuda.is_available():
                return torch.cuda.current_stream().cuda_stream
        except ImportError:
            pass
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def as_segments(segs):
    """Structured SEGMENT_DTYPE array from an array or (row_begin, row_count,
    user, iv_seq[, reserved]) tuples."""
    if isinstance(segs, np.ndarray) and segs.dtype == SEGMENT_DTYPE:
        return np.ascontiguousarray(segs)
    a = np.zeros(len(segs), SEGMENT_DTYPE)
    for i, s in enumerate(segs):
        a[i]["row_begin"], a[i]["row_count"], a[i]["user"], a[i]["iv_seq"] = s[0], s[1], s[2], s[3]
        if len(s) > 4:
            a[i]["reserved"] = s[4]
    return a


def _host_u8(x, n=None):
    a = np.frombuffer(bytes(x), np.uint8) if isinstance(x, (bytes, bytearray)) else np.ascontiguousarray(x, np.uint8)
    a = a.reshape(-1)
    if n is not None and a.size != n:
        raise ValueError(f"expected {n} bytes, got {a.size}")
    return a


class KeyTable:
    """Owns a gift_key_table handle."""

    def __init__(self, keys, n_users=None, stream=None):
        k = _host_u8(keys)
        if n_users is None:
            n_users = k.size // 32
        if k.size != 32 * n_users:
            raise ValueError("keys must be n_users * 32 bytes")
        h = ctypes.c_void_p()
        _check(lib().gift_key_table_create(k.ctypes.data, n_users, _stream(stream), ctypes.byref(h)))
        self.handle = h.value
        self.n_users = n_users

    @property
    def users(self):
        return lib().gift_key_table_users(self.handle)

    def destroy(self):
        if self.handle:
            h, self.handle = self.handle, None
            _check(lib().gift_key_table_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def key_table_create(keys, n_users=None, stream=None):
    return KeyTable(keys, n_users, stream)


def _table(segs, row_labels, verdicts):
    sg = as_segments(segs)
    t = _SegTable(sg.ctypes.data if len(sg) else None, len(sg), _ptr(row_labels), _ptr(verdicts))
    return t, sg


def _nonce(nonce_base, kt):
    nb = _host_u8(nonce_base)
    if kt is not None and nb.size != 12 * kt.n_users:
        raise ValueError("nonce_base must be n_users * 12 bytes")
    return nb


def seal(data, n_rows, row_bytes, segs, kt, nonce_base, out, tags, row_labels=None, verdicts=None, stream=None):
    """gift_seal.  data/out/tags/row_labels/verdicts are device buffers."""
    t = _Tensor(_ptr(data), n_rows, row_bytes)
    tab, keep = _table(segs, row_labels, verdicts)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_seal(ctypes.byref(t), ctypes.byref(tab), kt.handle, nb.ctypes.data, _ptr(out), _ptr(tags),
                           _stream(stream)))
    del keep


def open(data, n_rows, row_bytes, segs, kt, nonce_base, out, tags, verdicts, row_labels=None, stream=None):
    """gift_open.  verdicts (device int32[n_segs]) is required."""
    t = _Tensor(_ptr(data), n_rows, row_bytes)
    tab, keep = _table(segs, row_labels, verdicts)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_open(ctypes.byref(t), ctypes.byref(tab), kt.handle, nb.ctypes.data, _ptr(out), _ptr(tags),
                           _stream(stream)))
    del keep


def check_owner(segs, labels, n_rows, verdicts, stream=None):
    """gift_check_owner."""
    tab, keep = _table(segs, None, verdicts)
    _check(lib().gift_check_owner(ctypes.byref(tab), _ptr(labels), n_rows, _stream(stream)))
    del keep


def paged_kv(cache, cache_bytes, layer_stride, block_stride, part_stride, chunk_bytes, n_layers, n_parts, n_blocks):
    """gift_paged_kv for a device allocation (torch tensor or address)."""
    return _PagedKV(_ptr(cache), cache_bytes, layer_stride, block_stride, part_stride, chunk_bytes, n_layers, n_parts,
                    n_blocks)


def _requests(reqs):
    keep = [np.ascontiguousarray(b, np.uint32) for b, _, _ in reqs]
    arr = (_Request * max(len(reqs), 1))()
    for i, ((_, u, q), b) in enumerate(zip(reqs, keep)):
        arr[i] = _Request(b.ctypes.data if b.size else None, b.size, u, q)
    return arr, keep


def seal_paged(kv, reqs, kt, nonce_base, out, tags, block_labels=None, verdicts=None, stream=None):
    """gift_seal_paged.  kv from paged_kv(); reqs: list of (block_ids, user, iv_seq)."""
    arr, keep = _requests(reqs)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_seal_paged(ctypes.byref(kv), ctypes.addressof(arr) if reqs else None, len(reqs),
                                 _ptr(block_labels), kt.handle, nb.ctypes.data, _ptr(out), _ptr(tags), _ptr(verdicts),
                                 _stream(stream)))
    del keep


def open_paged(kv, reqs, kt, nonce_base, sealed, tags, verdicts, block_labels=None, stream=None):
    """gift_open_paged."""
    arr, keep = _requests(reqs)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_open_paged(ctypes.byref(kv), ctypes.addressof(arr) if reqs else None, len(reqs),
                                 _ptr(block_labels), kt.handle, nb.ctypes.data, _ptr(sealed), _ptr(tags),
                                 _ptr(verdicts), _stream(stream)))
    del keep


def token_encrypt(segs, tokens, nonces, n_tokens, kt, eos_token, out, stream=None):
    """gift_token_encrypt: tokens/nonces device u64[n_tokens], out device u8[n_tokens*16]."""
    tab, keep = _table(segs, None, None)
    _check(lib().gift_token_encrypt(ctypes.byref(tab), _ptr(tokens), _ptr(nonces), n_tokens, kt.handle, eos_token,
                                    _ptr(out), _stream(stream)))
    del keep


def token_decrypt(segs, blocks, n_tokens, kt, eos_token, tokens_out, nonces_out=None, stream=None):
    """gift_token_decrypt."""
    tab, keep = _table(segs, None, None)
    _check(lib().gift_token_decrypt(ctypes.byref(tab), _ptr(blocks), n_tokens, kt.handle, eos_token, _ptr(tokens_out),
                                    _ptr(nonces_out), _stream(stream)))
    del keep


def profile_next_call(before, after):
    """gift_profile_next_call: raw hipEvent_t handles (ints) or None."""
    _check(lib().gift_profile_next_call(before, after))


def raw_status(fn_name, *args):
    """Calls an entry point and returns its status instead of raising (tests)."""
    return getattr(lib(), fn_name)(*args)
