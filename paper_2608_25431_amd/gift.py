"""ctypes binding of libgift.so (include/gift.h): argument marshalling only.

Every entry point has the C name without the ``gift_`` prefix.  Device
buffers may be passed as torch tensors (their ``data_ptr()`` is used) or as
raw integer device addresses; host arrays are numpy arrays or bytes.  A
tensor passed as a device buffer must be a contiguous CUDA tensor of at
least the bytes the call touches, else ValueError is raised before the call
(the C ABI cannot see buffer sizes).  A non-OK status raises
:class:`GiftError`.  There is no fallback: if the HIP
library is not built, importing the binding's functions raises.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgift.so")

OK, E_INVALID, E_RANGE, E_OVERLAP, E_NONCE_REUSE, E_TOO_LARGE, E_HIP, E_NOMEM = 0, -1, -2, -3, -4, -5, -6, -7
E_REJECTED, E_RACE = -8, -9
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


class _Range(ctypes.Structure):
    _fields_ = [("addr", ctypes.c_uint64), ("bytes", ctypes.c_uint64)]


class _Request(ctypes.Structure):
    _fields_ = [("block_ids", ctypes.c_void_p), ("n_block_ids", ctypes.c_uint32), ("user", ctypes.c_uint32),
                ("iv_seq", ctypes.c_uint64)]


assert ctypes.sizeof(_Segment) == SEGMENT_DTYPE.itemsize == 32

EXPORTS = ("gift_key_table_create", "gift_key_table_users", "gift_key_table_destroy", "gift_seal", "gift_seal_noalloc",
           "gift_open",
           "gift_check_owner", "gift_seal_paged", "gift_open_paged", "gift_token_encrypt", "gift_token_decrypt", "gift_profile_next_call",
           "gift_status_string", "gift_last_error",
           # include/gift_ift.h
           "gift_own_create", "gift_own_destroy", "gift_own_register", "gift_own_release", "gift_own_units",
           "gift_own_flat_index", "gift_own_set", "gift_own_get", "gift_own_labels", "gift_own_ops",
           "gift_ift_add_residual", "gift_ift_add_bias", "gift_ift_find_max", "gift_ift_matmul",
           "gift_race_create", "gift_race_destroy", "gift_race_launch", "gift_race_wait", "gift_race_sync", "gift_race_sync_all",
           "gift_race_release")

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
        L.gift_seal_noalloc.argtypes = [ctypes.POINTER(_Tensor), ctypes.POINTER(_SegTable), P, P, P, P, P]
        L.gift_seal_noalloc.restype = st
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
        u32, u64 = ctypes.c_uint32, ctypes.c_uint64
        H = P
        for name, args in (
                ("gift_own_create", [ctypes.POINTER(ctypes.c_void_p)]), ("gift_own_destroy", [H]),
                ("gift_own_register", [H, P, u32, P, u32, u32]), ("gift_own_release", [H, P]),
                ("gift_own_units", [H, P, ctypes.POINTER(u64)]),
                ("gift_own_flat_index", [H, P, P, ctypes.POINTER(u64)]), ("gift_own_set", [H, P, u64, u64, u32]),
                ("gift_own_get", [H, P, u64, ctypes.POINTER(u32)]), ("gift_own_labels", [H, P, P, u64]),
                ("gift_ift_add_residual", [H, P, P, P, u64, u64, u32]),
                ("gift_ift_add_bias", [H, P, P, P, u64, u64, u32]),
                ("gift_ift_find_max", [H, P, P, u64, u64, u32, u32]),
                ("gift_ift_matmul", [H, P, P, P, u64, u64, u64, u32]),
                ("gift_race_create", [ctypes.POINTER(ctypes.c_void_p)]), ("gift_race_destroy", [H]),
                ("gift_race_launch", [H, u32, P, u32, P, u32, ctypes.POINTER(u64)]),
                ("gift_race_wait", [H, u32, u32, u64]), ("gift_race_sync", [H, u32]), ("gift_race_sync_all", [H]), ("gift_race_release", [H, _Range])):
            getattr(L, name).argtypes = args
            getattr(L, name).restype = st
        L.gift_own_ops.argtypes = [H]
        L.gift_own_ops.restype = u64
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


def _dev(x, nbytes, name):
    """Address of a device buffer of at least nbytes.  A torch tensor must be a
    contiguous CUDA tensor that large (a host buffer, or one too short, would
    make the kernels fault instead of failing here); an int is taken as a
    device address as is; None is NULL."""
    if x is None or isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        raise ValueError(f"{name}: a numpy array is host memory; pass a CUDA tensor or a device address")
    if hasattr(x, "data_ptr"):
        if not getattr(x, "is_cuda", False):
            raise ValueError(f"{name}: tensor must be on the GPU")
        if not x.is_contiguous():
            raise ValueError(f"{name}: tensor must be contiguous")
        have = x.numel() * x.element_size()
        if have < nbytes:
            raise ValueError(f"{name}: {have} bytes, the call needs {nbytes}")
        return x.data_ptr()
    raise TypeError(f"{name}: cannot take the address of {type(x)}")


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


def _table(segs, row_labels, verdicts, n_rows=0):
    sg = as_segments(segs)
    t = _SegTable(sg.ctypes.data if len(sg) else None, len(sg), _dev(row_labels, 4 * n_rows, "row_labels"),
                  _dev(verdicts, 4 * len(sg), "verdicts"))
    return t, sg


def _nonce(nonce_base, kt):
    nb = _host_u8(nonce_base)
    if kt is not None and nb.size != 12 * kt.n_users:
        raise ValueError("nonce_base must be n_users * 12 bytes")
    return nb


def seal(data, n_rows, row_bytes, segs, kt, nonce_base, out, tags, row_labels=None, verdicts=None, stream=None):
    """gift_seal.  data/out/tags/row_labels/verdicts are device buffers."""
    total = n_rows * row_bytes
    t = _Tensor(_dev(data, total, "data"), n_rows, row_bytes)
    tab, keep = _table(segs, row_labels, verdicts, n_rows)
    o, tg = _dev(out, total, "out"), _dev(tags, 16 * len(keep), "tags")
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_seal(ctypes.byref(t), ctypes.byref(tab), kt.handle, nb.ctypes.data, o, tg, _stream(stream)))
    del keep


def seal_noalloc(data, n_rows, row_bytes, segs, kt, nonce_base, out, tags, row_labels=None, verdicts=None,
                 stream=None):
    """gift_seal_noalloc: gift_seal on the device's fixed workspace (no
    device allocation; calls that overlap on one device race)."""
    total = n_rows * row_bytes
    t = _Tensor(_dev(data, total, "data"), n_rows, row_bytes)
    tab, keep = _table(segs, row_labels, verdicts, n_rows)
    o, tg = _dev(out, total, "out"), _dev(tags, 16 * len(keep), "tags")
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_seal_noalloc(ctypes.byref(t), ctypes.byref(tab), kt.handle, nb.ctypes.data, o, tg,
                                   _stream(stream)))
    del keep


def open(data, n_rows, row_bytes, segs, kt, nonce_base, out, tags, verdicts, row_labels=None, stream=None):
    """gift_open.  verdicts (device int32[n_segs]) is required."""
    total = n_rows * row_bytes
    t = _Tensor(_dev(data, total, "data"), n_rows, row_bytes)
    tab, keep = _table(segs, row_labels, verdicts, n_rows)
    o, tg = _dev(out, total, "out"), _dev(tags, 16 * len(keep), "tags")
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_open(ctypes.byref(t), ctypes.byref(tab), kt.handle, nb.ctypes.data, o, tg, _stream(stream)))
    del keep


def check_owner(segs, labels, n_rows, verdicts, stream=None):
    """gift_check_owner."""
    tab, keep = _table(segs, None, verdicts)
    _check(lib().gift_check_owner(ctypes.byref(tab), _dev(labels, 4 * n_rows, "labels"), n_rows, _stream(stream)))
    del keep


def paged_kv(cache, cache_bytes, layer_stride, block_stride, part_stride, chunk_bytes, n_layers, n_parts, n_blocks):
    """gift_paged_kv for a device allocation (torch tensor or address)."""
    return _PagedKV(_dev(cache, cache_bytes, "cache"), cache_bytes, layer_stride, block_stride, part_stride, chunk_bytes,
                    n_layers, n_parts, n_blocks)


def _requests(reqs):
    keep = [np.ascontiguousarray(b, np.uint32) for b, _, _ in reqs]
    arr = (_Request * max(len(reqs), 1))()
    for i, ((_, u, q), b) in enumerate(zip(reqs, keep)):
        arr[i] = _Request(b.ctypes.data if b.size else None, b.size, u, q)
    return arr, keep


def _paged_bufs(kv, keep, n, export, tags, verdicts, block_labels):
    total = kv.n_layers * kv.n_parts * kv.chunk_bytes * sum(int(b.size) for b in keep)
    return (_dev(export, total, "export buffer"), _dev(tags, 16 * n, "tags"), _dev(verdicts, 4 * n, "verdicts"),
            _dev(block_labels, 4 * kv.n_blocks, "block_labels"))


def seal_paged(kv, reqs, kt, nonce_base, out, tags, block_labels=None, verdicts=None, stream=None):
    """gift_seal_paged.  kv from paged_kv(); reqs: list of (block_ids, user, iv_seq)."""
    arr, keep = _requests(reqs)
    o, tg, vd, lb = _paged_bufs(kv, keep, len(reqs), out, tags, verdicts, block_labels)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_seal_paged(ctypes.byref(kv), ctypes.addressof(arr) if reqs else None, len(reqs), lb, kt.handle,
                                 nb.ctypes.data, o, tg, vd, _stream(stream)))
    del keep


def open_paged(kv, reqs, kt, nonce_base, sealed, tags, verdicts, block_labels=None, stream=None):
    """gift_open_paged."""
    arr, keep = _requests(reqs)
    sd, tg, vd, lb = _paged_bufs(kv, keep, len(reqs), sealed, tags, verdicts, block_labels)
    nb = _nonce(nonce_base, kt)
    _check(lib().gift_open_paged(ctypes.byref(kv), ctypes.addressof(arr) if reqs else None, len(reqs), lb, kt.handle,
                                 nb.ctypes.data, sd, tg, vd, _stream(stream)))
    del keep


def token_encrypt(segs, tokens, nonces, n_tokens, kt, eos_token, out, stream=None):
    """gift_token_encrypt: tokens/nonces device u64[n_tokens], out device u8[n_tokens*16]."""
    tab, keep = _table(segs, None, None)
    _check(lib().gift_token_encrypt(ctypes.byref(tab), _dev(tokens, 8 * n_tokens, "tokens"),
                                    _dev(nonces, 8 * n_tokens, "nonces"), n_tokens, kt.handle, eos_token,
                                    _dev(out, 16 * n_tokens, "out"), _stream(stream)))
    del keep


def token_decrypt(segs, blocks, n_tokens, kt, eos_token, tokens_out, nonces_out=None, stream=None):
    """gift_token_decrypt."""
    tab, keep = _table(segs, None, None)
    _check(lib().gift_token_decrypt(ctypes.byref(tab), _dev(blocks, 16 * n_tokens, "blocks"), n_tokens, kt.handle,
                                    eos_token, _dev(tokens_out, 8 * n_tokens, "tokens_out"),
                                    _dev(nonces_out, 8 * n_tokens, "nonces_out"), _stream(stream)))
    del keep


def profile_next_call(before, after):
    """gift_profile_next_call: raw hipEvent_t handles (ints) or None."""
    _check(lib().gift_profile_next_call(before, after))


def raw_status(fn_name, *args):
    """Calls an entry point and returns its status instead of raising (tests)."""
    return getattr(lib(), fn_name)(*args)


# --- include/gift_ift.h: host-side ownership records, IFT rules, race checks ---

def _check_host(s):
    # the host-only tracking entry points report through their status alone
    if s != OK:
        raise GiftError(s, status_string(s))


class Ownership:
    """Owns a gift_ownership handle (ownership records and IFT rules).

    Tensors are named by their base address (a torch tensor, numpy array or
    int); nothing is dereferenced."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check_host(lib().gift_own_create(ctypes.byref(h)))
        self.handle = h.value

    def destroy(self):
        if self.handle:
            h, self.handle = self.handle, None
            _check_host(lib().gift_own_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def register(self, base, shape, elem_size, odims=(0,)):
        sh = np.ascontiguousarray(shape, np.uint64)
        mask = 0
        for d in odims:
            mask |= 1 << d
        _check_host(lib().gift_own_register(self.handle, _ptr(base), sh.size, sh.ctypes.data, elem_size, mask))

    def release(self, base):
        _check_host(lib().gift_own_release(self.handle, _ptr(base)))

    def units(self, base):
        n = ctypes.c_uint64()
        _check_host(lib().gift_own_units(self.handle, _ptr(base), ctypes.byref(n)))
        return n.value

    def flat_index(self, base, subs):
        s = np.ascontiguousarray(subs, np.uint64)
        f = ctypes.c_uint64()
        _check_host(lib().gift_own_flat_index(self.handle, _ptr(base), s.ctypes.data if s.size else None,
                                              ctypes.byref(f)))
        return f.value

    def set(self, base, flat_begin, count, owner):
        _check_host(lib().gift_own_set(self.handle, _ptr(base), flat_begin, count, owner))

    def get(self, base, flat):
        o = ctypes.c_uint32()
        _check_host(lib().gift_own_get(self.handle, _ptr(base), flat, ctypes.byref(o)))
        return o.value

    def labels(self, base):
        n = self.units(base)
        out = np.empty(n, np.uint32)
        _check_host(lib().gift_own_labels(self.handle, _ptr(base), out.ctypes.data, n))
        return out

    @property
    def ops(self):
        return lib().gift_own_ops(self.handle)

    # IFT rules: return the status (OK or E_REJECTED) instead of raising, since
    # a refusal is an expected outcome of the monitor.
    def add_residual(self, out, inp, res, rows, cols, elem_size):
        return lib().gift_ift_add_residual(self.handle, _ptr(out), _ptr(inp), _ptr(res), rows, cols, elem_size)

    def add_bias(self, out, inp, bias, rows, cols, elem_size):
        return lib().gift_ift_add_bias(self.handle, _ptr(out), _ptr(inp), _ptr(bias), rows, cols, elem_size)

    def find_max(self, out, inp, rows, cols, in_elem_size, out_elem_size):
        return lib().gift_ift_find_max(self.handle, _ptr(out), _ptr(inp), rows, cols, in_elem_size, out_elem_size)

    def matmul(self, out, inp, weight, rows, k, n, elem_size):
        return lib().gift_ift_matmul(self.handle, _ptr(out), _ptr(inp), _ptr(weight), rows, k, n, elem_size)


def ranges(rs):
    """gift_range array (uint64 [n, 2]: addr, bytes) from (addr, bytes) pairs."""
    if isinstance(rs, np.ndarray) and rs.dtype == np.uint64 and rs.ndim == 2 and rs.shape[1] == 2:
        return np.ascontiguousarray(rs)
    return np.asarray(list(rs or ()), np.uint64).reshape(-1, 2)


class RaceChecker:
    """Owns a gift_race handle (launch-order checking across streams)."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check_host(lib().gift_race_create(ctypes.byref(h)))
        self.handle = h.value

    def destroy(self):
        if self.handle:
            h, self.handle = self.handle, None
            _check_host(lib().gift_race_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def launch(self, stream, reads=(), writes=()):
        """Returns (status, seq); reads/writes are (addr, bytes) pairs or a
        ranges() array."""
        r, w = ranges(reads), ranges(writes)
        seq = ctypes.c_uint64()
        s = lib().gift_race_launch(self.handle, stream, r.ctypes.data if len(r) else None, len(r),
                                   w.ctypes.data if len(w) else None, len(w), ctypes.byref(seq))
        return s, seq.value

    def wait(self, stream, on_stream, seq):
        """Returns the status (OK, or E_RANGE for a kernel not yet launched)."""
        return lib().gift_race_wait(self.handle, stream, on_stream, seq)

    def sync(self, stream):
        _check_host(lib().gift_race_sync(self.handle, stream))

    def sync_all(self):
        _check_host(lib().gift_race_sync_all(self.handle))

    def release(self, addr, nbytes):
        _check_host(lib().gift_race_release(self.handle, _Range(addr, nbytes)))
