"""Seeded synthetic workloads for the five benchmark configurations.

This module is the only code shared by the GPU path's tests/benchmark and the
CPU oracle's: it builds keys, nonce bases, segment tables, row labels, tamper
choices and tensor contents from counter-based splitmix64 streams.  It holds
none of the cipher's arithmetic.

Shapes follow the GIFT paper's serving workloads (Sec. 4.2: hidden-state rows
and paged KV blocks are the ownership units; Sec. 4.5: generated tokens are
exported per user):

  tiny          bf16 16 x 4096, 4 users, a seeded composition of the 16 rows
                into 4 segments.
  llama3_8b_kv  KV handoff of 64 requests from 16 users, sequence lengths
                uniform in [128, 2048]; one 16-token block holds 32 layers x
                (K,V) x 8 heads x 128 dims bf16, viewed as 32 rows of 64 KiB
                (one per layer); one segment per request.
  tamper        as llama3_8b_kv with 128 requests from 32 users; after
                sealing, 1% of segments get one flipped ciphertext bit and 1%
                one flipped tag bit; another 1% carry one relabelled row.
  decode_batch  1024 users owning 1-4 consecutive rows each of a bf16
                hidden-state tensor (hidden 8192) and of an int32 token
                buffer with the same ownership.
  llama3_70b_kv as llama3_8b_kv with 32 requests from 8 users, lengths
                uniform in [2048, 8192] and 80 layers; sealed in place with
                the owner check fused.

Tensor contents: bf16 values approximately N(0,1) (Irwin-Hall sum of four
16-bit uniforms, rounded to bf16), tokens uniform in a 128256-entry vocabulary.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

SEED_BASE = 0x6171F7
_M64 = (1 << 64) - 1

SEGMENT_DTYPE = np.dtype([("row_begin", "<u8"), ("row_count", "<u8"), ("user", "<u4"),
                          ("reserved", "<u4"), ("iv_seq", "<u8")])

# KV block geometry (bf16): 2 (K,V) x 8 KV heads x 128 head_dim x 16 tokens
KV_ROW_BYTES = 2 * 8 * 128 * 16 * 2
TOKENS_PER_BLOCK = 16
VOCAB = 128256


# ----------------------------------------------------------------------------
# counter-based splitmix64
# ----------------------------------------------------------------------------
def _sm64_np(x):
    x = (x + np.uint64(0x9E3779B97F4A7C15)).astype(np.uint64)
    x = ((x ^ (x >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)).astype(np.uint64)
    x = ((x ^ (x >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)).astype(np.uint64)
    return (x ^ (x >> np.uint64(31))).astype(np.uint64)


def _sm64_int(x):
    x = (x + 0x9E3779B97F4A7C15) & _M64
    x = ((x ^ (x >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & _M64
    return x ^ (x >> 31)


def stream_key(seed, domain):
    """64-bit key of one named random stream."""
    k = _sm64_int(seed & _M64)
    for ch in domain.encode():
        k = _sm64_int(k ^ ch)
    return k


def u64s(seed, domain, n, start=0):
    """n values of stream (seed, domain) at counters start..start+n-1."""
    with np.errstate(over="ignore"):
        idx = np.arange(start, start + n, dtype=np.uint64) + np.uint64(stream_key(seed, domain))
        return _sm64_np(idx)


def uniform_ints(seed, domain, n, lo, hi):
    """n integers uniform in [lo, hi] (inclusive), by rejection-free 128-bit
    multiply-shift of the 64-bit stream."""
    span = hi - lo + 1
    v = u64s(seed, domain, n)
    return np.array([lo + ((int(x) * span) >> 64) for x in v], dtype=np.int64)


def permutation(seed, domain, n):
    keys = u64s(seed, domain, n)
    return np.argsort(keys, kind="stable")


def random_bytes(seed, domain, nbytes):
    words = u64s(seed, domain, (nbytes + 7) // 8)
    return words.view(np.uint8)[:nbytes].copy()


# ----------------------------------------------------------------------------
# tensor contents (torch, identical on CPU and GPU)
# ----------------------------------------------------------------------------
def _torch_sm64(x):
    import torch
    # int64 arithmetic wraps modulo 2^64; >> on int64 is arithmetic, so mask
    # to make it logical.
    def c(v):
        return v - (1 << 64) if v >= (1 << 63) else v

    def lsr(v, k):
        return (v >> k) & ((1 << (64 - k)) - 1)

    x = x + c(0x9E3779B97F4A7C15)
    x = (x ^ lsr(x, 30)) * c(0xBF58476D1CE4E5B9)
    x = (x ^ lsr(x, 27)) * c(0x94D049BB133111EB)
    return x ^ lsr(x, 31)


_IH4_SCALE = np.float32(1.0 / (65536.0 * np.sqrt(4.0 / 12.0)))  # 1 / std of a sum of four 16-bit uniforms


def fill_bf16_normal(out_u8, seed, elem_offset=0, chunk_elems=1 << 26):
    """Writes approximately N(0,1) bf16 values for element indices
    elem_offset.. into the uint8 torch tensor out_u8 (length a multiple of 2)."""
    import torch
    n = out_u8.numel() // 2
    view = out_u8.view(torch.bfloat16)
    key = stream_key(seed, "bf16")
    keyc = key - (1 << 64) if key >= (1 << 63) else key
    for s in range(0, n, chunk_elems):
        m = min(chunk_elems, n - s)
        idx = torch.arange(elem_offset + s, elem_offset + s + m, dtype=torch.int64, device=out_u8.device) + keyc
        h = _torch_sm64(idx)
        acc = (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + ((h >> 48) & 0xFFFF)
        z = (acc - 131070).to(torch.float32) * float(_IH4_SCALE)
        view[s:s + m] = z.to(torch.bfloat16)
        del idx, h, acc, z


def fill_tokens(out_u8, seed, elem_offset=0, chunk_elems=1 << 26):
    """Writes int32 token ids uniform in [0, VOCAB) into out_u8."""
    import torch
    n = out_u8.numel() // 4
    view = out_u8.view(torch.int32)
    key = stream_key(seed, "tok")
    keyc = key - (1 << 64) if key >= (1 << 63) else key
    for s in range(0, n, chunk_elems):
        m = min(chunk_elems, n - s)
        idx = torch.arange(elem_offset + s, elem_offset + s + m, dtype=torch.int64, device=out_u8.device) + keyc
        h = (_torch_sm64(idx) >> 1) & ((1 << 62) - 1)
        view[s:s + m] = (h % VOCAB).to(torch.int32)


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------
@dataclass
class TensorSpec:
    name: str
    n_rows: int
    row_bytes: int
    dtype: str  # "bf16" | "i32"
    data_seed: int
    segs: np.ndarray  # SEGMENT_DTYPE
    labels: Optional[np.ndarray] = None  # uint32[n_rows] or None (no fused check)

    @property
    def nbytes(self):
        return self.n_rows * self.row_bytes

    def generate(self, device="cpu", byte_off=0, nbytes=None):
        """Tensor contents [byte_off, byte_off + nbytes) as a uint8 torch tensor."""
        import torch
        if nbytes is None:
            nbytes = self.nbytes - byte_off
        out = torch.empty(nbytes, dtype=torch.uint8, device=device)
        esz = 2 if self.dtype == "bf16" else 4
        assert byte_off % esz == 0 and nbytes % esz == 0
        if self.dtype == "bf16":
            fill_bf16_normal(out, self.data_seed, byte_off // esz)
        else:
            fill_tokens(out, self.data_seed, byte_off // esz)
        return out

    def seg_bytes(self, i):
        s = self.segs[i]
        return int(s["row_begin"]) * self.row_bytes, int(s["row_count"]) * self.row_bytes


@dataclass
class Workload:
    name: str
    seed: int
    n_users: int
    keys: np.ndarray        # uint8 [n_users, 32]
    nonce_base: np.ndarray  # uint8 [n_users, 12]
    tensors: List[TensorSpec]
    in_place: bool = False
    # tamper: list of (tensor index, segment index, kind, byte offset in the
    # tensor (kind "ct") or in the segment's tag (kind "tag"), bit)
    tamper: list = field(default_factory=list)
    # mixed-owner injections: (tensor index, segment index, row, new label)
    mixed: list = field(default_factory=list)

    @property
    def nbytes(self):
        return sum(t.nbytes for t in self.tensors)


def _keys(seed, n_users):
    return random_bytes(seed, "keys", 32 * n_users).reshape(n_users, 32), \
        random_bytes(seed, "nonce", 12 * n_users).reshape(n_users, 12)


class _IvCounter:
    """Per-user invocation counter: iv_seq values are never reused for a user."""

    def __init__(self):
        self.c = {}

    def next(self, u):
        v = self.c.get(u, 0)
        self.c[u] = v + 1
        return v


def _segments(rows_per_seg, users, ivc):
    segs = np.zeros(len(rows_per_seg), SEGMENT_DTYPE)
    r = 0
    for i, (n, u) in enumerate(zip(rows_per_seg, users)):
        segs[i]["row_begin"], segs[i]["row_count"], segs[i]["user"] = r, n, u
        segs[i]["iv_seq"] = ivc.next(int(u))
        r += n
    return segs, r


def _labels_for(segs, n_rows):
    lab = np.full(n_rows, 0xFFFFFFFF, np.uint32)
    for s in segs:
        lab[int(s["row_begin"]):int(s["row_begin"] + s["row_count"])] = s["user"]
    return lab


def tiny(seed=SEED_BASE + 1):
    n_users = 4
    keys, nb = _keys(seed, n_users)
    cuts = sorted((1 + permutation(seed, "cuts", 15))[:3].tolist())
    bounds = [0] + cuts + [16]
    rows = [bounds[i + 1] - bounds[i] for i in range(4)]
    segs, n_rows = _segments(rows, list(range(4)), _IvCounter())
    t = TensorSpec("hidden", n_rows, 4096 * 2, "bf16", stream_key(seed, "data0"), segs)
    return Workload("tiny", seed, n_users, keys, nb, [t])


def _kv(name, seed, n_req, n_users, lmin, lmax, layers):
    keys, nb = _keys(seed, n_users)
    users = uniform_ints(seed, "req_user", n_req, 0, n_users - 1)
    lens = uniform_ints(seed, "req_len", n_req, lmin, lmax)
    rows = [layers * ((int(l) + TOKENS_PER_BLOCK - 1) // TOKENS_PER_BLOCK) for l in lens]
    segs, n_rows = _segments(rows, users, _IvCounter())
    t = TensorSpec("kv", n_rows, KV_ROW_BYTES, "bf16", stream_key(seed, "data0"), segs)
    return Workload(name, seed, n_users, keys, nb, [t])


def llama3_8b_kv(seed=SEED_BASE + 2):
    return _kv("llama3_8b_kv", seed, 64, 16, 128, 2048, 32)


def tamper(seed=SEED_BASE + 3):
    w = _kv("tamper", seed, 128, 32, 128, 2048, 32)
    t = w.tensors[0]
    n = len(t.segs)
    k = -(-n // 100)  # ceil(1% of segments)
    order = permutation(seed, "tamper_pick", n)
    flip_ct = order[:k - k // 2] if k > 1 else order[:1]
    flip_tag = order[k - k // 2:k] if k > 1 else order[1:2]
    mixed = order[k:2 * k]
    r = u64s(seed, "tamper_pos", 4 * n)
    for j, i in enumerate(flip_ct):
        off, ln = t.seg_bytes(int(i))
        w.tamper.append((0, int(i), "ct", off + int(r[j] % np.uint64(ln)), int(r[n + j] % np.uint64(8))))
    for j, i in enumerate(flip_tag):
        w.tamper.append((0, int(i), "tag", int(r[2 * n + j] % np.uint64(16)), int(r[3 * n + j] % np.uint64(8))))
    lab = _labels_for(t.segs, t.n_rows)
    rm = u64s(seed, "mixed_pos", 2 * n)
    for j, i in enumerate(mixed):
        s = t.segs[int(i)]
        row = int(s["row_begin"]) + int(rm[j] % s["row_count"])
        other = (int(s["user"]) + 1 + int(rm[n + j] % np.uint64(w.n_users - 1))) % w.n_users
        lab[row] = other
        w.mixed.append((0, int(i), row, other))
    t.labels = lab
    return w


def decode_batch(seed=SEED_BASE + 4):
    n_users = 1024
    keys, nb = _keys(seed, n_users)
    order = permutation(seed, "user_order", n_users)
    rows = uniform_ints(seed, "user_rows", n_users, 1, 4)
    ivc = _IvCounter()
    rps = [int(rows[u]) for u in order]
    segs_h, n_rows = _segments(rps, order, ivc)
    segs_t, _ = _segments(rps, order, ivc)
    th = TensorSpec("hidden", n_rows, 8192 * 2, "bf16", stream_key(seed, "data0"), segs_h)
    tt = TensorSpec("tokens", n_rows, 4, "i32", stream_key(seed, "data1"), segs_t)
    return Workload("decode_batch", seed, n_users, keys, nb, [th, tt])


def llama3_70b_kv(seed=SEED_BASE + 5):
    w = _kv("llama3_70b_kv", seed, 32, 8, 2048, 8192, 80)
    w.in_place = True
    t = w.tensors[0]
    t.labels = _labels_for(t.segs, t.n_rows)
    return w


CONFIGS = {
    "tiny": tiny,
    "llama3_8b_kv": llama3_8b_kv,
    "tamper": tamper,
    "decode_batch": decode_batch,
    "llama3_70b_kv": llama3_70b_kv,
}


def get(name):
    return CONFIGS[name]()
