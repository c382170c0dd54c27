// gfx950 kernels for segmented, per-user AES-256-GCM and the owner check.
//
// Hot path (k_gcm_tiles): one workgroup of 1024 threads per CU, persistent
// over 2 MiB tiles.  Each lane handles one 16-byte block per 1024-block row:
//   - AES-256-CTR keystream from four T-tables in LDS, each replicated 32x so
//     that lane l reads copy (l mod 32) and a wave's random lookups never
//     collide in a bank; one v_perm_b32 forms each lookup address;
//   - one coalesced 16-byte load, XOR, 16-byte store;
//   - GHASH by per-lane Horner with M = H^1024: Y <- Y*M xor X, where the
//     multiply by the fixed M uses 32 nibble-indexed tables (8 KiB per user)
//     staged in LDS.
// Tiles are aligned to the END of their segment, so the block at distance d
// from the segment's last block contributes X*H^(d + 2) to the GHASH sum; a
// tile t contributes P_t * H^(t*T) with P_t = sum of X*H^(d_t + 2) over its
// own blocks (d_t: distance from the tile's end), and lane l of a full tile
// ends at distance (1023 - l) from the tile's end.  At tile end one leader
// wave per SIMD folds the lane partials of four waves with LDS tables of
// H^256 and applies the remaining per-lane power with one generic multiply,
// while the other waves prefetch the next tile.  The host cuts some tiles
// into row pieces (every tile when a call has fewer tiles than CUs, else up
// to one per CU at the queue's tail), whose partials meet by XOR.
//
// Around it: k_prologue (first kernel of a call: staged tables from pinned
// host memory, owner check, E_K(J0) xor H*L of one-tile segments),
// k_finalize (tags of longer segments), k_small (segments up to 1 KiB),
// zero-fill, the paged-call helpers, per-token encryption and key setup.
#include <hip/hip_runtime.h>

#include <stddef.h>

#include <mutex>

#include "gift_device.hpp"
#include "gift_internal.hpp"

namespace gift {

__constant__ AesConst c_aes = make_aes_const();

constexpr int32_t kVerdictOk = 0, kVerdictAuthFail = 1, kVerdictOwnerMixed = 2;

// LDS layout of k_gcm_tiles (bytes).
constexpr uint32_t kLdsGtab = 0;                    // 32 x 16 x 16 B GHASH tables of M
constexpr uint32_t kLdsAes = 8192;                  // T0/T1 (64 KiB) then T2/T3 (64 KiB)
constexpr uint32_t kLdsFold = kLdsAes + 131072;     // 32 x 16 x 16 B GHASH tables of W
constexpr uint32_t kLdsStage = kLdsFold + 8192;     // lane partials of the waves that are not leaders
// one 16 B slot per leader, then E_K(J0) xor H*L of a one-tile segment
constexpr uint32_t kLdsRed = kLdsStage + 16 * (kThreads - 64 * kLeaders);
constexpr uint32_t kLdsInfo = kLdsRed + 16 * (kLeaders + 1);  // TileInfo of the current tile

// The current tile's record in LDS, staged by the prefetch waves.
struct TileInfo {
  uint32_t g, s, trow, user;  // queue entry
  int32_t verdict;
  uint32_t next_k;  // queue entry claimed for the next tile
  uint32_t pad[2];
  uint4 fin;  // one-tile segment: E_K(J0) xor H*L from the prologue
  SegDesc desc;
  uint32_t rk[64];  // round keys (60 used)
};
constexpr uint32_t kLdsBytes = kLdsInfo + sizeof(TileInfo);
static_assert(kLdsBytes <= 160u * 1024u, "LDS of a gfx950 workgroup");

__device__ __forceinline__ uint32_t lds32(const uint8_t* base, uint32_t off) {
  return *(const uint32_t*)(base + off);
}
__device__ __forceinline__ uint4 lds128(const uint8_t* base, uint32_t off) { return *(const uint4*)(base + off); }

// T-table address of byte k of w for lane copy L: (x << 8) | (lane*4) in the
// first 64 KiB region (T0 at +0, T1 at +128) or, with the 0x10000 bit taken
// from L, the second region (T2 at +0, T3 at +128).
#define GIFT_SEL_A(k) (0x0c0c0000u | ((4u + (k)) << 8))
#define GIFT_SEL_B(k) (0x0c020000u | ((4u + (k)) << 8))
#define GIFT_T0(w, k) lds32(tt, __builtin_amdgcn_perm((w), L, GIFT_SEL_A(k)))
#define GIFT_T1(w, k) lds32(tt + 128, __builtin_amdgcn_perm((w), L, GIFT_SEL_A(k)))
#define GIFT_T2(w, k) lds32(tt, __builtin_amdgcn_perm((w), L, GIFT_SEL_B(k)))
#define GIFT_T3(w, k) lds32(tt + 128, __builtin_amdgcn_perm((w), L, GIFT_SEL_B(k)))

// AES-256 rounds R0..13 and the final round on a state that has been through
// rounds 1..R0-1 already.
template <int R0>
__device__ __forceinline__ void aes_rounds_lds(uint32_t& s0, uint32_t& s1, uint32_t& s2, uint32_t& s3,
                                               const uint32_t* rk, const uint8_t* tt, uint32_t L) {
#pragma unroll
  for (int r = R0; r < 14; r++) {
    // The LDS is the bottleneck: a wave that is forming addresses and issuing
    // its reads runs at raised priority, so the LDS queue is refilled as soon
    // as possible, and drops back while it combines results.
    __builtin_amdgcn_s_setprio(2);
    // all 16 lookups of the round are issued before any is combined, so a
    // wave keeps 16 LDS reads in flight
    const uint32_t a0 = GIFT_T0(s0, 0), a1 = GIFT_T1(s1, 1), a2 = GIFT_T2(s2, 2), a3 = GIFT_T3(s3, 3);
    const uint32_t b0 = GIFT_T0(s1, 0), b1 = GIFT_T1(s2, 1), b2 = GIFT_T2(s3, 2), b3 = GIFT_T3(s0, 3);
    const uint32_t c0 = GIFT_T0(s2, 0), c1 = GIFT_T1(s3, 1), c2 = GIFT_T2(s0, 2), c3 = GIFT_T3(s1, 3);
    const uint32_t d0 = GIFT_T0(s3, 0), d1 = GIFT_T1(s0, 1), d2 = GIFT_T2(s1, 2), d3 = GIFT_T3(s2, 3);
    __builtin_amdgcn_sched_group_barrier(0x0002, 16, 0);  // 16 address perms
    __builtin_amdgcn_sched_group_barrier(0x0100, 16, 0);  // 16 LDS reads
    __builtin_amdgcn_sched_group_barrier(0x0002, 8, 0);   // 8 xor3
    __builtin_amdgcn_s_setprio(0);
    s0 = xor3(xor3(a0, a1, a2), a3, rk[4 * r + 0]);
    s1 = xor3(xor3(b0, b1, b2), b3, rk[4 * r + 1]);
    s2 = xor3(xor3(c0, c1, c2), c3, rk[4 * r + 2]);
    s3 = xor3(xor3(d0, d1, d2), d3, rk[4 * r + 3]);
  }
  // Last round: S(x) is byte 0 of T2[x], byte 1 of T3[x], byte 2 of T0[x],
  // byte 3 of T1[x]; v_perm merges them, and the halves do not overlap so
  // OR = XOR.
#define GIFT_LAST(a, b, c, d, rkw)                                                              \
  xor3(__builtin_amdgcn_perm(GIFT_T3(b, 1), GIFT_T2(a, 0), 0x0c0c0500u),                        \
       __builtin_amdgcn_perm(GIFT_T1(d, 3), GIFT_T0(c, 2), 0x07020c0cu), (rkw))
  const uint32_t o0 = GIFT_LAST(s0, s1, s2, s3, rk[56]);
  const uint32_t o1 = GIFT_LAST(s1, s2, s3, s0, rk[57]);
  const uint32_t o2 = GIFT_LAST(s2, s3, s0, s1, rk[58]);
  const uint32_t o3 = GIFT_LAST(s3, s0, s1, s2, rk[59]);
#undef GIFT_LAST
  s0 = o0;
  s1 = o1;
  s2 = o2;
  s3 = o3;
}

// Counter-mode caching of rounds 1-2.  In a tile, lane l encrypts the counter
// blocks IV || BE32(c + kThreads*r) for rows r, so (kThreads >= 256) the
// counter's low 8 bits never change for the lane; the first three state columns are the IV (uniform).
// After round 1 only column 1 depends on counter bits 8..15 (one lookup per
// row); columns 2 and 3 depend on bits 16..31, which change at most twice per
// tile; column 0 is fixed.  Round 2 then has one varying lookup per column.
// So per row rounds 1-2 cost 5 lookups instead of 32.
struct CtrCache {
  uint32_t u1, u2, u3, in0;  // round-1 partial columns
  uint32_t in2, in3;         // round-1 columns 2, 3 for the current counter bits 16..31
  uint32_t w0, w1, w2, w3;   // round-2 partial columns
  uint32_t hi;               // counter bits 16..31 the cache was built for
};

__device__ __forceinline__ void ctr_cache_init(CtrCache& c, uint32_t k0, uint32_t k1, uint32_t k2, uint32_t c0,
                                               const uint32_t* rk, const uint8_t* tt, uint32_t L) {
  // every lane reads its own table copy, so these are equal across the wave
  const uint32_t u0 = __builtin_amdgcn_readfirstlane(xor3(GIFT_T0(k0, 0), GIFT_T1(k1, 1), GIFT_T2(k2, 2)) ^ rk[4]);
  c.u1 = __builtin_amdgcn_readfirstlane(xor3(GIFT_T0(k1, 0), GIFT_T1(k2, 1), GIFT_T3(k0, 3)) ^ rk[5]);
  c.u2 = __builtin_amdgcn_readfirstlane(xor3(GIFT_T0(k2, 0), GIFT_T2(k0, 2), GIFT_T3(k1, 3)) ^ rk[6]);
  c.u3 = __builtin_amdgcn_readfirstlane(xor3(GIFT_T1(k0, 1), GIFT_T2(k1, 2), GIFT_T3(k2, 3)) ^ rk[7]);
  c.in0 = u0 ^ GIFT_T3(bswap32(c0) ^ rk[3], 3);  // counter byte 15: fixed per lane
  c.hi = ~(c0 >> 16);                            // forces a refresh on first use
}

// Round-2 output for counter ctr (state after rounds 1 and 2).
__device__ __forceinline__ void ctr_rounds12(CtrCache& c, uint32_t ctr, uint32_t& x0, uint32_t& x1, uint32_t& x2,
                                             uint32_t& x3, const uint32_t* rk, const uint8_t* tt, uint32_t L) {
  const uint32_t s3 = bswap32(ctr) ^ rk[3];
  if ((ctr >> 16) != c.hi) {  // rare and per lane
    c.hi = ctr >> 16;
    c.in2 = c.u2 ^ GIFT_T1(s3, 1);
    c.in3 = c.u3 ^ GIFT_T0(s3, 0);
    c.w0 = xor3(GIFT_T0(c.in0, 0), GIFT_T2(c.in2, 2), GIFT_T3(c.in3, 3)) ^ rk[8];
    c.w1 = xor3(GIFT_T1(c.in2, 1), GIFT_T2(c.in3, 2), GIFT_T3(c.in0, 3)) ^ rk[9];
    c.w2 = xor3(GIFT_T0(c.in2, 0), GIFT_T1(c.in3, 1), GIFT_T2(c.in0, 2)) ^ rk[10];
    c.w3 = xor3(GIFT_T0(c.in3, 0), GIFT_T1(c.in0, 1), GIFT_T3(c.in2, 3)) ^ rk[11];
  }
  const uint32_t in1 = c.u1 ^ GIFT_T2(s3, 2);
  x0 = c.w0 ^ GIFT_T1(in1, 1);
  x1 = c.w1 ^ GIFT_T0(in1, 0);
  x2 = c.w2 ^ GIFT_T3(in1, 3);
  x3 = c.w3 ^ GIFT_T2(in1, 2);
}

// Y*M xor X with the 32 nibble tables of M in LDS: nibble q of Y (GCM bits
// 4q..4q+3; q even = high nibble of byte q/2) selects entry q*256 + v*16.
// 16 * (high nibble of byte k of w) and 16 * (low nibble of byte k of w),
// one SDWA instruction each (byte select on the source; for the low nibble
// the shifted byte is written to byte 0 of a zeroed result).
__device__ __forceinline__ uint32_t nib_hi16(uint32_t w, int k) {
  uint32_t r;
  switch (k) {
    case 0: asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 src1_sel:DWORD" : "=v"(r) : "v"(w), "v"(0xF0u)); break;
    case 1: asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD" : "=v"(r) : "v"(w), "v"(0xF0u)); break;
    case 2: asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD" : "=v"(r) : "v"(w), "v"(0xF0u)); break;
    default: asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD" : "=v"(r) : "v"(w), "v"(0xF0u)); break;
  }
  return r;
}
__device__ __forceinline__ uint32_t nib_lo16(uint32_t w, int k) {
  uint32_t r;
  switch (k) {
    case 0: asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0" : "=v"(r) : "v"(4u), "v"(w)); break;
    case 1: asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1" : "=v"(r) : "v"(4u), "v"(w)); break;
    case 2: asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2" : "=v"(r) : "v"(4u), "v"(w)); break;
    default: asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3" : "=v"(r) : "v"(4u), "v"(w)); break;
  }
  return r;
}

__device__ __forceinline__ u128 ghash_step_lds(const u128& y, const u128& x, const uint8_t* gt) {
  uint32_t a0 = x.w[0], a1 = x.w[1], a2 = x.w[2], a3 = x.w[3];
#pragma unroll
  for (int j = 0; j < 4; j++) {
    // eight table reads per word of Y in flight, then an xor tree
    const uint32_t w = y.w[j];
    uint4 e[8];
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const int q = 2 * (4 * j + k);
      e[2 * k] = lds128(gt + q * 256, nib_hi16(w, k));
      e[2 * k + 1] = lds128(gt + (q + 1) * 256, nib_lo16(w, k));
    }
    __builtin_amdgcn_sched_group_barrier(0x0002, 8, 1);  // addresses
    __builtin_amdgcn_sched_group_barrier(0x0100, 8, 1);  // 8 LDS reads
    __builtin_amdgcn_sched_group_barrier(0x0002, 16, 1); // xor3s
#pragma unroll
    for (int k = 0; k < 8; k += 2) {
      a0 = xor3(a0, e[k].x, e[k + 1].x);
      a1 = xor3(a1, e[k].y, e[k + 1].y);
      a2 = xor3(a2, e[k].z, e[k + 1].z);
      a3 = xor3(a3, e[k].w, e[k + 1].w);
    }
  }
  return u128{{a0, a1, a2, a3}};
}

// The same product for the tile end, one word of y (eight table reads) per
// loop iteration: the words rotate through w0, so nothing is indexed at run
// time, and the fold stays within the registers a call may clobber (more in
// flight would make it save callee-saved registers to scratch at every tile
// end).
__device__ __forceinline__ u128 ghash_step_lds_lean(const u128& y, const u128& x, const uint8_t* gt) {
  uint32_t a0 = x.w[0], a1 = x.w[1], a2 = x.w[2], a3 = x.w[3];
  uint32_t w0 = y.w[0], w1 = y.w[1], w2 = y.w[2], w3 = y.w[3];
#pragma unroll 1
  for (int j = 0; j < 4; j++) {
    const uint8_t* g = gt + j * 8 * 256;
    uint4 e[8];
#pragma unroll
    for (int k = 0; k < 4; k++) {
      e[2 * k] = lds128(g + (2 * k) * 256, nib_hi16(w0, k));
      e[2 * k + 1] = lds128(g + (2 * k + 1) * 256, nib_lo16(w0, k));
    }
#pragma unroll
    for (int k = 0; k < 8; k += 2) {
      a0 = xor3(a0, e[k].x, e[k + 1].x);
      a1 = xor3(a1, e[k].y, e[k + 1].y);
      a2 = xor3(a2, e[k].z, e[k + 1].z);
      a3 = xor3(a3, e[k].w, e[k + 1].w);
    }
    w0 = w1;
    w1 = w2;
    w2 = w3;
  }
  return u128{{a0, a1, a2, a3}};
}

__device__ __forceinline__ u128 load_block(const uint8_t* p, uint32_t n, bool aligned) {
  if (aligned && n == 16) {
    uint4 v = *(const uint4*)p;
    return u128{{v.x, v.y, v.z, v.w}};
  }
  u128 r = u128_zero();
#pragma unroll
  for (uint32_t k = 0; k < 16; k++)
    if (k < n) r.w[k >> 2] |= (uint32_t)p[k] << (8 * (k & 3));
  return r;
}

__device__ __forceinline__ void store_block(uint8_t* p, const u128& v, uint32_t n, bool aligned) {
  if (aligned && n == 16) {
    *(uint4*)p = make_uint4(v.w[0], v.w[1], v.w[2], v.w[3]);
    return;
  }
#pragma unroll
  for (uint32_t k = 0; k < 16; k++)
    if (k < n) p[k] = (uint8_t)(v.w[k >> 2] >> (8 * (k & 3)));
}

// keep the first n bytes of a block, zero the rest
__device__ __forceinline__ u128 mask_block(const u128& v, uint32_t n) {
  if (n >= 16) return v;
  u128 r = v;
#pragma unroll
  for (int j = 0; j < 4; j++) {
    int keep = (int)n - 4 * j;
    uint32_t m = keep >= 4 ? 0xFFFFFFFFu : (keep <= 0 ? 0u : ((1u << (8 * keep)) - 1u));
    r.w[j] &= m;
  }
  return r;
}

// Whole-block stream of the per-block kernel: every plaintext and ciphertext
// block passes through the caches once, so its 16-byte load and store carry
// the non-temporal hint.  Measured on llama3_8b_kv: seal kernel -0.75%.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint8_t* p) {
  const u32x4 t = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void st_stream(uint8_t* p, const uint4& v) {
  const u32x4 t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, (u32x4*)p);
}

__device__ __forceinline__ u128 ld_u128(const uint4* p) {
  uint4 v = *p;
  return u128{{v.x, v.y, v.z, v.w}};
}
__device__ __forceinline__ void st_u128(uint4* p, const u128& v) { *p = make_uint4(v.w[0], v.w[1], v.w[2], v.w[3]); }

// GHASH length block 0^64 || BE64(8*len) as block words.
__device__ __forceinline__ u128 length_block(uint64_t len) {
  uint64_t bits = len * 8ull;
  return u128{{0u, 0u, bswap32((uint32_t)(bits >> 32)), bswap32((uint32_t)bits)}};
}

// Tile end of a leader wave (see k_gcm_tiles): Horner over the staged lane
// partials of its waves in W (LDS tables), one multiply by the lane's power
// hp, then the wave sum into the leader's reduction slot.  Kept out of line,
// so that the main loop's register allocation does not see it (inlined, the
// kernel spills twice as many registers); the LDS regions arrive as byte
// offsets in the LDS address space, so every access is an LDS instruction.
typedef __attribute__((address_space(3))) uint8_t lds_byte;
__device__ __noinline__ void tile_fold(u128 v, uint32_t stage_off, uint32_t wt_off, u128 hp, uint32_t red_off,
                                       uint32_t lane) {
  constexpr int kFold = kThreads / 64 / kLeaders;
  const u128* stage = (const u128*)(lds_byte*)(uintptr_t)stage_off;
  const uint8_t* wt = (const uint8_t*)(lds_byte*)(uintptr_t)wt_off;
#pragma unroll 1
  for (int i = 1; i < kFold; i++) v = ghash_step_lds_lean(v, stage[64u * kLeaders * (i - 1)], wt);
  u128 z = gf_mul(v, hp);
#pragma unroll
  for (int j = 0; j < 4; j++) z.w[j] = wave_xor(z.w[j]);
  if (lane == 0) *(u128*)(lds_byte*)(uintptr_t)red_off = z;
}

// ---------------------------------------------------------------------------
// Per-block kernel over 2 MiB tiles of the non-small segments.
// ---------------------------------------------------------------------------
template <int MODE>
__global__ __launch_bounds__(kThreads) void k_gcm_tiles(GcmArgs a) {
  constexpr bool OPEN = (MODE & kModeOpen) != 0;
  constexpr bool GATHER = (MODE & kModeGather) != 0, SCATTER = (MODE & kModeScatter) != 0;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  __shared__ uint32_t tile_failed;  // open: the tag of the tile's one-tile segment did not match
  const uint32_t tid = threadIdx.x;
  uint8_t* tt = smem + kLdsAes;
  const uint8_t* gt = smem + kLdsGtab;
  u128* red = (u128*)(smem + kLdsRed);

  // Replicated T-tables: word w = region*16384 + x*64 + slot holds
  // T_{2*region + slot/32}[x] = rotl(Te0[x], 8*table).  Four consecutive
  // slots hold the same word, so each thread writes 16 bytes at a time.
  for (uint32_t q = tid; q < 8192u; q += kThreads) {
    const uint32_t w = 4u * q;
    const uint32_t region = w >> 14, x = (w >> 6) & 255u, slot = w & 63u;
    const uint32_t tab = 2u * region + (slot >> 5);
    const uint32_t v = c_aes.te0[x];
    const uint32_t sh = 8u * tab;
    const uint32_t r = (v << sh) | (v >> ((32u - sh) & 31u));
    ((uint4*)tt)[q] = make_uint4(r, r, r, r);
  }
  const uint32_t L = ((tid & 31u) << 2) | 0x10000u;  // this lane's table copy
  uint32_t cur_user = 0xFFFFFFFFu;  // user whose GHASH tables are in LDS
  TileInfo* ti = (TileInfo*)(smem + kLdsInfo);

  // Work queue over the host's tile order (longest tiles first): workgroup b
  // takes entry b first, then entries gridDim.x + (queue claims); the claim
  // is issued when a tile starts.  While the leader waves fold a tile's GHASH
  // partials, the other waves (the prefetch waves) load the next tile's
  // entry, descriptor, verdict, round keys and, for a new user, the tables of
  // M into LDS (nothing reads them then) and the tables of W into registers
  // (the fold still reads W), so no global-memory latency sits between two
  // tiles.  Every wave leaves the loop on the same entry.
  constexpr uint32_t kPf0 = 64u * kLeaders;  // first thread of the prefetch waves
  static_assert(kThreads - kPf0 > 593u, "prefetch roles");
  uint32_t claim = 0;  // thread kPf0: queue entry of the next tile
  bool pf_tabs = false;  // this thread holds entry j of the next user's W tables
  uint4 pf_w = make_uint4(0u, 0u, 0u, 0u);
  // thread kPf0 + j: j < 512 tables; 512 + i descriptor word i (i < 16);
  // 528 + i round-key word i (i < 64); 592 entry and verdict; 593 fin
  auto prefetch = [&](uint32_t k) {
    const uint32_t j = opaque(tid) - kPf0;
    const TileEnt e = k < a.n_ents ? a.tile_order[k] : TileEnt{kNoTile, 0u, 0u, 0u};
    if (j == 592u) {
      ti->g = e.g;
      ti->s = e.s;
      ti->trow = e.trow;
      ti->user = e.user;
    }
    if (e.g == kNoTile) return;
    const uint32_t u = e.user;
    if (j < 512u) {
      if (u != cur_user) {
        pf_tabs = true;
        ((uint4*)(smem + kLdsGtab))[j] = a.kt.gtab[(size_t)u * 512u + j];
        pf_w = a.kt.gtab_fold[(size_t)u * 512u + j];
      }
    } else if (j < 528u) {
      ((uint32_t*)&ti->desc)[j - 512u] = ((const uint32_t*)(a.segs + e.s))[j - 512u];
    } else if (j < 592u) {
      ti->rk[j - 528u] = a.kt.rk[(size_t)u * 64u + (j - 528u)];
    } else if (j == 592u) {
      ti->verdict = a.verdicts[e.s];
    } else if (j == 593u) {
      ti->fin = a.fin[e.s];  // meaningful for one-tile segments only
    }
  };
  auto commit = [&]() {
    if (pf_tabs) ((uint4*)(smem + kLdsFold))[tid - kPf0] = pf_w;
    // dead until the next prefetch (which the leader waves never run): not
    // carried across the tile
    pf_tabs = false;
    pf_w = make_uint4(0u, 0u, 0u, 0u);
  };
  if (tid >= kPf0) prefetch(blockIdx.x);

  for (;;) {
    commit();
    __syncthreads();  // the tile's record and tables are in LDS; the previous tile is done with them
    const uint32_t g = __builtin_amdgcn_readfirstlane(ti->g);
    if (g == kNoTile) break;
    // the thread index, recomputed per tile: per-lane values derived from it
    // are formed here, not hoisted to the kernel's start and held (or
    // spilled) across every tile
    const uint32_t tid_t = opaque(tid);
    if (tid_t == kPf0) claim = gridDim.x + atomicAdd(a.tile_counter, 1u);
    const uint32_t s = __builtin_amdgcn_readfirstlane(ti->s);
    const uint32_t trow = __builtin_amdgcn_readfirstlane(ti->trow);
    const uint32_t t = trow & 0xFFFFu;                                      // tile of the segment
    const int r0 = (int)((trow >> 16) & 0xFFu), r1 = (int)(trow >> 24);  // its rows in this entry
    const uint32_t user = __builtin_amdgcn_readfirstlane(ti->user);
    const int32_t verdict = (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)ti->verdict);
    cur_user = user;
    const uint32_t m = __builtin_amdgcn_readfirstlane(ti->desc.nblocks);
    const uint64_t off = ti->desc.byte_off, len = ti->desc.len;
    const uint32_t flags = __builtin_amdgcn_readfirstlane(ti->desc.flags);
    const bool aligned = (flags & kSegAligned) != 0;
    // a one-tile segment whose tile is cut into pieces gets its tag from the finalize pass
    const bool one = (flags & kSegOneTile) != 0 && r0 == 0 && r1 == kRows;
    if (one && tid_t == 0) red[kLeaders] = u128{{ti->fin.x, ti->fin.y, ti->fin.z, ti->fin.w}};  // for the tile end
    const int64_t base = (int64_t)m - (int64_t)(t + 1) * (int64_t)kTileBlocks;  // block index of virtual slot 0
    const int r_start = base < 0 ? (int)((uint64_t)(-base) / kThreads) : 0;
    const int r_lo = r_start > r0 ? r_start : r0;

    // paged side: block i of the segment lives in chunk i >> shift
    const uint64_t chunk0 = ti->desc.chunk0;
    const uint64_t cmask = (1ull << a.chunk_shift) - 1;
    auto paged = [&](uint64_t i) -> uint8_t* {
      return a.pbase + a.chunk_off[chunk0 + (i >> a.chunk_shift)] + ((i & cmask) << 4);
    };

    // Tile-uniform values are read from the tile record into SGPRs
    // (readfirstlane), so the per-block loop keeps no copy of the 60
    // round-key words in VGPRs.
    uint32_t rk[60];
#pragma unroll
    for (int i = 0; i < 60; i++) rk[i] = __builtin_amdgcn_readfirstlane(ti->rk[i]);
    const uint32_t k0 = __builtin_amdgcn_readfirstlane(ti->desc.iv[0]) ^ rk[0];
    const uint32_t k1 = __builtin_amdgcn_readfirstlane(ti->desc.iv[1]) ^ rk[1];
    const uint32_t k2 = __builtin_amdgcn_readfirstlane(ti->desc.iv[2]) ^ rk[2];

    u128 y = u128_zero();
    if (verdict != kVerdictOk) {
      // rejected before this call's data is touched: release zeros only.  A
      // scatter into the cache writes nothing at all: the request's table
      // names a block of another owner, which keeps its contents.
      if (!SCATTER) {
        for (int r = r_lo; r < r1; r++) {
          const int64_t i0 = base + (int64_t)r * kThreads + tid_t;
          if (i0 >= 0) {
            const uint64_t rem = len - 16ull * (uint64_t)i0;
            store_block(a.out + off + 16ull * (uint64_t)i0, u128_zero(), rem >= 16 ? 16u : (uint32_t)rem, aligned);
          }
        }
      }
    } else {
      CtrCache cc;
      const uint32_t c0 = 2u + (uint32_t)(base + (int64_t)tid_t);  // counter of this lane in row 0, mod 2^32
      ctr_cache_init(cc, k0, k1, k2, c0, rk, tt, L);

      // rows where every lane holds a whole block and the segment is 16-byte
      // aligned take the branch-free path
      const int r_full = base < 0 ? (int)(((uint64_t)(-base) + kThreads - 1) / kThreads) : 0;
      const int r_end_full = (t == 0 && (len & 15u)) ? r1 - (r1 == kRows ? 1 : 0) : r1;

      auto whole = [&](int r) { return aligned && r >= r_full && r < r_end_full; };
      // paged: a lane's chunk offset for the next whole-block row is loaded
      // one row ahead, so the gather or scatter address is ready when the row
      // starts
      constexpr bool PAGED = GATHER || SCATTER;
      auto chunk_of = [&](int r) -> uint64_t {
        const uint64_t i0 = (uint64_t)(base + (int64_t)r * kThreads + tid_t);
        return a.chunk_off[chunk0 + (i0 >> a.chunk_shift)];
      };
      uint64_t c_next = (PAGED && whole(r_lo)) ? chunk_of(r_lo) : 0;

      for (int r = r_lo; r < r1; r++) {
        // the whole-block rows load their input before the AES rounds, so the
        // HBM latency overlaps the keystream
        const bool fast = whole(r);
        const uint64_t c_cur = c_next;
        if (PAGED && whole(r + 1)) c_next = chunk_of(r + 1);
        const uint8_t* src = nullptr;
        uint8_t* dst = nullptr;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (fast) {
          // every lane's block index is >= 0 in these rows; pointer arithmetic
          // (not integers) keeps the global address space for the compiler
          const uint64_t i0 = (uint64_t)(base + (int64_t)r * kThreads + tid_t);
          uint8_t* pg = a.pbase + c_cur + ((i0 & cmask) << 4);
          src = GATHER ? pg : a.in + off + 16ull * i0;
          dst = SCATTER ? pg : a.out + off + 16ull * i0;
          v = ld_stream(src);
        }
        uint32_t x0, x1, x2, x3;
        ctr_rounds12(cc, c0 + (uint32_t)kThreads * (uint32_t)r, x0, x1, x2, x3, rk, tt, L);
        aes_rounds_lds<3>(x0, x1, x2, x3, rk, tt, L);
        u128 x;
        if (fast) {
          const uint4 o = make_uint4(v.x ^ x0, v.y ^ x1, v.z ^ x2, v.w ^ x3);
          st_stream(dst, o);
          x = OPEN ? u128{{v.x, v.y, v.z, v.w}} : u128{{o.x, o.y, o.z, o.w}};
        } else {
          x = u128_zero();
          const int64_t i0 = base + (int64_t)r * kThreads + tid_t;
          if (i0 >= 0) {
            const uint64_t boff = off + 16ull * (uint64_t)i0;
            const uint64_t rem = len - 16ull * (uint64_t)i0;
            const uint32_t n = rem >= 16 ? 16u : (uint32_t)rem;
            const u128 in = load_block(GATHER ? paged((uint64_t)i0) : a.in + boff, n, aligned);
            const u128 o = mask_block(u128{{in.w[0] ^ x0, in.w[1] ^ x1, in.w[2] ^ x2, in.w[3] ^ x3}}, n);
            store_block(SCATTER ? paged((uint64_t)i0) : a.out + boff, o, n, aligned);
            x = OPEN ? in : o;
          }
        }
        // GHASH table reads at a priority between the AES issue and combine
        // phases; the next AES round sets its own
        __builtin_amdgcn_s_setprio(1);
        y = ghash_step_lds(y, x, gt);
      }
    }  // verdict OK

    // Tile partial: lane tid_t contributes y * H^(kThreads + 1 - tid_t), its
    // distance from the tile end plus the H^2 that every block's GHASH term
    // carries.  Wave w = g + kLeaders*i (leader g, i < kFold) needs
    // H^(64*kLeaders*(kFold - 1 - i)) * H^(64*kLeaders + 1 - 64*g - lane): leader
    // g folds its waves by Horner in W = H^(64*kLeaders) from the LDS tables,
    // then multiplies once by the per-lane power.
    const bool fold = verdict == kVerdictOk;
    // the wave index is uniform: held in a scalar register, it frees vector
    // registers across the fold call
    const uint32_t tid_e = opaque(tid);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid_e >> 6), lane = tid_e & 63u;
    u128* stage = (u128*)(smem + kLdsStage);
    if (tid == kPf0) ti->next_k = claim;
    // the leaders fetch their lane's power before the barrier, so the load
    // overlaps the wait for the other waves
    u128 hp = u128_zero();
    if (fold && wave < (uint32_t)kLeaders)
      hp = ld_u128(a.kt.pow_h + (size_t)user * kHPowers + (64u * kLeaders + 1u - 64u * wave - lane));
    if (fold && wave >= (uint32_t)kLeaders) stage[tid_e - kPf0] = y;
    __syncthreads();
    if (wave >= (uint32_t)kLeaders) {
      prefetch(ti->next_k);  // overlaps the fold
    } else if (fold) {
      const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_byte*)smem;
      tile_fold(y, lds0 + kLdsStage + 16u * (wave * 64u + lane), lds0 + kLdsFold, hp, lds0 + kLdsRed + 16u * wave,
                lane);
    }
    __syncthreads();
    // wave 0 finishes the tile (fold, one and the row range are wave-uniform);
    // lane 0 writes
    if (wave == 0) {
      if (fold) {
        u128 p = red[0];
        for (int w = 1; w < kLeaders; w++) p = u128_xor(p, red[w]);
        if (r0 == 0 && r1 == kRows) {
          if (!one && lane == 0) st_u128(a.partials + g, p);
        } else {
          // a piece of a cut tile: its lane powers assumed rows up to the
          // tile's end, so it still carries H^(kThreads * (kRows - r1));
          // pieces meet in the tile's (zeroed) partial by XOR
          if (r1 < kRows) p = gf_mul_wave(p, ld_u128(a.kt.pow_hr + (size_t)user * kRows + (kRows - r1)), lane);
          if (lane == 0) {
            uint32_t* dst = (uint32_t*)(a.partials + g);
            for (int j = 0; j < 4; j++) atomicXor(dst + j, p.w[j]);
          }
        }
        if (one && lane == 0) {
          // S = P_0 xor H*L, tag = E_K(J0) xor S (the finalize pass skips this segment)
          const u128 tag = u128_xor(p, red[kLeaders]);
          if (!OPEN) {
            uint32_t* to = (uint32_t*)(a.tags_out + 16ull * s);
            for (int j = 0; j < 4; j++) to[j] = tag.w[j];
          } else {
            const uint32_t* tin = (const uint32_t*)(a.tags_in + 16ull * s);
            uint32_t diff = 0;
            for (int j = 0; j < 4; j++) diff |= tin[j] ^ tag.w[j];
            a.verdicts[s] = diff ? kVerdictAuthFail : kVerdictOk;
            tile_failed = diff != 0u;
          }
        }
      } else if (one && !OPEN && lane == 0) {
        uint32_t* to = (uint32_t*)(a.tags_out + 16ull * s);  // rejected: zero tag
        for (int j = 0; j < 4; j++) to[j] = 0u;
      }
    }
    // open of a contiguous tensor: a one-tile segment whose tag failed
    // releases zeros only.  Its tile is the whole segment, so the workgroup
    // zeroes it here (multi-tile and cut segments are zeroed by a later pass
    // once the finalize pass has their verdicts).
    if (OPEN && !GATHER && !SCATTER && one && fold) {
      __syncthreads();  // tile_failed is written
      if (tile_failed) {
        for (int r = r_lo; r < r1; r++) {
          const int64_t i0 = base + (int64_t)r * kThreads + tid_e;
          if (i0 >= 0) {
            const uint64_t rem = len - 16ull * (uint64_t)i0;
            store_block(a.out + off + 16ull * (uint64_t)i0, u128_zero(), rem >= 16 ? 16u : (uint32_t)rem, aligned);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Per-segment finalize of tiled segments: S = sum_t P_t H^(tT) xor H*L and
// tag = E_K(J0) xor S.  One wave per segment; lane l folds tiles l, l+64, ...
// H*L is a wave sum over the set bits of L (only its low 64 bits can be set)
// of the products H*x^(64+k); E_K(J0) reads a T-table copy in LDS.
// ---------------------------------------------------------------------------
template <bool OPEN>
__global__ __launch_bounds__(kFinLanes) void k_finalize(GcmArgs a) {
  __shared__ uint32_t te[256];
  const uint32_t s = blockIdx.x, lane = threadIdx.x;
  for (uint32_t i = lane; i < 256u; i += kFinLanes) te[i] = c_aes.te0[i];
  __syncthreads();
  const SegDesc sd = a.segs[s];
  if ((sd.flags & kSegSmall) || ((sd.flags & kSegOneTile) && !a.seg_cut[s])) return;
  const int32_t verdict = a.verdicts[s];
  if (verdict != kVerdictOk) {
    if (!OPEN && lane < 4) ((uint32_t*)(a.tags_out + 16ull * s))[lane] = 0u;
    return;
  }
  const uint32_t user = sd.user;
  const uint32_t tb = a.tile_base[s], nt = a.tile_base[s + 1] - tb;
  u128 z = u128_zero();
  if (lane < nt) {
    const uint32_t K = (nt - 1 - lane) / kFinLanes + 1;
    z = ld_u128(a.partials + tb + lane + (K - 1) * kFinLanes);
    if (K > 1) {
      const u128 hlt = ld_u128(a.kt.pow_hlt + user);
      for (int k = (int)K - 2; k >= 0; k--)
        z = u128_xor(gf_mul(z, hlt), ld_u128(a.partials + tb + lane + (uint32_t)k * kFinLanes));
    }
    if (lane > 0) z = gf_mul(z, ld_u128(a.kt.pow_ht + (size_t)user * kFinLanes + lane));
  }
  // H*L: bit 64+lane of L (GCM order) is bit 63-lane of the 64-bit length in bits
  const uint64_t lbits = sd.len * 8ull;
  if ((lbits >> (63 - lane)) & 1ull) z = u128_xor(z, ld_u128(a.kt.pow_hxl + (size_t)user * kHxLanes + lane));
#pragma unroll
  for (int j = 0; j < 4; j++) z.w[j] = wave_xor(z.w[j]);
  if (lane == 0) {
    const uint32_t j0[4] = {sd.iv[0], sd.iv[1], sd.iv[2], 0x01000000u};
    uint32_t e[4];
    aes256_encrypt_tab(a.kt.rk + (size_t)user * 64u, j0, e, te);
    const u128 tag = u128{{e[0] ^ z.w[0], e[1] ^ z.w[1], e[2] ^ z.w[2], e[3] ^ z.w[3]}};
    if (!OPEN) {
      uint32_t* to = (uint32_t*)(a.tags_out + 16ull * s);
      for (int j = 0; j < 4; j++) to[j] = tag.w[j];
    } else {
      const uint8_t* ti = a.tags_in + 16ull * s;
      uint32_t diff = 0;
#pragma unroll
      for (int k = 0; k < 16; k++) diff |= (uint32_t)ti[k] ^ ((tag.w[k >> 2] >> (8 * (k & 3))) & 0xFFu);
      a.verdicts[s] = diff ? kVerdictAuthFail : kVerdictOk;
    }
  }
}

// ---------------------------------------------------------------------------
// Segments of at most 64 blocks: one wave each, lane j owns block j and its
// GHASH term X_j * H^(m + 1 - j); lane 0 adds L*H.  Open decides the verdict
// before any plaintext is written.
// ---------------------------------------------------------------------------
template <bool OPEN>
__global__ __launch_bounds__(64) void k_small(GcmArgs a) {
  __shared__ uint32_t te[256];
  for (uint32_t i = threadIdx.x; i < 256u; i += 64u) te[i] = c_aes.te0[i];
  __syncthreads();
  const uint32_t s = a.small_list[blockIdx.x];
  const uint32_t j = threadIdx.x;
  const SegDesc sd = a.segs[s];
  const uint32_t m = sd.nblocks;
  const bool valid = j < m;
  const bool aligned = (sd.flags & kSegAligned) != 0;
  const uint64_t rem = valid ? sd.len - 16ull * j : 0;
  const uint32_t n = rem >= 16 ? 16u : (uint32_t)rem;
  uint8_t* dst = a.out + sd.byte_off + 16ull * j;
  const int32_t verdict = a.verdicts[s];
  if (verdict != kVerdictOk) {
    if (valid) store_block(dst, u128_zero(), n, aligned);
    if (!OPEN && j < 4) ((uint32_t*)(a.tags_out + 16ull * s))[j] = 0u;
    return;
  }
  const uint32_t user = sd.user;
  const uint32_t* rk = a.kt.rk + (size_t)user * 64u;
  u128 in = u128_zero(), o = u128_zero(), z = u128_zero();
  if (valid) {
    in = load_block(a.in + sd.byte_off + 16ull * j, n, aligned);
    const uint32_t cb[4] = {sd.iv[0], sd.iv[1], sd.iv[2], bswap32(2u + j)};
    uint32_t ks[4];
    aes256_encrypt_tab(rk, cb, ks, te);
    o = mask_block(u128{{in.w[0] ^ ks[0], in.w[1] ^ ks[1], in.w[2] ^ ks[2], in.w[3] ^ ks[3]}}, n);
    const u128 x = OPEN ? in : o;
    z = gf_mul(x, ld_u128(a.kt.pow_h + (size_t)user * kHPowers + (m + 1 - j)));
  }
  const u128 h = ld_u128((const uint4*)(a.kt.h + 4ull * user));
  if (j == 0) z = u128_xor(z, gf_mul(length_block(sd.len), h));
#pragma unroll
  for (int k = 0; k < 4; k++) z.w[k] = wave_xor(z.w[k]);
  uint32_t ok = 1;
  if (j == 0) {
    const uint32_t j0[4] = {sd.iv[0], sd.iv[1], sd.iv[2], 0x01000000u};
    uint32_t e[4];
    aes256_encrypt_tab(rk, j0, e, te);
    const u128 tag = u128{{e[0] ^ z.w[0], e[1] ^ z.w[1], e[2] ^ z.w[2], e[3] ^ z.w[3]}};
    if (!OPEN) {
      uint32_t* to = (uint32_t*)(a.tags_out + 16ull * s);
      for (int k = 0; k < 4; k++) to[k] = tag.w[k];
    } else {
      const uint8_t* ti = a.tags_in + 16ull * s;
      uint32_t diff = 0;
#pragma unroll
      for (int k = 0; k < 16; k++) diff |= (uint32_t)ti[k] ^ ((tag.w[k >> 2] >> (8 * (k & 3))) & 0xFFu);
      ok = diff == 0;
      a.verdicts[s] = ok ? kVerdictOk : kVerdictAuthFail;
    }
  }
  if (OPEN) ok = __builtin_amdgcn_readlane((int)ok, 0) != 0;
  if (valid) store_block(dst, ok ? o : u128_zero(), n, aligned);
}

// ---------------------------------------------------------------------------
// Segment-table expansion, by one workgroup of a call's first kernel: from
// the descriptors to the tables the GCM kernels read.
//   - tile_base: exclusive scan of the tiles of each segment (small segments
//     have none), tile_base[n] = all tiles;
//   - small_list: the small segments in table order;
//   - the cut: a tile runs on one CU, so with fewer tiles than CUs every
//     tile of more than p = ceil(all tile rows / CUs) rows is cut into
//     pieces of p rows; otherwise up to one tile per CU, the largest of more
//     than kPieceRows rows (in tile order within a row count), is cut into
//     pieces of kPieceRows rows.  Pieces are aligned to the tile's end; the
//     lowest may start below the tile's first row.  A one-tile segment
//     whose tile is cut is marked in seg_cut (its tag comes from the
//     finalize pass);
//   - the work queue: every whole tile and every piece, longest first (a
//     counting sort by the rows an entry runs), padded with kNoTile up to
//     cap entries.
// Each segment's tiles are split into runs of at most kRunTiles; threads
// take contiguous ranges of runs, so thread order is tile order.  Whole
// tiles and whole pieces take their slots by a scan over the threads, in
// tile order; the other entries (partial first tiles, remainder pieces) by
// LDS atomics, in no fixed order: which CU runs which entry changes no
// result.
// ---------------------------------------------------------------------------
constexpr int kExpandThreads = 1024;  // the most threads an expanding workgroup may have
constexpr int kPrologueThreads = 256;
constexpr uint32_t kRunTiles = 16;

__device__ __forceinline__ uint32_t tiles_in(uint32_t nblocks) {
  return (uint32_t)(((uint64_t)nblocks + kTileBlocks - 1) / kTileBlocks);
}

// Rows of tile t of a segment of m blocks (tiles aligned to its end: only the
// first tile, t = tiles - 1, can be partial).
__device__ __forceinline__ uint32_t tile_rows_of(uint32_t m, uint32_t t) {
  const int64_t base = (int64_t)m - (int64_t)(t + 1) * (int64_t)kTileBlocks;
  return base >= 0 ? (uint32_t)kRows : (uint32_t)kRows - (uint32_t)((uint64_t)(-base) / kThreads);
}

// Inclusive prefix sum over the wave's 64 lanes on the VALU's data-parallel
// primitives (no LDS round trips): row shifts by 1, 2, 4 and 8 scan each row
// of 16 lanes (a lane with no source adds 0), then the broadcasts of lane 15
// into rows 1 and 3 and of lane 31 into rows 2 and 3 carry the row totals up.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// The sum over the wave, in every lane.
__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(x), 63);
}

// Exclusive prefix sum of v over the workgroup in thread order; *total gets
// the sum of all.  wsum: one LDS word per wave.
__device__ uint32_t block_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  const uint32_t x = wave_incl_scan(v);
  __syncthreads();  // wsum is free
  if (lane == 63u) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (uint32_t w = 0; w < blockDim.x / 64u; w++) {
    const uint32_t c = wsum[w];
    before += w < wave ? c : 0u;
    all += c;
  }
  *total = all;
  return before + x - v;
}

// Exclusive prefix sums of three values at once (one pass of barriers).
__device__ uint3 block_scan3(uint3 v, uint3* wsum, uint3* total) {
  const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  const uint3 x = make_uint3(wave_incl_scan(v.x), wave_incl_scan(v.y), wave_incl_scan(v.z));
  __syncthreads();  // wsum is free
  if (lane == 63u) wsum[wave] = x;
  __syncthreads();
  uint3 before = make_uint3(0u, 0u, 0u), all = make_uint3(0u, 0u, 0u);
  for (uint32_t w = 0; w < blockDim.x / 64u; w++) {
    const uint3 c = wsum[w];
    if (w < wave) {
      before.x += c.x;
      before.y += c.y;
      before.z += c.z;
    }
    all.x += c.x;
    all.y += c.y;
    all.z += c.z;
  }
  *total = all;
  return make_uint3(before.x + x.x - v.x, before.y + x.y - v.y, before.z + x.z - v.z);
}

// Expansion by the calling workgroup (all its threads call it), from the
// per-segment brief records (the source may be host memory).  A one-tile
// segment whose tile is cut gets seg_cut = 1 (every segment gets its 0 or 1).
// The per-segment values the walks need sit in LDS for up to kInfoLds
// segments, else in x.info.
constexpr uint32_t kInfoLds = 1024;

__device__ void expand_tables(const SegBrief* brief, uint32_t n, const ExpandArgs& x) {
  __shared__ uint32_t hist[kRows + 1];    // tiles by rows
  __shared__ uint32_t cursor[kRows + 1];  // entries by rows run, then the next free slot of each
  __shared__ uint32_t wsum[kExpandThreads / 64];
  __shared__ uint3 wsum3[kExpandThreads / 64];
  __shared__ uint32_t first_seg[kExpandThreads];  // segment of each thread's first run
  __shared__ SegInfo info_lds[kInfoLds];
  __shared__ unsigned long long rows_all;
  __shared__ uint32_t c_piece, c_from, c_take, c_left, c_fine, c_ents, c_full_at, c_piece_at;
  const uint32_t tid = threadIdx.x, nt_ = blockDim.x, lane = tid & 63u;
  SegInfo* info = n <= kInfoLds ? info_lds : x.info;
  for (uint32_t i = tid; i <= (uint32_t)kRows; i += nt_) hist[i] = cursor[i] = 0u;
  first_seg[tid] = 0xFFFFFFFFu;
  if (tid == 0) rows_all = 0ull;

  // the brief records, two per 16-byte load, several loads in flight per
  // thread (the source may be host memory); flags as the descriptors have them
  {
    const uint4* src = (const uint4*)brief;
    const uint32_t n16 = (n + 1) / 2;
    constexpr int kInFlight = 8;
    auto note = [&](uint32_t i, uint32_t m, uint32_t user) {
      const bool small = m <= x.small_max;
      info[i].m = m;
      info[i].flags = small ? kSegSmall : (m <= kTileBlocks ? kSegOneTile : 0u);
      info[i].user = user;
      x.seg_cut[i] = 0u;
    };
    for (uint32_t i0 = tid; i0 < n16; i0 += kInFlight * nt_) {
      uint4 q[kInFlight];
#pragma unroll
      for (int k = 0; k < kInFlight; k++)
        if (i0 + k * nt_ < n16) q[k] = src[i0 + k * nt_];
#pragma unroll
      for (int k = 0; k < kInFlight; k++) {
        const uint32_t i = i0 + k * nt_;
        if (i >= n16) break;
        note(2 * i, q[k].x, q[k].y);
        if (2 * i + 1 < n) note(2 * i + 1, q[k].z, q[k].w);
      }
    }
  }
  __syncthreads();

  // segments [s0, s1) of this thread: count tiles, rows, small segments and runs
  const uint32_t per = (n + nt_ - 1) / nt_;
  const uint32_t s0 = min(n, tid * per), s1 = min(n, s0 + per);
  uint32_t my_tiles = 0, my_small = 0, my_runs = 0, my_whole = 0;
  unsigned long long my_rows = 0;
  for (uint32_t s = s0; s < s1; s++) {
    const uint32_t m = info[s].m;
    if (info[s].flags & kSegSmall) {
      my_small++;
      continue;
    }
    const uint32_t nt = tiles_in(m), r = tile_rows_of(m, nt - 1);
    my_tiles += nt;
    my_runs += (nt + kRunTiles - 1) / kRunTiles;
    my_rows += (unsigned long long)(nt - 1) * kRows + r;
    my_whole += nt - 1;
    atomicAdd(&hist[r], 1u);
  }
  // the whole tiles below each segment's first tile, and the rows, once per
  // wave.  The rows are read only with fewer tiles than CUs, when no thread
  // has 2^20 of them; capped there, the sums stay within 32 bits.
  my_whole = wave_sum(my_whole);
  const uint32_t rows_w = wave_sum((uint32_t)min(my_rows, 1ull << 20));
  if (lane == 0u) {
    if (my_whole) atomicAdd(&hist[kRows], my_whole);
    if (rows_w) atomicAdd(&rows_all, (unsigned long long)rows_w);
  }
  uint3 tot;
  const uint3 base0 = block_scan3(make_uint3(my_tiles, my_small, my_runs), wsum3, &tot);
  const uint32_t tb0 = base0.x, sm0 = base0.y, rn0 = base0.z;
  const uint32_t n_tiles = tot.x, n_runs = tot.z;
  const uint32_t per_r = (n_runs + nt_ - 1) / nt_;  // runs per thread
  {
    uint32_t tb = tb0, sm = sm0, rn = rn0;
    for (uint32_t s = s0; s < s1; s++) {
      x.tile_base[s] = tb;
      info[s].tb = tb;
      info[s].rb = rn;
      const SegInfo v = info[s];
      if (v.flags & kSegSmall) {
        x.small_list[sm++] = s;
        continue;
      }
      const uint32_t nt = tiles_in(v.m), nr = (nt + kRunTiles - 1) / kRunTiles;
      // this segment's runs fall in the run ranges of threads rn / per_r ..
      // (rn + nr - 1) / per_r; the lowest such segment starts a thread's range
      for (uint32_t c = rn / per_r; c <= (rn + nr - 1) / per_r; c++) atomicMin(&first_seg[c], s);
      tb += nt;
      rn += nr;
    }
  }
  if (tid == 0) x.tile_base[n] = n_tiles;
  __syncthreads();  // hist, rows_all, first_seg and the segment values complete

  // the cut (wave 0): with enough tiles, every tile of at least `from` rows
  // and the first `left` tiles of `take` rows, counted from the longest down
  // to at most cus tiles
  if (tid < 64u) {
    uint32_t piece = 0, from = kRows + 1, take = 0, left = 0, fine = 0;
    if (n_tiles > 0 && n_tiles < x.cus) {
      const unsigned long long p = (rows_all + x.cus - 1) / x.cus;
      if (p < (unsigned long long)kRows) {
        piece = (uint32_t)p;
        fine = 1;
      }
    } else if (n_tiles > 0) {
      piece = kPieceRows;
      // lane k holds rows kRows - k and kRows - 64 - k (those above kPieceRows)
      constexpr uint32_t kSpan = (uint32_t)(kRows - kPieceRows);
      static_assert(kSpan <= 128, "two row counts per lane");
      const uint32_t ra = kRows - lane, rb = kRows - 64u - lane;
      const uint32_t ha = lane < kSpan ? hist[ra] : 0u, hb = lane + 64u < kSpan ? hist[rb] : 0u;
      const uint32_t ia = wave_incl_scan(ha);  // tiles of at least ra rows
      const uint32_t tot_a = (uint32_t)__builtin_amdgcn_readlane((int)ia, 63);
      const uint32_t ib = tot_a + wave_incl_scan(hb);
      // from = the least row count whose tiles and all longer ones fit in cus
      const unsigned long long fa = __ballot(lane < kSpan && ia <= x.cus);
      const unsigned long long fb = __ballot(lane + 64u < kSpan && ib <= x.cus);
      uint32_t fit = 0;  // tiles of at least `from` rows
      if (fb) {
        const uint32_t k = 63u - (uint32_t)__clzll(fb);  // the highest lane: the fewest rows
        from = kRows - 64u - k;
        fit = (uint32_t)__builtin_amdgcn_readlane((int)ib, (int)k);
      } else if (fa) {
        const uint32_t k = 63u - (uint32_t)__clzll(fa);
        from = kRows - k;
        fit = (uint32_t)__builtin_amdgcn_readlane((int)ia, (int)k);
      }
      left = x.cus - fit;
      if (left) {
        // the longest row count below from that has tiles (above kPieceRows)
        const unsigned long long ta = __ballot(lane < kSpan && ra < from && ha > 0u);
        const unsigned long long tb = __ballot(lane + 64u < kSpan && rb < from && hb > 0u);
        if (ta)
          take = kRows + 1u - (uint32_t)__ffsll((unsigned long long)ta);
        else if (tb)
          take = kRows - 63u - (uint32_t)__ffsll((unsigned long long)tb);
      }
    }
    if (tid == 0) {
      c_piece = piece;
      c_from = from;
      c_take = take;
      c_left = take ? left : 0u;
      c_fine = fine;
    }
  }
  __syncthreads();
  const uint32_t piece = c_piece, from = c_from, take = c_take, left = c_left;
  const bool fine = c_fine != 0;

  // rank in tile order of each segment's first tile of `take` rows
  auto takes_of = [&](uint32_t m, uint32_t nt) -> uint32_t {
    return (take == (uint32_t)kRows ? nt - 1 : 0u) + (tile_rows_of(m, nt - 1) == take ? 1u : 0u);
  };
  if (left) {
    uint32_t mine = 0, all;
    for (uint32_t s = s0; s < s1; s++)
      if (!(info[s].flags & kSegSmall)) mine += takes_of(info[s].m, tiles_in(info[s].m));
    uint32_t rank = block_scan(mine, wsum, &all);
    for (uint32_t s = s0; s < s1; s++) {
      info[s].tk = rank;
      if (!(info[s].flags & kSegSmall)) rank += takes_of(info[s].m, tiles_in(info[s].m));
    }
    __syncthreads();
  }
  // The tiles of a segment are t = 0 .. nt - 1 from its end; all have kRows
  // rows but the first, t = nt - 1, which has r1 rows.  A run [t0, t1) holds
  // nf whole tiles (t < fe), of which the first nc are cut, and maybe the
  // partial first tile.
  struct RunPlan {
    uint32_t nf, nc;  // whole tiles, cut whole tiles (a prefix of them)
    bool part;        // holds the partial first tile
    bool part_cut;
    uint32_t r1;      // its rows
  };
  auto plan_run = [&](const SegInfo& v, uint32_t t0, uint32_t t1) -> RunPlan {
    RunPlan q;
    const uint32_t nt = tiles_in(v.m);
    q.r1 = tile_rows_of(v.m, nt - 1);
    const uint32_t fe = q.r1 == (uint32_t)kRows ? nt : nt - 1;  // whole tiles are t < fe
    const uint32_t fend = min(t1, fe);
    q.nf = fend > t0 ? fend - t0 : 0u;
    // whole tiles are cut: all of them (a fine cut, or kRows >= from), else
    // those whose rank among the tiles of `take` = kRows rows is below left
    if (fine || (uint32_t)kRows >= from) {
      q.nc = q.nf;
    } else if (take == (uint32_t)kRows && left > v.tk) {
      const uint32_t cend = min(fend, left - v.tk);  // t < left - tk
      q.nc = cend > t0 ? cend - t0 : 0u;
    } else {
      q.nc = 0;
    }
    q.part = q.r1 < (uint32_t)kRows && nt - 1 >= t0 && nt - 1 < t1;
    q.part_cut = q.part && (fine ? q.r1 > piece : (q.r1 >= from || (q.r1 == take && left > v.tk)));
    return q;
  };

  // runs [r_lo, r_hi) of this thread, from the segment holding run r_lo;
  // visit(s, v, t0, t1): tiles t0 .. t1 - 1 of segment s (values v)
  const uint32_t r_lo = min(n_runs, tid * per_r), r_hi = min(n_runs, r_lo + per_r);
  auto walk = [&](auto&& visit) {
    if (r_lo >= r_hi) return;
    uint32_t s = first_seg[tid];
    SegInfo v = info[s];
    uint32_t run = r_lo - v.rb;  // run of s
    for (uint32_t k = r_lo; k < r_hi; k++) {
      while ((v.flags & kSegSmall) || run * kRunTiles >= tiles_in(v.m)) {  // on to the next tiled segment
        s++;
        run = 0;
        v = info[s];
      }
      const uint32_t t0 = run * kRunTiles;
      visit(s, v, t0, min(tiles_in(v.m), t0 + kRunTiles));
      run++;
    }
  };
  // Count the entries by the rows each runs.  Uncut whole tiles (kRows
  // rows) and whole pieces get slots by thread order, which is tile order;
  // the other lengths (partial tiles, the remainders of cut tiles) by LDS
  // atomics.
  const uint32_t rem_full = piece ? (uint32_t)kRows % piece : 0u;  // remainder piece of a cut whole tile
  uint32_t my_full = 0, my_pieces = 0;
  walk([&](uint32_t s, const SegInfo& v, uint32_t t0, uint32_t t1) {
    const RunPlan q = plan_run(v, t0, t1);
    my_full += q.nf - q.nc;
    if (q.nc) {
      my_pieces += q.nc * ((uint32_t)kRows / piece);
      if (rem_full) atomicAdd(&cursor[rem_full], q.nc);
    }
    if (q.part) {
      if (!q.part_cut) {
        atomicAdd(&cursor[q.r1], 1u);
      } else {
        my_pieces += q.r1 / piece;
        if (q.r1 % piece) atomicAdd(&cursor[q.r1 % piece], 1u);
      }
    }
    // a one-tile segment has one run: this thread owns its entry
    if ((v.flags & kSegOneTile) && (q.nc || q.part_cut)) x.seg_cut[s] = 1u;
  });
  uint3 tot2;
  const uint3 b2 = block_scan3(make_uint3(my_full, my_pieces, 0u), wsum3, &tot2);
  const uint32_t full0 = b2.x, piece0 = b2.y, n_full = tot2.x, n_pieces = tot2.y;
  if (tid < 64u) {  // start of each length's run, longest first: lane k holds rows kRows - k and kRows - 64 - k
    const uint32_t ka = kRows - lane, kb = kRows - 64u - lane;
    const bool has_b = kRows > 64 + (int)lane;
    const uint32_t ca = cursor[ka] + (ka == (uint32_t)kRows ? n_full : 0u) + (ka == piece ? n_pieces : 0u);
    const uint32_t cb = has_b ? cursor[kb] + (kb == piece ? n_pieces : 0u) : 0u;
    const uint32_t ia = wave_incl_scan(ca), tot_a = (uint32_t)__builtin_amdgcn_readlane((int)ia, 63);
    const uint32_t ib = tot_a + wave_incl_scan(cb);
    // the atomics of a length start after its slots taken in thread order
    cursor[ka] = ia - ca + (ka == (uint32_t)kRows ? n_full : 0u) + (ka == piece ? n_pieces : 0u);
    if (has_b) cursor[kb] = ib - cb + (kb == piece ? n_pieces : 0u);
    if (ka == (uint32_t)kRows) c_full_at = ia - ca;  // first slot of the whole tiles
    if (ka == piece) c_piece_at = ia - ca;           // first slot of the whole pieces
    if (has_b && kb == piece) c_piece_at = ib - cb;
    if (lane == 63u) c_ents = ib;
  }
  __syncthreads();
  uint32_t at_full = c_full_at + full0, at_piece = (n_pieces ? c_piece_at : 0u) + piece0;
  walk([&](uint32_t s, const SegInfo& v, uint32_t t0, uint32_t t1) {
    const RunPlan q = plan_run(v, t0, t1);
    const uint32_t user = v.user, g0 = v.tb;
    auto put = [&](uint32_t pos, uint32_t t, uint32_t r0, uint32_t r1) {
      if (pos < x.cap) x.order[pos] = TileEnt{g0 + t, s, t | (r0 << 16) | (r1 << 24), user};
    };
    // pieces [r1 - piece, r1) from the tile's end down; the lowest may start
    // below the tile's first row lo
    auto pieces = [&](uint32_t t, uint32_t rows) {
      const uint32_t lo = (uint32_t)kRows - rows;
      for (uint32_t r1 = kRows; r1 > lo; r1 -= min(r1, piece)) {
        const uint32_t r0 = r1 > piece ? r1 - piece : 0u, len = r1 - max(r0, lo);
        put(len == piece ? at_piece++ : atomicAdd(&cursor[len], 1u), t, r0, r1);
      }
    };
    // a cut whole tile: kRows / piece whole pieces, then the remainder, if any
    const uint32_t per_tile = q.nc ? (uint32_t)kRows / piece : 0u;
    for (uint32_t t = t0; t < t0 + q.nc; t++) {
      for (uint32_t k = 0; k < per_tile; k++) put(at_piece++, t, kRows - (k + 1) * piece, kRows - k * piece);
      if (rem_full) put(atomicAdd(&cursor[rem_full], 1u), t, 0u, rem_full);
    }
    for (uint32_t t = t0 + q.nc; t < t0 + q.nf; t++) put(at_full++, t, 0u, kRows);
    if (q.part) {
      const uint32_t t = tiles_in(v.m) - 1;
      if (q.part_cut)
        pieces(t, q.r1);
      else
        put(atomicAdd(&cursor[q.r1], 1u), t, 0u, kRows);
    }
  });
  const uint32_t ents = c_ents;
  for (uint32_t k = ents + tid; k < x.cap; k += nt_) x.order[k] = TileEnt{kNoTile, 0u, 0u, 0u};
  if (tid == 0 && x.n_ents) *x.n_ents = ents;
}

// The expansion alone, for the library's test hook.
__global__ __launch_bounds__(kExpandThreads) void k_expand(const SegBrief* brief, uint32_t n, ExpandArgs x) {
  expand_tables(brief, n, x);
}

// ---------------------------------------------------------------------------
// First kernel of a call.  It copies the call's staged tables (descriptors,
// zero ranges, zeroed queue head, block ids) from the mapped host ring into
// device scratch, zeroes the tile partials, settles every segment's first
// verdict -- with labels, the owner check (OWNER_MIXED iff some row label
// differs from the segment's user; the sentinels never equal a user), else
// OK -- and forms E_K(J0) xor H*L of one-tile segments.  With an expansion,
// workgroup 0 builds the tile tables and the work queue meanwhile from the
// brief records; the other workgroups read descriptors and block ids where
// the copy reads them, so no part waits on another.
// ---------------------------------------------------------------------------
struct PrologueArgs {
  uint4* dst;
  const uint4* src;  // nullptr: the tables are in dst already
  size_t n16;        // 16-byte words of staged tables
  const SegDesc* segs;  // where the descriptors are readable now (src or dst)
  uint32_t n;
  const uint32_t* labels;
  const uint32_t* bids;
  int32_t* verdicts;
  KeyTableDev kt;
  uint4* fin;
  uint4* zero;
  uint32_t n_zero;
  bool expand;
  const SegBrief* brief;  // where the brief records are readable now
  ExpandArgs x;
};

__global__ __launch_bounds__(kPrologueThreads) void k_prologue(PrologueArgs a) {
  __shared__ uint32_t te[256];
  const bool ex = a.expand && a.n > 0;
  if (ex && blockIdx.x == 0) {
    expand_tables(a.brief, a.n, a.x);
    if (gridDim.x > 1) return;  // the other workgroups do the rest
    __syncthreads();
  }
  // the other workgroups (all of them without an expansion, or workgroup 0
  // after it when it is alone)
  const bool sep = ex && gridDim.x > 1;
  const uint32_t wg = sep ? blockIdx.x - 1 : blockIdx.x, n_wg = sep ? gridDim.x - 1 : gridDim.x;
  const size_t gsz = (size_t)n_wg * blockDim.x, me = (size_t)wg * blockDim.x + threadIdx.x;
  if (a.src)
    for (size_t i = me; i < a.n16; i += gsz) a.dst[i] = a.src[i];
  for (size_t i = me; i < a.n_zero; i += gsz) a.zero[i] = make_uint4(0u, 0u, 0u, 0u);
  if (!a.verdicts) return;
  const SegDesc* segs = a.segs;
  if (a.fin) {
    for (uint32_t i = threadIdx.x; i < 256u; i += blockDim.x) te[i] = c_aes.te0[i];
    __syncthreads();
  }
  for (uint32_t s = wg; s < a.n; s += n_wg) {
    if (a.fin && threadIdx.x < 64u && (segs[s].flags & kSegOneTile)) {
      // GCM a one-tile segment needs besides its tile: E_K(J0) xor H*L,
      // J0 = IV || BE32(1), H*L a wave sum over the set bits of the length
      // block (only its low 64 bits can be set) of the products H*x^(64+k)
      const uint32_t lane = threadIdx.x, user = segs[s].user;
      u128 z = u128_zero();
      if (((segs[s].len * 8ull) >> (63 - lane)) & 1ull) z = ld_u128(a.kt.pow_hxl + (size_t)user * kHxLanes + lane);
#pragma unroll
      for (int j = 0; j < 4; j++) z.w[j] = wave_xor(z.w[j]);
      if (lane == 0) {
        const uint32_t j0[4] = {segs[s].iv[0], segs[s].iv[1], segs[s].iv[2], 0x01000000u};
        uint32_t e[4];
        aes256_encrypt_tab(a.kt.rk + (size_t)user * 64u, j0, e, te);
        a.fin[s] = make_uint4(e[0] ^ z.w[0], e[1] ^ z.w[1], e[2] ^ z.w[2], e[3] ^ z.w[3]);
      }
    }
    int bad = 0;
    if (a.labels) {
      const uint64_t rb = segs[s].row_begin, rc = segs[s].row_count;
      const uint32_t user = segs[s].user;
      for (uint64_t r = threadIdx.x; r < rc; r += blockDim.x) bad |= a.labels[a.bids ? a.bids[rb + r] : rb + r] != user;
      bad = __syncthreads_or(bad);
    }
    if (threadIdx.x == 0) a.verdicts[s] = bad ? kVerdictOwnerMixed : kVerdictOk;
  }
}

// ---------------------------------------------------------------------------
// Zero-fill of uncovered rows and of rejected segments.
// ---------------------------------------------------------------------------
// Zero-fill of uncovered rows and (open) of segments whose verdict is not OK.
// The host cuts ranges into pieces of at most kZeroPieceBytes; a workgroup
// takes whole pieces, so nothing loops over all ranges per thread.
__global__ __launch_bounds__(256) void k_zero_ranges(uint8_t* out, const ZeroRange* __restrict__ rs, uint32_t n,
                                                     const int32_t* __restrict__ verdicts) {
  for (uint32_t i = blockIdx.x; i < n; i += gridDim.x) {
    const ZeroRange z = rs[i];
    if (z.seg >= 0 && verdicts[z.seg] == kVerdictOk) continue;
    uint8_t* p = out + z.off;
    uint64_t head = (16u - ((uintptr_t)p & 15u)) & 15u;
    if (head > z.len) head = z.len;
    for (uint64_t b = threadIdx.x; b < head; b += blockDim.x) p[b] = 0;
    const uint64_t mid = (z.len - head) / 16u;
    uint4* q = (uint4*)(p + head);
    for (uint64_t k = threadIdx.x; k < mid; k += blockDim.x) q[k] = make_uint4(0u, 0u, 0u, 0u);
    for (uint64_t b = head + 16u * mid + threadIdx.x; b < z.len; b += blockDim.x) p[b] = 0;
  }
}

__global__ __launch_bounds__(256) void k_wipe(uint8_t* p, size_t bytes) {
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < bytes; i += gsz) p[i] = 0;
}


// ---------------------------------------------------------------------------
// Per-token encryption (token || nonce as one block under the owner's key,
// the end-of-sequence token as the all-0xFF block).  The work is cut into
// chunks of 64 tokens of one segment: chunk_base[s] is the first chunk of
// segment s (an exclusive scan of ceil(row_count / 64), chunk_base[n_segs] =
// n_chunks), and a workgroup of 64 threads takes one chunk at a time,
// finding its segment by binary search.  Outputs of uncovered tokens were
// zeroed before this launch.
// ---------------------------------------------------------------------------
template <bool DECRYPT>
__global__ __launch_bounds__(kTokenChunk) void k_tokens(const SegDesc* __restrict__ segs,
                                                        const uint32_t* __restrict__ chunk_base, uint32_t n_segs,
                                                        uint32_t n_chunks,
                                               const uint64_t* __restrict__ tokens,
                                               const uint64_t* __restrict__ nonces,
                                               const uint8_t* __restrict__ blocks_in, uint8_t* __restrict__ blocks_out,
                                               uint64_t* __restrict__ tokens_out, uint64_t* __restrict__ nonces_out,
                                               uint64_t eos_token, KeyTableDev kt) {
  __shared__ uint32_t tab[256];
  __shared__ uint8_t isb[256];
  for (uint32_t i = threadIdx.x; i < 256u; i += blockDim.x) {
    tab[i] = DECRYPT ? c_aes.td0[i] : c_aes.te0[i];
    isb[i] = c_aes.inv_sbox[i];
  }
  __syncthreads();
  for (uint32_t b = blockIdx.x; b < n_chunks; b += gridDim.x) {
    // The segment of chunk b, chunk_base[lo] <= b < chunk_base[hi] throughout,
    // by a 64-way search: lane l tests split point lo + l * step; chunk_base
    // increases (every segment has a chunk), so the lanes that pass form a
    // prefix, lane 0 always among them, and the last of them bounds the next
    // interval.  Two rounds of loads for 4,096 segments instead of twelve.
    uint32_t lo = 0, hi = n_segs;
    while (hi - lo > 1u) {
      const uint32_t step = (hi - lo + 63u) / 64u;
      const uint32_t p = lo + threadIdx.x * step;
      const unsigned long long pass = __ballot(p < hi && chunk_base[p] <= b);
      lo += (63u - (uint32_t)__clzll(pass)) * step;
      hi = min(hi, lo + step);
    }
    const uint32_t s = lo;
    const uint64_t rb = segs[s].row_begin, rc = segs[s].row_count;
    const uint32_t user = segs[s].user;
    const uint64_t i = (uint64_t)kTokenChunk * (b - chunk_base[s]) + threadIdx.x;
    if (i < rc) {
      const uint64_t r = rb + i;
      if (!DECRYPT) {
        const uint64_t t = tokens[r], n = nonces[r];
        uint32_t o[4];
        if (t == eos_token) {
          o[0] = o[1] = o[2] = o[3] = 0xFFFFFFFFu;
        } else {
          const uint32_t blk[4] = {(uint32_t)t, (uint32_t)(t >> 32), (uint32_t)n, (uint32_t)(n >> 32)};
          aes256_encrypt_tab(kt.rk + 64ull * user, blk, o, tab);
        }
        *(uint4*)(blocks_out + 16ull * r) = make_uint4(o[0], o[1], o[2], o[3]);
      } else {
        const uint4 b = *(const uint4*)(blocks_in + 16ull * r);
        uint64_t t, n;
        if ((b.x & b.y & b.z & b.w) == 0xFFFFFFFFu) {
          t = eos_token;
          n = 0;
        } else {
          const uint32_t blk[4] = {b.x, b.y, b.z, b.w};
          uint32_t p[4];
          aes256_decrypt_tab(kt.dk + 64ull * user, blk, p, tab, isb);
          t = (uint64_t)p[0] | ((uint64_t)p[1] << 32);
          n = (uint64_t)p[2] | ((uint64_t)p[3] << 32);
        }
        tokens_out[r] = t;
        if (nonces_out) nonces_out[r] = n;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Paged KV: offsets of a segment's chunks in stream order (for each block of
// its table, each layer, each part), and zeroing of rejected segments' chunks.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_chunk_table(const SegDesc* __restrict__ segs, uint32_t n,
                                                     const uint32_t* __restrict__ bids, uint32_t n_layers,
                                                     uint32_t n_parts, uint64_t ls, uint64_t bs, uint64_t ps,
                                                     uint64_t* __restrict__ chunk_off) {
  const uint64_t per_block = (uint64_t)n_layers * n_parts;
  for (uint32_t s = blockIdx.x; s < n; s += gridDim.x) {
    const uint64_t bid0 = segs[s].row_begin, nchunks = segs[s].row_count * per_block, c0 = segs[s].chunk0;
    for (uint64_t c = threadIdx.x; c < nchunks; c += blockDim.x) {
      const uint64_t j = c / per_block, rem = c % per_block;
      const uint64_t l = rem / n_parts, p = rem % n_parts;
      chunk_off[c0 + c] = l * ls + (uint64_t)bids[bid0 + j] * bs + p * ps;
    }
  }
}

// Open: zero the output of segments that failed, tile by tile.  A workgroup
// takes whole tiles of kTileBlocks blocks (the GCM kernel's tiles, found
// through tile_base), so the work per workgroup is bounded.  Contiguous
// output (chunk_off == nullptr): every segment whose verdict is not OK.
// Through block tables: only requests that failed authentication -- their
// blocks passed the label check, so they are the request's own; a request
// rejected by the label check writes nothing.
__global__ __launch_bounds__(256) void k_zero_failed(const SegDesc* __restrict__ segs, uint32_t n,
                                                     const uint32_t* __restrict__ tile_base, uint32_t n_tiles,
                                                     const int32_t* __restrict__ verdicts,
                                                     const uint64_t* __restrict__ chunk_off, uint8_t* base,
                                                     uint32_t chunk_shift) {
  const uint64_t cmask = (1ull << chunk_shift) - 1;
  for (uint32_t g = blockIdx.x; g < n_tiles; g += gridDim.x) {
    uint32_t lo = 0, hi = n;  // tile_base[lo] <= g < tile_base[hi]
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (tile_base[mid] <= g)
        lo = mid;
      else
        hi = mid;
    }
    const int32_t v = verdicts[lo];
    if (chunk_off ? v != kVerdictAuthFail : v == kVerdictOk) continue;
    const uint64_t m = segs[lo].nblocks;
    const uint64_t t = g - tile_base[lo];
    // tiles are aligned to the end of the segment, as in k_gcm_tiles
    const uint64_t end = m - t * (uint64_t)kTileBlocks;
    const uint64_t begin = end > kTileBlocks ? end - kTileBlocks : 0;
    if (chunk_off) {
      const uint64_t c0 = segs[lo].chunk0;
      for (uint64_t i = begin + threadIdx.x; i < end; i += blockDim.x)
        *(uint4*)(base + chunk_off[c0 + (i >> chunk_shift)] + ((i & cmask) << 4)) = make_uint4(0u, 0u, 0u, 0u);
    } else {
      const uint64_t len = segs[lo].len;
      uint8_t* p = base + segs[lo].byte_off;
      const bool aligned = (segs[lo].flags & kSegAligned) != 0;
      for (uint64_t i = begin + threadIdx.x; i < end; i += blockDim.x) {
        const uint64_t rem = len - 16ull * i;
        store_block(p + 16ull * i, u128_zero(), rem >= 16 ? 16u : (uint32_t)rem, aligned);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Key-table setup.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_key_sched(const uint8_t* __restrict__ keys, KeyTableDev kt) {
  const uint32_t u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= kt.n_users) return;
  uint32_t rk[60];
  aes256_key_schedule(keys + 32ull * u, rk, c_aes);
  for (int i = 0; i < 60; i++) kt.rk[64ull * u + i] = rk[i];
  for (int i = 60; i < 64; i++) kt.rk[64ull * u + i] = 0u;
  uint32_t dk[60];
  aes256_dec_key_schedule(rk, dk);
  for (int i = 0; i < 60; i++) kt.dk[64ull * u + i] = dk[i];
  for (int i = 60; i < 64; i++) kt.dk[64ull * u + i] = 0u;
  const uint32_t zero[4] = {0u, 0u, 0u, 0u};
  uint32_t h[4];
  aes256_encrypt_words(rk, zero, h, c_aes);
  for (int i = 0; i < 4; i++) kt.h[4ull * u + i] = h[i];
}

constexpr uint32_t kPowersPerUser = kHPowers + kFinLanes + 1 + kHxLanes + kRows;

__global__ __launch_bounds__(256) void k_key_powers(KeyTableDev kt) {
  const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t u = idx / kPowersPerUser;
  const uint32_t j = (uint32_t)(idx % kPowersPerUser);
  if (u >= kt.n_users) return;
  const u128 h = ld_u128((const uint4*)(kt.h + 4ull * u));
  if (j < (uint32_t)kHPowers) {
    st_u128(kt.pow_h + u * kHPowers + j, gf_pow(h, j));
  } else if (j < (uint32_t)(kHPowers + kFinLanes)) {
    const uint32_t l = j - kHPowers;
    st_u128(kt.pow_ht + u * kFinLanes + l, gf_pow(h, (uint64_t)l * kTileBlocks));
  } else if (j == (uint32_t)(kHPowers + kFinLanes)) {
    st_u128(kt.pow_hlt + u, gf_pow(h, (uint64_t)kFinLanes * kTileBlocks));
  } else if (j < (uint32_t)(kHPowers + kFinLanes + 1 + kHxLanes)) {
    const uint32_t k = j - (kHPowers + kFinLanes + 1);
    st_u128(kt.pow_hxl + u * kHxLanes + k, gf_mul(h, gf_xpow_elem(64 + (int)k)));
  } else {
    const uint32_t k = j - (kHPowers + kFinLanes + 1 + kHxLanes);
    st_u128(kt.pow_hr + u * kRows + k, gf_pow(h, (uint64_t)k * kThreads));
  }
}

// Nibble tables of M = H^kThreads (gtab) and W = H^(64 * kLeaders)
// (gtab_fold): entry [q][v] = (v placed at GCM bits 4q..4q+3, MSB first) * M,
// built from the four products x^(4q+k) * M.
__global__ __launch_bounds__(256) void k_key_gtab(KeyTableDev kt) {
  const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t u = idx / 64u;
  const int q = (int)(idx % 32u);
  const bool fold = (idx % 64u) >= 32u;
  if (u >= kt.n_users) return;
  const u128 h = ld_u128((const uint4*)(kt.h + 4ull * u));
  const u128 mm = gf_pow(h, fold ? (uint64_t)(64 * kLeaders) : (uint64_t)kThreads);
  uint4* tab = (fold ? kt.gtab_fold : kt.gtab) + u * 512u;
  u128 b[4];
  for (int k = 0; k < 4; k++) b[k] = gf_mul(gf_xpow_elem(4 * q + k), mm);
  for (int v = 0; v < 16; v++) {
    u128 e = u128_zero();
    for (int k = 0; k < 4; k++)
      if (v & (8 >> k)) e = u128_xor(e, b[k]);
    st_u128(tab + (uint64_t)q * 16u + v, e);
  }
}

// ---------------------------------------------------------------------------
// Launch wrappers.
// ---------------------------------------------------------------------------
static inline uint32_t cdiv(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }

hipError_t launch_key_setup(const uint8_t* keys_dev, KeyTableDev kt, hipStream_t s) {
  hipLaunchKernelGGL(k_key_sched, dim3(cdiv(kt.n_users, 64)), dim3(64), 0, s, keys_dev, kt);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_key_powers, dim3(cdiv((uint64_t)kt.n_users * kPowersPerUser, 256)), dim3(256), 0, s, kt);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_key_gtab, dim3(cdiv((uint64_t)kt.n_users * 64u, 256)), dim3(256), 0, s, kt);
  return hipGetLastError();
}



hipError_t launch_gcm_tiles(const GcmArgs& a, int mode, uint32_t grid, hipStream_t s) {
  if (a.n_ents == 0) return hipSuccess;
  const uint32_t g = a.n_ents < grid ? a.n_ents : grid;
  switch (mode) {
    case 0: hipLaunchKernelGGL(k_gcm_tiles<0>, dim3(g), dim3(kThreads), 0, s, a); break;
    case kModeOpen: hipLaunchKernelGGL(k_gcm_tiles<kModeOpen>, dim3(g), dim3(kThreads), 0, s, a); break;
    case kModeGather: hipLaunchKernelGGL(k_gcm_tiles<kModeGather>, dim3(g), dim3(kThreads), 0, s, a); break;
    case kModeOpen | kModeScatter:
      hipLaunchKernelGGL(k_gcm_tiles<kModeOpen | kModeScatter>, dim3(g), dim3(kThreads), 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gcm_small(const GcmArgs& a, bool open, hipStream_t s) {
  if (a.n_small == 0) return hipSuccess;
  if (open)
    hipLaunchKernelGGL(k_small<true>, dim3(a.n_small), dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL(k_small<false>, dim3(a.n_small), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gcm_finalize(const GcmArgs& a, bool open, hipStream_t s) {
  if (a.n_multi == 0) return hipSuccess;
  if (open)
    hipLaunchKernelGGL(k_finalize<true>, dim3(a.n_segs), dim3(kFinLanes), 0, s, a);
  else
    hipLaunchKernelGGL(k_finalize<false>, dim3(a.n_segs), dim3(kFinLanes), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_zero_ranges(uint8_t* out, const ZeroRange* r, uint32_t n, const int32_t* verdicts, uint32_t grid,
                              hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (grid > n) grid = n;
  hipLaunchKernelGGL(k_zero_ranges, dim3(grid), dim3(256), 0, s, out, r, n, verdicts);
  return hipGetLastError();
}

hipError_t launch_tokens(const SegDesc* segs, const uint32_t* chunk_base, uint32_t n_segs, uint32_t n_chunks,
                         bool decrypt, const uint64_t* tokens, const uint64_t* nonces, const uint8_t* blocks_in,
                         uint8_t* blocks_out, uint64_t* tokens_out, uint64_t* nonces_out, uint64_t eos_token,
                         KeyTableDev kt, hipStream_t s) {
  if (n_segs == 0 || n_chunks == 0) return hipSuccess;
  const uint32_t grid = n_chunks < 65535u ? n_chunks : 65535u;
  if (decrypt)
    hipLaunchKernelGGL(k_tokens<true>, dim3(grid), dim3(kTokenChunk), 0, s, segs, chunk_base, n_segs, n_chunks,
                       tokens, nonces, blocks_in, blocks_out, tokens_out, nonces_out, eos_token, kt);
  else
    hipLaunchKernelGGL(k_tokens<false>, dim3(grid), dim3(kTokenChunk), 0, s, segs, chunk_base, n_segs, n_chunks,
                       tokens, nonces, blocks_in, blocks_out, tokens_out, nonces_out, eos_token, kt);
  return hipGetLastError();
}

hipError_t launch_chunk_table(const SegDesc* segs, uint32_t n_segs, const uint32_t* bids, uint32_t n_layers,
                              uint32_t n_parts, uint64_t layer_stride, uint64_t block_stride, uint64_t part_stride,
                              uint64_t* chunk_off, hipStream_t s) {
  if (n_segs == 0) return hipSuccess;
  const uint32_t grid = n_segs < 65535u ? n_segs : 65535u;
  hipLaunchKernelGGL(k_chunk_table, dim3(grid), dim3(256), 0, s, segs, n_segs, bids, n_layers, n_parts, layer_stride,
                     block_stride, part_stride, chunk_off);
  return hipGetLastError();
}

hipError_t launch_zero_failed(const SegDesc* segs, uint32_t n_segs, const uint32_t* tile_base, uint32_t n_tiles,
                              const int32_t* verdicts, const uint64_t* chunk_off, uint8_t* base, uint32_t chunk_shift,
                              uint32_t grid, hipStream_t s) {
  if (n_segs == 0 || n_tiles == 0) return hipSuccess;
  if (grid > n_tiles) grid = n_tiles;
  hipLaunchKernelGGL(k_zero_failed, dim3(grid), dim3(256), 0, s, segs, n_segs, tile_base, n_tiles, verdicts,
                     chunk_off, base, chunk_shift);
  return hipGetLastError();
}


hipError_t launch_expand(const SegBrief* brief, uint32_t n_segs, const ExpandArgs& x, hipStream_t s) {
  if (n_segs == 0) return hipSuccess;
  hipLaunchKernelGGL(k_expand, dim3(1), dim3(kExpandThreads), 0, s, brief, n_segs, x);
  return hipGetLastError();
}

hipError_t launch_prologue(void* dst, const void* src, size_t bytes, uint32_t n_segs, uint64_t bids_off,
                           const uint32_t* labels, int32_t* verdicts, const KeyTableDev* kt, uint4* fin,
                           uint4* zero, uint32_t n_zero, uint64_t brief_off, const ExpandArgs* ex, hipStream_t s) {
  if (bytes & 15u) return hipErrorInvalidValue;
  const size_t n16 = src ? bytes / 16 : 0;
  const bool expand = ex != nullptr && n_segs > 0;
  if (n16 == 0 && !verdicts && n_zero == 0 && !expand) return hipSuccess;
  if (n16 && (((uintptr_t)dst | (uintptr_t)src) & 15u)) return hipErrorInvalidValue;
  if (expand && (brief_off & 15u || brief_off + 8ull * (n_segs + 1) > bytes)) return hipErrorInvalidValue;
  const uint8_t* rd = src ? (const uint8_t*)src : (const uint8_t*)dst;  // where the tables are readable now
  uint64_t grid = cdiv(n16 > n_zero ? n16 : n_zero, kPrologueThreads);
  if (verdicts && n_segs > grid) grid = n_segs;
  if (grid > 1024u) grid = 1024u;
  if (grid == 0) grid = 1;
  if (expand) grid += 1;  // workgroup 0 expands the segment table
  PrologueArgs a{};
  a.dst = (uint4*)dst;
  a.src = (const uint4*)src;
  a.n16 = n16;
  a.segs = (const SegDesc*)rd;
  a.n = n_segs;
  a.labels = labels;
  a.bids = bids_off == kNoBids ? nullptr : (const uint32_t*)(rd + bids_off);
  a.verdicts = verdicts;
  a.kt = kt ? *kt : KeyTableDev{};
  a.fin = kt ? fin : nullptr;
  a.zero = zero;
  a.n_zero = n_zero;
  a.expand = expand;
  if (expand) {
    a.x = *ex;
    a.brief = (const SegBrief*)(rd + brief_off);
  }
  hipLaunchKernelGGL(k_prologue, dim3((uint32_t)grid), dim3(kPrologueThreads), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fixed workspace of gift_seal_noalloc.  Each device holds its own copy of
// the array at its own address; host code never uses the array's name (a
// host-side stand-in), only the address hipGetSymbolAddress gives for the
// current device, looked up once per device at set-up.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

static std::mutex g_scratch_mu;
static uint8_t* g_scratch_addr[kStaticScratchDevices] = {nullptr};

hipError_t static_scratch_setup(int dev) {
  if (dev < 0 || dev >= kStaticScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_addr[dev]) return hipSuccess;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (ptr == nullptr || ((uintptr_t)ptr & 255u)) return hipErrorInvalidSymbol;
  g_scratch_addr[dev] = (uint8_t*)ptr;
  return hipSuccess;
}

uint8_t* static_scratch(int dev) {
  if (dev < 0 || dev >= kStaticScratchDevices) return nullptr;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  return g_scratch_addr[dev];
}

hipError_t launch_wipe(void* p, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  uint32_t grid = cdiv(bytes, 256u * 16u);
  if (grid > 4096u) grid = 4096u;
  hipLaunchKernelGGL(k_wipe, dim3(grid), dim3(256), 0, s, (uint8_t*)p, bytes);
  return hipGetLastError();
}

}  // namespace gift
