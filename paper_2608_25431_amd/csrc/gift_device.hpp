// Device-side building blocks for segmented AES-256-GCM on gfx950:
// compile-time AES tables, the AES-256 key schedule, a table-free AES block
// function for setup/finalize work, GF(2^128) arithmetic in GCM bit order,
// and small wave-level helpers.  The per-block hot loop lives in
// gift_kernels.hip and uses LDS-resident tables instead.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gift {

// ---------------------------------------------------------------------------
// AES constants, generated at compile time from the field definition
// (FIPS-197 Sec. 4.2 and Sec. 5.1.1): the S-box is the affine image of the
// multiplicative inverse in GF(2^8) mod x^8+x^4+x^3+x+1.  Here the inverse
// is a^254 and the affine map is b ^ rotl(b,1) ^ rotl(b,2) ^ rotl(b,3) ^
// rotl(b,4) ^ 0x63.
// ---------------------------------------------------------------------------
constexpr uint8_t xt(uint8_t a) { return (uint8_t)((a << 1) ^ ((a & 0x80) ? 0x1b : 0)); }
constexpr uint8_t gmul(uint8_t a, uint8_t b) {
  uint8_t p = 0;
  for (int i = 0; i < 8; i++) {
    if (b & 1) p ^= a;
    a = xt(a);
    b >>= 1;
  }
  return p;
}
constexpr uint8_t rotl8(uint8_t b, int s) { return (uint8_t)((b << s) | (b >> (8 - s))); }
constexpr uint8_t ginv(uint8_t a) {
  // a^254 = a^-1 for a != 0 (the multiplicative group has order 255); 0 -> 0
  uint8_t r = 1, base = a;
  int e = 254;
  while (e) {
    if (e & 1) r = gmul(r, base);
    base = gmul(base, base);
    e >>= 1;
  }
  return a ? r : 0;
}
constexpr uint8_t sbox_of(uint8_t a) {
  uint8_t b = ginv(a);
  return (uint8_t)(b ^ rotl8(b, 1) ^ rotl8(b, 2) ^ rotl8(b, 3) ^ rotl8(b, 4) ^ 0x63);
}

struct AesConst {
  uint8_t sbox[256];
  uint8_t inv_sbox[256];
  // Te0[x]: the MixColumns image of S(x) placed in row 0, as a little-endian
  // column word: bytes (2S, S, S, 3S).  Rows 1..3 are byte rotations.
  uint32_t te0[256];
  // Td0[x]: the InvMixColumns image of S^-1(x) in row 0: bytes
  // (0e, 09, 0d, 0b) * S^-1(x).  Rows 1..3 are byte rotations.
  uint32_t td0[256];
};

constexpr AesConst make_aes_const() {
  AesConst c{};
  for (int x = 0; x < 256; x++) {
    uint8_t s = sbox_of((uint8_t)x);
    c.sbox[x] = s;
    c.inv_sbox[s] = (uint8_t)x;
    c.te0[x] = (uint32_t)gmul(s, 2) | ((uint32_t)s << 8) | ((uint32_t)s << 16) | ((uint32_t)gmul(s, 3) << 24);
  }
  for (int x = 0; x < 256; x++) {
    uint8_t v = c.inv_sbox[x];
    c.td0[x] = (uint32_t)gmul(v, 0x0e) | ((uint32_t)gmul(v, 0x09) << 8) | ((uint32_t)gmul(v, 0x0d) << 16) |
               ((uint32_t)gmul(v, 0x0b) << 24);
  }
  return c;
}

__device__ __forceinline__ uint32_t rotl32(uint32_t x, int s) { return (x << s) | (x >> ((32 - s) & 31)); }
__device__ __forceinline__ uint32_t bswap32(uint32_t x) { return __builtin_bswap32(x); }
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}
// a ^ (b & c) in one v_bitop3_b32
__device__ __forceinline__ uint32_t xor_and(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x78);
}

// x, unknown to the optimiser from here on: values derived from it are
// computed where they are used, not hoisted across a loop and held in
// registers (or spilled) until then
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// ---------------------------------------------------------------------------
// AES-256 key schedule (FIPS-197 Sec. 5.2, Nk = 8, Nr = 14).  Words are
// little-endian u32 of the schedule bytes, so word c of round r XORs
// directly into state column c.
// ---------------------------------------------------------------------------
__device__ inline void aes256_key_schedule(const uint8_t* __restrict__ key, uint32_t rk[60],
                                           const AesConst& C) {
  for (int i = 0; i < 8; i++)
    rk[i] = (uint32_t)key[4 * i] | ((uint32_t)key[4 * i + 1] << 8) | ((uint32_t)key[4 * i + 2] << 16) |
            ((uint32_t)key[4 * i + 3] << 24);
  uint8_t rc = 1;
  for (int i = 8; i < 60; i++) {
    uint32_t t = rk[i - 1];
    if ((i & 7) == 0 || (i & 7) == 4) {
      if ((i & 7) == 0) t = (t >> 8) | (t << 24);  // RotWord on LE bytes
      t = (uint32_t)C.sbox[t & 0xff] | ((uint32_t)C.sbox[(t >> 8) & 0xff] << 8) |
          ((uint32_t)C.sbox[(t >> 16) & 0xff] << 16) | ((uint32_t)C.sbox[t >> 24] << 24);
      if ((i & 7) == 0) {
        t ^= rc;
        rc = xt(rc);
      }
    }
    rk[i] = rk[i - 8] ^ t;
  }
}

// One AES-256 block from tables in global/constant memory.  Used only where
// a few blocks per segment are needed (E_K(J0), H, small segments).
// State words are columns (little-endian), as above.
__device__ inline void aes256_encrypt_words(const uint32_t* __restrict__ rk, const uint32_t in[4], uint32_t out[4],
                                            const AesConst& C) {
  uint32_t s0 = in[0] ^ rk[0], s1 = in[1] ^ rk[1], s2 = in[2] ^ rk[2], s3 = in[3] ^ rk[3];
#define GIFT_TE(w, k) rotl32(C.te0[((w) >> (8 * (k))) & 0xff], 8 * (k))
  for (int r = 1; r < 14; r++) {
    uint32_t t0 = GIFT_TE(s0, 0) ^ GIFT_TE(s1, 1) ^ GIFT_TE(s2, 2) ^ GIFT_TE(s3, 3) ^ rk[4 * r + 0];
    uint32_t t1 = GIFT_TE(s1, 0) ^ GIFT_TE(s2, 1) ^ GIFT_TE(s3, 2) ^ GIFT_TE(s0, 3) ^ rk[4 * r + 1];
    uint32_t t2 = GIFT_TE(s2, 0) ^ GIFT_TE(s3, 1) ^ GIFT_TE(s0, 2) ^ GIFT_TE(s1, 3) ^ rk[4 * r + 2];
    uint32_t t3 = GIFT_TE(s3, 0) ^ GIFT_TE(s0, 1) ^ GIFT_TE(s1, 2) ^ GIFT_TE(s2, 3) ^ rk[4 * r + 3];
    s0 = t0;
    s1 = t1;
    s2 = t2;
    s3 = t3;
  }
#undef GIFT_TE
#define GIFT_SB(w, k) ((uint32_t)C.sbox[((w) >> (8 * (k))) & 0xff] << (8 * (k)))
  out[0] = (GIFT_SB(s0, 0) | GIFT_SB(s1, 1) | GIFT_SB(s2, 2) | GIFT_SB(s3, 3)) ^ rk[56];
  out[1] = (GIFT_SB(s1, 0) | GIFT_SB(s2, 1) | GIFT_SB(s3, 2) | GIFT_SB(s0, 3)) ^ rk[57];
  out[2] = (GIFT_SB(s2, 0) | GIFT_SB(s3, 1) | GIFT_SB(s0, 2) | GIFT_SB(s1, 3)) ^ rk[58];
  out[3] = (GIFT_SB(s3, 0) | GIFT_SB(s0, 1) | GIFT_SB(s1, 2) | GIFT_SB(s2, 3)) ^ rk[59];
#undef GIFT_SB
}

// The same cipher with its table passed in (typically a copy in LDS, where
// per-lane lookups are cheap, unlike the constant segment): te0 as in
// AesConst, and S(x) is byte 1 of te0[x].
__device__ inline void aes256_encrypt_tab(const uint32_t* __restrict__ rk, const uint32_t in[4], uint32_t out[4],
                                          const uint32_t* te0) {
  uint32_t s0 = in[0] ^ rk[0], s1 = in[1] ^ rk[1], s2 = in[2] ^ rk[2], s3 = in[3] ^ rk[3];
#define GIFT_TE(w, k) rotl32(te0[((w) >> (8 * (k))) & 0xffu], 8 * (k))
  for (int r = 1; r < 14; r++) {
    const uint32_t t0 = GIFT_TE(s0, 0) ^ GIFT_TE(s1, 1) ^ GIFT_TE(s2, 2) ^ GIFT_TE(s3, 3) ^ rk[4 * r + 0];
    const uint32_t t1 = GIFT_TE(s1, 0) ^ GIFT_TE(s2, 1) ^ GIFT_TE(s3, 2) ^ GIFT_TE(s0, 3) ^ rk[4 * r + 1];
    const uint32_t t2 = GIFT_TE(s2, 0) ^ GIFT_TE(s3, 1) ^ GIFT_TE(s0, 2) ^ GIFT_TE(s1, 3) ^ rk[4 * r + 2];
    const uint32_t t3 = GIFT_TE(s3, 0) ^ GIFT_TE(s0, 1) ^ GIFT_TE(s1, 2) ^ GIFT_TE(s2, 3) ^ rk[4 * r + 3];
    s0 = t0;
    s1 = t1;
    s2 = t2;
    s3 = t3;
  }
#undef GIFT_TE
#define GIFT_SB(w, k) (((te0[((w) >> (8 * (k))) & 0xffu] >> 8) & 0xffu) << (8 * (k)))
  out[0] = (GIFT_SB(s0, 0) | GIFT_SB(s1, 1) | GIFT_SB(s2, 2) | GIFT_SB(s3, 3)) ^ rk[56];
  out[1] = (GIFT_SB(s1, 0) | GIFT_SB(s2, 1) | GIFT_SB(s3, 2) | GIFT_SB(s0, 3)) ^ rk[57];
  out[2] = (GIFT_SB(s2, 0) | GIFT_SB(s3, 1) | GIFT_SB(s0, 2) | GIFT_SB(s1, 3)) ^ rk[58];
  out[3] = (GIFT_SB(s3, 0) | GIFT_SB(s0, 1) | GIFT_SB(s1, 2) | GIFT_SB(s2, 3)) ^ rk[59];
#undef GIFT_SB
}

// Equivalent inverse cipher with td0 and the inverse S-box passed in.
__device__ inline void aes256_decrypt_tab(const uint32_t* __restrict__ dk, const uint32_t in[4], uint32_t out[4],
                                          const uint32_t* td0, const uint8_t* isb) {
  uint32_t s0 = in[0] ^ dk[56], s1 = in[1] ^ dk[57], s2 = in[2] ^ dk[58], s3 = in[3] ^ dk[59];
#define GIFT_TD(w, k) rotl32(td0[((w) >> (8 * (k))) & 0xffu], 8 * (k))
  for (int r = 13; r >= 1; r--) {
    const uint32_t t0 = GIFT_TD(s0, 0) ^ GIFT_TD(s3, 1) ^ GIFT_TD(s2, 2) ^ GIFT_TD(s1, 3) ^ dk[4 * r + 0];
    const uint32_t t1 = GIFT_TD(s1, 0) ^ GIFT_TD(s0, 1) ^ GIFT_TD(s3, 2) ^ GIFT_TD(s2, 3) ^ dk[4 * r + 1];
    const uint32_t t2 = GIFT_TD(s2, 0) ^ GIFT_TD(s1, 1) ^ GIFT_TD(s0, 2) ^ GIFT_TD(s3, 3) ^ dk[4 * r + 2];
    const uint32_t t3 = GIFT_TD(s3, 0) ^ GIFT_TD(s2, 1) ^ GIFT_TD(s1, 2) ^ GIFT_TD(s0, 3) ^ dk[4 * r + 3];
    s0 = t0;
    s1 = t1;
    s2 = t2;
    s3 = t3;
  }
#undef GIFT_TD
#define GIFT_ISB(w, k) ((uint32_t)isb[((w) >> (8 * (k))) & 0xffu] << (8 * (k)))
  out[0] = (GIFT_ISB(s0, 0) | GIFT_ISB(s3, 1) | GIFT_ISB(s2, 2) | GIFT_ISB(s1, 3)) ^ dk[0];
  out[1] = (GIFT_ISB(s1, 0) | GIFT_ISB(s0, 1) | GIFT_ISB(s3, 2) | GIFT_ISB(s2, 3)) ^ dk[1];
  out[2] = (GIFT_ISB(s2, 0) | GIFT_ISB(s1, 1) | GIFT_ISB(s0, 2) | GIFT_ISB(s3, 3)) ^ dk[2];
  out[3] = (GIFT_ISB(s3, 0) | GIFT_ISB(s2, 1) | GIFT_ISB(s1, 2) | GIFT_ISB(s0, 3)) ^ dk[3];
#undef GIFT_ISB
}

// InvMixColumns of one column word (FIPS-197 Sec. 5.3.3), used to derive the
// round keys of the equivalent inverse cipher (Sec. 5.3.5).
__device__ inline uint32_t inv_mix_column(uint32_t w) {
  const uint8_t a0 = w & 0xff, a1 = (w >> 8) & 0xff, a2 = (w >> 16) & 0xff, a3 = w >> 24;
  const uint8_t b0 = gmul(a0, 0x0e) ^ gmul(a1, 0x0b) ^ gmul(a2, 0x0d) ^ gmul(a3, 0x09);
  const uint8_t b1 = gmul(a0, 0x09) ^ gmul(a1, 0x0e) ^ gmul(a2, 0x0b) ^ gmul(a3, 0x0d);
  const uint8_t b2 = gmul(a0, 0x0d) ^ gmul(a1, 0x09) ^ gmul(a2, 0x0e) ^ gmul(a3, 0x0b);
  const uint8_t b3 = gmul(a0, 0x0b) ^ gmul(a1, 0x0d) ^ gmul(a2, 0x09) ^ gmul(a3, 0x0e);
  return (uint32_t)b0 | ((uint32_t)b1 << 8) | ((uint32_t)b2 << 16) | ((uint32_t)b3 << 24);
}

// Round keys of the equivalent inverse cipher: dw[i] = w[i] for rounds 0 and
// 14, InvMixColumns(w[i]) for rounds 1..13 (FIPS-197 Sec. 5.3.5).
__device__ inline void aes256_dec_key_schedule(const uint32_t rk[60], uint32_t dk[60]) {
  for (int i = 0; i < 60; i++) dk[i] = (i < 4 || i >= 56) ? rk[i] : inv_mix_column(rk[i]);
}

// One AES-256 block decryption with the equivalent inverse cipher: start
// with round key 14, then for rounds 13..1 InvSubBytes + InvShiftRows +
// InvMixColumns (the Td tables) + dw[round], finally InvSubBytes +
// InvShiftRows + dw[0].  InvShiftRows takes row r of output column c from
// input column c - r.
__device__ inline void aes256_decrypt_words(const uint32_t* __restrict__ dk, const uint32_t in[4], uint32_t out[4],
                                            const AesConst& C) {
  uint32_t s0 = in[0] ^ dk[56], s1 = in[1] ^ dk[57], s2 = in[2] ^ dk[58], s3 = in[3] ^ dk[59];
#define GIFT_TD(w, k) rotl32(C.td0[((w) >> (8 * (k))) & 0xff], 8 * (k))
  for (int r = 13; r >= 1; r--) {
    uint32_t t0 = GIFT_TD(s0, 0) ^ GIFT_TD(s3, 1) ^ GIFT_TD(s2, 2) ^ GIFT_TD(s1, 3) ^ dk[4 * r + 0];
    uint32_t t1 = GIFT_TD(s1, 0) ^ GIFT_TD(s0, 1) ^ GIFT_TD(s3, 2) ^ GIFT_TD(s2, 3) ^ dk[4 * r + 1];
    uint32_t t2 = GIFT_TD(s2, 0) ^ GIFT_TD(s1, 1) ^ GIFT_TD(s0, 2) ^ GIFT_TD(s3, 3) ^ dk[4 * r + 2];
    uint32_t t3 = GIFT_TD(s3, 0) ^ GIFT_TD(s2, 1) ^ GIFT_TD(s1, 2) ^ GIFT_TD(s0, 3) ^ dk[4 * r + 3];
    s0 = t0;
    s1 = t1;
    s2 = t2;
    s3 = t3;
  }
#undef GIFT_TD
#define GIFT_ISB(w, k) ((uint32_t)C.inv_sbox[((w) >> (8 * (k))) & 0xff] << (8 * (k)))
  out[0] = (GIFT_ISB(s0, 0) | GIFT_ISB(s3, 1) | GIFT_ISB(s2, 2) | GIFT_ISB(s1, 3)) ^ dk[0];
  out[1] = (GIFT_ISB(s1, 0) | GIFT_ISB(s0, 1) | GIFT_ISB(s3, 2) | GIFT_ISB(s2, 3)) ^ dk[1];
  out[2] = (GIFT_ISB(s2, 0) | GIFT_ISB(s1, 1) | GIFT_ISB(s0, 2) | GIFT_ISB(s3, 3)) ^ dk[2];
  out[3] = (GIFT_ISB(s3, 0) | GIFT_ISB(s2, 1) | GIFT_ISB(s1, 2) | GIFT_ISB(s0, 3)) ^ dk[3];
#undef GIFT_ISB
}

// ---------------------------------------------------------------------------
// GF(2^128) in GCM bit order (SP 800-38D Sec. 6.3): a block is 16 bytes,
// bit 0 = MSB of byte 0 = coefficient of x^0.  In registers a block is four
// little-endian words w[0..3] (bytes 0..15 in memory order).
// ---------------------------------------------------------------------------
struct u128 {
  uint32_t w[4];
};

__device__ __forceinline__ u128 u128_zero() { return u128{{0u, 0u, 0u, 0u}}; }
__device__ __forceinline__ u128 u128_xor(const u128& a, const u128& b) {
  return u128{{a.w[0] ^ b.w[0], a.w[1] ^ b.w[1], a.w[2] ^ b.w[2], a.w[3] ^ b.w[3]}};
}

// General product of two field elements (SP 800-38D Sec. 6.3 defines it bit
// by bit).  Computed on big-endian words so that "rightshift of the bit
// string" is a plain 128-bit right shift.  ~0.8k VALU ops (one bit-field
// extract and four v_bitop3 per bit of x); used only outside the per-block
// loop.
__device__ inline u128 gf_mul(const u128& x, const u128& y) {
  // 8-bit comb: V_j = y * x^j for j < 8, then Horner over the bytes of x
  // from the highest powers down, z <- z * x^8 xor sum_j x_(8n+j) V_j.  In
  // the MSB-first word order a multiply by x is a right shift by one bit, and
  // the bits x^128..x^135 that a shift by 8 pushes out fold back as
  // x^m * (1 + x + x^2 + x^7), i.e. 0xE1 << (17 + k) for pushed-out bit k.
  uint32_t V[8][4];
  V[0][0] = bswap32(y.w[0]);
  V[0][1] = bswap32(y.w[1]);
  V[0][2] = bswap32(y.w[2]);
  V[0][3] = bswap32(y.w[3]);
#pragma unroll
  for (int j = 1; j < 8; j++) {
    const uint32_t carry = 0u - (V[j - 1][3] & 1u);
    V[j][3] = __builtin_amdgcn_alignbit(V[j - 1][2], V[j - 1][3], 1);
    V[j][2] = __builtin_amdgcn_alignbit(V[j - 1][1], V[j - 1][2], 1);
    V[j][1] = __builtin_amdgcn_alignbit(V[j - 1][0], V[j - 1][1], 1);
    V[j][0] = (V[j - 1][0] >> 1) ^ (0xE1000000u & carry);
  }
  uint32_t z0 = 0, z1 = 0, z2 = 0, z3 = 0;
#pragma unroll
  for (int n = 15; n >= 0; n--) {
    const uint32_t t = z3 & 0xFFu;
    z3 = __builtin_amdgcn_alignbit(z2, z3, 8);
    z2 = __builtin_amdgcn_alignbit(z1, z2, 8);
    z1 = __builtin_amdgcn_alignbit(z0, z1, 8);
    z0 = xor3(xor3(z0 >> 8, t << 17, t << 22), t << 23, t << 24);
    const uint32_t xw = x.w[n >> 2];
#pragma unroll
    for (int j = 0; j < 8; j++) {
      const uint32_t m = 0u - ((xw >> (8 * (n & 3) + 7 - j)) & 1u);  // coefficient of x^(8n+j)
      z0 = xor_and(z0, V[j][0], m);
      z1 = xor_and(z1, V[j][1], m);
      z2 = xor_and(z2, V[j][2], m);
      z3 = xor_and(z3, V[j][3], m);
    }
  }
  return u128{{bswap32(z0), bswap32(z1), bswap32(z2), bswap32(z3)}};
}

// The element x^p (only bit p set).
__device__ inline u128 gf_xpow_elem(int p) {
  u128 r = u128_zero();
  int byte = p >> 3, bit = 7 - (p & 7);
  r.w[byte >> 2] = (uint32_t)(1u << bit) << (8 * (byte & 3));
  return r;
}

// h^e by square-and-multiply.
__device__ inline u128 gf_pow(const u128& h, uint64_t e) {
  u128 r = gf_xpow_elem(0);  // multiplicative identity
  u128 b = h;
  while (e) {
    if (e & 1) r = gf_mul(r, b);
    e >>= 1;
    if (e) b = gf_mul(b, b);
  }
  return r;
}

// XOR over the 64 lanes of a wave, returned wave-uniform.  Within each row of
// 16 lanes, DPP combines lanes 1 apart and 2 apart (quad permutations), then
// mirrored half rows and mirrored rows, after which every lane holds its
// row's XOR; the four rows are read out with readlane.  No LDS round trips (a
// shuffle butterfly takes six dependent ones).  Every lane of the wave must
// be active.
__device__ __forceinline__ uint32_t wave_xor(uint32_t v) {
  v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true);   // quad_perm [1,0,3,2]
  v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true);   // quad_perm [2,3,0,1]
  v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, true);  // row_half_mirror
  v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, true);  // row_mirror
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 0) ^ (uint32_t)__builtin_amdgcn_readlane((int)v, 16) ^
         (uint32_t)__builtin_amdgcn_readlane((int)v, 32) ^ (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
}

// The same product computed by a whole wave, x and y wave-uniform, returned
// wave-uniform: lane n < 16 takes byte n of x, i.e. the sum over j < 8 of
// x_(8n+j) * y * x^(8n+j), starting from y * x^(8n) (n shifts by 8, each
// folding the pushed-out byte back as in gf_mul), and the 16 partial sums are
// XORed across the lanes' row.  About a quarter of gf_mul's instructions in
// the wave's critical path.  Every lane of the wave must be active.
__device__ inline u128 gf_mul_wave(const u128& x, const u128& y, uint32_t lane) {
  uint32_t v0 = bswap32(y.w[0]), v1 = bswap32(y.w[1]), v2 = bswap32(y.w[2]), v3 = bswap32(y.w[3]);
  const uint32_t n = lane & 15u;
#pragma unroll 1
  for (uint32_t k = 0; k < n; k++) {
    const uint32_t t = v3 & 0xFFu;
    v3 = __builtin_amdgcn_alignbit(v2, v3, 8);
    v2 = __builtin_amdgcn_alignbit(v1, v2, 8);
    v1 = __builtin_amdgcn_alignbit(v0, v1, 8);
    v0 = xor3(xor3(v0 >> 8, t << 17, t << 22), t << 23, t << 24);
  }
  // byte n of x, by shifts of its two halves (an index into x.w would go
  // through private memory)
  const uint64_t lo = ((uint64_t)x.w[1] << 32) | x.w[0], hi = ((uint64_t)x.w[3] << 32) | x.w[2];
  const uint32_t xb = lane < 16u ? (uint32_t)(((n & 8u) ? hi : lo) >> (8u * (n & 7u))) & 0xFFu : 0u;
  uint32_t z0 = 0, z1 = 0, z2 = 0, z3 = 0;
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const uint32_t m = 0u - ((xb >> (7 - j)) & 1u);  // coefficient of x^(8n+j)
    z0 = xor_and(z0, v0, m);
    z1 = xor_and(z1, v1, m);
    z2 = xor_and(z2, v2, m);
    z3 = xor_and(z3, v3, m);
    if (j < 7) {  // v <- v * x: a right shift by one bit, folding x^128 back as 0xE1
      const uint32_t carry = 0u - (v3 & 1u);
      v3 = __builtin_amdgcn_alignbit(v2, v3, 1);
      v2 = __builtin_amdgcn_alignbit(v1, v2, 1);
      v1 = __builtin_amdgcn_alignbit(v0, v1, 1);
      v0 = (v0 >> 1) ^ (0xE1000000u & carry);
    }
  }
  return u128{{bswap32(wave_xor(z0)), bswap32(wave_xor(z1)), bswap32(wave_xor(z2)), bswap32(wave_xor(z3))}};
}

}  // namespace gift
