/*
 * GCM with a 96-bit IV, 128-bit tag and no additional data, written out from
 * NIST SP 800-38D.  Test infrastructure only (see gift_oracle.h).
 *
 * Bit strings follow Sec. 6.1/6.3: bit 0 of a 128-bit block is the most
 * significant bit of byte 0.
 */
#include <string.h>

#include "gift_oracle.h"

/* Sec. 6.3, Algorithm 1: Z = X * Y in GF(2^128), R = 11100001 || 0^120. */
void oracle_gf128_mul(const uint8_t x[16], const uint8_t y[16], uint8_t z[16]) {
  uint8_t zz[16] = {0}, v[16];
  memcpy(v, y, 16);
  for (int i = 0; i < 128; i++) {
    int xi = (x[i / 8] >> (7 - (i % 8))) & 1;
    if (xi)
      for (int k = 0; k < 16; k++) zz[k] ^= v[k];
    int lsb = v[15] & 1; /* LSB_1(V_i): the last bit of the string */
    for (int k = 15; k > 0; k--) v[k] = (uint8_t)((v[k] >> 1) | (v[k - 1] << 7));
    v[0] >>= 1;
    if (lsb) v[0] ^= 0xE1;
  }
  memcpy(z, zz, 16);
}

/* Sec. 6.4, Algorithm 2: Y_i = (Y_{i-1} xor X_i) * H over m whole blocks. */
void oracle_ghash(const uint8_t h[16], const uint8_t* x, size_t nblocks, uint8_t y[16]) {
  uint8_t acc[16] = {0};
  for (size_t i = 0; i < nblocks; i++) {
    for (int k = 0; k < 16; k++) acc[k] ^= x[16 * i + k];
    oracle_gf128_mul(acc, h, acc);
  }
  memcpy(y, acc, 16);
}

/* Sec. 6.2: inc32 increments the rightmost 32 bits modulo 2^32 (big-endian). */
static void inc32(uint8_t cb[16]) {
  for (int k = 15; k >= 12; k--) {
    cb[k]++;
    if (cb[k] != 0) break;
  }
}

/* Sec. 6.5, Algorithm 3: GCTR.  A final partial block uses the leading bytes
 * of its cipher output. */
void oracle_gctr(const uint8_t w[240], const uint8_t icb[16], const uint8_t* x, size_t len, uint8_t* y) {
  uint8_t cb[16], ks[16];
  memcpy(cb, icb, 16);
  for (size_t off = 0; off < len; off += 16) {
    oracle_aes256_cipher(w, cb, ks);
    size_t n = (len - off < 16) ? (len - off) : 16;
    for (size_t k = 0; k < n; k++) y[off + k] = (uint8_t)(x[off + k] ^ ks[k]);
    inc32(cb);
  }
}

/* GHASH_H(C || 0^u || 0^64 || [len(C)]_64) as Algorithm 2 over the padded
 * string, fed one block at a time. */
static void ghash_c_len(const uint8_t h[16], const uint8_t* c, size_t len, uint8_t s[16]) {
  uint8_t acc[16] = {0}, blk[16];
  for (size_t off = 0; off < len; off += 16) {
    size_t n = (len - off < 16) ? (len - off) : 16;
    memset(blk, 0, 16);
    memcpy(blk, c + off, n);
    for (int k = 0; k < 16; k++) acc[k] ^= blk[k];
    oracle_gf128_mul(acc, h, acc);
  }
  memset(blk, 0, 16); /* [len(A)]_64 = 0 */
  uint64_t bits = (uint64_t)len * 8u;
  for (int k = 0; k < 8; k++) blk[15 - k] = (uint8_t)(bits >> (8 * k));
  for (int k = 0; k < 16; k++) acc[k] ^= blk[k];
  oracle_gf128_mul(acc, h, acc);
  memcpy(s, acc, 16);
}

/* Sec. 7.1, Algorithm 4 with a 96-bit IV: J0 = IV || 0^31 || 1. */
void oracle_gcm_ae(const uint8_t key[32], const uint8_t iv[12], const uint8_t* p, size_t len, uint8_t* c,
                   uint8_t tag[16]) {
  uint8_t w[240], zero[16] = {0}, h[16], j0[16], icb[16], s[16], ej0[16];
  oracle_aes256_key_expansion(key, w);
  oracle_aes256_cipher(w, zero, h);
  memcpy(j0, iv, 12);
  j0[12] = 0;
  j0[13] = 0;
  j0[14] = 0;
  j0[15] = 1;
  memcpy(icb, j0, 16);
  inc32(icb);
  oracle_gctr(w, icb, p, len, c);
  ghash_c_len(h, c, len, s);
  oracle_aes256_cipher(w, j0, ej0); /* GCTR_K(J0, S) for one block */
  for (int k = 0; k < 16; k++) tag[k] = (uint8_t)(ej0[k] ^ s[k]);
}

/* Sec. 7.2, Algorithm 5: returns 1 and writes P when T' = T, else 0. */
int oracle_gcm_ad(const uint8_t key[32], const uint8_t iv[12], const uint8_t* c, size_t len, const uint8_t tag[16],
                  uint8_t* p) {
  uint8_t w[240], zero[16] = {0}, h[16], j0[16], icb[16], s[16], ej0[16], t2[16];
  oracle_aes256_key_expansion(key, w);
  oracle_aes256_cipher(w, zero, h);
  memcpy(j0, iv, 12);
  j0[12] = 0;
  j0[13] = 0;
  j0[14] = 0;
  j0[15] = 1;
  ghash_c_len(h, c, len, s);
  oracle_aes256_cipher(w, j0, ej0);
  int diff = 0;
  for (int k = 0; k < 16; k++) {
    t2[k] = (uint8_t)(ej0[k] ^ s[k]);
    diff |= t2[k] ^ tag[k];
  }
  if (diff) return 0;
  memcpy(icb, j0, 16);
  inc32(icb);
  oracle_gctr(w, icb, c, len, p);
  return 1;
}
