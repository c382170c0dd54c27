/*
 * AES-256 block cipher, written out from FIPS-197.
 * Test infrastructure only (see gift_oracle.h).
 *
 * The state is the 4x4 byte array of FIPS-197 Sec. 3.4, held as st[r + 4c]
 * (row r, column c), which is exactly the order of the input bytes.
 * Nothing here is tabulated by hand: the S-box is built at first use from
 * the multiplicative inverse in GF(2^8) and the affine map of Sec. 5.1.1,
 * and the round constants are successive powers of x (Sec. 5.2).
 */
#include <pthread.h>
#include <string.h>

#include "gift_oracle.h"

/* FIPS-197 Sec. 4.2.1: multiplication by x modulo m(x) = x^8+x^4+x^3+x+1 */
static uint8_t xtime(uint8_t a) { return (uint8_t)((a << 1) ^ ((a & 0x80) ? 0x1b : 0x00)); }

/* FIPS-197 Sec. 4.2: product of two field elements by repeated xtime */
static uint8_t gf8_mul(uint8_t a, uint8_t b) {
  uint8_t p = 0;
  while (b) {
    if (b & 1) p ^= a;
    a = xtime(a);
    b >>= 1;
  }
  return p;
}

static uint8_t g_sbox[256], g_inv_sbox[256];
static pthread_once_t g_sbox_once = PTHREAD_ONCE_INIT;

/* FIPS-197 Sec. 5.1.1: S(a) = affine(inverse(a)), inverse(0) = 0,
 * b'_i = b_i ^ b_(i+4) ^ b_(i+5) ^ b_(i+6) ^ b_(i+7) ^ c_i with c = 0x63. */
static void build_sbox(void) {
  for (int a = 0; a < 256; a++) {
    uint8_t inv = 0;
    if (a != 0) {
      for (int b = 1; b < 256; b++) {
        if (gf8_mul((uint8_t)a, (uint8_t)b) == 1) {
          inv = (uint8_t)b;
          break;
        }
      }
    }
    uint8_t s = 0;
    for (int i = 0; i < 8; i++) {
      int bit = ((inv >> i) ^ (inv >> ((i + 4) & 7)) ^ (inv >> ((i + 5) & 7)) ^ (inv >> ((i + 6) & 7)) ^
                 (inv >> ((i + 7) & 7)) ^ (0x63 >> i)) &
                1;
      s |= (uint8_t)(bit << i);
    }
    g_sbox[a] = s;
  }
  for (int a = 0; a < 256; a++) g_inv_sbox[g_sbox[a]] = (uint8_t)a;
}

static void ensure_sbox(void) { pthread_once(&g_sbox_once, build_sbox); }

void oracle_aes_sbox(uint8_t sbox[256], uint8_t inv_sbox[256]) {
  ensure_sbox();
  memcpy(sbox, g_sbox, 256);
  memcpy(inv_sbox, g_inv_sbox, 256);
}

/* FIPS-197 Sec. 5.2, Nk = 8, Nr = 14: 60 words w[0..59], word i at w + 4i. */
void oracle_aes256_key_expansion(const uint8_t key[32], uint8_t w[240]) {
  ensure_sbox();
  memcpy(w, key, 32);
  uint8_t rcon = 0x01; /* x^(i/Nk - 1), starting at x^0 */
  for (int i = 8; i < 60; i++) {
    uint8_t t[4];
    memcpy(t, w + 4 * (i - 1), 4);
    if (i % 8 == 0) {
      uint8_t r = t[0]; /* RotWord */
      t[0] = t[1];
      t[1] = t[2];
      t[2] = t[3];
      t[3] = r;
      for (int k = 0; k < 4; k++) t[k] = g_sbox[t[k]]; /* SubWord */
      t[0] ^= rcon;
      rcon = xtime(rcon);
    } else if (i % 8 == 4) {
      for (int k = 0; k < 4; k++) t[k] = g_sbox[t[k]];
    }
    for (int k = 0; k < 4; k++) w[4 * i + k] = (uint8_t)(w[4 * (i - 8) + k] ^ t[k]);
  }
}

/* Sec. 5.1.4: XOR column c with round-key word w[4*round + c] */
static void add_round_key(uint8_t st[16], const uint8_t w[240], int round) {
  for (int c = 0; c < 4; c++)
    for (int r = 0; r < 4; r++) st[r + 4 * c] ^= w[16 * round + 4 * c + r];
}

static void sub_bytes(uint8_t st[16]) {
  for (int i = 0; i < 16; i++) st[i] = g_sbox[st[i]];
}

static void inv_sub_bytes(uint8_t st[16]) {
  for (int i = 0; i < 16; i++) st[i] = g_inv_sbox[st[i]];
}

/* Sec. 5.1.2: row r rotates left by r: s'[r][c] = s[r][(c + r) mod 4] */
static void shift_rows(uint8_t st[16]) {
  uint8_t t[16];
  for (int r = 0; r < 4; r++)
    for (int c = 0; c < 4; c++) t[r + 4 * c] = st[r + 4 * ((c + r) % 4)];
  memcpy(st, t, 16);
}

/* Sec. 5.3.1: s'[r][(c + r) mod 4] = s[r][c] */
static void inv_shift_rows(uint8_t st[16]) {
  uint8_t t[16];
  for (int r = 0; r < 4; r++)
    for (int c = 0; c < 4; c++) t[r + 4 * ((c + r) % 4)] = st[r + 4 * c];
  memcpy(st, t, 16);
}

/* Sec. 5.1.3: each column times the fixed matrix with rows
 * (02 03 01 01), (01 02 03 01), (01 01 02 03), (03 01 01 02). */
static void mix_columns(uint8_t st[16]) {
  for (int c = 0; c < 4; c++) {
    uint8_t a0 = st[4 * c], a1 = st[4 * c + 1], a2 = st[4 * c + 2], a3 = st[4 * c + 3];
    st[4 * c + 0] = (uint8_t)(gf8_mul(a0, 2) ^ gf8_mul(a1, 3) ^ a2 ^ a3);
    st[4 * c + 1] = (uint8_t)(a0 ^ gf8_mul(a1, 2) ^ gf8_mul(a2, 3) ^ a3);
    st[4 * c + 2] = (uint8_t)(a0 ^ a1 ^ gf8_mul(a2, 2) ^ gf8_mul(a3, 3));
    st[4 * c + 3] = (uint8_t)(gf8_mul(a0, 3) ^ a1 ^ a2 ^ gf8_mul(a3, 2));
  }
}

/* Sec. 5.3.3: inverse matrix rows (0e 0b 0d 09), (09 0e 0b 0d), (0d 09 0e 0b), (0b 0d 09 0e) */
static void inv_mix_columns(uint8_t st[16]) {
  for (int c = 0; c < 4; c++) {
    uint8_t a0 = st[4 * c], a1 = st[4 * c + 1], a2 = st[4 * c + 2], a3 = st[4 * c + 3];
    st[4 * c + 0] = (uint8_t)(gf8_mul(a0, 0x0e) ^ gf8_mul(a1, 0x0b) ^ gf8_mul(a2, 0x0d) ^ gf8_mul(a3, 0x09));
    st[4 * c + 1] = (uint8_t)(gf8_mul(a0, 0x09) ^ gf8_mul(a1, 0x0e) ^ gf8_mul(a2, 0x0b) ^ gf8_mul(a3, 0x0d));
    st[4 * c + 2] = (uint8_t)(gf8_mul(a0, 0x0d) ^ gf8_mul(a1, 0x09) ^ gf8_mul(a2, 0x0e) ^ gf8_mul(a3, 0x0b));
    st[4 * c + 3] = (uint8_t)(gf8_mul(a0, 0x0b) ^ gf8_mul(a1, 0x0d) ^ gf8_mul(a2, 0x09) ^ gf8_mul(a3, 0x0e));
  }
}

/* Sec. 5.1 Cipher with Nr = 14 */
void oracle_aes256_cipher(const uint8_t w[240], const uint8_t in[16], uint8_t out[16]) {
  ensure_sbox();
  uint8_t st[16];
  memcpy(st, in, 16);
  add_round_key(st, w, 0);
  for (int round = 1; round < 14; round++) {
    sub_bytes(st);
    shift_rows(st);
    mix_columns(st);
    add_round_key(st, w, round);
  }
  sub_bytes(st);
  shift_rows(st);
  add_round_key(st, w, 14);
  memcpy(out, st, 16);
}

/* Sec. 5.3 InvCipher with Nr = 14 */
void oracle_aes256_inv_cipher(const uint8_t w[240], const uint8_t in[16], uint8_t out[16]) {
  ensure_sbox();
  uint8_t st[16];
  memcpy(st, in, 16);
  add_round_key(st, w, 14);
  for (int round = 13; round >= 1; round--) {
    inv_shift_rows(st);
    inv_sub_bytes(st);
    add_round_key(st, w, round);
    inv_mix_columns(st);
  }
  inv_shift_rows(st);
  inv_sub_bytes(st);
  add_round_key(st, w, 0);
  memcpy(out, st, 16);
}
