/*
 * Segmented, per-user seal/open and the owner-label check, as the plain
 * definition.  Test infrastructure only (see gift_oracle.h).
 *
 * Semantics (GIFT paper):
 *   - Sec. 3, workflow steps 5-6: before data leaves the protected domain,
 *     every byte is encrypted under its owner's key; here each owner segment
 *     is one GCM message under its user's key and its own IV.
 *   - Sec. 3, step 3: manipulated ownership metadata must produce only a
 *     decryption failure; here open returns AUTH_FAIL for the segment and
 *     releases none of its bytes.
 *   - Sec. 4.2: ownership is recorded per contiguous segment (a row range);
 *     memory not covered by any record is never released (zero here).
 *   - Sec. 4.3, rule step 5: all non-parameter sources of a segment must
 *     share one owner; a row label that differs from the segment's user
 *     (including the parameter and unowned sentinels) rejects the segment.
 */
#include <stdlib.h>
#include <string.h>

#include "gift_oracle.h"

/* (2^32 - 2) blocks of 16 bytes: the most one GCM invocation may encrypt
 * (SP 800-38D Sec. 5.2.1.1). */
#define MAX_SEG_BYTES ((((uint64_t)1 << 32) - 2) * 16)

void oracle_segment_iv(const uint8_t nonce_base[12], uint64_t iv_seq, uint8_t iv[12]) {
  memcpy(iv, nonce_base, 12);
  for (int k = 0; k < 8; k++) iv[11 - k] ^= (uint8_t)(iv_seq >> (8 * k));
}

static int cmp_u64pair(const void* a, const void* b) {
  const uint64_t* x = (const uint64_t*)a;
  const uint64_t* y = (const uint64_t*)b;
  if (x[0] != y[0]) return x[0] < y[0] ? -1 : 1;
  if (x[1] != y[1]) return x[1] < y[1] ? -1 : 1;
  return 0;
}

/* Validation shared by the entry points.  check_keys: 0 = owner check only
 * (no key set, no cipher): user range, GCM length limit and nonce reuse are
 * not checked; 1 = GCM entry points: all checks; 2 = per-token block cipher:
 * user range only (no IV, no GCM length). */
static int validate(uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs, uint32_t n_segs,
                    uint32_t n_users, int check_keys) {
  if (n_segs > 0 && segs == NULL) return ORACLE_E_INVALID;
  if (row_bytes == 0) return ORACLE_E_INVALID;
  for (uint32_t i = 0; i < n_segs; i++) {
    const oracle_segment* s = &segs[i];
    if (s->row_count == 0 || s->reserved != 0) return ORACLE_E_INVALID;
    if (s->user == ORACLE_LABEL_PARAM || s->user == ORACLE_LABEL_UNOWNED) return ORACLE_E_INVALID;
    if (s->row_begin > n_rows || s->row_count > n_rows - s->row_begin) return ORACLE_E_RANGE;
    if (check_keys && s->user >= n_users) return ORACLE_E_RANGE;
    /* row_count * row_bytes without overflow, then the GCM length limit */
    if (check_keys == 1 && s->row_count > MAX_SEG_BYTES / row_bytes) return ORACLE_E_TOO_LARGE;
  }
  if (n_segs > 1) {
    uint64_t* v = (uint64_t*)malloc(sizeof(uint64_t) * 2 * n_segs);
    for (uint32_t i = 0; i < n_segs; i++) {
      v[2 * i] = segs[i].row_begin;
      v[2 * i + 1] = segs[i].row_count;
    }
    qsort(v, n_segs, 2 * sizeof(uint64_t), cmp_u64pair);
    for (uint32_t i = 1; i < n_segs; i++) {
      if (v[2 * i] < v[2 * (i - 1)] + v[2 * (i - 1) + 1]) {
        free(v);
        return ORACLE_E_OVERLAP;
      }
    }
    if (check_keys == 1) {
      for (uint32_t i = 0; i < n_segs; i++) {
        v[2 * i] = segs[i].user;
        v[2 * i + 1] = segs[i].iv_seq;
      }
      qsort(v, n_segs, 2 * sizeof(uint64_t), cmp_u64pair);
      for (uint32_t i = 1; i < n_segs; i++) {
        if (v[2 * i] == v[2 * (i - 1)] && v[2 * i + 1] == v[2 * (i - 1) + 1]) {
          free(v);
          return ORACLE_E_NONCE_REUSE;
        }
      }
    }
    free(v);
  }
  return ORACLE_OK;
}

static int segment_mixed(const oracle_segment* s, const uint32_t* labels) {
  if (labels == NULL) return 0;
  for (uint64_t r = s->row_begin; r < s->row_begin + s->row_count; r++)
    if (labels[r] != s->user) return 1;
  return 0;
}

/* Zero every row that no segment covers (Sec. 4.2, unowned memory). */
static void zero_uncovered(uint8_t* out, uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs,
                           uint32_t n_segs) {
  uint8_t* covered = (uint8_t*)calloc(n_rows ? n_rows : 1, 1);
  for (uint32_t i = 0; i < n_segs; i++)
    for (uint64_t r = segs[i].row_begin; r < segs[i].row_begin + segs[i].row_count; r++) covered[r] = 1;
  for (uint64_t r = 0; r < n_rows; r++)
    if (!covered[r]) memset(out + r * row_bytes, 0, row_bytes);
  free(covered);
}

int oracle_seal(const uint8_t* data, uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs,
                uint32_t n_segs, const uint32_t* labels, const uint8_t* keys, uint32_t n_users,
                const uint8_t* nonce_base, uint8_t* out, uint8_t* tags, int32_t* verdicts) {
  if ((n_rows > 0 && (data == NULL || out == NULL)) || (n_segs > 0 && (tags == NULL || keys == NULL ||
                                                                       nonce_base == NULL)))
    return ORACLE_E_INVALID;
  int st = validate(n_rows, row_bytes, segs, n_segs, n_users, 1);
  if (st != ORACLE_OK) return st;
  for (uint32_t i = 0; i < n_segs; i++) {
    const oracle_segment* s = &segs[i];
    uint64_t off = s->row_begin * row_bytes, len = s->row_count * row_bytes;
    if (segment_mixed(s, labels)) {
      memset(out + off, 0, len);
      memset(tags + 16 * (size_t)i, 0, 16);
      if (verdicts) verdicts[i] = ORACLE_SEG_OWNER_MIXED;
      continue;
    }
    uint8_t iv[12];
    oracle_segment_iv(nonce_base + 12 * (size_t)s->user, s->iv_seq, iv);
    oracle_gcm_ae(keys + 32 * (size_t)s->user, iv, data + off, len, out + off, tags + 16 * (size_t)i);
    if (verdicts) verdicts[i] = ORACLE_SEG_OK;
  }
  zero_uncovered(out, n_rows, row_bytes, segs, n_segs);
  return ORACLE_OK;
}

int oracle_open(const uint8_t* data, uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs,
                uint32_t n_segs, const uint32_t* labels, const uint8_t* keys, uint32_t n_users,
                const uint8_t* nonce_base, uint8_t* out, const uint8_t* tags, int32_t* verdicts) {
  if ((n_rows > 0 && (data == NULL || out == NULL)) ||
      (n_segs > 0 && (tags == NULL || keys == NULL || nonce_base == NULL || verdicts == NULL)))
    return ORACLE_E_INVALID;
  int st = validate(n_rows, row_bytes, segs, n_segs, n_users, 1);
  if (st != ORACLE_OK) return st;
  for (uint32_t i = 0; i < n_segs; i++) {
    const oracle_segment* s = &segs[i];
    uint64_t off = s->row_begin * row_bytes, len = s->row_count * row_bytes;
    if (segment_mixed(s, labels)) {
      memset(out + off, 0, len);
      verdicts[i] = ORACLE_SEG_OWNER_MIXED;
      continue;
    }
    uint8_t iv[12];
    oracle_segment_iv(nonce_base + 12 * (size_t)s->user, s->iv_seq, iv);
    if (oracle_gcm_ad(keys + 32 * (size_t)s->user, iv, data + off, len, tags + 16 * (size_t)i, out + off)) {
      verdicts[i] = ORACLE_SEG_OK;
    } else {
      memset(out + off, 0, len);
      verdicts[i] = ORACLE_SEG_AUTH_FAIL;
    }
  }
  zero_uncovered(out, n_rows, row_bytes, segs, n_segs);
  return ORACLE_OK;
}

int oracle_check_owner(const oracle_segment* segs, uint32_t n_segs, const uint32_t* labels, uint64_t n_rows,
                       int32_t* verdicts) {
  if (labels == NULL || (n_segs > 0 && verdicts == NULL)) return ORACLE_E_INVALID;
  int st = validate(n_rows, 1, segs, n_segs, 0, 0);
  if (st != ORACLE_OK) return st;
  for (uint32_t i = 0; i < n_segs; i++)
    verdicts[i] = segment_mixed(&segs[i], labels) ? ORACLE_SEG_OWNER_MIXED : ORACLE_SEG_OK;
  return ORACLE_OK;
}

/* GIFT Sec. 4.5: token obfuscation -- token || random nonce through the block
 * cipher under the owner's key; a special ciphertext for end-of-sequence. */
int oracle_token_encrypt(const oracle_segment* segs, uint32_t n_segs, uint64_t n_tokens, const uint64_t* tokens,
                         const uint64_t* nonces, const uint8_t* keys, uint32_t n_users, uint64_t eos_token,
                         uint8_t* out) {
  if ((n_tokens > 0 && (tokens == NULL || nonces == NULL || out == NULL)) || (n_segs > 0 && keys == NULL))
    return ORACLE_E_INVALID;
  int st = validate(n_tokens, 1, segs, n_segs, n_users, 2);
  if (st != ORACLE_OK) return st;
  memset(out, 0, 16 * (size_t)n_tokens);
  for (uint32_t i = 0; i < n_segs; i++) {
    uint8_t w[240];
    oracle_aes256_key_expansion(keys + 32 * (size_t)segs[i].user, w);
    for (uint64_t r = segs[i].row_begin; r < segs[i].row_begin + segs[i].row_count; r++) {
      if (tokens[r] == eos_token) {
        memset(out + 16 * r, ORACLE_EOS_BYTE, 16);
        continue;
      }
      uint8_t blk[16];
      for (int k = 0; k < 8; k++) {
        blk[k] = (uint8_t)(tokens[r] >> (8 * k));
        blk[8 + k] = (uint8_t)(nonces[r] >> (8 * k));
      }
      oracle_aes256_cipher(w, blk, out + 16 * r);
    }
  }
  return ORACLE_OK;
}

int oracle_token_decrypt(const oracle_segment* segs, uint32_t n_segs, uint64_t n_tokens, const uint8_t* blocks,
                         const uint8_t* keys, uint32_t n_users, uint64_t eos_token, uint64_t* tokens_out,
                         uint64_t* nonces_out) {
  if ((n_tokens > 0 && (blocks == NULL || tokens_out == NULL)) || (n_segs > 0 && keys == NULL))
    return ORACLE_E_INVALID;
  int st = validate(n_tokens, 1, segs, n_segs, n_users, 2);
  if (st != ORACLE_OK) return st;
  for (uint64_t r = 0; r < n_tokens; r++) {
    tokens_out[r] = 0;
    if (nonces_out) nonces_out[r] = 0;
  }
  for (uint32_t i = 0; i < n_segs; i++) {
    uint8_t w[240];
    oracle_aes256_key_expansion(keys + 32 * (size_t)segs[i].user, w);
    for (uint64_t r = segs[i].row_begin; r < segs[i].row_begin + segs[i].row_count; r++) {
      int eos = 1;
      for (int k = 0; k < 16; k++) eos &= blocks[16 * r + k] == ORACLE_EOS_BYTE;
      if (eos) {
        tokens_out[r] = eos_token;
        continue;
      }
      uint8_t p[16];
      oracle_aes256_inv_cipher(w, blocks + 16 * r, p);
      uint64_t t = 0, n = 0;
      for (int k = 0; k < 8; k++) {
        t |= (uint64_t)p[k] << (8 * k);
        n |= (uint64_t)p[8 + k] << (8 * k);
      }
      tokens_out[r] = t;
      if (nonces_out) nonces_out[r] = n;
    }
  }
  return ORACLE_OK;
}
