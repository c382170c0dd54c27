/*
 * CPU oracle for segmented, per-user AES-256-GCM seal/open and the
 * owner-label check.
 *
 * TEST INFRASTRUCTURE ONLY.  This code is the plain, slow, obviously-correct
 * definition that the GPU library is checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or constant with the GPU library: the S-box,
 * the round constants and the GHASH reduction are recomputed here from their
 * mathematical definitions.
 *
 * Sources followed:
 *   - AES-256: FIPS-197 (Sec. 4.2 field arithmetic, Sec. 5.1 Cipher,
 *     Sec. 5.1.1 S-box construction, Sec. 5.2 KeyExpansion with Nk=8, Nr=14,
 *     Sec. 5.3 InvCipher).
 *   - GCM: NIST SP 800-38D (Sec. 6.2 inc32, Sec. 6.3 Algorithm 1 (bitwise
 *     multiply in GF(2^128)), Sec. 6.4 Algorithm 2 GHASH, Sec. 6.5 Algorithm 3
 *     GCTR, Sec. 7.1 Algorithm 4 GCM-AE, Sec. 7.2 Algorithm 5 GCM-AD), with a
 *     96-bit IV, a 128-bit tag and no additional authenticated data.
 *   - Token encryption: the GIFT paper, Sec. 4.5 (a 64-bit token extended to
 *     128 bits with a random nonce and enciphered as one block under the
 *     owner's key; a special ciphertext marks the end of the sequence).
 *   - Segment semantics: the GIFT paper, Sec. 3 (system workflow, steps 3-6:
 *     per-owner keys; manipulated ownership metadata must yield only a
 *     decryption failure; every exported byte is encrypted under its owner's
 *     key), Sec. 4.2 (ownership recorded per contiguous segment; unowned
 *     memory is never released) and Sec. 4.3 (rule step 5: all non-parameter
 *     sources of a segment must share one owner).
 *
 * Parity status: every function here is pinned by CPU tests against
 * independent facts (OpenSSL's AES/GCM, closed forms in GF(2^128), field
 * axioms, brute force on tiny tensors); none is "parity unpinned".
 */
#ifndef GIFT_ORACLE_H
#define GIFT_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes (same numeric contract as the library's) ---- */
#define ORACLE_OK 0
#define ORACLE_E_INVALID -1    /* null pointer, zero row_bytes, empty segment, bad sentinel/reserved */
#define ORACLE_E_RANGE -2      /* rows beyond the tensor, user beyond the key set */
#define ORACLE_E_OVERLAP -3    /* two segments share a row */
#define ORACLE_E_NONCE_REUSE -4 /* two segments share (user, iv_seq) */
#define ORACLE_E_TOO_LARGE -5  /* segment longer than (2^32-2) blocks */

/* per-segment verdicts */
#define ORACLE_SEG_OK 0
#define ORACLE_SEG_AUTH_FAIL 1
#define ORACLE_SEG_OWNER_MIXED 2

#define ORACLE_LABEL_PARAM 0xFFFFFFFEu
#define ORACLE_LABEL_UNOWNED 0xFFFFFFFFu

/* one owner segment: a contiguous row range of one user (paper Sec. 4.2) */
typedef struct {
  uint64_t row_begin;
  uint64_t row_count;
  uint32_t user;
  uint32_t reserved; /* must be 0 */
  uint64_t iv_seq;
} oracle_segment;

/* ---- AES-256 (FIPS-197) ---- */
void oracle_aes_sbox(uint8_t sbox[256], uint8_t inv_sbox[256]);
void oracle_aes256_key_expansion(const uint8_t key[32], uint8_t w[240]);
void oracle_aes256_cipher(const uint8_t w[240], const uint8_t in[16], uint8_t out[16]);
void oracle_aes256_inv_cipher(const uint8_t w[240], const uint8_t in[16], uint8_t out[16]);

/* ---- GCM pieces (SP 800-38D) ---- */
void oracle_gf128_mul(const uint8_t x[16], const uint8_t y[16], uint8_t z[16]);
void oracle_ghash(const uint8_t h[16], const uint8_t* x, size_t nblocks, uint8_t y[16]);
void oracle_gctr(const uint8_t w[240], const uint8_t icb[16], const uint8_t* x, size_t len, uint8_t* y);
void oracle_gcm_ae(const uint8_t key[32], const uint8_t iv[12], const uint8_t* p, size_t len,
                   uint8_t* c, uint8_t tag[16]);
/* returns 1 when the tag verifies (p holds the plaintext), 0 on FAIL (p untouched) */
int oracle_gcm_ad(const uint8_t key[32], const uint8_t iv[12], const uint8_t* c, size_t len,
                  const uint8_t tag[16], uint8_t* p);

/* IV of a segment: nonce_base[user] XOR (0^32 || BE64(iv_seq)) */
void oracle_segment_iv(const uint8_t nonce_base[12], uint64_t iv_seq, uint8_t iv[12]);

/* ---- segmented semantics ----
 * data/out: n_rows*row_bytes host bytes (out may equal data).
 * keys: n_users*32 bytes; nonce_base: n_users*12 bytes.
 * labels: n_rows u32 or NULL (no owner check).
 * tags: n_segs*16 bytes.  verdicts: n_segs int32 (may be NULL for seal).
 * Validation order: per segment in caller order (INVALID, then RANGE, then
 * TOO_LARGE), then OVERLAP over all segments, then NONCE_REUSE.
 * Rows that no segment covers are zero in out.  A rejected segment has zero
 * output bytes (and a zero tag on seal). */
int oracle_seal(const uint8_t* data, uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs,
                uint32_t n_segs, const uint32_t* labels, const uint8_t* keys, uint32_t n_users,
                const uint8_t* nonce_base, uint8_t* out, uint8_t* tags, int32_t* verdicts);
int oracle_open(const uint8_t* data, uint64_t n_rows, uint64_t row_bytes, const oracle_segment* segs,
                uint32_t n_segs, const uint32_t* labels, const uint8_t* keys, uint32_t n_users,
                const uint8_t* nonce_base, uint8_t* out, const uint8_t* tags, int32_t* verdicts);
/* Owner check only: writes verdicts (OK / OWNER_MIXED). */
int oracle_check_owner(const oracle_segment* segs, uint32_t n_segs, const uint32_t* labels,
                       uint64_t n_rows, int32_t* verdicts);

/* ---- paged KV cache (GIFT Sec. 4.2 KV blocks, Sec. 4.5 index tables) ----
 * cache: host copy of the cache allocation (cache_bytes bytes).  Chunk
 * (layer l, block b, part p) = cache[l*ls + b*bs + p*ps, + chunk_bytes).
 * A request's stream is its chunks for each block of its table, each layer,
 * each part, in that order; it is one GCM message.  Seal writes request i's
 * ciphertext at out + (sum of earlier requests' lengths).  With
 * block_labels, a request holding a block labelled with anyone else is
 * rejected: zero ciphertext and tag on seal; on open nothing is written
 * into the cache (its table names another owner's block, which must keep
 * its contents).  Open scatters verified plaintext into the table's chunks
 * and zeroes the chunks of requests that fail authentication.
 * Validation: geometry (INVALID: chunk a power of two >= 16, strides multiples
 * of 16, counts >= 1, strided dimensions that do not overlap), then per
 * request in order: INVALID (empty table, sentinel user), RANGE (block id,
 * user, chunk beyond cache_bytes), TOO_LARGE; then OVERLAP (a block id twice
 * in the call); then NONCE_REUSE. */
typedef struct {
  uint64_t cache_bytes;
  uint64_t layer_stride, block_stride, part_stride;
  uint64_t chunk_bytes;
  uint32_t n_layers, n_parts;
  uint64_t n_blocks;
} oracle_paged_kv;

typedef struct {
  const uint32_t* block_ids;
  uint32_t n_block_ids;
  uint32_t user;
  uint64_t iv_seq;
} oracle_request;

int oracle_seal_paged(const uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* reqs, uint32_t n_reqs,
                      const uint32_t* block_labels, const uint8_t* keys, uint32_t n_users, const uint8_t* nonce_base,
                      uint8_t* out, uint8_t* tags, int32_t* verdicts);
int oracle_open_paged(uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* reqs, uint32_t n_reqs,
                      const uint32_t* block_labels, const uint8_t* keys, uint32_t n_users, const uint8_t* nonce_base,
                      const uint8_t* in, const uint8_t* tags, int32_t* verdicts);

/* ---- per-token encryption (GIFT Sec. 4.5) ----
 * Token i (a row of a token buffer; segments index tokens) of user u:
 *   block = LE64(tokens[i]) || LE64(nonces[i]);  out[i] = CIPH_Ku(block)
 * except tokens[i] == eos_token, whose ciphertext is the reserved block of
 * sixteen 0xFF bytes (for every key).  Tokens covered by no segment give a
 * zero block.  Decryption inverts this: the reserved block gives eos_token
 * (nonce 0); other blocks give the first 8 bytes of CIPH^-1 as the token and
 * the last 8 as the nonce; uncovered tokens give 0.  Validation: INVALID,
 * RANGE (rows, users) and OVERLAP as for the tensor entry points; iv_seq is
 * unused. */
#define ORACLE_EOS_BYTE 0xFF
int oracle_token_encrypt(const oracle_segment* segs, uint32_t n_segs, uint64_t n_tokens, const uint64_t* tokens,
                         const uint64_t* nonces, const uint8_t* keys, uint32_t n_users, uint64_t eos_token,
                         uint8_t* out);
int oracle_token_decrypt(const oracle_segment* segs, uint32_t n_segs, uint64_t n_tokens, const uint8_t* blocks,
                         const uint8_t* keys, uint32_t n_users, uint64_t eos_token, uint64_t* tokens_out,
                         uint64_t* nonces_out);

#ifdef __cplusplus
}
#endif
#endif
