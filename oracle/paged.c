/*
 * Paged-KV seal/open as the plain definition: gather the request's chunks in
 * stream order, run the GCM oracle on the gathered message, place the result.
 * Test infrastructure only (see gift_oracle.h).
 *
 * GIFT Sec. 4.2: PagedAttention splits the KV cache into blocks and ownership
 * is recorded per KV block; Sec. 4.5: block tables are kept by the monitor;
 * Sec. 2.2: a manipulated block table makes a request read another user's
 * KV -- here the per-block labels reject such a request.
 */
#include <stdlib.h>
#include <string.h>

#include "gift_oracle.h"

#define MAX_SEG_BYTES ((((uint64_t)1 << 32) - 2) * 16)

static uint64_t chunk_offset(const oracle_paged_kv* kv, uint64_t l, uint64_t b, uint64_t p) {
  return l * kv->layer_stride + b * kv->block_stride + p * kv->part_stride;
}

static int cmp_u64(const void* a, const void* b) {
  uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* geometry: sort the three (stride, count) pairs; each stride with count > 1
 * must be at least the extent of what it contains */
static int geometry_ok(const oracle_paged_kv* kv) {
  uint64_t cb = kv->chunk_bytes;
  if (cb < 16 || (cb & (cb - 1))) return 0;
  if ((kv->layer_stride % 16) || (kv->block_stride % 16) || (kv->part_stride % 16)) return 0;
  if (kv->n_layers == 0 || kv->n_parts == 0 || kv->n_blocks == 0) return 0;
  uint64_t st[3] = {kv->layer_stride, kv->block_stride, kv->part_stride};
  uint64_t ct[3] = {kv->n_layers, kv->n_blocks, kv->n_parts};
  for (int i = 0; i < 3; i++) /* selection sort by stride */
    for (int j = i + 1; j < 3; j++)
      if (st[j] < st[i]) {
        uint64_t t = st[i];
        st[i] = st[j];
        st[j] = t;
        t = ct[i];
        ct[i] = ct[j];
        ct[j] = t;
      }
  unsigned __int128 extent = cb;
  for (int i = 0; i < 3; i++) {
    if (ct[i] <= 1) continue;
    if ((unsigned __int128)st[i] < extent) return 0;
    extent += (unsigned __int128)st[i] * (ct[i] - 1);
    if (extent >> 64) return 0;
  }
  return 1;
}

static int validate_paged(const oracle_paged_kv* kv, const oracle_request* reqs, uint32_t n, uint32_t n_users) {
  if (!geometry_ok(kv)) return ORACLE_E_INVALID;
  uint64_t per_block = (uint64_t)kv->n_layers * kv->n_parts * kv->chunk_bytes;
  unsigned __int128 fixed = (unsigned __int128)kv->layer_stride * (kv->n_layers - 1) +
                            (unsigned __int128)kv->part_stride * (kv->n_parts - 1) + kv->chunk_bytes;
  uint64_t total = 0;
  for (uint32_t i = 0; i < n; i++) {
    const oracle_request* r = &reqs[i];
    if (r->n_block_ids == 0 || r->block_ids == NULL) return ORACLE_E_INVALID;
    if (r->user == ORACLE_LABEL_PARAM || r->user == ORACLE_LABEL_UNOWNED) return ORACLE_E_INVALID;
    uint32_t maxb = 0;
    for (uint32_t j = 0; j < r->n_block_ids; j++)
      if (r->block_ids[j] > maxb) maxb = r->block_ids[j];
    if (maxb >= kv->n_blocks) return ORACLE_E_RANGE;
    if (r->user >= n_users) return ORACLE_E_RANGE;
    if ((unsigned __int128)kv->block_stride * maxb + fixed > kv->cache_bytes) return ORACLE_E_RANGE;
    if ((unsigned __int128)per_block * r->n_block_ids > MAX_SEG_BYTES) return ORACLE_E_TOO_LARGE;
    total += r->n_block_ids;
  }
  uint64_t* v = (uint64_t*)malloc(sizeof(uint64_t) * 2 * (total + n + 1));
  uint64_t k = 0;
  for (uint32_t i = 0; i < n; i++)
    for (uint32_t j = 0; j < reqs[i].n_block_ids; j++) v[k++] = reqs[i].block_ids[j];
  qsort(v, k, sizeof(uint64_t), cmp_u64);
  for (uint64_t j = 1; j < k; j++)
    if (v[j] == v[j - 1]) {
      free(v);
      return ORACLE_E_OVERLAP;
    }
  /* (user, iv_seq) pairs: user in the high bits would collide, so compare pairs directly */
  for (uint32_t i = 0; i < n; i++)
    for (uint32_t j = i + 1; j < n; j++)
      if (reqs[i].user == reqs[j].user && reqs[i].iv_seq == reqs[j].iv_seq) {
        free(v);
        return ORACLE_E_NONCE_REUSE;
      }
  free(v);
  return ORACLE_OK;
}

static int request_mixed(const oracle_request* r, const uint32_t* labels) {
  if (labels == NULL) return 0;
  for (uint32_t j = 0; j < r->n_block_ids; j++)
    if (labels[r->block_ids[j]] != r->user) return 1;
  return 0;
}

/* the request's stream: for each block of its table, each layer, each part */
static void gather(const uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* r, uint8_t* dst) {
  uint64_t o = 0;
  for (uint32_t j = 0; j < r->n_block_ids; j++)
    for (uint64_t l = 0; l < kv->n_layers; l++)
      for (uint64_t p = 0; p < kv->n_parts; p++) {
        memcpy(dst + o, cache + chunk_offset(kv, l, r->block_ids[j], p), kv->chunk_bytes);
        o += kv->chunk_bytes;
      }
}

static void scatter(uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* r, const uint8_t* src) {
  uint64_t o = 0;
  for (uint32_t j = 0; j < r->n_block_ids; j++)
    for (uint64_t l = 0; l < kv->n_layers; l++)
      for (uint64_t p = 0; p < kv->n_parts; p++) {
        if (src)
          memcpy(cache + chunk_offset(kv, l, r->block_ids[j], p), src + o, kv->chunk_bytes);
        else
          memset(cache + chunk_offset(kv, l, r->block_ids[j], p), 0, kv->chunk_bytes);
        o += kv->chunk_bytes;
      }
}

int oracle_seal_paged(const uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* reqs, uint32_t n,
                      const uint32_t* block_labels, const uint8_t* keys, uint32_t n_users, const uint8_t* nonce_base,
                      uint8_t* out, uint8_t* tags, int32_t* verdicts) {
  if (kv == NULL || (n > 0 && (reqs == NULL || cache == NULL || keys == NULL || nonce_base == NULL || out == NULL ||
                               tags == NULL)))
    return ORACLE_E_INVALID;
  int st = validate_paged(kv, reqs, n, n_users);
  if (st != ORACLE_OK) return st;
  uint64_t per_block = (uint64_t)kv->n_layers * kv->n_parts * kv->chunk_bytes, off = 0;
  for (uint32_t i = 0; i < n; i++) {
    const oracle_request* r = &reqs[i];
    uint64_t len = per_block * r->n_block_ids;
    if (request_mixed(r, block_labels)) {
      memset(out + off, 0, len);
      memset(tags + 16 * (size_t)i, 0, 16);
      if (verdicts) verdicts[i] = ORACLE_SEG_OWNER_MIXED;
    } else {
      uint8_t* msg = (uint8_t*)malloc(len);
      gather(cache, kv, r, msg);
      uint8_t iv[12];
      oracle_segment_iv(nonce_base + 12 * (size_t)r->user, r->iv_seq, iv);
      oracle_gcm_ae(keys + 32 * (size_t)r->user, iv, msg, len, out + off, tags + 16 * (size_t)i);
      free(msg);
      if (verdicts) verdicts[i] = ORACLE_SEG_OK;
    }
    off += len;
  }
  return ORACLE_OK;
}

int oracle_open_paged(uint8_t* cache, const oracle_paged_kv* kv, const oracle_request* reqs, uint32_t n,
                      const uint32_t* block_labels, const uint8_t* keys, uint32_t n_users, const uint8_t* nonce_base,
                      const uint8_t* in, const uint8_t* tags, int32_t* verdicts) {
  if (kv == NULL || (n > 0 && (reqs == NULL || cache == NULL || keys == NULL || nonce_base == NULL || in == NULL ||
                               tags == NULL || verdicts == NULL)))
    return ORACLE_E_INVALID;
  int st = validate_paged(kv, reqs, n, n_users);
  if (st != ORACLE_OK) return st;
  uint64_t per_block = (uint64_t)kv->n_layers * kv->n_parts * kv->chunk_bytes, off = 0;
  for (uint32_t i = 0; i < n; i++) {
    const oracle_request* r = &reqs[i];
    uint64_t len = per_block * r->n_block_ids;
    if (request_mixed(r, block_labels)) {
      /* Rejected at launch (Sec. 4.1, malicious behaviour detection): the
       * request's table names a block of another owner, so the open runs
       * for none of its chunks and writes nothing -- that owner's block
       * keeps its contents, and the manipulation shows only as this
       * request's failure (Sec. 3, workflow step 3). */
      verdicts[i] = ORACLE_SEG_OWNER_MIXED;
    } else {
      uint8_t* msg = (uint8_t*)malloc(len);
      uint8_t iv[12];
      oracle_segment_iv(nonce_base + 12 * (size_t)r->user, r->iv_seq, iv);
      if (oracle_gcm_ad(keys + 32 * (size_t)r->user, iv, in + off, len, tags + 16 * (size_t)i, msg)) {
        scatter(cache, kv, r, msg);
        verdicts[i] = ORACLE_SEG_OK;
      } else {
        scatter(cache, kv, r, NULL);
        verdicts[i] = ORACLE_SEG_AUTH_FAIL;
      }
      free(msg);
    }
    off += len;
  }
  return ORACLE_OK;
}
