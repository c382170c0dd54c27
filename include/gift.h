/*
 * gift.h -- ownership-segmented, per-user AES-256-GCM seal/open of
 * GPU-resident tensors, and the owner-label check, for AMD Instinct MI355X
 * (gfx950).
 *
 * This library is the data-parallel part of "encryption-as-isolation" from
 * the GIFT paper (Sec. 3, System overview): each user's data that leaves the
 * protected domain is encrypted under that user's own key, so a framework
 * that mixes or misroutes ciphertexts learns nothing and can only cause a
 * decryption failure.  Ownership is recorded per contiguous segment of rows
 * (Sec. 4.2, Ownership Segmentation).  The paper does not name a cipher; this
 * library uses AES-256-GCM (FIPS-197, NIST SP 800-38D) with a 96-bit IV, a
 * 16-byte tag and no additional authenticated data.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Memory: pointers documented "device" are HIP device pointers on the
 *   current device; "host" pointers are ordinary host memory that the call
 *   reads before it returns (the caller may reuse it right away).  The
 *   caller owns every buffer it passes.  The library owns the key-table
 *   handle, one pinned host staging ring per device (8 MiB) and device
 *   scratch kept per (device, stream) for later calls (at most 16 buffers
 *   per device, each as large as the largest call on its stream needed; held
 *   until the process ends).  Calls on one stream reuse its buffer in stream
 *   order; a buffer moves to another stream only after its last use.  A
 *   call that reuses a buffer also makes its stream wait for the buffer's
 *   last use, since one handle can name different streams (a handle reused
 *   after hipStreamDestroy, hipStreamPerThread in each thread).
 * - Errors: a call returns GIFT_OK or a negative gift_status.  Argument
 *   errors are detected on the host before anything is enqueued; when a call
 *   returns an error no GPU work was enqueued and no output was touched.
 * - Asynchrony: all GPU work is enqueued on `stream` (NULL = the null
 *   stream).  Outputs (ciphertext, plaintext, tags, verdicts) are valid once
 *   the stream reaches the end of the call -- the analogue of the paper's
 *   rule that keys are selected only after the device-to-host copy of the
 *   data has been waited for (Sec. 4.1, Insight 3).  Calls on different
 *   streams are independent; overlapping calls on one output buffer race.
 * - Tensor layout: `data` holds n_rows rows of row_bytes bytes each,
 *   contiguous, row-major.  Bytes are encrypted in memory order; no dtype is
 *   interpreted.
 * - Segment i of a table covers bytes [row_begin*row_bytes,
 *   (row_begin+row_count)*row_bytes) and is one GCM message under the key of
 *   `user` with IV = nonce_base[user] XOR (0^32 || BE64(iv_seq)).  tags[i]
 *   and verdicts[i] follow the caller's order of segments.
 * - Rows covered by no segment are written as zero in `out` (Sec. 4.2:
 *   memory without an ownership record is never released).
 * - Thread safety: every entry point may be called concurrently from
 *   several host threads; a key table may be shared by several streams.
 */
#ifndef GIFT_H
#define GIFT_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GIFT_OK = 0,
  GIFT_E_INVALID = -1,     /* null pointer, zero row_bytes, empty segment, reserved != 0,
                              sentinel user, partial overlap of out and data */
  GIFT_E_RANGE = -2,       /* segment rows beyond n_rows, user >= n_users */
  GIFT_E_OVERLAP = -3,     /* two segments share a row */
  GIFT_E_NONCE_REUSE = -4, /* two segments of one call share (user, iv_seq) */
  GIFT_E_TOO_LARGE = -5,   /* segment longer than (2^32-2)*16 bytes (SP 800-38D Sec. 5.2.1.1) */
  GIFT_E_HIP = -6,         /* a HIP runtime call failed */
  GIFT_E_NOMEM = -7,       /* device or pinned host allocation failed */
  GIFT_E_REJECTED = -8,    /* an IFT rule refused a launch (include/gift_ift.h) */
  GIFT_E_RACE = -9         /* a launch would race with another stream (include/gift_ift.h) */
} gift_status;

/* per-segment verdicts, int32 */
enum { GIFT_SEG_OK = 0, GIFT_SEG_AUTH_FAIL = 1, GIFT_SEG_OWNER_MIXED = 2 };

/* Row-label sentinels (Sec. 4.2 / Sec. 3 step 0): rows holding model
 * parameters, and rows with no ownership record.  Neither is a valid user. */
#define GIFT_LABEL_PARAM 0xFFFFFFFEu
#define GIFT_LABEL_UNOWNED 0xFFFFFFFFu

/* A tensor in device memory: n_rows rows of row_bytes bytes, contiguous. */
typedef struct {
  void* data; /* device */
  uint64_t n_rows;
  uint64_t row_bytes;
} gift_tensor;

/* One owner segment (32 bytes): a contiguous row range owned by one user
 * (Sec. 4.2, ownership record = subscripts of the ownership dimension +
 * owner ID).  iv_seq makes the IV unique; the caller must never reuse a
 * (user, iv_seq) pair across calls either. */
typedef struct {
  uint64_t row_begin;
  uint64_t row_count; /* >= 1 */
  uint32_t user;      /* < n_users of the key table */
  uint32_t reserved;  /* must be 0 */
  uint64_t iv_seq;
} gift_segment;

/* The segments of one call.  segs is a host array in any order (segments
 * must not overlap).  row_labels (device, n_rows u32, or NULL) enables the
 * fused owner check in gift_seal/gift_open.  verdicts (device, n_segs int32)
 * receives one verdict per segment; it may be NULL for gift_seal only. */
typedef struct {
  const gift_segment* segs; /* host */
  uint32_t n_segs;
  const uint32_t* row_labels; /* device or NULL */
  int32_t* verdicts;          /* device or NULL (seal only) */
} gift_segment_table;

/* Opaque, immutable, device-resident per-user key material. */
typedef struct gift_key_table_s* gift_key_table;

/*
 * Expands n_users AES-256 keys (host, n_users*32 bytes; user u's key at
 * keys + 32*u) into device-resident key material: the FIPS-197 key schedule
 * (and that of the equivalent inverse cipher), the GHASH key H = E_K(0^128)
 * and the per-user tables of powers of H the kernels use.  The paper keeps user keys in the monitor's protected memory
 * (Sec. 3, step 0); here that memory is the GPU's.  The expansion runs on
 * `stream`; the table may be used by later work on that stream at once, and
 * on other streams after the caller has synchronised with it.  Host copies
 * of the keys are wiped before return.
 * Errors: GIFT_E_INVALID (null keys/out, n_users == 0 or >= GIFT_LABEL_PARAM),
 * GIFT_E_NOMEM, GIFT_E_HIP.
 */
gift_status gift_key_table_create(const uint8_t* keys, uint32_t n_users, hipStream_t stream,
                                  gift_key_table* out);

/* Number of users of a key table (0 for NULL). */
uint32_t gift_key_table_users(gift_key_table kt);

/* Zeroes the device key material and frees it.  Synchronises the device
 * first, so no enqueued call may still use the table.  NULL is a no-op. */
gift_status gift_key_table_destroy(gift_key_table kt);

/*
 * Seal (encrypt + authenticate) each segment of `t` under its owner's key
 * (Sec. 3, steps 5-6: data is encrypted with its owners' keys before it is
 * returned to the untrusted framework).
 *   t          tensor to seal (device data).
 *   st         segments; st->row_labels enables the fused owner check:
 *              a segment whose rows carry any label other than its user
 *              (including the sentinels) is rejected -- its bytes in `out`
 *              and its tag are zeroed and its verdict is OWNER_MIXED
 *              (Sec. 4.3, rule step 5; Sec. 4.1, launch rejection).
 *   kt         key table with n_users > every segment's user.
 *   nonce_base host, n_users*12 bytes.
 *   out        device, n_rows*row_bytes bytes; may equal t->data (in place)
 *              but must not partially overlap it.
 *   tags       device, n_segs*16 bytes, written.
 * Errors: see gift_status; all detected before any work is enqueued.
 */
gift_status gift_seal(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt,
                      const uint8_t* nonce_base, void* out, uint8_t* tags, hipStream_t stream);

/*
 * gift_seal for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, semantics, validation and outputs as gift_seal, but it calls no
 * hipMalloc, hipFree, hipHostMalloc or hipEventCreate: its device workspace
 * is a fixed array of GIFT_NOALLOC_WORKSPACE_BYTES in the library's code
 * object, one per device (held until the process ends), and its tables go
 * through a staging ring allocated up front.  Both are set up by
 * gift_key_table_create on the key table's device, so a key table must have
 * been created on the current device first.
 *   Limit: the call's workspace (64 B per segment, 16 B per 2 MiB tile and per
 *   queue entry, 32 B per zero range and 4 MiB of uncovered rows, ...) must
 *   fit GIFT_NOALLOC_WORKSPACE_BYTES, and its staged tables half of that;
 *   otherwise it returns GIFT_E_NOMEM before enqueuing anything.  The
 *   benchmark workloads need at most about 1 MiB.
 *   Every call on a device shares that device's workspace and leaves its
 *   contents there; each call sets what must start at zero itself.  Calls
 *   ordered on one stream are safe; calls that overlap on one device (other
 *   streams, or host threads on different streams) race on the workspace.
 */
#define GIFT_NOALLOC_WORKSPACE_BYTES (8u << 20)
gift_status gift_seal_noalloc(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt,
                              const uint8_t* nonce_base, void* out, uint8_t* tags, hipStream_t stream);

/*
 * Open (verify + decrypt) each segment of the sealed tensor `t`.  A segment
 * whose tag does not verify -- wrong key, wrong user, wrong iv_seq, moved or
 * modified ciphertext or tag -- gets verdict AUTH_FAIL and zero bytes in
 * `out`: manipulated ownership metadata yields only a decryption failure
 * (Sec. 3, step 3).  With st->row_labels, mixed segments get OWNER_MIXED and
 * zero bytes.
 *   tags       device, n_segs*16 bytes, read.
 *   st->verdicts is required.
 * Plaintext of a failing segment may exist in `out` transiently while the
 * stream runs; it is zeroed before the call's work completes on the stream.
 */
gift_status gift_open(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt,
                      const uint8_t* nonce_base, void* out, const uint8_t* tags, hipStream_t stream);

/*
 * Owner-label check alone (Sec. 4.3, rule step 5; Sec. 3: each private byte
 * must have a single owner): verdicts[i] = OWNER_MIXED if any row of segment
 * i has labels[r] != segs[i].user, else OK.  labels: device, n_rows u32.
 * st->verdicts is required; st->row_labels is ignored.  Users are not
 * checked against a key set and iv_seq is not used.
 */
gift_status gift_check_owner(const gift_segment_table* st, const uint32_t* labels, uint64_t n_rows,
                             hipStream_t stream);

/*
 * Paged KV cache (GIFT Sec. 4.2: PagedAttention splits the cache into KV
 * blocks and ownership is recorded per block; Sec. 4.5: the monitor keeps
 * the block tables in its own memory).  The cache is one device allocation;
 * the chunk of (layer l, block id b, part p) -- p selects K/V planes when they
 * are stored apart -- is the chunk_bytes bytes at
 *     base + l*layer_stride + b*block_stride + p*part_stride.
 * Requirements (else GIFT_E_INVALID): base 16-byte aligned; chunk_bytes a
 * power of two >= 16; strides multiples of 16; n_layers, n_parts, n_blocks
 * >= 1; and the three strided dimensions do not overlap: sorted by stride,
 * each stride is at least the extent of everything inside it (the chunk,
 * then each smaller dimension times its count).  cache_bytes bounds every
 * chunk the call touches (GIFT_E_RANGE).
 */
typedef struct {
  void* base; /* device */
  uint64_t cache_bytes;
  uint64_t layer_stride, block_stride, part_stride; /* bytes */
  uint64_t chunk_bytes;
  uint32_t n_layers, n_parts;
  uint64_t n_blocks; /* block ids are < n_blocks */
} gift_paged_kv;

/* One request's KV: its block table (host, in sequence order) and owner.
 * Its sealed stream is the chunks in the order: for each block of the table,
 * for each layer, for each part -- one GCM message under the user's key and
 * IV nonce_base[user] XOR (0^32 || BE64(iv_seq)). */
typedef struct {
  const uint32_t* block_ids; /* host */
  uint32_t n_block_ids;      /* >= 1 */
  uint32_t user;
  uint64_t iv_seq;
} gift_request;

/*
 * Seal requests straight out of a paged cache into a contiguous export
 * buffer (KV handoff or swap-out): request i's ciphertext is written at
 * out + sum_{j<i} len_j, len_j = n_block_ids_j * n_layers * n_parts *
 * chunk_bytes, in caller order; tags[i] is its tag.
 *   block_labels  device, n_blocks u32, or NULL: when given, a request whose
 *                 table holds a block labelled with anyone else (including
 *                 the sentinels) is rejected -- zero ciphertext and tag,
 *                 verdict OWNER_MIXED (Sec. 4.3 rule step 5; this is the
 *                 check that stops a manipulated block table from exporting
 *                 another user's KV under the wrong key, Sec. 2.2).
 *   verdicts      device, n_reqs int32, or NULL.
 *   out           device; must not overlap the cache allocation.
 * A block id may appear only once in the whole call (GIFT_E_OVERLAP).
 */
gift_status gift_seal_paged(const gift_paged_kv* kv, const gift_request* reqs, uint32_t n_reqs,
                            const uint32_t* block_labels, gift_key_table kt, const uint8_t* nonce_base, void* out,
                            uint8_t* tags, int32_t* verdicts, hipStream_t stream);

/*
 * Open a contiguous sealed buffer (laid out as gift_seal_paged writes it)
 * into the paged cache: request i's plaintext is scattered into the chunks
 * of its block table (which may differ from the blocks it was sealed from,
 * e.g. on swap-in).  A request that fails authentication (AUTH_FAIL) has
 * every chunk of its table zeroed (its blocks passed the label check, so they
 * are its own).  A request rejected by the label check (OWNER_MIXED) writes
 * nothing into the cache: its table names a block of another owner, whose
 * contents stay as they were, so a manipulated table shows only as this
 * request's failure (Sec. 3, workflow step 3; Sec. 4.1, launch rejection).
 *   in        device, the sealed buffer; must not overlap the cache.
 *   tags      device, n_reqs*16 bytes.  verdicts: device, required.
 */
gift_status gift_open_paged(const gift_paged_kv* kv, const gift_request* reqs, uint32_t n_reqs,
                            const uint32_t* block_labels, gift_key_table kt, const uint8_t* nonce_base,
                            const void* in, const uint8_t* tags, int32_t* verdicts, hipStream_t stream);

/*
 * Per-token encryption with obfuscation (GIFT Sec. 4.5, "Token
 * encryption").  Tokens are encrypted one by one with a block cipher, not as
 * one stream, so that the untrusted framework can still append tokens and
 * split sequences; appending a random nonce keeps identical tokens from
 * giving identical ciphertexts.  For token i owned by user u (segments index
 * tokens: row r of a segment is token r):
 *     out[i] = AES-256_Ku( LE64(tokens[i]) || LE64(nonces[i]) )   (16 bytes)
 * and a token equal to eos_token is written as the reserved end-of-sequence
 * ciphertext, sixteen 0xFF bytes, whatever the key, so the framework can
 * recognise the end of generation.  Tokens covered by no segment give a zero
 * block.
 *   tokens, nonces  device, n_tokens u64 each; the nonces are the caller's
 *                   random draws (the library draws no randomness).
 *   out             device, n_tokens*16 bytes.
 *   st              segments over token indices; iv_seq, row_labels and
 *                   verdicts are not used; users must be < n_users.
 * Errors: GIFT_E_INVALID, GIFT_E_RANGE, GIFT_E_OVERLAP as for gift_seal;
 * GIFT_E_TOO_LARGE past 2^32 - 1 chunks of 64 tokens of one segment (about
 * 2^38 tokens).
 */
gift_status gift_token_encrypt(const gift_segment_table* st, const uint64_t* tokens, const uint64_t* nonces,
                               uint64_t n_tokens, gift_key_table kt, uint64_t eos_token, uint8_t* out,
                               hipStream_t stream);

/*
 * Inverse of gift_token_encrypt: the reserved all-0xFF block gives
 * eos_token (nonce 0); any other block gives the first 8 bytes of its AES-256
 * decryption under the owner's key as the token and the last 8 as the nonce
 * (the nonce is removed, Sec. 4.5).  A block cipher carries no
 * authentication: a block decrypted under the wrong key yields an unrelated
 * token, which the caller can range-check against its vocabulary.  Tokens
 * covered by no segment give 0.
 *   blocks      device, n_tokens*16 bytes.
 *   tokens_out  device, n_tokens u64; nonces_out device, n_tokens u64, or NULL.
 * Errors as for gift_token_encrypt.
 */
gift_status gift_token_decrypt(const gift_segment_table* st, const uint8_t* blocks, uint64_t n_tokens,
                               gift_key_table kt, uint64_t eos_token, uint64_t* tokens_out, uint64_t* nonces_out,
                               hipStream_t stream);

/*
 * Profiling hook for benchmark harnesses.  On the calling host thread, the
 * next gift_seal, gift_open, gift_seal_paged or gift_open_paged that
 * launches the per-block kernel records
 * `before` on its stream immediately before that launch and `after`
 * immediately after it, so hipEventElapsedTime(before, after) is that
 * kernel's duration; the hook is then cleared.  Both events must have been
 * created on the current device; NULL, NULL clears the hook.
 * Errors: GIFT_E_INVALID if exactly one event is NULL.
 */
gift_status gift_profile_next_call(hipEvent_t before, hipEvent_t after);

/* Static description of a status code. */
const char* gift_status_string(gift_status s);

/* Message of the last failing call on this host thread ("" if none). */
const char* gift_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GIFT_H */
