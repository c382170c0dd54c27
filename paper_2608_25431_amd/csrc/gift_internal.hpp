// Types shared by the host runtime (gift_host.cpp) and the kernels
// (gift_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gift.h"

namespace gift {

// Work decomposition of the per-block kernel: one workgroup per CU (its LDS
// tables fill most of the CU's 160 KiB), kThreads lanes each owning one
// 16-byte block of every kThreads-block row, kRows rows per tile.
#ifndef GIFT_THREADS
#define GIFT_THREADS 1024
#endif
#ifndef GIFT_ROWS
#define GIFT_ROWS (131072 / GIFT_THREADS)
#endif
constexpr int kThreads = GIFT_THREADS;
constexpr int kRows = GIFT_ROWS;
constexpr uint32_t kTileBlocks = (uint32_t)kThreads * kRows;  // 2 MiB per tile by default
static_assert(kThreads % 64 == 0 && kThreads <= 1024, "workgroup size");
constexpr uint32_t kSmallMaxBlocks = 64;                   // segments up to 1 KiB: one wave each
constexpr int kHPowers = kThreads + 2;                     // H^0 .. H^(kThreads+1) per user
constexpr int kHxLanes = 64;                               // H * x^(64+k), k < 64, per user
constexpr int kFinLanes = 64;                              // lanes of the per-segment finalize
// Tile end of the per-block kernel: one leader wave per SIMD folds the lane
// partials of kThreads / 64 / kLeaders waves with W = H^(64 * kLeaders).
constexpr int kLeaders = 4;
static_assert(kThreads % (64 * kLeaders) == 0, "waves per leader");

// kSegOneTile: a tiled segment of at most kTileBlocks blocks; unless its tile
// is cut into pieces, the tile kernel writes its tag (open: its verdict)
// itself and the finalize pass skips it.
enum : uint32_t { kSegAligned = 1u, kSegSmall = 2u, kSegOneTile = 4u };

// Device descriptor of one segment (64 B), built on the host.
struct SegDesc {
  uint64_t byte_off;   // first byte of the segment in the tensor
  uint64_t len;        // bytes (>= 1)
  uint64_t row_begin;  // rows, for the owner check
  uint64_t row_count;
  uint32_t iv[3];      // IV as little-endian words of its 12 bytes
  uint32_t user;
  uint32_t nblocks;    // ceil(len / 16), <= 2^32 - 2
  uint32_t flags;      // kSegAligned | kSegSmall
  uint64_t chunk0;     // paged calls: index of the segment's first chunk in the chunk table
};
static_assert(sizeof(SegDesc) == 64, "SegDesc layout");

// A byte range of `out` to zero: always (seg < 0) or when the verdict of
// segment `seg` is not OK.
struct ZeroRange {
  uint64_t off;
  uint64_t len;
  int32_t seg;
  uint32_t pad[3];
};
static_assert(sizeof(ZeroRange) == 32, "ZeroRange layout");
constexpr uint64_t kZeroPieceBytes = 4ull << 20;  // zero ranges are cut into pieces of at most this size

// Per-user key material in device memory, one allocation.
struct KeyTableDev {
  uint32_t* rk;      // [n_users][64] round-key words (60 used)
  uint32_t* dk;      // [n_users][64] equivalent-inverse-cipher round keys (60 used)
  uint32_t* h;       // [n_users][4]  H = E_K(0^128)
  uint4* gtab;       // [n_users][32][16] 4-bit GHASH tables of M = H^kThreads
  uint4* gtab_fold;  // [n_users][32][16] 4-bit GHASH tables of W = H^(64 * kLeaders)
  uint4* pow_h;      // [n_users][kHPowers] H^k
  uint4* pow_ht;     // [n_users][kFinLanes] H^(k * kTileBlocks)
  uint4* pow_hlt;    // [n_users] H^(kFinLanes * kTileBlocks)
  uint4* pow_hxl;    // [n_users][kHxLanes] H * x^(64+k): the products H * L needs
  uint4* pow_hr;     // [n_users][kRows] H^(k * kThreads): a tile piece ending k rows before its tile's end
  uint32_t n_users;
};

// One entry of the tile kernel's work queue: rows [r0, r1) of tile g (in
// tile_base numbering), which is tile t of segment s counted from the
// segment's end; user is the segment's user.  trow packs t (bits 0-15), r0
// (16-23) and r1 (24-31).  A whole tile has r0 = 0, r1 = kRows; a tile that
// the expansion kernel cuts has one entry per piece of rows instead.
struct TileEnt {
  uint32_t g, s, trow, user;
};
static_assert(sizeof(TileEnt) == 16, "TileEnt layout");
static_assert(kRows <= 255, "rows fit a byte of TileEnt::trow");
constexpr int kPieceRows = kRows / 4;  // rows of the pieces cut at the queue's tail
constexpr uint32_t kNoTile = 0xFFFFFFFFu;

// Addressing of k_gcm_tiles: contiguous tensor, or a paged cache on the
// input side (seal: gather) or the output side (open: scatter).
enum : int { kModeOpen = 1, kModeGather = 2, kModeScatter = 4 };

struct GcmArgs {
  const uint8_t* in;
  uint8_t* out;
  // paged calls: chunk c of a segment starts at pbase + chunk_off[chunk0 + c]
  // and holds 2^chunk_shift blocks
  const uint64_t* chunk_off;
  uint8_t* pbase;
  uint32_t chunk_shift;
  const SegDesc* segs;
  uint32_t n_segs;
  const uint32_t* tile_base;   // [n_segs + 1] first tile of each segment (small ones: 0 tiles)
  const uint32_t* small_list;  // [n_small] indices of small segments
  uint32_t n_tiles;
  uint32_t n_ents;             // capacity of the work queue (tiles, some cut into pieces; kNoTile after the last)
  uint32_t n_small;
  uint32_t n_multi;            // nonzero: launch the finalize pass (some segment may have more than one entry)
  uint4* partials;             // [n_tiles] GHASH partial of each tile
  const uint4* fin;            // [n_segs] E_K(J0) xor H*L of one-tile segments (from the prologue)
  const TileEnt* tile_order;   // [n_ents] tiles and pieces in the order the workgroups claim them
  const uint32_t* seg_cut;     // [n_segs] 1: a one-tile segment cut into pieces (the finalize pass forms its tag)
  uint32_t* tile_counter;      // work-queue head, zeroed with the staged tables
  int32_t* verdicts;           // [n_segs]
  uint8_t* tags_out;           // seal: [n_segs][16]
  const uint8_t* tags_in;      // open: [n_segs][16]
  KeyTableDev kt;
};

// Fixed per-device workspace of gift_seal_noalloc (gift_kernels.hip): a
// __device__ array of kStaticScratchBytes in the library's code object.
// static_scratch_setup(dev) looks up its address on device dev, which must be
// current, once (the key-table constructor calls it); static_scratch(dev)
// returns that address, or nullptr before set-up.
constexpr size_t kStaticScratchBytes = GIFT_NOALLOC_WORKSPACE_BYTES;
constexpr int kStaticScratchDevices = 64;
hipError_t static_scratch_setup(int dev);
uint8_t* static_scratch(int dev);

// Launch wrappers (gift_kernels.hip).  All enqueue on `s` and return the
// launch status.
hipError_t launch_key_setup(const uint8_t* keys_dev, KeyTableDev kt, hipStream_t s);
// Outputs of the segment-table expansion (see launch_prologue): tile_base
// [n + 1] (exclusive scan of each segment's tiles), the small-segment list,
// and the work queue of cap entries; *n_ents (device, may be NULL) gets the
// number of entries; seg_cut marks the one-tile segments whose tile it cuts.
// A tile runs on one CU, so:
// - with fewer tiles than cus, every tile of more than p = ceil(tile rows of
//   all tiles / cus) rows is cut into pieces of p rows;
// - otherwise up to cus tiles of more than kPieceRows rows, the largest
//   first (in tile order within a row count), are cut into pieces of
//   kPieceRows rows, which sort to the tail of the queue, so that the
//   workgroups, which run at slightly different speeds, finish together.
// The queue holds every whole tile and every piece, longest first, padded
// with kNoTile entries up to cap.
// The host stages one brief record per segment beside the descriptors: what
// the expansion reads of a segment (8 B instead of its 64-B descriptor).  A
// segment is small when it has at most the call's small_max blocks (0 in
// calls without a small-segment path) and one-tile when it is not small and
// has at most kTileBlocks blocks, as its descriptor's flags say.
struct SegBrief {
  uint32_t nblocks, user;
};
static_assert(sizeof(SegBrief) == 8, "SegBrief layout");
// Per-segment values of the expansion: blocks, flags, user, first tile,
// first run (runs of up to 16 tiles), cut rank of its first candidate tile.
struct SegInfo {
  uint32_t m, flags, user, tb, rb, tk;
};
struct ExpandArgs {
  uint32_t* tile_base;
  uint32_t* small_list;
  TileEnt* order;
  uint32_t cap;
  uint32_t cus;
  uint32_t* n_ents;
  SegInfo* info;      // [n] scratch, used when the call has more segments than the expansion keeps in LDS
  uint32_t* seg_cut;  // [n] out: 1 for a one-tile segment whose tile is cut (its tag comes from the finalize pass)
  uint32_t small_max;  // blocks of the largest small segment (0: the call has no small-segment path)
};
// First kernel of a call.  Copies bytes of staged tables from src (the
// mapped host ring; nullptr: they are in dst already) to dst, zeroes the
// n_zero tile partials at zero (pieces of a cut tile XOR theirs into them),
// and, when verdicts is not NULL, writes each segment's first verdict: the
// owner check against labels (indexed by row, or by the block ids at byte
// bids_off of the tables for paged calls) or OK without labels.  With a key
// table it also writes fin[s] = E_K(J0) xor H*L of every one-tile segment s.
// The descriptors sit at byte 0 of the tables.  With ex, one workgroup runs
// the segment-table expansion into *ex meanwhile, from the brief records at
// byte brief_off of the tables.
constexpr uint64_t kNoBids = ~0ull;
hipError_t launch_prologue(void* dst, const void* src, size_t bytes, uint32_t n_segs, uint64_t bids_off,
                           const uint32_t* labels, int32_t* verdicts, const KeyTableDev* kt, uint4* fin,
                           uint4* zero, uint32_t n_zero, uint64_t brief_off, const ExpandArgs* ex, hipStream_t s);
// The expansion alone, on brief records in device memory: the library's test
// hook.
hipError_t launch_expand(const SegBrief* brief, uint32_t n_segs, const ExpandArgs& x, hipStream_t s);
// Entries the work queue can hold: a tail cut adds at most
// kRows / kPieceRows - 1 entries for each of at most cus tiles; a fine cut
// (pieces of p >= all rows / cus rows) at most all rows / p <= cus entries
// beyond one per tile.
inline uint64_t queue_capacity(uint32_t n_tiles, uint32_t cus) {
  return (uint64_t)n_tiles + (uint64_t)(kRows / kPieceRows - 1) * cus;
}
hipError_t launch_gcm_tiles(const GcmArgs& a, int mode, uint32_t grid, hipStream_t s);
hipError_t launch_gcm_small(const GcmArgs& a, bool open, hipStream_t s);
hipError_t launch_gcm_finalize(const GcmArgs& a, bool open, hipStream_t s);
hipError_t launch_zero_ranges(uint8_t* out, const ZeroRange* r, uint32_t n, const int32_t* verdicts, uint32_t grid,
                              hipStream_t s);
hipError_t launch_wipe(void* p, size_t bytes, hipStream_t s);
// Paged calls: chunk offsets from the block tables (segment rows index bids).
hipError_t launch_chunk_table(const SegDesc* segs, uint32_t n_segs, const uint32_t* bids, uint32_t n_layers,
                              uint32_t n_parts, uint64_t layer_stride, uint64_t block_stride, uint64_t part_stride,
                              uint64_t* chunk_off, hipStream_t s);
// Open: zeroes the output of failed segments tile by tile -- contiguous
// (chunk_off NULL, base = out): every segment whose verdict is not OK;
// through block tables (base = the cache): requests whose verdict is
// AUTH_FAIL only (a request rejected by the label check writes nothing).
hipError_t launch_zero_failed(const SegDesc* segs, uint32_t n_segs, const uint32_t* tile_base, uint32_t n_tiles,
                              const int32_t* verdicts, const uint64_t* chunk_off, uint8_t* base, uint32_t chunk_shift,
                              uint32_t grid, hipStream_t s);
// Per-token block encryption (decrypt == true: the inverse).  Rows of the
// descriptors are token indices.
// tokens per workgroup of the token kernel (chunks never span two segments)
constexpr uint32_t kTokenChunk = 64;
hipError_t launch_tokens(const SegDesc* segs, const uint32_t* chunk_base, uint32_t n_segs, uint32_t n_chunks,
                         bool decrypt, const uint64_t* tokens, const uint64_t* nonces, const uint8_t* blocks_in,
                         uint8_t* blocks_out, uint64_t* tokens_out, uint64_t* nonces_out, uint64_t eos_token,
                         KeyTableDev kt, hipStream_t s);

}  // namespace gift
