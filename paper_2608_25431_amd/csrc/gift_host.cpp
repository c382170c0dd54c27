// Host runtime of the C ABI in include/gift.h: argument validation, IV
// derivation, segment descriptors, pinned staging, stream-ordered scratch
// and kernel launches.  Every data-dependent step runs in the kernels of
// gift_kernels.hip; this file only decides what to launch.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <deque>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "gift.h"
#include "gift_ift.h"
#include "gift_internal.hpp"

using namespace gift;

namespace gift {

namespace {

// Tile rows of tile t of a segment of m blocks.  Tiles are aligned to the
// segment's end, so only a segment's first tile can be partial; its rows
// below kRows - tile_rows hold no blocks.
uint32_t tile_rows(uint64_t m, uint32_t t) {
  const int64_t base = (int64_t)m - (int64_t)(t + 1) * (int64_t)kTileBlocks;
  return base >= 0 ? (uint32_t)kRows : (uint32_t)kRows - (uint32_t)((uint64_t)(-base) / kThreads);
}

uint32_t tiles_of(const SegDesc& d) { return (uint32_t)(((uint64_t)d.nblocks + kTileBlocks - 1) / kTileBlocks); }

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

// What the host decides for a call's launches, from per-segment counts only
// (the tile tables and the work queue are built on the device by
// launch_expand): the queue's capacity, the tile kernel's grid and whether
// the finalize pass may have work.
struct QueuePlan {
  uint64_t cap = 0;
  uint32_t grid = 0;
  bool finalize = false;
};

QueuePlan plan_queue(uint32_t n_tiles, uint64_t tile_rows_all, uint32_t n_multi, uint32_t one_rows_max, uint32_t cus) {
  QueuePlan q;
  if (n_tiles == 0 || cus == 0) return q;
  q.cap = queue_capacity(n_tiles, cus);
  // the expansion kernel's cut: with fewer tiles than CUs, tiles of more than
  // ceil(rows / cus) rows; otherwise tiles of more than kPieceRows rows at most
  const bool fine = n_tiles < cus;
  const uint64_t p = fine ? (tile_rows_all + cus - 1) / cus : (uint64_t)kPieceRows;
  const uint64_t cut_above = (fine && p >= (uint64_t)kRows) ? (uint64_t)kRows : p;
  // every entry runs at least one row, so entries <= rows; extra workgroups
  // find no entry and leave
  q.grid = fine ? (uint32_t)std::min<uint64_t>(cus, tile_rows_all) : cus;
  q.finalize = n_multi > 0 || (uint64_t)one_rows_max > cut_above;
  return q;
}

// Test hook, not part of the C ABI: runs the expansion kernel on host
// descriptors and copies its tables back (seg_cut[n], tile_base[n + 1],
// small list[n], cap queue entries and their count).  Synchronous; it
// allocates device buffers of its own.
int expand_for_test(const SegDesc* descs, uint32_t n, uint32_t cus, uint32_t* seg_cut, uint32_t* tile_base,
                    uint32_t* small_list, TileEnt* order, uint32_t cap, uint32_t* n_ents) {
  if (n == 0) return (int)hipErrorInvalidValue;
  std::vector<SegBrief> brief(n + 1);  // an even count: the kernel reads them two at a time
  for (uint32_t i = 0; i < n; i++) brief[i] = SegBrief{descs[i].nblocks, descs[i].user};
  const size_t o_tb = align_up(sizeof(SegBrief) * (n + 1)), o_sl = o_tb + align_up(4ull * (n + 1)),
               o_si = o_sl + align_up(4ull * n), o_sc = o_si + align_up(sizeof(SegInfo) * n),
               o_to = o_sc + align_up(4ull * n), o_ne = o_to + align_up(sizeof(TileEnt) * (cap ? cap : 1)),
               bytes = o_ne + 256;
  uint8_t* m = nullptr;
  hipError_t e = hipMalloc((void**)&m, bytes);
  if (e != hipSuccess) return (int)e;
  e = hipMemset(m, 0, bytes);
  if (e == hipSuccess) e = hipMemcpy(m, brief.data(), sizeof(SegBrief) * (n + 1), hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = launch_expand((const SegBrief*)m, n,
                      ExpandArgs{(uint32_t*)(m + o_tb), (uint32_t*)(m + o_sl), (TileEnt*)(m + o_to), cap, cus,
                                 (uint32_t*)(m + o_ne), (SegInfo*)(m + o_si), (uint32_t*)(m + o_sc), kSmallMaxBlocks},
                      nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(seg_cut, m + o_sc, 4ull * n, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(tile_base, m + o_tb, 4ull * (n + 1), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(small_list, m + o_sl, 4ull * n, hipMemcpyDeviceToHost);
  if (e == hipSuccess && cap) e = hipMemcpy(order, m + o_to, sizeof(TileEnt) * cap, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(n_ents, m + o_ne, 4, hipMemcpyDeviceToHost);
  hipError_t e2 = hipFree(m);
  return (int)(e != hipSuccess ? e : e2);
}

}  // namespace gift

struct gift_key_table_s {
  int device;
  uint32_t n_users;
  void* mem;
  size_t bytes;
  KeyTableDev dev;
};

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_prof_before = nullptr, g_prof_after = nullptr;

gift_status fail(gift_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

gift_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? GIFT_E_NOMEM : GIFT_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Events the library records only to learn on the host that enqueued work
// has finished with a buffer (a staging slot, a call's scratch): no timing,
// and no system-scope fence when the event completes, which would write back
// and invalidate the caches after the preceding kernel (about 6 us of idle
// queue per event); the host reads none of the results through them.
constexpr unsigned kPollEvent = hipEventDisableTiming | hipEventDisableSystemFence;

constexpr uint64_t kMaxSegBytes = ((1ull << 32) - 2) * 16ull;  // SP 800-38D Sec. 5.2.1.1
constexpr int kMaxDevices = 64;

int device_cus(int dev) {
  static std::mutex mu;
  static int cus[kMaxDevices] = {0};
  std::lock_guard<std::mutex> g(mu);
  if (dev < 0 || dev >= kMaxDevices) return 256;
  if (cus[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    // the expansion sums tile rows in 32 bits, exactly while fewer tiles
    // than CUs hold fewer than 2^20 rows: at most 8191 CUs
    cus[dev] = v < 4096 ? v : 4096;
  }
  return cus[dev];
}

// An event of the staging ring's pool and the number of times it has been
// recorded.  The ring records a pooled event again only after its previous
// recording has completed, so a holder that remembers the generation it saw
// knows, when the count has moved on, that the work it waited for is done.
struct PoolEvent {
  hipEvent_t ev = nullptr;
  std::atomic<uint64_t> gen{0};
};
// A recording of a pooled event: (event, generation), or none.
struct EventMark {
  PoolEvent* pe = nullptr;
  uint64_t gen = 0;
};

// Pinned host staging ring per device.  A call's descriptors are copied
// here and read into device scratch by the call's first kernel (a DMA copy
// would make the compute queue wait for the copy engine, ~30 us per call).
// The call enqueues all its kernels inside upload(), and one pooled event
// recorded behind the last of them guards the slot: the slot is reused only
// after that event has completed.  The same recording marks the end of the
// call's use of its scratch (ScratchLease::release), so a call puts one
// event, not two, into the queue (each costs the queue a few microseconds,
// and one between two kernels stalls the second).
class Staging {
 public:
  static constexpr size_t kCap = 8u << 20;
  static constexpr size_t kMaxStaged = kCap / 2;  // larger tables take a private synchronous path

  // Allocates the ring and a pool of kEvents events, once; the key-table
  // constructor calls it, so a call that may not allocate finds them ready.
  hipError_t prepare() {
    std::lock_guard<std::mutex> g(mu_);
    hipError_t e = ring();
    while (e == hipSuccess && n_events_ < kEvents) {
      PoolEvent* pe = nullptr;
      e = new_event(&pe);
      if (e == hipSuccess) free_ev_.push_back(pe);
    }
    return e;
  }

  // Copies bytes into the ring, then consume(src) enqueues on s the kernel
  // that reads them and the rest of the call's work: src is the copy's
  // device address, or nullptr when the bytes were DMA-copied to dst instead
  // (no device address for the ring, or a table too large for it).  The
  // pooled event recorded behind that work is returned in *mark (none for
  // empty or very large tables).  With no_alloc the call creates nothing: it
  // needs a prepared ring with a device address and at most kMaxStaged
  // bytes, and when every pooled event is in flight it waits for the oldest
  // slot and takes its event.
  template <class F>
  hipError_t upload(void* dst, const void* src, size_t bytes, hipStream_t s, F&& consume, bool no_alloc = false,
                    EventMark* mark = nullptr) {
    std::lock_guard<std::mutex> g(mu_);
    if (mark) *mark = EventMark{};
    if (bytes == 0) return consume((const void*)nullptr);
    if (no_alloc && (base_ == nullptr || dbase_ == nullptr || bytes > kMaxStaged || (bytes & 15u)))
      return hipErrorNotInitialized;
    if (bytes > kMaxStaged) {  // rare: very large tables take a private synchronous path
      void* tmp = nullptr;
      hipError_t e = hipHostMalloc(&tmp, bytes, hipHostMallocDefault);
      if (e != hipSuccess) return e;
      memcpy(tmp, src, bytes);
      e = hipMemcpyAsync(dst, tmp, bytes, hipMemcpyHostToDevice, s);
      hipError_t e2 = hipStreamSynchronize(s);
      (void)hipHostFree(tmp);
      if (e == hipSuccess) e = e2;
      return e != hipSuccess ? e : consume((const void*)nullptr);
    }
    if (base_ == nullptr) {
      hipError_t e = ring();
      if (e != hipSuccess) return e;
    }
    size_t need = (bytes + 255) & ~(size_t)255;
    if (head_ + need > kCap) head_ = 0;
    // retire finished slots oldest first, stopping at the first still in
    // flight (one query per call in the usual single-stream case); a slot in
    // flight that overlaps [head_, head_ + need) must finish first
    while (!live_.empty() && (live_.front().done || hipEventQuery(live_.front().pe->ev) == hipSuccess)) {
      free_ev_.push_back(live_.front().pe);
      live_.pop_front();
    }
    for (Slot& sl : live_)
      if (!sl.done && sl.off < head_ + need && head_ < sl.off + sl.len) {
        hipError_t e = hipEventSynchronize(sl.pe->ev);
        if (e != hipSuccess) return e;
        sl.done = true;
      }
    memcpy(base_ + head_, src, bytes);
    hipError_t e;
    if (dbase_ && !(bytes & 15u)) {
      e = consume((const void*)(dbase_ + head_));
    } else {
      e = hipMemcpyAsync(dst, base_ + head_, bytes, hipMemcpyHostToDevice, s);
      if (e == hipSuccess) e = consume((const void*)nullptr);
    }
    if (e != hipSuccess) {
      (void)hipStreamSynchronize(s);  // the slot may still be read: let it drain
      return e;
    }
    if (free_ev_.empty() && no_alloc && !live_.empty()) {
      // every pooled event is in flight: the oldest slot's event is the next free
      e = hipEventSynchronize(live_.front().pe->ev);
      if (e != hipSuccess) {
        (void)hipStreamSynchronize(s);
        return e;
      }
      free_ev_.push_back(live_.front().pe);
      live_.pop_front();
    }
    PoolEvent* pe = nullptr;
    if (!free_ev_.empty()) {
      pe = free_ev_.back();
      free_ev_.pop_back();
    } else if (no_alloc) {
      (void)hipStreamSynchronize(s);
      return hipErrorNotInitialized;
    } else {
      e = new_event(&pe);
      if (e != hipSuccess) {
        (void)hipStreamSynchronize(s);
        return e;
      }
    }
    // the generation moves on before the recording: a holder of the old one
    // sees a completed recording either way
    const uint64_t gen = pe->gen.fetch_add(1) + 1;
    e = hipEventRecord(pe->ev, s);
    if (e != hipSuccess) {
      (void)hipStreamSynchronize(s);
      free_ev_.push_back(pe);
      return e;
    }
    live_.push_back(Slot{head_, need, pe, false});
    head_ += need;
    if (mark) *mark = EventMark{pe, gen};
    return hipSuccess;
  }

 private:
  static constexpr int kEvents = 64;
  // the pinned, mapped ring and its device address (mu_ held)
  hipError_t ring() {
    if (base_ != nullptr) return hipSuccess;
    hipError_t e = hipHostMalloc((void**)&base_, kCap, hipHostMallocMapped);
    if (e != hipSuccess) {
      base_ = nullptr;
      return e;
    }
    if (hipHostGetDevicePointer((void**)&dbase_, base_, 0) != hipSuccess) dbase_ = nullptr;
    return hipSuccess;
  }
  struct Slot {
    size_t off, len;
    PoolEvent* pe;
    bool done;  // its event has completed
  };
  // a new pooled event (mu_ held, or before the ring is shared)
  hipError_t new_event(PoolEvent** out) {
    hipEvent_t ev;
    hipError_t e = hipEventCreateWithFlags(&ev, kPollEvent);
    if (e != hipSuccess) return e;
    pool_.emplace_back();
    pool_.back().ev = ev;
    n_events_++;
    *out = &pool_.back();
    return hipSuccess;
  }
  std::mutex mu_;
  uint8_t* base_ = nullptr;
  uint8_t* dbase_ = nullptr;  // base_ as the device addresses it (mapped pinned memory)
  size_t head_ = 0;
  std::deque<Slot> live_;  // in allocation order
  std::deque<PoolEvent> pool_;  // stable addresses: holders keep pointers
  std::vector<PoolEvent*> free_ev_;
  int n_events_ = 0;  // events created so far
};

Staging* staging_for(int dev) {
  static Staging st[kMaxDevices];
  return (dev >= 0 && dev < kMaxDevices) ? &st[dev] : nullptr;
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Device scratch of the calls (descriptors, tile queue, partials, ...),
// cached per (device, stream) instead of allocated and freed on every call.
// Work on one stream runs in order, so the buffer of an earlier call on the
// same stream can serve the next call at once: its first use there (the
// descriptor upload) runs behind everything the earlier call enqueued.  A
// handle does not always name one stream, though: the next stream created
// after hipStreamDestroy can get the destroyed one's handle while its work is
// still in flight, and hipStreamPerThread names a different stream in each
// thread.  So a call that takes over a buffer also makes its stream wait for
// the event recorded behind the buffer's last use (a no-op wait when that use
// was on the same stream).  A
// lease holds the entry's lock until its call has enqueued all its work, so
// two host threads on one stream cannot interleave their uses of the buffer.
// The event behind a call's last work (the call's pooled staging event,
// else the entry's own, recorded when the lease ends) guards the rare cases
// where a buffer is replaced (it is too small) or handed to another stream:
// the host waits for its last use first.  A pooled event is held with the
// generation it was recorded under: once the ring has recorded it again (for
// any stream), that use has completed and nothing waits on it.  When every entry of the device is busy on other
// streams, a call falls back to stream-ordered allocation.
struct ScratchEntry {
  std::mutex mu;
  bool bound = false;  // stream is valid
  hipStream_t stream = nullptr;
  uint8_t* ptr = nullptr;
  size_t cap = 0;
  hipEvent_t done = nullptr;   // recorded at the end of a call that staged nothing
  EventMark mark;              // else the call's staging event marks the last use of ptr
  bool recorded = false;       // done or mark marks the last use of ptr
  bool unsure = false;    // a use is not covered by done: synchronise the device first
};

constexpr int kScratchEntries = 16;

struct ScratchTable {
  std::mutex mu;
  ScratchEntry e[kScratchEntries];
};

ScratchTable* scratch_table(int dev) {
  // never destroyed: device memory outlives static destruction order
  static ScratchTable* t[kMaxDevices] = {nullptr};
  static std::mutex mu;
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> g(mu);
  if (!t[dev]) t[dev] = new ScratchTable;
  return t[dev];
}

class ScratchLease {
 public:
  ScratchLease() = default;
  ScratchLease(const ScratchLease&) = delete;
  ScratchLease& operator=(const ScratchLease&) = delete;
  ~ScratchLease() { (void)release(); }

  // A buffer of at least `bytes` for work enqueued on `s` by this call.
  hipError_t acquire(int dev, hipStream_t s, size_t bytes) {
    s_ = s;
    ScratchTable* tab = scratch_table(dev);
    if (!tab) return hipErrorInvalidDevice;
    for (int attempt = 0; attempt < 4 && !e_; attempt++) {
      ScratchEntry* mine = nullptr;
      {
        std::lock_guard<std::mutex> g(tab->mu);
        for (ScratchEntry& x : tab->e)
          if (x.bound && x.stream == s) mine = &x;
        if (!mine) {
          // an unbound entry, else one that no call holds (its stream's
          // last use must finish before the buffer changes hands)
          for (ScratchEntry& x : tab->e)
            if (!x.bound && x.mu.try_lock()) {
              e_ = &x;
              break;
            }
          for (int i = 0; i < kScratchEntries && !e_; i++)
            if (tab->e[i].mu.try_lock()) e_ = &tab->e[i];
          if (e_) {
            lk_ = std::unique_lock<std::mutex>(e_->mu, std::adopt_lock);
            e_->bound = true;
            e_->stream = s;
          }
        }
      }
      if (e_) {
        // taken over from another stream (or fresh): its last use there
        // must finish before this call's work may touch the buffer
        hipError_t w = settle(*e_);
        if (w != hipSuccess) return w;
      }
      if (mine) {
        std::unique_lock<std::mutex> l(mine->mu);
        if (mine->bound && mine->stream == s) {  // still ours after the wait
          e_ = mine;
          lk_ = std::move(l);
          // the handle may name another stream than the buffer's last use did
          hipError_t w = hipSuccess;
          if (e_->unsure) {
            w = settle(*e_);
          } else if (e_->recorded) {
            hipEvent_t ev = last_event(*e_);
            if (ev) w = hipStreamWaitEvent(s, ev, 0);
          }
          if (w != hipSuccess) return w;
        }
      } else if (!e_) {
        break;  // every entry is busy on another stream
      }
    }
    if (!e_) {
      hipError_t r = hipMallocAsync((void**)&ptr, bytes, s);
      owned_ = r == hipSuccess;
      return r;
    }
    if (e_->cap < bytes) {
      hipError_t w = settle(*e_);
      if (w != hipSuccess) return w;
      if (e_->ptr) {
        w = hipFree(e_->ptr);
        e_->ptr = nullptr;
        e_->cap = 0;
        if (w != hipSuccess) return w;
      }
      const size_t cap = std::max(bytes, (size_t)1 << 20);
      w = hipMalloc((void**)&e_->ptr, cap);
      if (w != hipSuccess) {
        e_->ptr = nullptr;
        return w;
      }
      e_->cap = cap;
    }
    if (!e_->done) {
      hipError_t w = hipEventCreateWithFlags(&e_->done, kPollEvent);
      if (w != hipSuccess) {
        e_->done = nullptr;
        return w;
      }
    }
    ptr = e_->ptr;
    return hipSuccess;
  }

  // Ends the call's use of the buffer, after its last enqueued work: marked
  // by the call's staging event (m), else by the entry's event, recorded now.
  hipError_t release(EventMark m = EventMark{}) {
    hipError_t r = hipSuccess;
    if (owned_) {
      r = hipFreeAsync(ptr, s_);
      owned_ = false;
    } else if (e_) {
      if (ptr) {
        e_->mark = m;
        if (!m.pe) r = hipEventRecord(e_->done, s_);
        e_->recorded = r == hipSuccess;
        e_->unsure = r != hipSuccess;
      }
      lk_.unlock();
      e_ = nullptr;
    }
    ptr = nullptr;
    return r;
  }

  uint8_t* ptr = nullptr;

 private:
  // waits until no enqueued work uses the entry's buffer
  static hipError_t settle(ScratchEntry& x) {
    if (x.unsure) {
      hipError_t w = hipDeviceSynchronize();
      if (w != hipSuccess) return w;
      x.unsure = false;
      x.recorded = false;
    }
    if (x.recorded) {
      hipEvent_t ev = last_event(x);
      hipError_t w = ev ? hipEventSynchronize(ev) : hipSuccess;
      if (w != hipSuccess) return w;
      x.recorded = false;
    }
    return hipSuccess;
  }

  // the event that still marks the entry's last use, or nullptr when that
  // use has certainly completed (its pooled event was recorded again since)
  static hipEvent_t last_event(const ScratchEntry& x) {
    if (!x.mark.pe) return x.done;
    return x.mark.pe->gen.load() == x.mark.gen ? x.mark.pe->ev : nullptr;
  }

  ScratchEntry* e_ = nullptr;
  std::unique_lock<std::mutex> lk_;
  hipStream_t s_ = nullptr;
  bool owned_ = false;
};



struct Plan {
  std::vector<SegDesc> descs;
  std::vector<ZeroRange> zr;  // rows no segment covers
  uint32_t n_tiles = 0;
  uint32_t n_small = 0;
  uint32_t n_multi = 0;        // segments of more than one tile
  uint64_t tile_rows = 0;      // tile rows of all tiles
  uint32_t one_rows_max = 0;   // most tile rows of a one-tile segment
};

enum class Check { kOwner, kGcm, kBlock };

// Checks segments in caller order (INVALID, RANGE, TOO_LARGE), then overlap,
// then (user, iv_seq) reuse.  kOwner (owner check): users are not
// range-checked, the GCM length limit does not apply and iv_seq is unused.
// kBlock (per-token block cipher): users are range-checked; there is no IV.
gift_status check_segments(const gift_segment* segs, uint32_t n, uint64_t n_rows, uint64_t row_bytes,
                           uint32_t n_users, Check mode) {
  const bool keys = mode != Check::kOwner, gcm = mode == Check::kGcm;
  for (uint32_t i = 0; i < n; i++) {
    const gift_segment& s = segs[i];
    if (s.row_count == 0 || s.reserved != 0)
      return fail(GIFT_E_INVALID, "segment %u: row_count must be >= 1 and reserved 0", i);
    if (s.user == GIFT_LABEL_PARAM || s.user == GIFT_LABEL_UNOWNED)
      return fail(GIFT_E_INVALID, "segment %u: user id is a label sentinel", i);
    if (s.row_begin > n_rows || s.row_count > n_rows - s.row_begin)
      return fail(GIFT_E_RANGE, "segment %u: rows [%llu, +%llu) exceed n_rows %llu", i,
                  (unsigned long long)s.row_begin, (unsigned long long)s.row_count, (unsigned long long)n_rows);
    if (keys && s.user >= n_users)
      return fail(GIFT_E_RANGE, "segment %u: user %u >= n_users %u", i, s.user, n_users);
    if (gcm && s.row_count > kMaxSegBytes / row_bytes)
      return fail(GIFT_E_TOO_LARGE, "segment %u: longer than (2^32-2)*16 bytes", i);
  }
  if (n > 1) {
    std::vector<std::pair<uint64_t, uint64_t>> v(n);
    for (uint32_t i = 0; i < n; i++) v[i] = {segs[i].row_begin, segs[i].row_count};
    // tables usually arrive in row order: sort only when they do not
    if (!std::is_sorted(v.begin(), v.end())) std::sort(v.begin(), v.end());
    for (uint32_t i = 1; i < n; i++)
      if (v[i].first < v[i - 1].first + v[i - 1].second)
        return fail(GIFT_E_OVERLAP, "segments overlap at row %llu", (unsigned long long)v[i].first);
    if (gcm) {
      // a reuse needs a user that owns two segments; with every user once
      // (a bitmap over the key set) there is nothing to sort
      bool repeat = true;  // (a key set far larger than the table: just sort)
      if ((uint64_t)n_users <= 64ull * n + 4096) {
        std::vector<uint8_t> seen(n_users, 0);
        repeat = false;
        for (uint32_t i = 0; i < n && !repeat; i++) repeat = seen[segs[i].user]++ != 0;
      }
      if (repeat) {
        for (uint32_t i = 0; i < n; i++) v[i] = {segs[i].user, segs[i].iv_seq};
        std::sort(v.begin(), v.end());
        for (uint32_t i = 1; i < n; i++)
          if (v[i] == v[i - 1])
            return fail(GIFT_E_NONCE_REUSE, "two segments share user %llu and iv_seq %llu",
                        (unsigned long long)v[i].first, (unsigned long long)v[i].second);
      }
    }
  }
  return GIFT_OK;
}

// Descriptors, zero ranges of uncovered rows, and per-segment work counts.
void build_plan(const gift_segment* segs, uint32_t n, uint64_t n_rows, uint64_t row_bytes, const uint8_t* nonce_base,
                const void* in, const void* out, Plan& P) {
  P.descs.resize(n);
  std::vector<std::pair<uint64_t, uint64_t>> cover(n);
  for (uint32_t i = 0; i < n; i++) {
    const gift_segment& s = segs[i];
    SegDesc& d = P.descs[i];
    memset(&d, 0, sizeof d);
    d.byte_off = s.row_begin * row_bytes;
    d.len = s.row_count * row_bytes;
    d.row_begin = s.row_begin;
    d.row_count = s.row_count;
    d.user = s.user;
    const uint64_t nb = (d.len + 15) / 16;
    d.nblocks = (uint32_t)nb;
    if (nonce_base) {
      uint8_t iv[12];
      memcpy(iv, nonce_base + 12ull * s.user, 12);
      for (int k = 0; k < 8; k++) iv[11 - k] ^= (uint8_t)(s.iv_seq >> (8 * k));
      for (int w = 0; w < 3; w++)
        d.iv[w] = (uint32_t)iv[4 * w] | ((uint32_t)iv[4 * w + 1] << 8) | ((uint32_t)iv[4 * w + 2] << 16) |
                  ((uint32_t)iv[4 * w + 3] << 24);
    }
    const bool aligned = ((((uintptr_t)in + d.byte_off) | ((uintptr_t)out + d.byte_off)) & 15u) == 0;
    const bool small = nb <= kSmallMaxBlocks;
    const bool one = !small && nb <= kTileBlocks;
    d.flags = (aligned ? kSegAligned : 0u) | (small ? kSegSmall : 0u) | (one ? kSegOneTile : 0u);
    if (small) {
      P.n_small++;
    } else {
      const uint32_t nt = tiles_of(d), r = tile_rows(nb, nt - 1);
      P.n_tiles += nt;
      P.tile_rows += (uint64_t)(nt - 1) * kRows + r;
      if (one) P.one_rows_max = std::max(P.one_rows_max, r);
    }
    if (!small && !one) P.n_multi++;
    cover[i] = {s.row_begin, s.row_count};
  }
  if (!std::is_sorted(cover.begin(), cover.end())) std::sort(cover.begin(), cover.end());
  uint64_t cur = 0;
  for (auto& c : cover) {
    if (c.first > cur) P.zr.push_back(ZeroRange{cur * row_bytes, (c.first - cur) * row_bytes, -1, {0, 0, 0}});
    cur = c.first + c.second;
  }
  if (cur < n_rows) P.zr.push_back(ZeroRange{cur * row_bytes, (n_rows - cur) * row_bytes, -1, {0, 0, 0}});
  // pieces of at most kZeroPieceBytes, so that one workgroup takes one piece
  std::vector<ZeroRange> pieces;
  pieces.reserve(P.zr.size());
  for (const ZeroRange& z : P.zr)
    for (uint64_t o = 0; o < z.len; o += kZeroPieceBytes)
      pieces.push_back(ZeroRange{z.off + o, std::min(kZeroPieceBytes, z.len - o), z.seg, {0, 0, 0}});
  P.zr.swap(pieces);
}

gift_status current_device(int* dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  return GIFT_OK;
}

// no_alloc: the call's scratch is the device's fixed workspace
// (static_scratch) instead of a leased buffer, and its tables go through the
// prepared staging ring; nothing is allocated or created.
template <bool OPEN>
gift_status run_gcm(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt, const uint8_t* nonce_base,
                    void* out, uint8_t* tags_out, const uint8_t* tags_in, hipStream_t stream, bool no_alloc = false) {
  g_last_error.clear();
  if (!t || !st || !kt) return fail(GIFT_E_INVALID, "null tensor, segment table or key table");
  const uint32_t n = st->n_segs;
  if (t->n_rows > 0 && (!t->data || !out)) return fail(GIFT_E_INVALID, "null data or out");
  if (n > 0 && (!st->segs || !nonce_base || (OPEN ? !tags_in : !tags_out)))
    return fail(GIFT_E_INVALID, "null segs, nonce_base or tags");
  if (OPEN && n > 0 && !st->verdicts) return fail(GIFT_E_INVALID, "gift_open needs st->verdicts");
  if (t->row_bytes == 0) return fail(GIFT_E_INVALID, "row_bytes must be >= 1");
  if (t->n_rows > UINT64_MAX / t->row_bytes) return fail(GIFT_E_INVALID, "tensor size overflows");
  const uint64_t total = t->n_rows * t->row_bytes;
  if (out != t->data && total > 0) {
    const uintptr_t a = (uintptr_t)t->data, b = (uintptr_t)out;
    if (a < b + total && b < a + total) return fail(GIFT_E_INVALID, "out partially overlaps data");
  }
  gift_status sv = check_segments(st->segs, n, t->n_rows, t->row_bytes, kt->n_users, Check::kGcm);
  if (sv != GIFT_OK) return sv;
  if (total == 0) return GIFT_OK;

  // the profiling hook applies to this call only
  hipEvent_t prof_before = g_prof_before, prof_after = g_prof_after;
  g_prof_before = g_prof_after = nullptr;
  int dev;
  if ((sv = current_device(&dev)) != GIFT_OK) return sv;
  if (dev != kt->device) return fail(GIFT_E_INVALID, "key table belongs to device %d, current is %d", kt->device, dev);

  Plan P;
  build_plan(st->segs, n, t->n_rows, t->row_bytes, nonce_base, t->data, out, P);
  const uint32_t cus = (uint32_t)device_cus(dev);
  const QueuePlan Q = plan_queue(P.n_tiles, P.tile_rows, P.n_multi, P.one_rows_max, cus);

  // scratch: the staged tables (descs | brief records | zero ranges | queue
  // head), then what the device builds and fills (tile_base | small list |
  // segment values | cut marks | work queue | partials | verdicts | one-tile tag masks)
  const size_t o_desc = 0;
  const size_t o_br = o_desc + align256(sizeof(SegDesc) * n);
  const size_t o_zr = o_br + align256(sizeof(SegBrief) * (n + 1));
  const size_t o_qh = o_zr + align256(sizeof(ZeroRange) * P.zr.size());
  const size_t o_st = o_qh + 256;  // end of the staged tables
  const size_t o_tb = o_st;
  const size_t o_sl = o_tb + align256(4ull * (n + 1));
  const size_t o_si = o_sl + align256(4ull * (n ? n : 1));
  const size_t o_sc = o_si + align256(sizeof(SegInfo) * (n ? n : 1));
  const size_t o_to = o_sc + align256(4ull * (n ? n : 1));
  const size_t o_pt = o_to + align256(sizeof(TileEnt) * (Q.cap ? Q.cap : 1));
  const size_t o_vd = o_pt + align256(16ull * (P.n_tiles ? P.n_tiles : 1));
  const size_t o_fn = o_vd + align256(4ull * (n ? n : 1));
  const size_t bytes = o_fn + align256(16ull * (n ? n : 1));
  ScratchLease lease;
  uint8_t* scratch = nullptr;
  hipError_t e = hipSuccess;
  if (no_alloc) {
    if (bytes > kStaticScratchBytes || o_st > Staging::kMaxStaged)
      return fail(GIFT_E_NOMEM,
                  "gift_seal_noalloc: the call needs %zu bytes of workspace (%zu of them staged tables); the fixed "
                  "workspace holds %zu (%zu staged)",
                  bytes, o_st, kStaticScratchBytes, Staging::kMaxStaged);
    scratch = static_scratch(dev);
    if (!scratch) return fail(GIFT_E_INVALID, "gift_seal_noalloc: no workspace on device %d (create a key table there first)", dev);
  } else {
    e = lease.acquire(dev, stream, bytes);
    if (e != hipSuccess) return hip_fail(e, "device scratch");
    scratch = lease.ptr;
  }

  std::vector<uint8_t> host(o_st);  // zero-filled: the queue head starts at 0
  if (n) memcpy(host.data() + o_desc, P.descs.data(), sizeof(SegDesc) * n);
  {
    SegBrief* br = (SegBrief*)(host.data() + o_br);
    for (uint32_t i = 0; i < n; i++) br[i] = SegBrief{P.descs[i].nblocks, P.descs[i].user};
  }
  if (!P.zr.empty()) memcpy(host.data() + o_zr, P.zr.data(), sizeof(ZeroRange) * P.zr.size());
  int32_t* verdicts = st->verdicts ? st->verdicts : (int32_t*)(scratch + o_vd);
  Staging* sg = staging_for(dev);
  if (!sg) return fail(GIFT_E_INVALID, "device index %d unsupported", dev);
  // the prologue copies the tables, settles the verdicts (owner check),
  // zeroes the tile partials (pieces of a cut tile XOR theirs into them) and
  // expands the segment table on the device
  const ExpandArgs ex{(uint32_t*)(scratch + o_tb), (uint32_t*)(scratch + o_sl), (TileEnt*)(scratch + o_to),
                      (uint32_t)Q.cap, cus, nullptr, (SegInfo*)(scratch + o_si), (uint32_t*)(scratch + o_sc),
                      kSmallMaxBlocks};
  const SegDesc* d_desc = (const SegDesc*)(scratch + o_desc);
  gift_status rs = GIFT_OK;
  EventMark call_ev;  // the event recorded behind the call's last kernel
  // the call's kernels after the prologue, enqueued while the staging slot is
  // held, so that the one event behind the last of them frees the slot (an
  // event between two kernels costs the queue several microseconds)
  auto rest = [&]() -> hipError_t {
    if (n > 0) {
      GcmArgs a{};  // zero-initialised: no field is left undefined
      a.in = (const uint8_t*)t->data;
      a.out = (uint8_t*)out;
      a.chunk_off = nullptr;
      a.pbase = nullptr;
      a.chunk_shift = 0;
      a.segs = d_desc;
      a.n_segs = n;
      a.tile_base = (const uint32_t*)(scratch + o_tb);
      a.small_list = (const uint32_t*)(scratch + o_sl);
      a.n_tiles = P.n_tiles;
      a.n_ents = (uint32_t)Q.cap;
      a.n_small = P.n_small;
      a.n_multi = Q.finalize ? 1u : 0u;
      a.partials = (uint4*)(scratch + o_pt);
      a.fin = (const uint4*)(scratch + o_fn);
      a.tile_order = (const TileEnt*)(scratch + o_to);
      a.seg_cut = (const uint32_t*)(scratch + o_sc);
      a.tile_counter = (uint32_t*)(scratch + o_qh);
      a.verdicts = verdicts;
      a.tags_out = tags_out;
      a.tags_in = tags_in;
      a.kt = kt->dev;
      if (prof_before && P.n_tiles > 0) {
        e = hipEventRecord(prof_before, stream);
        if (e != hipSuccess) {
          rs = hip_fail(e, "profiling event");
          return e;
        }
      }
      e = launch_gcm_tiles(a, OPEN ? kModeOpen : 0, Q.grid, stream);
      if (e != hipSuccess) {
        rs = hip_fail(e, "gcm launch");
        return e;
      }
      if (prof_after && P.n_tiles > 0) {
        e = hipEventRecord(prof_after, stream);
        if (e != hipSuccess) {
          rs = hip_fail(e, "profiling event");
          return e;
        }
      }
      e = launch_gcm_small(a, OPEN, stream);
      if (e == hipSuccess) e = launch_gcm_finalize(a, OPEN, stream);
      // open: segments that failed are zeroed after their verdicts are known;
      // without a finalize pass every verdict came from a kernel that zeroed
      // its own failed segments (the small-segment kernel, or the tile kernel
      // for an uncut one-tile segment)
      if (e == hipSuccess && OPEN && Q.finalize)
        e = launch_zero_failed(d_desc, n, a.tile_base, P.n_tiles, verdicts, nullptr, (uint8_t*)out, 0u, cus * 4u,
                               stream);
      if (e != hipSuccess) {
        rs = hip_fail(e, "gcm launch");
        return e;
      }
    }
    if (!P.zr.empty()) {
      e = launch_zero_ranges((uint8_t*)out, (const ZeroRange*)(scratch + o_zr), (uint32_t)P.zr.size(), verdicts,
                             (uint32_t)device_cus(dev) * 4u, stream);
      if (e != hipSuccess) {
        rs = hip_fail(e, "zero-fill launch");
        return e;
      }
    }
    return hipSuccess;
  };
  e = sg->upload(
      scratch, host.data(), o_st, stream,
      [&](const void* src) {
        hipError_t r = launch_prologue(scratch, src, o_st, n, kNoBids, st->row_labels, n ? verdicts : nullptr,
                                       &kt->dev, (uint4*)(scratch + o_fn), (uint4*)(scratch + o_pt), P.n_tiles, o_br,
                                       n ? &ex : nullptr, stream);
        if (r != hipSuccess) {
          rs = hip_fail(r, "prologue launch");
          return r;
        }
        return rest();
      },
      no_alloc, &call_ev);
  if (e != hipSuccess && rs == GIFT_OK) rs = hip_fail(e, "staging upload");
  e = lease.release(call_ev);
  if (rs == GIFT_OK && e != hipSuccess) rs = hip_fail(e, "device scratch release");
  return rs;
}

// ---------------------------------------------------------------------------
// Paged KV calls.
// ---------------------------------------------------------------------------
bool mul_ok(uint64_t a, uint64_t b, uint64_t* r) { return !__builtin_mul_overflow(a, b, r); }
bool add_ok(uint64_t a, uint64_t b, uint64_t* r) { return !__builtin_add_overflow(a, b, r); }

// Geometry rules of gift_paged_kv (see gift.h).
gift_status check_paged_geometry(const gift_paged_kv* kv) {
  const uint64_t cb = kv->chunk_bytes;
  if (!kv->base || ((uintptr_t)kv->base & 15u)) return fail(GIFT_E_INVALID, "paged: base null or not 16-byte aligned");
  if (cb < 16 || (cb & (cb - 1))) return fail(GIFT_E_INVALID, "paged: chunk_bytes must be a power of two >= 16");
  if ((kv->layer_stride | kv->block_stride | kv->part_stride) & 15u)
    return fail(GIFT_E_INVALID, "paged: strides must be multiples of 16");
  if (kv->n_layers == 0 || kv->n_parts == 0 || kv->n_blocks == 0)
    return fail(GIFT_E_INVALID, "paged: n_layers, n_parts and n_blocks must be >= 1");
  struct Dim {
    uint64_t stride, count;
  } dims[3] = {{kv->layer_stride, kv->n_layers}, {kv->block_stride, kv->n_blocks}, {kv->part_stride, kv->n_parts}};
  std::sort(dims, dims + 3, [](const Dim& x, const Dim& y) { return x.stride < y.stride; });
  uint64_t extent = cb;
  for (const Dim& d : dims) {
    if (d.count <= 1) continue;
    uint64_t span;
    if (d.stride < extent || !mul_ok(d.stride, d.count - 1, &span) || !add_ok(span, extent, &extent))
      return fail(GIFT_E_INVALID, "paged: strided dimensions overlap");
  }
  return GIFT_OK;
}

template <bool OPEN>
gift_status run_paged(const gift_paged_kv* kv, const gift_request* reqs, uint32_t n, const uint32_t* labels,
                      gift_key_table kt, const uint8_t* nonce_base, const void* in, void* out, uint8_t* tags_out,
                      const uint8_t* tags_in, int32_t* verdicts_user, hipStream_t stream) {
  g_last_error.clear();
  if (!kv || !kt) return fail(GIFT_E_INVALID, "null cache description or key table");
  if (n > 0 && (!reqs || !nonce_base || (OPEN ? (!in || !tags_in || !verdicts_user) : (!out || !tags_out))))
    return fail(GIFT_E_INVALID, "null requests, nonce_base, buffer, tags or verdicts");
  gift_status sv = check_paged_geometry(kv);
  if (sv != GIFT_OK) return sv;
  const uint64_t per_block_chunks = (uint64_t)kv->n_layers * kv->n_parts;
  uint64_t per_block_bytes;
  if (!mul_ok(per_block_chunks, kv->chunk_bytes, &per_block_bytes)) return fail(GIFT_E_INVALID, "paged: sizes overflow");
  // fixed part of the farthest chunk: last layer and part
  uint64_t fixed = kv->chunk_bytes, t1, t2;
  if (!mul_ok(kv->layer_stride, kv->n_layers - 1, &t1) || !mul_ok(kv->part_stride, kv->n_parts - 1, &t2) ||
      !add_ok(fixed, t1, &fixed) || !add_ok(fixed, t2, &fixed))
    return fail(GIFT_E_RANGE, "paged: chunks exceed the cache");
  uint64_t total_bytes = 0, total_bids = 0;
  for (uint32_t i = 0; i < n; i++) {
    const gift_request& r = reqs[i];
    if (r.n_block_ids == 0 || !r.block_ids) return fail(GIFT_E_INVALID, "request %u: empty block table", i);
    if (r.user == GIFT_LABEL_PARAM || r.user == GIFT_LABEL_UNOWNED)
      return fail(GIFT_E_INVALID, "request %u: user id is a label sentinel", i);
    uint32_t maxb = 0;
    for (uint32_t j = 0; j < r.n_block_ids; j++) maxb = r.block_ids[j] > maxb ? r.block_ids[j] : maxb;
    if (maxb >= kv->n_blocks) return fail(GIFT_E_RANGE, "request %u: block id %u >= n_blocks", i, maxb);
    if (r.user >= kt->n_users) return fail(GIFT_E_RANGE, "request %u: user %u >= n_users", i, r.user);
    uint64_t far;
    if (!mul_ok(kv->block_stride, maxb, &far) || !add_ok(far, fixed, &far) || far > kv->cache_bytes)
      return fail(GIFT_E_RANGE, "request %u: chunks exceed cache_bytes", i);
    uint64_t len;
    if (!mul_ok(per_block_bytes, r.n_block_ids, &len) || len > kMaxSegBytes)
      return fail(GIFT_E_TOO_LARGE, "request %u: longer than (2^32-2)*16 bytes", i);
    if (!add_ok(total_bytes, len, &total_bytes)) return fail(GIFT_E_INVALID, "paged: sizes overflow");
    total_bids += r.n_block_ids;
  }
  {
    std::vector<uint32_t> all;
    all.reserve(total_bids);
    for (uint32_t i = 0; i < n; i++) all.insert(all.end(), reqs[i].block_ids, reqs[i].block_ids + reqs[i].n_block_ids);
    std::sort(all.begin(), all.end());
    for (size_t j = 1; j < all.size(); j++)
      if (all[j] == all[j - 1]) return fail(GIFT_E_OVERLAP, "block id %u appears twice", all[j]);
    std::vector<std::pair<uint64_t, uint64_t>> v(n);
    for (uint32_t i = 0; i < n; i++) v[i] = {reqs[i].user, reqs[i].iv_seq};
    std::sort(v.begin(), v.end());
    for (uint32_t i = 1; i < n; i++)
      if (v[i] == v[i - 1])
        return fail(GIFT_E_NONCE_REUSE, "two requests share user %llu and iv_seq %llu", (unsigned long long)v[i].first,
                    (unsigned long long)v[i].second);
  }
  const void* flat = OPEN ? in : out;
  if (total_bytes > 0) {
    const uintptr_t a0 = (uintptr_t)kv->base, b0 = (uintptr_t)flat;
    if (a0 < b0 + total_bytes && b0 < a0 + kv->cache_bytes)
      return fail(GIFT_E_INVALID, "the contiguous buffer overlaps the cache allocation");
    if (b0 & 15u) return fail(GIFT_E_INVALID, "the contiguous buffer must be 16-byte aligned");
  }
  if (n == 0) return GIFT_OK;
  int dev;
  if ((sv = current_device(&dev)) != GIFT_OK) return sv;
  if (dev != kt->device) return fail(GIFT_E_INVALID, "key table belongs to device %d, current is %d", kt->device, dev);

  // descriptors: rows = positions in the uploaded block-id array
  std::vector<SegDesc> descs(n);
  uint64_t boff = 0, bpos = 0, cpos = 0;
  uint32_t n_tiles = 0, n_multi = 0, one_rows_max = 0;
  uint64_t tile_rows_all = 0;
  for (uint32_t i = 0; i < n; i++) {
    const gift_request& r = reqs[i];
    SegDesc& d = descs[i];
    memset(&d, 0, sizeof d);
    d.byte_off = boff;
    d.len = per_block_bytes * r.n_block_ids;
    d.row_begin = bpos;
    d.row_count = r.n_block_ids;
    d.user = r.user;
    d.nblocks = (uint32_t)(d.len / 16);
    d.flags = kSegAligned | (d.nblocks <= kTileBlocks ? kSegOneTile : 0u);
    if (d.nblocks > kTileBlocks) n_multi++;
    d.chunk0 = cpos;
    uint8_t iv[12];
    memcpy(iv, nonce_base + 12ull * r.user, 12);
    for (int k = 0; k < 8; k++) iv[11 - k] ^= (uint8_t)(r.iv_seq >> (8 * k));
    for (int w = 0; w < 3; w++)
      d.iv[w] = (uint32_t)iv[4 * w] | ((uint32_t)iv[4 * w + 1] << 8) | ((uint32_t)iv[4 * w + 2] << 16) |
                ((uint32_t)iv[4 * w + 3] << 24);
    const uint32_t nt = tiles_of(d), rows = tile_rows(d.nblocks, nt - 1);
    n_tiles += nt;
    tile_rows_all += (uint64_t)(nt - 1) * kRows + rows;
    if (nt == 1) one_rows_max = std::max(one_rows_max, rows);
    boff += d.len;
    bpos += r.n_block_ids;
    cpos += per_block_chunks * r.n_block_ids;
  }
  uint32_t shift = 0;
  while ((16ull << shift) < kv->chunk_bytes) shift++;
  const uint32_t cus = (uint32_t)device_cus(dev);
  const QueuePlan Q = plan_queue(n_tiles, tile_rows_all, n_multi, one_rows_max, cus);

  // scratch: the staged tables (descs | brief records | block ids | queue
  // head), then what the device builds and fills (tile_base | small list |
  // segment values | cut marks | work queue | partials | verdicts | chunk offsets | one-tile tag masks)
  const size_t o_desc = 0;
  const size_t o_br = o_desc + align256(sizeof(SegDesc) * n);
  const size_t o_bid = o_br + align256(sizeof(SegBrief) * (n + 1));
  const size_t o_qh = o_bid + align256(4ull * total_bids);
  const size_t o_st = o_qh + 256;  // end of the staged tables
  const size_t o_tb = o_st;
  const size_t o_sl = o_tb + align256(4ull * (n + 1));
  const size_t o_si = o_sl + align256(4ull * n);
  const size_t o_sc = o_si + align256(sizeof(SegInfo) * n);
  const size_t o_to = o_sc + align256(4ull * n);
  const size_t o_pt = o_to + align256(sizeof(TileEnt) * (Q.cap ? Q.cap : 1));
  const size_t o_vd = o_pt + align256(16ull * (n_tiles ? n_tiles : 1));
  const size_t o_ck = o_vd + align256(4ull * n);
  const size_t o_fn = o_ck + align256(8ull * cpos);
  const size_t bytes = o_fn + align256(16ull * (n ? n : 1));
  ScratchLease lease;
  hipError_t e = lease.acquire(dev, stream, bytes);
  if (e != hipSuccess) return hip_fail(e, "device scratch");
  uint8_t* scratch = lease.ptr;
  std::vector<uint8_t> host(o_st);  // zero-filled: the queue head starts at 0
  memcpy(host.data() + o_desc, descs.data(), sizeof(SegDesc) * n);
  {
    SegBrief* br = (SegBrief*)(host.data() + o_br);
    for (uint32_t i = 0; i < n; i++) br[i] = SegBrief{descs[i].nblocks, descs[i].user};
  }
  {
    uint32_t* bp = (uint32_t*)(host.data() + o_bid);
    for (uint32_t i = 0; i < n; i++) {
      memcpy(bp, reqs[i].block_ids, 4ull * reqs[i].n_block_ids);
      bp += reqs[i].n_block_ids;
    }
  }
  int32_t* verdicts = verdicts_user ? verdicts_user : (int32_t*)(scratch + o_vd);
  Staging* sg = staging_for(dev);
  // the prologue copies the tables, settles the verdicts (owner check by
  // block id), zeroes the tile partials and expands the segment table
  const ExpandArgs ex{(uint32_t*)(scratch + o_tb), (uint32_t*)(scratch + o_sl), (TileEnt*)(scratch + o_to),
                      (uint32_t)Q.cap, cus, nullptr, (SegInfo*)(scratch + o_si), (uint32_t*)(scratch + o_sc), 0u};
  gift_status rs = GIFT_OK;
  EventMark call_ev;  // the event recorded behind the call's last kernel
  const SegDesc* d_desc = (const SegDesc*)(scratch + o_desc);
  const uint32_t* d_bid = (const uint32_t*)(scratch + o_bid);
  uint64_t* d_ck = (uint64_t*)(scratch + o_ck);
  // the call's kernels after the prologue, enqueued while the staging slot is
  // held (one event behind the last of them frees the slot)
  auto rest = [&]() -> hipError_t {
    e = launch_chunk_table(d_desc, n, d_bid, kv->n_layers, kv->n_parts, kv->layer_stride, kv->block_stride,
                           kv->part_stride, d_ck, stream);
    if (e != hipSuccess) {
      rs = hip_fail(e, "paged expansion");
      return e;
    }
    GcmArgs a{};  // zero-initialised: no field is left undefined
    a.in = (const uint8_t*)in;
    a.out = (uint8_t*)out;
    a.chunk_off = d_ck;
    a.pbase = (uint8_t*)kv->base;
    a.chunk_shift = shift;
    a.segs = d_desc;
    a.n_segs = n;
    a.tile_base = (const uint32_t*)(scratch + o_tb);
    a.small_list = (const uint32_t*)(scratch + o_sl);
    a.n_tiles = n_tiles;
    a.n_ents = (uint32_t)Q.cap;
    a.n_multi = Q.finalize ? 1u : 0u;
    a.n_small = 0;
    a.partials = (uint4*)(scratch + o_pt);
    a.fin = (const uint4*)(scratch + o_fn);
    a.tile_order = (const TileEnt*)(scratch + o_to);
    a.seg_cut = (const uint32_t*)(scratch + o_sc);
    a.tile_counter = (uint32_t*)(scratch + o_qh);
    a.verdicts = verdicts;
    a.tags_out = tags_out;
    a.tags_in = tags_in;
    a.kt = kt->dev;
    if (g_prof_before) {
      e = hipEventRecord(g_prof_before, stream);
      if (e != hipSuccess) {
        rs = hip_fail(e, "profiling event");
        return e;
      }
    }
    e = launch_gcm_tiles(a, OPEN ? (kModeOpen | kModeScatter) : kModeGather, Q.grid, stream);
    if (e == hipSuccess && g_prof_after) e = hipEventRecord(g_prof_after, stream);
    if (e == hipSuccess) e = launch_gcm_finalize(a, OPEN, stream);
    if (e == hipSuccess && OPEN)
      e = launch_zero_failed(d_desc, n, (const uint32_t*)(scratch + o_tb), n_tiles, verdicts, d_ck,
                             (uint8_t*)kv->base, shift, cus * 4u, stream);
    if (e != hipSuccess) {
      rs = hip_fail(e, "paged gcm launch");
      return e;
    }
    return hipSuccess;
  };
  e = sg ? sg->upload(scratch, host.data(), o_st, stream,
                      [&](const void* src) {
                        hipError_t r = launch_prologue(scratch, src, o_st, n, o_bid, labels, verdicts, &kt->dev,
                                                       (uint4*)(scratch + o_fn), (uint4*)(scratch + o_pt), n_tiles,
                                                       o_br, &ex, stream);
                        if (r != hipSuccess) {
                          rs = hip_fail(r, "prologue launch");
                          return r;
                        }
                        return rest();
                      },
                      false, &call_ev)
         : hipErrorInvalidDevice;
  if (e != hipSuccess && rs == GIFT_OK) rs = hip_fail(e, "staging upload");
  g_prof_before = g_prof_after = nullptr;
  e = lease.release(call_ev);
  if (rs == GIFT_OK && e != hipSuccess) rs = hip_fail(e, "device scratch release");
  return rs;
}

}  // namespace

extern "C" {

gift_status gift_seal_paged(const gift_paged_kv* kv, const gift_request* reqs, uint32_t n_reqs,
                            const uint32_t* block_labels, gift_key_table kt, const uint8_t* nonce_base, void* out,
                            uint8_t* tags, int32_t* verdicts, hipStream_t stream) {
  return run_paged<false>(kv, reqs, n_reqs, block_labels, kt, nonce_base, nullptr, out, tags, nullptr, verdicts,
                          stream);
}

gift_status gift_open_paged(const gift_paged_kv* kv, const gift_request* reqs, uint32_t n_reqs,
                            const uint32_t* block_labels, gift_key_table kt, const uint8_t* nonce_base,
                            const void* in, const uint8_t* tags, int32_t* verdicts, hipStream_t stream) {
  return run_paged<true>(kv, reqs, n_reqs, block_labels, kt, nonce_base, in, nullptr, nullptr, tags, verdicts, stream);
}


const char* gift_status_string(gift_status s) {
  switch (s) {
    case GIFT_OK: return "ok";
    case GIFT_E_INVALID: return "invalid argument";
    case GIFT_E_RANGE: return "segment or user out of range";
    case GIFT_E_OVERLAP: return "segments overlap";
    case GIFT_E_NONCE_REUSE: return "(user, iv_seq) reused within the call";
    case GIFT_E_TOO_LARGE: return "segment exceeds the GCM length limit";
    case GIFT_E_HIP: return "HIP runtime error";
    case GIFT_E_NOMEM: return "out of memory";
    case GIFT_E_REJECTED: return "IFT rule rejected the kernel launch";
    case GIFT_E_RACE: return "launch races with an unfinished kernel on another stream";
  }
  return "unknown status";
}

const char* gift_last_error(void) { return g_last_error.c_str(); }

uint32_t gift_key_table_users(gift_key_table kt) { return kt ? kt->n_users : 0u; }

gift_status gift_profile_next_call(hipEvent_t before, hipEvent_t after) {
  if ((before == nullptr) != (after == nullptr)) return fail(GIFT_E_INVALID, "pass both events or neither");
  g_prof_before = before;
  g_prof_after = after;
  return GIFT_OK;
}

gift_status gift_key_table_create(const uint8_t* keys, uint32_t n_users, hipStream_t stream, gift_key_table* out) {
  g_last_error.clear();
  if (!keys || !out) return fail(GIFT_E_INVALID, "null keys or out");
  if (n_users == 0 || n_users >= GIFT_LABEL_PARAM) return fail(GIFT_E_INVALID, "n_users out of range");
  *out = nullptr;
  int dev;
  gift_status sv = current_device(&dev);
  if (sv != GIFT_OK) return sv;
  const uint64_t u = n_users;
  const size_t o_rk = 0;
  const size_t o_dk = o_rk + align256(u * 64 * 4);
  const size_t o_h = o_dk + align256(u * 64 * 4);
  const size_t o_gt = o_h + align256(u * 16);
  const size_t o_gf = o_gt + align256(u * 512 * 16);
  const size_t o_ph = o_gf + align256(u * 512 * 16);
  const size_t o_pt = o_ph + align256(u * kHPowers * 16);
  const size_t o_pl = o_pt + align256(u * kFinLanes * 16);
  const size_t o_px = o_pl + align256(u * 16);
  const size_t o_pr = o_px + align256(u * kHxLanes * 16);
  const size_t bytes = o_pr + align256(u * kRows * 16);
  uint8_t* mem = nullptr;
  hipError_t e = hipMalloc((void**)&mem, bytes);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(key table)");
  uint8_t* kdev = nullptr;
  e = hipMalloc((void**)&kdev, 32ull * u);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return hip_fail(e, "hipMalloc(keys)");
  }
  gift_key_table kt = new gift_key_table_s;
  kt->device = dev;
  kt->n_users = n_users;
  kt->mem = mem;
  kt->bytes = bytes;
  kt->dev.rk = (uint32_t*)(mem + o_rk);
  kt->dev.dk = (uint32_t*)(mem + o_dk);
  kt->dev.h = (uint32_t*)(mem + o_h);
  kt->dev.gtab = (uint4*)(mem + o_gt);
  kt->dev.gtab_fold = (uint4*)(mem + o_gf);
  kt->dev.pow_h = (uint4*)(mem + o_ph);
  kt->dev.pow_ht = (uint4*)(mem + o_pt);
  kt->dev.pow_hlt = (uint4*)(mem + o_pl);
  kt->dev.pow_hxl = (uint4*)(mem + o_px);
  kt->dev.pow_hr = (uint4*)(mem + o_pr);
  kt->dev.n_users = n_users;
  // The copy reads the caller's buffer; synchronising before return means no
  // copy of the keys outlives the call on the host side of the library.
  e = hipMemcpyAsync(kdev, keys, 32ull * u, hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = launch_key_setup(kdev, kt->dev, stream);
  if (e == hipSuccess) e = launch_wipe(kdev, 32ull * u, stream);
  hipError_t e2 = hipStreamSynchronize(stream);
  (void)hipFree(kdev);
  if (e == hipSuccess) e = e2;
  // set-up of this device for gift_seal_noalloc: the fixed workspace's
  // address and the staging ring with its event pool
  if (e == hipSuccess) e = static_scratch_setup(dev);
  if (e == hipSuccess) {
    Staging* sg = staging_for(dev);
    e = sg ? sg->prepare() : hipErrorInvalidDevice;
  }
  if (e != hipSuccess) {
    (void)hipFree(mem);
    delete kt;
    return hip_fail(e, "key table setup");
  }
  *out = kt;
  return GIFT_OK;
}

gift_status gift_key_table_destroy(gift_key_table kt) {
  g_last_error.clear();
  if (!kt) return GIFT_OK;
  int prev = -1;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(kt->device);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemset(kt->mem, 0, kt->bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  hipError_t e2 = hipFree(kt->mem);
  if (prev >= 0) (void)hipSetDevice(prev);
  delete kt;
  if (e != hipSuccess) return hip_fail(e, "key table wipe");
  if (e2 != hipSuccess) return hip_fail(e2, "key table free");
  return GIFT_OK;
}

gift_status gift_seal(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt, const uint8_t* nonce_base,
                      void* out, uint8_t* tags, hipStream_t stream) {
  return run_gcm<false>(t, st, kt, nonce_base, out, tags, nullptr, stream);
}

gift_status gift_seal_noalloc(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt,
                              const uint8_t* nonce_base, void* out, uint8_t* tags, hipStream_t stream) {
  return run_gcm<false>(t, st, kt, nonce_base, out, tags, nullptr, stream, true);
}

gift_status gift_open(const gift_tensor* t, const gift_segment_table* st, gift_key_table kt, const uint8_t* nonce_base,
                      void* out, const uint8_t* tags, hipStream_t stream) {
  return run_gcm<true>(t, st, kt, nonce_base, out, nullptr, tags, stream);
}

gift_status gift_check_owner(const gift_segment_table* st, const uint32_t* labels, uint64_t n_rows,
                             hipStream_t stream) {
  g_last_error.clear();
  if (!st || !labels) return fail(GIFT_E_INVALID, "null segment table or labels");
  const uint32_t n = st->n_segs;
  if (n > 0 && (!st->segs || !st->verdicts)) return fail(GIFT_E_INVALID, "null segs or verdicts");
  gift_status sv = check_segments(st->segs, n, n_rows, 1, 0, Check::kOwner);
  if (sv != GIFT_OK) return sv;
  if (n == 0) return GIFT_OK;
  int dev;
  if ((sv = current_device(&dev)) != GIFT_OK) return sv;
  Plan P;
  build_plan(st->segs, n, n_rows, 1, nullptr, nullptr, nullptr, P);
  const size_t bytes = sizeof(SegDesc) * n;
  ScratchLease lease;
  hipError_t e = lease.acquire(dev, stream, bytes);
  if (e != hipSuccess) return hip_fail(e, "device scratch");
  SegDesc* d = (SegDesc*)lease.ptr;
  Staging* sg = staging_for(dev);
  EventMark call_ev;  // the event recorded behind the prologue
  e = sg ? sg->upload(d, P.descs.data(), bytes, stream,
                      [&](const void* src) {
                        return launch_prologue(d, src, bytes, n, kNoBids, labels, st->verdicts, nullptr, nullptr,
                                               nullptr, 0u, 0u, nullptr, stream);
                      },
                      false, &call_ev)
         : hipErrorInvalidDevice;
  hipError_t e2 = lease.release(call_ev);
  if (e != hipSuccess) return hip_fail(e, "check_owner");
  if (e2 != hipSuccess) return hip_fail(e2, "device scratch release");
  return GIFT_OK;
}

// Per-token encryption (GIFT Sec. 4.5), both directions.
static gift_status run_tokens(bool decrypt, const gift_segment_table* st, uint64_t n_tokens, gift_key_table kt,
                              uint64_t eos_token, const uint64_t* tokens, const uint64_t* nonces,
                              const uint8_t* blocks_in, uint8_t* blocks_out, uint64_t* tokens_out,
                              uint64_t* nonces_out, hipStream_t stream) {
  g_last_error.clear();
  if (!st || !kt) return fail(GIFT_E_INVALID, "null segment table or key table");
  const uint32_t n = st->n_segs;
  if (n > 0 && !st->segs) return fail(GIFT_E_INVALID, "null segs");
  if (n_tokens > 0 && (decrypt ? (!blocks_in || !tokens_out) : (!tokens || !nonces || !blocks_out)))
    return fail(GIFT_E_INVALID, "null token buffers");
  if (n_tokens > UINT64_MAX / 16) return fail(GIFT_E_INVALID, "token count overflows");
  gift_status sv = check_segments(st->segs, n, n_tokens, 1, kt->n_users, Check::kBlock);
  if (sv != GIFT_OK) return sv;
  if (n_tokens == 0) return GIFT_OK;
  int dev;
  if ((sv = current_device(&dev)) != GIFT_OK) return sv;
  if (dev != kt->device) return fail(GIFT_E_INVALID, "key table belongs to device %d, current is %d", kt->device, dev);
  Plan P;
  build_plan(st->segs, n, n_tokens, 1, nullptr, nullptr, nullptr, P);
  // staged: the descriptors, then the first 64-token chunk of each segment
  // (an exclusive scan; the token kernel's work items are these chunks)
  const size_t o_cb = sizeof(SegDesc) * n;
  const size_t staged = o_cb + ((4ull * (n + 1) + 15) & ~(size_t)15);
  std::vector<uint8_t> host(n > 0 ? staged : 0);
  uint64_t n_chunks = 0;
  if (n > 0) {
    memcpy(host.data(), P.descs.data(), o_cb);
    uint32_t* cb = (uint32_t*)(host.data() + o_cb);
    for (uint32_t i = 0; i < n; i++) {
      cb[i] = (uint32_t)n_chunks;
      n_chunks += (st->segs[i].row_count + kTokenChunk - 1) / kTokenChunk;
      if (n_chunks > UINT32_MAX) return fail(GIFT_E_TOO_LARGE, "more than 2^32 - 1 chunks of %u tokens", kTokenChunk);
    }
    cb[n] = (uint32_t)n_chunks;
  }
  SegDesc* d = nullptr;
  hipError_t e = hipSuccess;
  ScratchLease lease;
  if (n > 0) {
    e = lease.acquire(dev, stream, staged);
    if (e != hipSuccess) return hip_fail(e, "device scratch");
    d = (SegDesc*)lease.ptr;
  }
  // uncovered tokens (rows no segment covers) get zero output: only when the
  // plan has such gaps is the output cleared first, the token kernel then
  // overwrites every covered entry
  const bool gaps = !P.zr.empty();
  EventMark call_ev;  // the event recorded behind the call's last kernel
  auto rest = [&]() -> hipError_t {
    hipError_t r = hipSuccess;
    if (gaps)
      r = decrypt ? launch_wipe(tokens_out, 8ull * n_tokens, stream) : launch_wipe(blocks_out, 16ull * n_tokens, stream);
    if (r == hipSuccess && gaps && decrypt && nonces_out) r = launch_wipe(nonces_out, 8ull * n_tokens, stream);
    if (r == hipSuccess)
      r = launch_tokens(d, (const uint32_t*)((const uint8_t*)d + o_cb), n, (uint32_t)n_chunks, decrypt, tokens,
                        nonces, blocks_in, blocks_out, tokens_out, nonces_out, eos_token, kt->dev, stream);
    return r;
  };
  if (n > 0) {
    // the token kernels are enqueued while the staging slot is held (one
    // event behind the last of them frees the slot)
    Staging* sg = staging_for(dev);
    e = sg ? sg->upload(d, host.data(), staged, stream,
                        [&](const void* src) {
                          hipError_t r = launch_prologue(d, src, staged, n, kNoBids, nullptr, nullptr, nullptr,
                                                         nullptr, nullptr, 0u, 0u, nullptr, stream);
                          return r != hipSuccess ? r : rest();
                        },
                        false, &call_ev)
           : hipErrorInvalidDevice;
  } else {
    e = rest();
  }
  hipError_t e2 = lease.release(call_ev);
  if (e != hipSuccess) return hip_fail(e, "token kernels");
  if (e2 != hipSuccess) return hip_fail(e2, "device scratch release");
  return GIFT_OK;
}

gift_status gift_token_encrypt(const gift_segment_table* st, const uint64_t* tokens, const uint64_t* nonces,
                               uint64_t n_tokens, gift_key_table kt, uint64_t eos_token, uint8_t* out,
                               hipStream_t stream) {
  return run_tokens(false, st, n_tokens, kt, eos_token, tokens, nonces, nullptr, out, nullptr, nullptr, stream);
}

gift_status gift_token_decrypt(const gift_segment_table* st, const uint8_t* blocks, uint64_t n_tokens,
                               gift_key_table kt, uint64_t eos_token, uint64_t* tokens_out, uint64_t* nonces_out,
                               hipStream_t stream) {
  return run_tokens(true, st, n_tokens, kt, eos_token, nullptr, nullptr, blocks, nullptr, tokens_out, nonces_out,
                    stream);
}

}  // extern "C"
