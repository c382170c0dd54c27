// Host-side ownership tracking: ownership records and IFT rules (GIFT
// Sec. 4.2-4.3) and launch-order checking (Sec. 4.4).  Declared in
// include/gift_ift.h.  No HIP calls.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <new>
#include <unordered_map>
#include <vector>

#include "gift_ift.h"

namespace {

bool mul_ok(uint64_t a, uint64_t b, uint64_t* r) { return !__builtin_mul_overflow(a, b, r); }

// One tensor record (Sec. 4.2): base, shape, element size, ownership
// dimensions; the second-level index is the dense owner array over the odim
// subscripts.
struct TensorRec {
  uintptr_t base = 0;
  uint64_t bytes = 0;
  uint32_t ndim = 0;
  uint64_t shape[GIFT_MAX_DIMS] = {0};
  uint32_t elem = 0;
  uint32_t odim_mask = 0;
  std::vector<uint64_t> radix;  // sizes of the odim dimensions, in order
  std::vector<uint32_t> owner;  // one entry per unit
};

}  // namespace

struct gift_ownership_s {
  std::map<uintptr_t, TensorRec> tensors;  // first-level index: base address
  uint64_t ops = 0;                        // record operations done by IFT rules
};

struct gift_race_s {
  struct Access {
    uint32_t stream;
    uint64_t seq;
  };
  struct Interval {
    uint64_t end;
    bool has_writer = false;
    Access writer{0, 0};
    std::vector<Access> readers;  // last reader per stream
  };
  using Clock = std::map<uint32_t, uint64_t>;  // stream -> last kernel known finished
  struct Stream {
    uint64_t issued = 0;     // kernels launched on the stream
    uint64_t completed = 0;  // kernels known finished by a host synchronisation
    Clock view;              // kernels of other streams ordered before the next launch here
    // view in effect from a sequence number on: (first seq, view), ascending
    std::vector<std::pair<uint64_t, Clock>> history;
  };
  std::map<uint64_t, Interval> ivs;  // keyed by start; disjoint
  std::unordered_map<uint32_t, Stream> streams;

  static void merge(Clock& into, const Clock& from) {
    for (const auto& kv : from) {
      uint64_t& v = into[kv.first];
      v = std::max(v, kv.second);
    }
  }
  // the view kernel seq of stream st was launched under
  const Clock* view_of(const Stream& st, uint64_t seq) const {
    const Clock* c = nullptr;
    for (const auto& h : st.history) {
      if (h.first > seq) break;
      c = &h.second;
    }
    return c;
  }
  // Views recorded for kernels that are now complete are never needed again
  // except the newest one, which still applies to later sequence numbers.
  static void prune(Stream& st) {
    size_t keep = 0;
    while (keep + 1 < st.history.size() && st.history[keep + 1].first <= st.completed) keep++;
    if (keep > 0) st.history.erase(st.history.begin(), st.history.begin() + (ptrdiff_t)keep);
  }
  // has kernel a finished before the next kernel launched on `stream` starts?
  bool ordered(const Access& a, uint32_t stream) {
    if (a.stream == stream) return true;
    if (a.seq <= streams[a.stream].completed) return true;
    const Clock& v = streams[stream].view;
    auto it = v.find(a.stream);
    return it != v.end() && a.seq <= it->second;
  }
  // ensure an interval boundary at x (no-op if x is a boundary or uncovered)
  void split(uint64_t x) {
    auto it = ivs.upper_bound(x);
    if (it == ivs.begin()) return;
    --it;
    if (it->first < x && x < it->second.end) {
      Interval right = it->second;
      it->second.end = x;
      ivs.emplace(x, right);
    }
  }
  // iterate intervals overlapping [a, b)
  template <typename F>
  void each(uint64_t a, uint64_t b, F f) const {
    if (a >= b) return;
    auto it = ivs.upper_bound(a);
    if (it != ivs.begin()) --it;
    for (; it != ivs.end() && it->first < b; ++it)
      if (it->second.end > a) f(it->second);
  }
};

extern "C" {

// ---------------------------------------------------------------------------
// ownership records
// ---------------------------------------------------------------------------
gift_status gift_own_create(gift_ownership* out) {
  if (!out) return GIFT_E_INVALID;
  *out = new (std::nothrow) gift_ownership_s;
  return *out ? GIFT_OK : GIFT_E_NOMEM;
}

gift_status gift_own_destroy(gift_ownership h) {
  delete h;
  return GIFT_OK;
}

gift_status gift_own_register(gift_ownership h, const void* base, uint32_t ndim, const uint64_t* shape,
                              uint32_t elem_size, uint32_t odim_mask) {
  if (!h || !base || !shape || ndim == 0 || ndim > GIFT_MAX_DIMS || elem_size == 0) return GIFT_E_INVALID;
  if (odim_mask >> ndim) return GIFT_E_INVALID;
  TensorRec r;
  r.base = (uintptr_t)base;
  r.ndim = ndim;
  r.elem = elem_size;
  r.odim_mask = odim_mask;
  uint64_t n = elem_size, units = 1;
  for (uint32_t d = 0; d < ndim; d++) {
    if (shape[d] == 0 || !mul_ok(n, shape[d], &n)) return GIFT_E_INVALID;
    r.shape[d] = shape[d];
    if (odim_mask & (1u << d)) {
      if (!mul_ok(units, shape[d], &units)) return GIFT_E_INVALID;
      r.radix.push_back(shape[d]);
    }
  }
  if (r.base + n < r.base) return GIFT_E_INVALID;
  r.bytes = n;
  // overlap with the neighbouring records
  auto it = h->tensors.lower_bound(r.base);
  if (it != h->tensors.end() && it->first < r.base + r.bytes) return GIFT_E_OVERLAP;
  if (it != h->tensors.begin()) {
    --it;
    if (it->first + it->second.bytes > r.base) return GIFT_E_OVERLAP;
  }
  try {
    r.owner.assign(units, GIFT_LABEL_UNOWNED);
  } catch (const std::bad_alloc&) {
    return GIFT_E_NOMEM;
  }
  h->tensors.emplace(r.base, std::move(r));
  return GIFT_OK;
}

gift_status gift_own_release(gift_ownership h, const void* base) {
  if (!h) return GIFT_E_INVALID;
  return h->tensors.erase((uintptr_t)base) ? GIFT_OK : GIFT_E_INVALID;
}

static TensorRec* find(gift_ownership h, const void* base) {
  if (!h) return nullptr;
  auto it = h->tensors.find((uintptr_t)base);
  return it == h->tensors.end() ? nullptr : &it->second;
}

gift_status gift_own_units(gift_ownership h, const void* base, uint64_t* n_units) {
  TensorRec* r = find(h, base);
  if (!r || !n_units) return GIFT_E_INVALID;
  *n_units = r->owner.size();
  return GIFT_OK;
}

gift_status gift_own_flat_index(gift_ownership h, const void* base, const uint64_t* subs, uint64_t* flat) {
  TensorRec* r = find(h, base);
  if (!r || !flat || (!subs && !r->radix.empty())) return GIFT_E_INVALID;
  uint64_t f = 0;
  for (size_t k = 0; k < r->radix.size(); k++) {
    if (subs[k] >= r->radix[k]) return GIFT_E_RANGE;
    f = f * r->radix[k] + subs[k];
  }
  *flat = f;
  return GIFT_OK;
}

gift_status gift_own_set(gift_ownership h, const void* base, uint64_t flat_begin, uint64_t count, uint32_t owner) {
  TensorRec* r = find(h, base);
  if (!r) return GIFT_E_INVALID;
  const uint64_t n = r->owner.size();
  if (flat_begin > n || count > n - flat_begin) return GIFT_E_RANGE;
  std::fill(r->owner.begin() + flat_begin, r->owner.begin() + flat_begin + count, owner);
  return GIFT_OK;
}

gift_status gift_own_get(gift_ownership h, const void* base, uint64_t flat, uint32_t* owner) {
  TensorRec* r = find(h, base);
  if (!r || !owner) return GIFT_E_INVALID;
  if (flat >= r->owner.size()) return GIFT_E_RANGE;
  *owner = r->owner[flat];
  return GIFT_OK;
}

gift_status gift_own_labels(gift_ownership h, const void* base, uint32_t* labels, uint64_t n_units) {
  TensorRec* r = find(h, base);
  if (!r || (!labels && n_units)) return GIFT_E_INVALID;
  if (n_units != r->owner.size()) return GIFT_E_RANGE;
  if (n_units) memcpy(labels, r->owner.data(), 4 * n_units);
  return GIFT_OK;
}

uint64_t gift_own_ops(gift_ownership h) { return h ? h->ops : 0; }

// --- IFT rules -------------------------------------------------------------
static bool is_matrix(const TensorRec* r, uint64_t rows, uint64_t cols, uint32_t elem) {
  return r && r->ndim == 2 && r->shape[0] == rows && r->shape[1] == cols && r->elem == elem && r->odim_mask == 1u;
}
static bool is_rows_vector(const TensorRec* r, uint64_t rows, uint32_t elem) {
  return r && r->ndim == 1 && r->shape[0] == rows && r->elem == elem && r->odim_mask == 1u;
}
static bool elems_are(const TensorRec* r, uint32_t ndim, const uint64_t* shape, uint32_t elem) {
  if (!r || r->ndim != ndim || r->elem != elem) return false;
  for (uint32_t d = 0; d < ndim; d++)
    if (r->shape[d] != shape[d]) return false;
  return true;
}
// rule step 4: every unit of a parameter input is parameter-owned (one check)
static bool all_param(gift_ownership h, const TensorRec* r) {
  h->ops++;
  for (uint32_t o : r->owner)
    if (o != GIFT_LABEL_PARAM) return false;
  return true;
}
// Rule step 5 over rows: out[i] <- owner shared by the non-parameter sources
// (one or two row-owned tensors).  The shared owner may be the parameter
// label (data derived from parameters alone); unowned memory is never read.
// All rows are checked before any record changes.
static gift_status propagate_rows(gift_ownership h, TensorRec* out, const TensorRec* a, const TensorRec* b,
                                  uint64_t rows) {
  std::vector<uint32_t> next(rows);
  for (uint64_t i = 0; i < rows; i++) {
    const uint32_t oa = a->owner[i];
    h->ops++;
    if (b) {
      const uint32_t ob = b->owner[i];
      h->ops++;
      if (ob != oa) return GIFT_E_REJECTED;
    }
    if (oa == GIFT_LABEL_UNOWNED) return GIFT_E_REJECTED;
    next[i] = oa;
  }
  for (uint64_t i = 0; i < rows; i++) {
    out->owner[i] = next[i];
    h->ops++;
  }
  return GIFT_OK;
}

gift_status gift_ift_add_residual(gift_ownership h, const void* out, const void* in, const void* res, uint64_t rows,
                                  uint64_t cols, uint32_t elem_size) {
  if (!h) return GIFT_E_INVALID;
  TensorRec *o = find(h, out), *x = find(h, in), *rr = find(h, res);  // step 1
  if (!is_matrix(o, rows, cols, elem_size) || !is_matrix(x, rows, cols, elem_size) ||
      !is_matrix(rr, rows, cols, elem_size))  // step 2
    return GIFT_E_REJECTED;
  if (rr == x || rr == o) return GIFT_E_REJECTED;  // step 3: only out == in may alias
  return propagate_rows(h, o, x, rr, rows);         // step 5 (no parameter inputs)
}

gift_status gift_ift_add_bias(gift_ownership h, const void* out, const void* in, const void* bias, uint64_t rows,
                              uint64_t cols, uint32_t elem_size) {
  if (!h) return GIFT_E_INVALID;
  TensorRec *o = find(h, out), *x = find(h, in), *b = find(h, bias);
  const uint64_t bshape[1] = {cols};
  if (!is_matrix(o, rows, cols, elem_size) || !is_matrix(x, rows, cols, elem_size) ||
      !elems_are(b, 1, bshape, elem_size))
    return GIFT_E_REJECTED;
  if (b == x || b == o) return GIFT_E_REJECTED;
  if (!all_param(h, b)) return GIFT_E_REJECTED;  // step 4
  return propagate_rows(h, o, x, nullptr, rows);
}

gift_status gift_ift_find_max(gift_ownership h, const void* out, const void* in, uint64_t rows, uint64_t cols,
                              uint32_t in_elem_size, uint32_t out_elem_size) {
  if (!h) return GIFT_E_INVALID;
  TensorRec *o = find(h, out), *x = find(h, in);
  if (!is_rows_vector(o, rows, out_elem_size) || !is_matrix(x, rows, cols, in_elem_size)) return GIFT_E_REJECTED;
  if (o == x) return GIFT_E_REJECTED;
  return propagate_rows(h, o, x, nullptr, rows);
}

gift_status gift_ift_matmul(gift_ownership h, const void* out, const void* in, const void* weight, uint64_t rows,
                            uint64_t k, uint64_t n, uint32_t elem_size) {
  if (!h) return GIFT_E_INVALID;
  TensorRec *o = find(h, out), *x = find(h, in), *w = find(h, weight);
  const uint64_t wshape[2] = {k, n};
  if (!is_matrix(o, rows, n, elem_size) || !is_matrix(x, rows, k, elem_size) || !elems_are(w, 2, wshape, elem_size))
    return GIFT_E_REJECTED;
  if (o == x || o == w || x == w) return GIFT_E_REJECTED;
  if (!all_param(h, w)) return GIFT_E_REJECTED;
  return propagate_rows(h, o, x, nullptr, rows);
}

// ---------------------------------------------------------------------------
// launch-order checking
// ---------------------------------------------------------------------------
gift_status gift_race_create(gift_race* out) {
  if (!out) return GIFT_E_INVALID;
  *out = new (std::nothrow) gift_race_s;
  return *out ? GIFT_OK : GIFT_E_NOMEM;
}

gift_status gift_race_destroy(gift_race h) {
  delete h;
  return GIFT_OK;
}

gift_status gift_race_launch(gift_race h, uint32_t stream, const gift_range* reads, uint32_t n_reads,
                             const gift_range* writes, uint32_t n_writes, uint64_t* seq) {
  if (!h || (n_reads && !reads) || (n_writes && !writes)) return GIFT_E_INVALID;
  for (uint32_t i = 0; i < n_reads; i++)
    if (reads[i].addr + reads[i].bytes < reads[i].addr) return GIFT_E_INVALID;
  for (uint32_t i = 0; i < n_writes; i++)
    if (writes[i].addr + writes[i].bytes < writes[i].addr) return GIFT_E_INVALID;
  // check
  bool race = false;
  auto other_pending = [&](const gift_race_s::Access& a) { return !h->ordered(a, stream); };
  for (uint32_t i = 0; i < n_reads && !race; i++)
    h->each(reads[i].addr, reads[i].addr + reads[i].bytes, [&](const gift_race_s::Interval& iv) {
      if (iv.has_writer && other_pending(iv.writer)) race = true;
    });
  for (uint32_t i = 0; i < n_writes && !race; i++)
    h->each(writes[i].addr, writes[i].addr + writes[i].bytes, [&](const gift_race_s::Interval& iv) {
      if (iv.has_writer && other_pending(iv.writer)) race = true;
      for (const auto& r : iv.readers)
        if (other_pending(r)) race = true;
    });
  if (race) return GIFT_E_RACE;
  // record
  const uint64_t s = ++h->streams[stream].issued;
  auto touch = [&](uint64_t a, uint64_t b, bool write) {
    if (a >= b) return;
    h->split(a);
    h->split(b);
    // fill gaps in [a, b) with fresh intervals
    uint64_t cur = a;
    auto it = h->ivs.lower_bound(a);
    std::vector<std::pair<uint64_t, uint64_t>> gaps;
    for (; it != h->ivs.end() && it->first < b; ++it) {
      if (it->first > cur) gaps.push_back({cur, it->first});
      cur = it->second.end;
    }
    if (cur < b) gaps.push_back({cur, b});
    for (auto& g : gaps) {
      gift_race_s::Interval iv;
      iv.end = g.second;
      h->ivs.emplace(g.first, iv);
    }
    for (it = h->ivs.lower_bound(a); it != h->ivs.end() && it->first < b; ++it) {
      gift_race_s::Interval& iv = it->second;
      if (write) {
        iv.has_writer = true;
        iv.writer = {stream, s};
        iv.readers.clear();
      } else {
        bool found = false;
        for (auto& r : iv.readers)
          if (r.stream == stream) {
            r.seq = s;
            found = true;
          }
        if (!found) iv.readers.push_back({stream, s});
      }
    }
  };
  for (uint32_t i = 0; i < n_reads; i++) touch(reads[i].addr, reads[i].addr + reads[i].bytes, false);
  for (uint32_t i = 0; i < n_writes; i++) touch(writes[i].addr, writes[i].addr + writes[i].bytes, true);
  if (seq) *seq = s;
  return GIFT_OK;
}

gift_status gift_race_wait(gift_race h, uint32_t stream, uint32_t on_stream, uint64_t seq) {
  if (!h) return GIFT_E_INVALID;
  auto& src = h->streams[on_stream];
  if (seq > src.issued) return GIFT_E_RANGE;
  if (seq == 0 || on_stream == stream) return GIFT_OK;
  gift_race_s::Clock v = h->streams[stream].view;
  if (const gift_race_s::Clock* c = h->view_of(src, seq)) gift_race_s::merge(v, *c);
  uint64_t& mine = v[on_stream];
  mine = std::max(mine, seq);
  auto& dst = h->streams[stream];
  dst.view = v;
  if (!dst.history.empty() && dst.history.back().first == dst.issued + 1)
    dst.history.back().second = std::move(v);
  else
    dst.history.emplace_back(dst.issued + 1, std::move(v));
  return GIFT_OK;
}

gift_status gift_race_sync(gift_race h, uint32_t stream) {
  if (!h) return GIFT_E_INVALID;
  auto& st = h->streams[stream];
  st.completed = st.issued;
  // what the stream waited on has finished too
  const gift_race_s::Clock v = st.view;
  for (const auto& kv : v) {
    uint64_t& c = h->streams[kv.first].completed;
    c = std::max(c, kv.second);
  }
  for (auto& kv : h->streams) gift_race_s::prune(kv.second);
  return GIFT_OK;
}

gift_status gift_race_sync_all(gift_race h) {
  if (!h) return GIFT_E_INVALID;
  // every recorded access has finished, so none can conflict with a later
  // launch: the records and the stream views are dropped (sequence numbers go on)
  for (auto& kv : h->streams) {
    kv.second.completed = kv.second.issued;
    kv.second.view.clear();
    kv.second.history.clear();
  }
  h->ivs.clear();
  return GIFT_OK;
}

gift_status gift_race_release(gift_race h, gift_range r) {
  if (!h || r.addr + r.bytes < r.addr) return GIFT_E_INVALID;
  if (r.bytes == 0) return GIFT_OK;
  h->split(r.addr);
  h->split(r.addr + r.bytes);
  auto it = h->ivs.lower_bound(r.addr);
  while (it != h->ivs.end() && it->first < r.addr + r.bytes) it = h->ivs.erase(it);
  return GIFT_OK;
}

}  // extern "C"
