/*
 * gift_ift.h -- host-side ownership tracking for the GPU data path:
 * ownership records (GIFT Sec. 4.2), IFT rules for four example kernels
 * (Sec. 4.3) and launch-order checking against read-write and write-write
 * races (Sec. 4.4).  These are plain C++ state machines in libgift.so; they
 * make no HIP call and need no GPU.  Row labels produced here are what
 * gift_seal / gift_check_owner consume (include/gift.h).
 *
 * Statuses are those of gift.h, including the two that only these calls
 * return:
 *   GIFT_E_REJECTED (-8): an IFT rule refused the launch (ownership mixing,
 *                          a read of unowned memory, a non-parameter weight,
 *                          a shape or aliasing mismatch, an unknown tensor);
 *                          no record was changed.
 *   GIFT_E_RACE     (-9):  the launch would race with an unfinished kernel
 *                          on another stream; nothing was recorded.
 * Handles are not thread-safe: the paper drives each stream's tracking from
 * its own thread, and a caller sharing a handle across threads must lock it.
 */
#ifndef GIFT_IFT_H
#define GIFT_IFT_H

#include <stdint.h>

#include "gift.h"

#ifdef __cplusplus
extern "C" {
#endif

#define GIFT_MAX_DIMS 8

/* ------------------------------------------------------------------------
 * Ownership records (Sec. 4.2).  A two-level index: base address -> tensor
 * record (base, shape, element size, ownership-related dimensions "odim");
 * subscripts of the odim dimensions -> owner (a user ID, GIFT_LABEL_PARAM for
 * model parameters, or GIFT_LABEL_UNOWNED).  Ownership units of a tensor are
 * numbered by the mixed-radix index of their odim subscripts, in dimension
 * order ("flat index"): rows of a matrix with odim = {0}; (layer, block,
 * head) triples of a 5-D KV tensor with odim = {0, 1, 3}; one unit if
 * odim is empty.
 * ------------------------------------------------------------------------ */
typedef struct gift_ownership_s* gift_ownership;

gift_status gift_own_create(gift_ownership* out);
gift_status gift_own_destroy(gift_ownership h);

/* Registers a tensor (the device allocation at base; its bytes are
 * prod(shape) * elem_size).  odim_mask bit d marks dimension d as
 * ownership-related.  Every unit starts unowned.
 * Errors: GIFT_E_INVALID (null, ndim 0 or > GIFT_MAX_DIMS, zero sizes, mask
 * beyond ndim, overflow), GIFT_E_OVERLAP (overlaps a registered tensor). */
gift_status gift_own_register(gift_ownership h, const void* base, uint32_t ndim, const uint64_t* shape,
                              uint32_t elem_size, uint32_t odim_mask);

/* Forgets a tensor's record: its memory becomes unowned (Sec. 4.2: records
 * are cleared when the tensor is released).  GIFT_E_INVALID if unknown. */
gift_status gift_own_release(gift_ownership h, const void* base);

/* Number of ownership units of a tensor. */
gift_status gift_own_units(gift_ownership h, const void* base, uint64_t* n_units);

/* Flat index of odim subscripts (subs: one value per odim dimension, in
 * dimension order).  GIFT_E_RANGE if a subscript is out of its dimension. */
gift_status gift_own_flat_index(gift_ownership h, const void* base, const uint64_t* subs, uint64_t* flat);

/* Sets units [flat_begin, flat_begin + count) to owner; reads one unit. */
gift_status gift_own_set(gift_ownership h, const void* base, uint64_t flat_begin, uint64_t count, uint32_t owner);
gift_status gift_own_get(gift_ownership h, const void* base, uint64_t flat, uint32_t* owner);

/* Copies the owners of all units (n_units entries, host) -- for a row-owned
 * tensor these are the row labels gift_seal and gift_check_owner take. */
gift_status gift_own_labels(gift_ownership h, const void* base, uint32_t* labels, uint64_t n_units);

/* Record operations performed by the IFT rules so far (Sec. 4.1, Insight 2:
 * the FFN AddBias example costs 2*B + 1 of them for B rows). */
uint64_t gift_own_ops(gift_ownership h);

/* ------------------------------------------------------------------------
 * IFT rules (Sec. 4.3).  Each follows the rule steps of the paper:
 * (1) find the records of the tensors by base address; (2) check that their
 * shapes match the kernel arguments; (3) check that tensors occupy distinct
 * memory unless the kernel allows the alias (an in-place output); (4) check
 * that parameter inputs are parameter-owned; (5) for every row, check that
 * the non-parameter sources share one owner and give that owner to the output
 * row.  The shared owner may be GIFT_LABEL_PARAM (rows computed from
 * parameters alone stay parameter-owned); an unowned source row is refused,
 * since unowned memory may not be read.  Either every row propagates or
 * nothing changes (GIFT_E_REJECTED).  Matrices are row-major [rows, cols]
 * tensors with odim = {0}; bias and weight may have any odim and must be all
 * parameter-owned.  The operation counter also counts the checks made by a
 * launch that is then rejected.
 * ------------------------------------------------------------------------ */
/* out[i,:] = in[i,:] + res[i,:]; out may alias in (in place). */
gift_status gift_ift_add_residual(gift_ownership h, const void* out, const void* in, const void* res, uint64_t rows,
                                  uint64_t cols, uint32_t elem_size);
/* out[i,:] = in[i,:] + bias[:] (bias: [cols], parameter); out may alias in. */
gift_status gift_ift_add_bias(gift_ownership h, const void* out, const void* in, const void* bias, uint64_t rows,
                              uint64_t cols, uint32_t elem_size);
/* out[i] = argmax_j in[i,j] (out: [rows] of out_elem_size bytes). */
gift_status gift_ift_find_max(gift_ownership h, const void* out, const void* in, uint64_t rows, uint64_t cols,
                              uint32_t in_elem_size, uint32_t out_elem_size);
/* out[i,:] = in[i,:] x weight (in: [rows, k], weight: [k, n] parameter,
 * out: [rows, n]); no aliasing. */
gift_status gift_ift_matmul(gift_ownership h, const void* out, const void* in, const void* weight, uint64_t rows,
                            uint64_t k, uint64_t n, uint32_t elem_size);

/* ------------------------------------------------------------------------
 * Launch-order checking (Sec. 4.4, concurrency control).  Memory segments
 * are byte ranges.  Each range remembers its last writer kernel and its last
 * reader kernel per stream, as (stream, sequence number); each stream
 * remembers the last kernel known complete.  A kernel is complete once a
 * synchronisation of its stream (or of the device) has been recorded after
 * its launch.  A launch is refused (GIFT_E_RACE, nothing recorded) if
 *   - it reads a range whose last writer is on another stream and not
 *     complete (read-write race), or
 *   - it writes a range whose last writer or any reader is on another stream
 *     and not complete (write-write / write-read race),
 * unless that kernel is ordered before the launch by the device itself:
 * kernels on one stream are ordered, and a stream that waits on an event
 * recorded after kernel k of another stream (gift_race_wait) runs its later
 * kernels after k and after everything k was ordered after (transitively).
 * Stream waits are how the collective-operation order of Sec. 4.4 (a
 * receiver reading a buffer between two writers on another stream) is
 * admitted without a host synchronisation.
 * ------------------------------------------------------------------------ */
typedef struct {
  uint64_t addr;
  uint64_t bytes;
} gift_range;

typedef struct gift_race_s* gift_race;

gift_status gift_race_create(gift_race* out);
gift_status gift_race_destroy(gift_race h);
/* Checks and records a launch on `stream`; *seq receives its sequence
 * number on that stream (1, 2, ...).  Empty ranges are ignored. */
gift_status gift_race_launch(gift_race h, uint32_t stream, const gift_range* reads, uint32_t n_reads,
                             const gift_range* writes, uint32_t n_writes, uint64_t* seq);
/* Stream `stream` waits for kernel `seq` of `on_stream` (hipStreamWaitEvent on
 * an event recorded right after that kernel).  seq 0 or on_stream == stream
 * is a no-op; GIFT_E_RANGE if seq has not been launched on on_stream. */
gift_status gift_race_wait(gift_race h, uint32_t stream, uint32_t on_stream, uint64_t seq);
/* Every kernel launched on `stream` so far is complete (stream
 * synchronisation, a blocking copy on that stream), and so is every kernel the
 * stream has waited on. */
gift_status gift_race_sync(gift_race h, uint32_t stream);
/* Every kernel launched so far is complete (device synchronisation).  No
 * recorded access can conflict with a later launch any more, so the per-range
 * records are dropped here: memory stays bounded in a long-running server
 * that synchronises the device now and then. */
gift_status gift_race_sync_all(gift_race h);
/* The range was freed: its records are dropped. */
gift_status gift_race_release(gift_race h, gift_range r);

#ifdef __cplusplus
}
#endif
#endif /* GIFT_IFT_H */
