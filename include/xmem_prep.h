/* xmem_prep.h -- C ABI of the trace-preparation steps upstream of the Memory
 * Simulator: lifecycle pairing of raw allocator events and time-window
 * attribution of the blocks to operators (the Analyzer, Section 3.2), and
 * category-based retiming into the Simulator's event words (the Memory
 * Orchestrator, Section 3.3).
 *
 * All calls are batched over independent traces in CSR layout, run entirely
 * in the library's HIP kernels on the caller's stream, allocate nothing and
 * do not synchronise.  Every pointer named d_* is device memory owned by the
 * caller.  Call-level errors are returned (XMEM_E* of xmem.h); a batch whose
 * offsets turn out invalid on the device is reported through *d_status. */
#ifndef XMEM_PREP_H
#define XMEM_PREP_H

#include <stddef.h>
#include <stdint.h>

#include "xmem.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One allocator instant event as the profiler records it (Section 3.2, the
 * cpu_instant_event stream): bytes > 0 allocates `bytes` at `addr`, bytes < 0
 * frees the block at `addr`, bytes == 0 is ignored.  24 bytes. */
typedef struct {
  int64_t ts;
  uint64_t addr;
  int64_t bytes;
} xmem_raw_event;

/* A memory block (Section 3.2): an allocation and its deallocation.  t_free
 * is XMEM_PERSISTENT for a block that is never freed.  32 bytes. */
#define XMEM_PERSISTENT INT64_MAX
typedef struct {
  int64_t size;
  int64_t t_alloc;
  int64_t t_free;
  int32_t category; /* xmem_block_category */
  int32_t pad;
} xmem_block;

/* Block roles the Orchestrator retimes (Section 3.3). */
typedef enum {
  XMEM_CAT_OTHER = 0,     /* activations, temporaries: lifetime kept */
  XMEM_CAT_PARAMETER = 1, /* model.to(device): persistent */
  XMEM_CAT_BATCH = 2,     /* batch data: freed at the iteration boundary after it, or its own free if earlier */
  XMEM_CAT_GRADIENT = 3,  /* freed at the first zero_grad after its allocation; persistent if none */
  XMEM_CAT_OPTIMIZER = 4  /* optimizer states: persistent */
} xmem_block_category;

/* An execution window of the profile (Section 3.2): a python_function call of
 * a high-level component (a model layer, the data loader, optimizer.step ...)
 * or a cpu_op operator.  A trace's windows are listed by start time (a window
 * that starts with its parent comes after it), are properly nested, and name
 * their enclosing window by its index in the trace (an earlier index, or -1
 * for a root).  32 bytes. */
typedef struct {
  int64_t start;    /* the window is [start, end], both ends included */
  int64_t end;
  int32_t parent;
  int32_t kind;     /* XMEM_WIN_COMPONENT or XMEM_WIN_OPERATOR */
  int32_t category; /* xmem_block_category of the blocks an operator produces */
  int32_t pad;
} xmem_window;
#define XMEM_WIN_COMPONENT 0
#define XMEM_WIN_OPERATOR 1

/* Largest n_records any call accepts (record indices are 32-bit). */
#define XMEM_PREP_MAX_RECORDS ((int64_t)0xFFFFFFF0)

/* Device workspace bytes for a call over n_traces traces and n_records
 * records: n_records = total raw events for xmem_lifecycles, the larger of
 * total blocks and total windows for xmem_attribute, 2 x total blocks for
 * xmem_orchestrate.  0 for invalid arguments. */
size_t xmem_prep_workspace_bytes(int64_t n_traces, int64_t n_records);

/* Lifecycle pairing (Section 3.2).  Each trace's raw events are taken in
 * stream order: an allocation opens a block at its address; the next event
 * at that address closes it if it is a free (the block's t_free is that
 * event's ts) or, if it is another allocation, leaves it persistent.  A free
 * at an address with no open block is dropped and counted.  Blocks come out
 * in allocation order.
 *   d_raw            : xmem_raw_event[total_raw], trace t at
 *                      [d_raw_offsets[t], d_raw_offsets[t+1]).
 *   d_category       : int32[total_raw] or NULL; a block takes the value of
 *                      its allocation event (0 when NULL).
 *   d_raw_offsets    : int64[n_traces+1], 0-based, non-decreasing, last ==
 *                      total_raw.
 *   d_blocks         : xmem_block[total_raw] (room for the worst case).
 *   d_block_offsets  : int64[n_traces+1], written.
 *   d_unmatched_frees: int64[n_traces] or NULL, written.
 *   d_status         : int32[1], written: 0, or XMEM_T_BAD_BATCH when the
 *                      offsets are invalid (then every block offset is 0).
 *   d_workspace      : >= xmem_prep_workspace_bytes(n_traces, total_raw),
 *                      256-byte aligned.
 * Returns XMEM_OK, XMEM_EINVAL (null pointer, negative count, total_raw >
 * XMEM_PREP_MAX_RECORDS), XMEM_EWORKSPACE or XMEM_EHIP. */
int xmem_lifecycles(const xmem_raw_event* d_raw, const int32_t* d_category, const int64_t* d_raw_offsets,
                    int64_t n_traces, int64_t total_raw, xmem_block* d_blocks, int64_t* d_block_offsets,
                    int64_t* d_unmatched_frees, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                    void* hip_stream);

/* Time-window attribution (Section 3.2).  A block is linked to an operator
 * window that contains its allocation time, trying the operators that do from
 * the innermost outward: it links if (i) its free is no later than the
 * window's end, or (ii) its free is later than the end of the operator's
 * nearest enclosing component window (persistent blocks outlive every
 * window).  Blocks linked by (ii) are the operator's products and take its
 * category; blocks linked by (i) are its temporaries (XMEM_CAT_OTHER).
 * Blocks with no link are filtered out; the rest keep their order.
 *   d_blocks, d_block_offsets: a batch as xmem_lifecycles writes it.
 *   d_windows, d_window_offsets: each trace's windows (xmem_window), CSR.
 *   d_kept           : xmem_block[total_blocks] (room for the worst case).
 *   d_kept_offsets   : int64[n_traces+1], written.
 *   d_block_window   : int32[total_blocks] or NULL: for every input block, the
 *                      index within its trace of the window it links to, or -1.
 *   d_status         : as for xmem_lifecycles (block or window offsets
 *                      invalid -> XMEM_T_BAD_BATCH, kept offsets 0).
 *   d_workspace      : >= xmem_prep_workspace_bytes(n_traces,
 *                      max(total_blocks, total_windows)).
 * Returns as xmem_lifecycles. */
int xmem_attribute(const xmem_block* d_blocks, const int64_t* d_block_offsets, int64_t n_traces,
                   int64_t total_blocks, const xmem_window* d_windows, const int64_t* d_window_offsets,
                   int64_t total_windows, xmem_block* d_kept, int64_t* d_kept_offsets, int32_t* d_block_window,
                   int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* hip_stream);

/* Orchestration (Section 3.3).  Each block's free is retimed by category
 * (xmem_block_category; a free earlier than the allocation moves to it);
 * then every allocation and every non-persistent free is put in time order,
 * at equal times frees of earlier blocks first, then allocations, then frees
 * of blocks allocated at that time, and within each the blocks' order.  The
 * result is written as the Simulator's event words (xmem.h): an allocation
 * is its size, a free is XMEM_EVENT_FREE_BIT | the index of its allocation's
 * word within the trace.
 *   d_blocks, d_block_offsets: a batch as xmem_lifecycles writes it, with
 *                      categories set; trace t's blocks in allocation order.
 *   d_step_ts, d_step_offsets: ascending iteration-start timestamps
 *                      (profiler.step()) of each trace, CSR (int64[n+1]).
 *   d_zero_grad_ts, d_zero_grad_offsets: ascending optimizer.zero_grad()
 *                      timestamps of each trace, CSR.
 *   d_events         : uint64[2 * total_blocks] (room for the worst case).
 *   d_event_offsets  : int64[n_traces+1], written.
 *   d_status         : as for xmem_lifecycles (block, step or zero_grad
 *                      offsets invalid -> XMEM_T_BAD_BATCH, event offsets 0).
 *   d_workspace      : >= xmem_prep_workspace_bytes(n_traces, 2*total_blocks).
 * Returns as xmem_lifecycles. */
int xmem_orchestrate(const xmem_block* d_blocks, const int64_t* d_block_offsets, int64_t n_traces,
                     int64_t total_blocks, const int64_t* d_step_ts, const int64_t* d_step_offsets,
                     const int64_t* d_zero_grad_ts, const int64_t* d_zero_grad_offsets, uint64_t* d_events,
                     int64_t* d_event_offsets, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                     void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* XMEM_PREP_H */
