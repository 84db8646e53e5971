/*
 * xmem.h -- C ABI of libxmem_replay.so: batched replay of tensor allocate/free
 * traces through a model of a two-level caching GPU allocator, on one AMD
 * Instinct MI355X (gfx950).
 *
 * The operation is the Memory Simulator of xMem (Shi, Pezaros, Elkhatib,
 * "xMem: A CPU-Based Approach for Accurate Estimation of GPU Memory in Deep
 * Learning Training Workloads", Middleware '25), Section 3.4: each trace is an
 * orchestrated, chronologically ordered sequence of memory-block events; the
 * simulator replays it through (i) size round-up, (ii) segment requests,
 * (iii) best-fit-with-coalescing block management (search, split, merge),
 * (iv) caching of freed blocks and (v) device-level OOM after reclamation, and
 * reports the tensor and segment memory time series, whose maxima are the
 * estimated peaks.  Section 2.2 (Tensors, Segments) gives the rounding example
 * (512 B) and the segment example (2 MB for a 1 MB tensor); Section 6.4 (iii)
 * gives the 20 MB-for-10 MB example.
 *
 * Everything here is plain C: no torch types.  All buffers passed to the
 * replay entry points are DEVICE memory owned by the caller, except `params`,
 * which is a host pointer read during the call and not retained.  The library
 * keeps no state between calls and is re-entrant.
 */
#ifndef XMEM_H
#define XMEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define XMEM_ABI_VERSION 1u

/* ------------------------------------------------------------------------
 * Event word (uint64), one per event, traces concatenated (CSR layout).
 *
 *   ALLOC: bit 63 = 0, bits [62:0] = requested bytes s.
 *          s == 0 is a no-op allocation (it still has a handle that may be
 *          freed once).  s > XMEM_MAX_REQUEST_BYTES is malformed
 *          (XMEM_T_BAD_EVENT).
 *   FREE : bit 63 = 1, bits [31:0] = h, the index *within the same trace* of
 *          the ALLOC event whose block is released; bits [62:32] must be 0
 *          (else XMEM_T_BAD_EVENT).  h must satisfy h < (index of this
 *          event), event h must be an ALLOC, and h must not have been freed
 *          before (else XMEM_T_BAD_FREE).
 *
 * An ALLOC that is never freed stays live until the end of the trace
 * (Section 3.2: blocks without a deallocation are persistent).
 * ---------------------------------------------------------------------- */
#define XMEM_EVENT_FREE_BIT       (1ull << 63)
#define XMEM_MAX_REQUEST_BYTES    (1ull << 48)
#define XMEM_MAX_TRACE_EVENTS     ((int64_t)0x7fffffff)
/* Segment bytes ever created in one pool; a request that would pass it stops
 * the trace with XMEM_T_OVERFLOW.  Since allocated <= reserved <= the sum over
 * both pools, every reported byte count stays below 2^62. */
#define XMEM_POOL_CREATED_LIMIT   (1ll << 61)

static inline uint64_t xmem_event_alloc(uint64_t bytes) { return bytes & ~XMEM_EVENT_FREE_BIT; }
static inline uint64_t xmem_event_free(uint32_t alloc_index) { return XMEM_EVENT_FREE_BIT | (uint64_t)alloc_index; }

/* ------------------------------------------------------------------------
 * Allocator parameters.  Every constant of the allocator model is a field;
 * the defaults are the values the paper states or exemplifies.
 *
 * Request r = round_bytes * ceil(s / round_bytes)            (Section 3.4 (i)).
 * Pool       = SMALL if r <= small_max_bytes else LARGE.
 * New segment size when no cached free block fits           (Section 3.4 (ii),
 * Section 2.2.2 "2MB for a 1MB tensor", Section 6.4 "20MB for a 10MB tensor"):
 *   SMALL                      -> small_segment_bytes
 *   LARGE, r < min_large_alloc -> mid_segment_bytes
 *   LARGE, r >= min_large_alloc-> large_round_bytes * ceil(r / large_round_bytes)
 * Split (Section 3.4 (iii)): the front r bytes of the chosen block are used;
 * the remainder becomes a free block iff remainder >= split_min_{pool}_bytes,
 * otherwise the whole block is handed out.
 * Capacity (Section 3.4 (iv)-(v)): a segment request with
 * reserved + S > device_capacity_bytes first releases every segment that is
 * one whole free block (both pools); if still reserved + S > capacity the
 * trace stops with XMEM_T_OOM.  INT64_MAX means unbounded.
 *
 * Flags, bits [5:0] (XMEM_FLAGS_CHUNKS_MASK): with unbounded capacity, the
 * events of each pool of a trace may be replayed in several chunks at once.
 * The value k sets the grain: a pool gets about k x (its events / the mean
 * trace length) chunks, at most k.  0 = k chosen from the number of traces
 * (64512 / n_traces, at most 63; 2 when that is below 16, and 1 from 16384
 * traces on; a single trace of 2^20 events or more: 127, of at most 4096
 * events: 1; two traces of 2^20 events or more on average: 63, replayed in
 * rounds on per-chunk paged sets), 1 = one serial replay per pool, at most
 * 63.  Results are
 * identical for
 * every value; only the speed and the workspace size differ.  All other bits
 * are reserved and must be 0.
 *
 * Validity (else XMEM_EINVAL): abi_version == XMEM_ABI_VERSION, flags as above;
 * round_bytes a power of two in [1, 2^30]; small_max, small_segment,
 * mid_segment, min_large_alloc, large_round in [1, 2^40] and multiples of
 * round_bytes; small_max <= small_segment; min_large_alloc <= mid_segment;
 * split_min_small, split_min_large in [1, 2^40]; device_capacity >= 1.
 * ---------------------------------------------------------------------- */
typedef struct {
  uint32_t abi_version;           /* XMEM_ABI_VERSION                          */
  uint32_t flags;                 /* bits [5:0]: chunks per pool (0 = automatic) */
  int64_t  round_bytes;           /* 512        Section 2.2.1, 3.4 (i)         */
  int64_t  small_max_bytes;       /* 1 MiB (inclusive)                         */
  int64_t  small_segment_bytes;   /* 2 MiB      Section 2.2.2                  */
  int64_t  mid_segment_bytes;     /* 20 MiB     Section 6.4 (iii)              */
  int64_t  min_large_alloc_bytes; /* 10 MiB                                    */
  int64_t  large_round_bytes;     /* 2 MiB                                     */
  int64_t  split_min_small_bytes; /* 512        split whenever not exact       */
  int64_t  split_min_large_bytes; /* 512; preset PYTORCH_LIKE: 1 MiB + 1       */
  int64_t  device_capacity_bytes; /* INT64_MAX = unbounded                     */
} xmem_allocator_params;

enum { XMEM_PRESET_PAPER = 0, XMEM_PRESET_PYTORCH_LIKE = 1 };
#define XMEM_FLAGS_CHUNKS_MASK 0x3Fu

/* ------------------------------------------------------------------------
 * Per-trace result (96 bytes).  "Allocated" is the tensor series: the sum of
 * rounded request sizes r of live handles.  "Reserved" is the segment series:
 * the sum of sizes of segments currently held (Section 3.4, last paragraph).
 * All values describe the state after event stop_event-1 (or after the last
 * event when the trace ran to completion).
 * ---------------------------------------------------------------------- */
typedef struct {
  int64_t peak_allocated;         /* max over events of allocated               */
  int64_t peak_reserved;          /* max over events of reserved                */
  int64_t peak_allocated_event;   /* first event reaching the peak; -1 if 0     */
  int64_t peak_reserved_event;    /* first event reaching the peak; -1 if 0     */
  int64_t final_allocated;
  int64_t final_reserved;
  int64_t segments_created;
  int64_t segments_released;
  int64_t max_free_blocks_small;  /* max over events of #free blocks, SMALL pool */
  int64_t max_free_blocks_large;  /* same, LARGE pool                            */
  int64_t stop_event;             /* -1, or index (within trace) of the event that stopped it */
  int32_t status;                 /* XMEM_T_*                                    */
  int32_t reserved_;              /* 0                                           */
} xmem_trace_result;

/* per-trace status */
enum {
  XMEM_T_OK = 0,
  XMEM_T_OOM = 1,        /* capacity exceeded after reclamation                 */
  XMEM_T_BAD_FREE = 2,   /* free of a non-alloc, of a later event, or double free */
  XMEM_T_BAD_EVENT = 3,  /* undecodable word (size > 2^48, nonzero free bits)   */
  XMEM_T_OVERFLOW = 4,   /* segment bytes created in one pool would pass 2^61   */
  XMEM_T_BAD_BATCH = 5,  /* offsets array rejected on the device (async form)   */
  XMEM_T_ABORTED = 6     /* the chunked replay stopped at its safety time limit
                            (a wavefront waited 20 s for a task while no chain
                            finished) before this trace was done; the results
                            are not valid.  Not expected in practice.          */
};

/* call-level return codes */
enum {
  XMEM_OK = 0,
  XMEM_EINVAL = -1,      /* null pointer, negative count, invalid params        */
  XMEM_EOFFSETS = -2,    /* offsets[0] != 0, decreasing, trace too long, or offsets[n] != total */
  XMEM_EHIP = -3,        /* a HIP runtime call failed                           */
  XMEM_ENOMEM = -4,      /* device allocation failed (sync form only)           */
  XMEM_EWORKSPACE = -5,  /* workspace null or smaller than xmem_workspace_bytes */
  XMEM_ESCRATCH = -6     /* xmem_replay_batch_noalloc: the batch needs more workspace
                            than XMEM_NOALLOC_SCRATCH_BYTES                      */
};

/* Fill *p with the defaults of a preset.  Returns XMEM_OK or XMEM_EINVAL. */
int xmem_default_params(xmem_allocator_params* p, int preset);

/* XMEM_OK if *p is valid (rules above), else XMEM_EINVAL.  Host only. */
int xmem_validate_params(const xmem_allocator_params* p);

/* Bytes of device workspace xmem_replay_batch_ex needs for this batch:
 * about 86 bytes per event plus, for batches of 32 traces or more, a fixed
 * 268 MB of paged free-block sets for pools whose free blocks outgrow the
 * replay kernel's LDS table (less for fewer traces), plus the chunked
 * replay's task queue and chunk states (at most about 810 MB); for a single
 * trace, or two averaging 2^20 events or more, the chunks' own paged sets
 * instead, up to 8.4 MB per pool and chunk (one trace of 16.8M events:
 * 3.6 GB in all); for three or four traces averaging 2^20 events or more,
 * both (up to 4.2 GB of paged sets, for pools that spill).
 * Returns 0 on invalid arguments. */
size_t xmem_workspace_bytes(int64_t n_traces, int64_t total_events,
                            const xmem_allocator_params* params);

/* Synchronous replay (Section 3.4).
 *   d_events   : device, uint64[offsets[n_traces]], event words, trace t is
 *                d_events[offsets[t] .. offsets[t+1]).
 *   d_offsets  : device, int64[n_traces+1], offsets[0] == 0, non-decreasing,
 *                each trace at most XMEM_MAX_TRACE_EVENTS events.
 *   n_traces   : >= 0.
 *   params     : host pointer, validated.
 *   d_out      : device, xmem_trace_result[n_traces], written.
 * Copies the offsets to the host to validate them, allocates and frees its
 * own workspace, runs on the null stream and synchronises it.
 * Returns XMEM_OK or a negative XMEM_E* code; per-trace problems are reported
 * in d_out[t].status / stop_event and never fail the call. */
int xmem_replay_batch(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                      const xmem_allocator_params* params, xmem_trace_result* d_out);

/* Asynchronous replay on `hip_stream` (a hipStream_t; NULL = null stream).
 *   total_events     : must equal offsets[n_traces] (checked on the device).
 *   d_reserved_series: device int64[total_events] or NULL.  Entry e receives
 *                      the reserved bytes after event e of its trace, or -1
 *                      for events at or after the trace's stop_event.
 *   d_workspace      : device, >= xmem_workspace_bytes(...) bytes, 256-byte
 *                      aligned; contents are scratch (no initialisation needed).
 * No host synchronisation, no allocation.  Host-checkable errors are returned
 * immediately; if the offsets turn out invalid on the device, every trace is
 * reported with status XMEM_T_BAD_BATCH and stop_event 0. */
int xmem_replay_batch_ex(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                         int64_t total_events, const xmem_allocator_params* params,
                         xmem_trace_result* d_out, int64_t* d_reserved_series,
                         void* d_workspace, size_t workspace_bytes, void* hip_stream);

/* Same as xmem_replay_batch_ex, for measurement: additionally records the
 * caller-created events phase_events[0..XMEM_PHASE_EVENTS) (hipEvent_t) on
 * the stream at the phase boundaries:
 *   [0] before the plan and link-clearing kernel,
 *   [1] before the event-stream pass (decode, round, link, tensor series),
 *   [2] before the chunk planner of the chunked replay (nothing in between
 *       [2] and [3] for the serial replay),
 *   [3] before the allocator replay kernel (the segment series: the chunk
 *       scheduler, the serial replay, or the rounds of a batch of a few
 *       traces), the dominant kernel,
 *   [4] after it, before the fallback kernels (paged sets, 64-bit fields),
 *   [5] before the per-trace finalisation,
 *   [6] before the optional series expansion,
 *   [7] after the last kernel.
 * phase_events may be NULL (then it is exactly xmem_replay_batch_ex); else
 * n_phase_events must be >= XMEM_PHASE_EVENTS (XMEM_EINVAL otherwise). */
#define XMEM_PHASE_EVENTS 8
int xmem_replay_batch_ex_timed(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                               int64_t total_events, const xmem_allocator_params* params,
                               xmem_trace_result* d_out, int64_t* d_reserved_series,
                               void* d_workspace, size_t workspace_bytes, void* hip_stream,
                               void* const* phase_events, int n_phase_events);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): xmem_replay_batch_ex
 * with its workspace in a fixed area of XMEM_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on, from the first call on that GPU until
 * the process ends.  Same arguments, results and series as
 * xmem_replay_batch_ex, without the workspace; it runs on the current device,
 * whose stream hip_stream (a hipStream_t; NULL = null stream) must be.
 * When the workspace xmem_replay_batch_ex would take does not fit, the
 * batch is replayed serially (flags' chunk grain ignored) with fewer paged-set
 * slots, which changes only the speed; a batch that does not fit even then
 * (about 2.8 million events in all, fewer with many traces) is rejected with
 * XMEM_ESCRATCH before any device work.  Calls on one GPU share the area:
 * calls that overlap in time on the same GPU (on different streams or from
 * different threads) race and corrupt each other's results; calls ordered on
 * one stream are safe.  The first call on a GPU takes the area's device
 * address (hipGetSymbolAddress); no call allocates or frees device memory.
 * Returns as xmem_replay_batch_ex, plus XMEM_ESCRATCH. */
#define XMEM_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
int xmem_replay_batch_noalloc(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                              int64_t total_events, const xmem_allocator_params* params, xmem_trace_result* d_out,
                              int64_t* d_reserved_series, void* hip_stream);

/* OOM prediction (Section 4.1, Eq. (1)): an estimate predicts an out-of-
 * memory failure on a device whose maximum memory is M_max when the estimated
 * peak exceeds it, OOM-hat = [M-hat_peak > M_max].  The estimated peak is the
 * peak of the segment (reserved) series, the maximum Section 3.4 reports.
 *   d_results  : device, xmem_trace_result[n_traces], as a replay wrote them
 *                (read only).
 *   n_traces   : >= 0.
 *   m_max_bytes: the device's maximum memory in bytes, >= 0.
 *   d_flags    : device, int32[n_traces], written: 1 when the trace's replay
 *                stopped with XMEM_T_OOM (the simulated allocator failed at
 *                its own device_capacity_bytes, Section 3.4 (v)) or ran to
 *                completion with peak_reserved > m_max_bytes; 0 when it ran to
 *                completion with peak_reserved <= m_max_bytes; -1 when it
 *                stopped for any other reason (no estimate).  Replays meant for
 *                this test run with device_capacity_bytes unbounded or equal to
 *                m_max_bytes.
 * Asynchronous on hip_stream (a hipStream_t; NULL = null stream); allocates
 * nothing.  Returns XMEM_OK, XMEM_EINVAL (negative count or m_max, a null
 * pointer with n_traces > 0) or XMEM_EHIP. */
int xmem_oom_predicted(const xmem_trace_result* d_results, int64_t n_traces, int64_t m_max_bytes, int32_t* d_flags,
                       void* hip_stream);

/* Static description of a return code or status; never NULL. */
const char* xmem_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* XMEM_H */
