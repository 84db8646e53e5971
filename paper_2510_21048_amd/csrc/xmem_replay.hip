// xmem_replay.hip -- batched replay of allocate/free traces through the caching
// allocator model of xMem's Memory Simulator (Section 3.4), for gfx950.
//
// Pipeline of one call (all on the caller's stream, no host synchronisation):
//   k_plan      one workgroup checks the offsets, counts stream tiles per
//               trace (2048 events each) and their prefix, resets stop words;
//               the other workgroups zero the cross-tile link words.
//   k_stream    one workgroup per tile: decodes and validates each event word,
//               rounds the request (Section 3.4 (i)), classifies its pool,
//               links every allocation to its first free (inside the tile
//               through LDS; from a later tile by a plain store of an inverted
//               index), writes a 16-bit code per event, and reduces the tile's
//               allocated-bytes deltas under the monoid (sum, max prefix, first
//               argmax) -- the tensor series -- with a DPP wavefront scan.
//   k_cross_check  per tile: the frees of allocations in earlier tiles; an
//               allocation named by several frees is linked to the first, and
//               its trace stops at the second (double free).
//   k_replay_fast  one wavefront per allocator chain: the segment series.  A
//               chain is one (trace, pool) pair when the capacity is unbounded
//               (the pools never interact), else one trace.  The chain walks
//               the annotated stream in 64-event tiles with a one-tile
//               prefetch.  Each free block is one packed key (size, address)
//               held unordered in an LDS table (768 per pool; paged sorted sets
//               in HBM beyond): best fit (Section 3.4 (iii)) is a masked wavefront
//               minimum, splits and merges rewrite one slot, a new segment is
//               requested only when nothing fits (Section 3.4 (ii), (iv)), and
//               under a capacity idle segments are released before OOM is
//               declared (Section 3.4 (v)).  Allocated blocks reach their free
//               through a per-event mailbox (or lane registers for the last two
//               tiles).  The chain records only change points: each
//               reserved-bytes change and each new maximum of its free-block
//               count.  Keys hold 31-bit sizes and addresses (in granules);
//               a chain that needs more hands itself over to
//   k_replay_wide  the same replay with 64-bit fields (sorted VGPR table).
//   Under unbounded capacity the chains are cut into chunks replayed at once
//   (the chunk planner and the chunk scheduler below) with results identical
//   to the serial replay.
//   k_finalize  one wavefront per trace: resolves the stop event, combines
//               tile monoids up to it (re-reducing a partial tile; lanes, then
//               a DPP wavefront scan), and reads the change points as of the
//               stop (under a capacity, each lane over every 64th of them).
//   k_series    optional per-event reserved series, expanded from change points.
//
// Address model: each pool has its own bump pointer in units of the rounding
// granule; segments are laid out in creation order with a one-unit gap after
// each, so a free block ending exactly at a block's start, or starting exactly
// at its end, is its physical neighbour in the same segment.  Only the order
// of addresses within a pool is observable (best-fit ties), and creation order
// is preserved.  A per-pool table of created segments (bases ascending) tells
// whether a free block is a whole, idle segment.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "xmem.h"

// The workspace of xmem_replay_batch_noalloc (one copy per GPU, held until the process ends).
static __device__ __align__(256) unsigned char scratch[XMEM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 256;

constexpr int kStreamThreads = 256;
constexpr int kPerThread = 8;
constexpr int64_t kTile = kStreamThreads * kPerThread;  // events per stream tile
constexpr int kWave = 64;
constexpr int kLdsEntries = 512;                         // the 64-bit kernel: overflow entries per pool held in LDS

constexpr uint64_t kFreeBit = 1ull << 63;
constexpr uint64_t kMaxRequest = 1ull << 48;

// the op word of an event, rebuilt from its event word and code by annotate()
constexpr int kKindShift = 62;
constexpr uint64_t kKindAlloc = 1, kKindFree = 2;
constexpr uint64_t kPoolBit = 1ull << 61;
constexpr uint64_t kUnitsMask = (1ull << 61) - 1;

constexpr uint64_t kNoStop = ~0ull;

struct Derived {
  int shift;             // log2(round_bytes)
  uint64_t small_max_u, small_seg_u, mid_seg_u, min_large_u, large_round_u;
  uint64_t large_round_mask;  // large_round_u - 1 when it is a power of two (no division), else 0
  uint64_t split_min_u[2];
  uint64_t cap_u;        // floor(capacity / round)
  uint64_t limit_u;      // 2^61 / round: segment units ever created per pool
  int split_pools;       // pools replayed as independent chains
};

struct TilePart { int64_t s, m, i; };                  // i < 0: empty
struct TileInfo { int64_t base; int32_t t0, cnt, t, len; };  // a stream tile: its trace's first event, its offset and length in the trace, the trace and its length
struct ResRec { int64_t reserved; int32_t event, created, released, pad; };
struct MfRec { int32_t event, value; };
struct ChainHdr { int64_t stop; int32_t status, n_res, n_mf, pad; int64_t pad2; };
struct alignas(16) Blk { uint64_t a, s; };             // address, size, in units
struct ChunkRes { int64_t reserved; int32_t event, created; };  // a chunk's reserved change point
// chunked replay: per-chain progress, and what one chunk's replay reported
// per chain: frontier chunk, records stitched, running max free count, delta keys on top of the frontier's base state
// (few traces) mode: 0 first chunk, 1 speculative rounds, 2 the rest in one piece;
// big: on the paged sets; rounds: speculative rounds taken
// resume: 1 + the event a chain's first chunk spilled at, for its first round on the paged sets (0: none)
struct CCtl { int32_t f, done, n_res, n_mf, runmax, nd, mode, big, rounds, resume; };
// per chunk: stop, status, records, segments created, largest free-block count
struct CHdr { int64_t stop; int32_t status, n_res, n_mf, changed, maxc, pad; };
constexpr int kMaxDelta = 64;               // delta keys: the new segments of one chunk
constexpr int64_t kDeltaWords = kMaxDelta + 8;  // keys, then bump, created_u, reserved_u, created; then the
                                                // current round's chunks that created segments (a bit each)
constexpr int kRoundMask = kMaxDelta + 4;
constexpr int kMaxChunks = 63;
// one or two long traces (2^20 events or more on average) on the paged-set rounds (no
// scheduler): traces x chunks at most 127, so 2 x 127 workgroups of one wavefront, one per CU;
// the cut planner's share table has room for a single trace's 127 chunks.  Two such traces run
// there as fast as on the scheduler when no pool spills, and about 10x faster when their pools
// outgrow the LDS table (the scheduler hands those to the serial paged kernel); three or four
// would get 42 or 31 chunks each, 1.4-1.9x slower than the scheduler's 63 when none spills
constexpr int kMaxComboChunks = 127;
constexpr int64_t kFineEvents = 1 << 20;
constexpr int64_t kLongFewTraces = 2;
inline bool long_few(int64_t T, int64_t N) { return T >= 1 && T <= kLongFewTraces && N / T >= kFineEvents; }
constexpr int kCutSlots = kMaxComboChunks + 1;
// chunk end state: the free-table keys, then bump, created_u, reserved_u, (count | created << 32)
constexpr int kStateKeys = 768;
constexpr int64_t kStateWords = kStateKeys + 8;
constexpr int kSpecRounds = 8;  // speculative rounds before the rest of a chain is replayed in one piece
// the chunk planner's blocks: kPlanPer consecutive events per thread
constexpr int kPlanThreads = 256;
constexpr int kPlanPer = 8;
constexpr int64_t kPlanBlock = kPlanThreads * kPlanPer;
struct PlanAgg;
struct PlanChain;
// chunk scheduler control words, each in a 128-byte line of its own
constexpr int kQLine = 32;
constexpr int kQHead = 0;            // tickets drawn
constexpr int kQResv = kQLine;       // slots reserved by producers
constexpr int kQDone = 2 * kQLine;   // chains finished
constexpr int kQAbort = 3 * kQLine;  // set when a wavefront gave up waiting (safety time limit)
constexpr int kQFin = 4 * kQLine;    // tasks finished
constexpr int kQWords = 5 * kQLine;
// the scheduler's safety limit: a wavefront gives up after this long with no task running and no
// queue progress (a lost task would otherwise keep every waiting wavefront spinning)
constexpr uint64_t kSchedLimitSeconds = 20;

struct Ws {
  int32_t* ctl;          // [0]: offsets rejected
  int64_t* tile_base;    // T+1
  TilePart* tile_part;   // <= T + N/kTile + 1
  TileInfo* tinfo;       // per stream tile
  uint64_t* scnt;        // per stream tile: (trace << 32) | its frees that linked their allocations, listed in its mailbox slots
  uint64_t* stop_bad;    // T: (event << 8 | status), min over malformed events
  ChainHdr* hdr;         // 2T: [trace][pool]
  uint16_t* code;        // N: per event: kind, pool, and for an allocation freed in its own stream tile, that free's offset
  uint32_t* lx;          // N: per allocation freed from a later stream tile: ~ index of its first such free (0 = none)
  const uint64_t* ev;    // the caller's event words (set by the host after carving)
  Blk* mbox;             // N: block of the alloc, delivered to the slot of its free
  ResRec* res;           // N: reserved change points (pool 0 / single chain from the front, pool 1 from the back)
  MfRec* mf;             // N: free-count maxima (pool 0 front, pool 1 back)
  Blk* ovf;              // N: free blocks past the table capacity (pool 0 front, pool 1 back)
  Blk* segs;             // N: segments created (base, size) (pool 0 front, pool 1 back)
  uint64_t* big;         // paged-chain slots: sorted key pages of the chains replayed by k_replay_big
  // chunked replay (chunks > 1 only)
  int64_t* pblk_base;    // T+1: each trace's first planner block
  PlanAgg* pagg;         // per planner block: own events, coverage and never-freed run of each pool
  int64_t* ppre;         // per planner block: 4 prefixes (own events of pool 0, 1; coverage of pool 0, 1)
  PlanChain* pchain;     // 2T: a chain's own events, gap and chunk count
  uint64_t* pshare;      // 2T x (chunks + 1): smallest clean key per share; [chunks]: last key short of share 1
  int32_t* cbound;       // 2T x (chunks + 1): chunk boundaries (event indices) of each chain
  int32_t* cnum;         // 2T: chunks of each chain
  int32_t* cown;         // 2T x (chunks + 1): the chain's own events before each boundary
  CCtl* cctl;            // 2T
  CHdr* chdr;            // 2T x chunks
  uint64_t* cst;         // 2T x chunks x kStateWords: end state of each chunk
  uint32_t* cg;          // paged chunks: 2T x chunks x 64: choice summary of each chunk (k_chunk_stitch)
  uint64_t* cdel;        // 2T x kDeltaWords: the frontier's delta keys and counters (certified chunks)
  // the chunk scheduler (many traces): the task queue, its control words, pending tasks per chain
  uint64_t* cq;          // cq_cap task words
  uint32_t* cqc;         // kQWords control words (tickets, reservations, chains done, abort flag)
  int32_t* cpend;        // 6T: [0, 2T) tasks of the chain's current round not yet finished; [2T, 4T) the
                         // round's first chunk that stopped, or in a large pool created segments (none: past
                         // the last); [4T, 6T) the round's first chunk neither queued nor given up yet
  int64_t cq_cap;
  int chunks;
  // chunked replay on the paged sets (a few traces only: every (chain, chunk) has its own slot)
  uint64_t* bslot;       // 2T x chunks x bslot_keys: working pages
  uint64_t* bstate;      // 2T x chunks x bstate_words: end state (scalars, then both sets' keys in order)
  int32_t bcap;          // directory entries per set (0: no chunked paged replay)
  int64_t bslot_keys, bstate_keys, bstate_words;
  int32_t nbig;          // paged-chain slots: workgroups of k_replay_big
};

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// paged-chain slots (see k_replay_big): keys per slot, and slots for T traces
constexpr int64_t kBigSlotKeysHost = 4 * (2048 + 2) * 64;
inline int64_t big_slots(int64_t T) { return 2 * T < 64 ? 2 * T : 64; }
// chunked replay on the paged sets: at most this many (chain, chunk) slots (one or two long
// traces: 2 x kMaxComboChunks); a set's
// directory holds N / 16 + 8 pages (a pool never has more free blocks than its trace
// has events), at most the serial kernel's 4096
constexpr int64_t kBigChunkMax = 128;
constexpr int64_t kBigDirMaxHost = 4096;
// the batch's rounds run on the paged-set kernels alone (few traces) rather than the scheduler
inline bool combo_main(int64_t T, int64_t N, int K) {
  return K > 1 && (2 * T * K <= kBigChunkMax || (long_few(T, N) && T * K <= kMaxComboChunks));
}
// up to four traces averaging 2^20 events or more that run the scheduler keep paged slots as
// well: a pool that spills there takes the paged-set rounds afterwards, not the serial paged
// kernel (at 63 chunks: 8 x 63 slots of at most 8.4 MB)
constexpr int64_t kSpillRoundTraces = 4;
inline bool combo_after(int64_t T, int64_t N, int K) {
  return K > 1 && !combo_main(T, N, K) && T <= kSpillRoundTraces && N / T >= kFineEvents;
}
inline int32_t bigc_cap(int64_t T, int64_t N, int K) {
  if (!combo_main(T, N, K) && !combo_after(T, N, K)) return 0;
  const int64_t c = N / 16 + 8;
  return (int32_t)(c < kBigDirMaxHost ? c : kBigDirMaxHost);
}

inline size_t carve(void* base, int64_t T, int64_t N, int K, Ws* w, int64_t nbig = -1) {
  if (nbig < 0) nbig = big_slots(T);
  const int64_t max_tiles = T + N / kTile + 1;
  size_t o = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) { char* p = b ? b + o : nullptr; o += align256(bytes); return p; };
  Ws x;
  x.ctl = reinterpret_cast<int32_t*>(take(256));
  x.tile_base = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (T + 1)));
  x.tile_part = reinterpret_cast<TilePart*>(take(sizeof(TilePart) * max_tiles));
  x.tinfo = reinterpret_cast<TileInfo*>(take(sizeof(TileInfo) * max_tiles));
  x.scnt = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * max_tiles));
  x.stop_bad = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * T));
  x.hdr = reinterpret_cast<ChainHdr*>(take(sizeof(ChainHdr) * 2 * T));
  x.code = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * N));
  x.lx = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * N));
  x.ev = nullptr;
  x.mbox = reinterpret_cast<Blk*>(take(sizeof(Blk) * N));
  x.res = reinterpret_cast<ResRec*>(take(sizeof(ResRec) * N));
  x.mf = reinterpret_cast<MfRec*>(take(sizeof(MfRec) * N));
  x.ovf = reinterpret_cast<Blk*>(take(sizeof(Blk) * N));
  x.segs = reinterpret_cast<Blk*>(take(sizeof(Blk) * N));
  x.big = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * kBigSlotKeysHost * nbig));
  x.nbig = (int32_t)nbig;
  x.chunks = K;
  x.pblk_base = x.ppre = nullptr;
  x.pagg = nullptr;
  x.pchain = nullptr;
  x.pshare = nullptr;
  x.cbound = x.cnum = x.cown = nullptr;
  x.cctl = nullptr;
  x.chdr = nullptr;
  x.cst = nullptr;
  x.cg = nullptr;
  x.cdel = nullptr;
  x.cq = nullptr;
  x.cqc = nullptr;
  x.cpend = nullptr;
  x.cq_cap = 0;
  x.bslot = x.bstate = nullptr;
  x.bcap = bigc_cap(T, N, K);
  x.bslot_keys = x.bstate_keys = x.bstate_words = 0;
  if (x.bcap > 0) {
    x.bslot_keys = 2 * (int64_t)(x.bcap + 2) * 64;
    const int64_t keys = (int64_t)x.bcap * 64 < N + 64 ? (int64_t)x.bcap * 64 : N + 64;
    x.bstate_keys = keys;
    x.bstate_words = 8 + 2 * keys;
    x.bslot = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * x.bslot_keys * 2 * T * K));
    x.bstate = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * x.bstate_words * 2 * T * K));
  }
  if (K > 1) {
    const int64_t blocks = T + N / kPlanBlock + 1;  // planner blocks: at most one partial block per trace
    x.pblk_base = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (T + 1)));
    x.pagg = reinterpret_cast<PlanAgg*>(take(96 * blocks));
    x.ppre = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * 4 * blocks));
    x.pchain = reinterpret_cast<PlanChain*>(take(32 * 2 * T));
    x.pshare = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * 2 * T * (K + 1)));
    x.cbound = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 2 * T * (K + 1)));
    x.cnum = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 2 * T));
    x.cown = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 2 * T * (K + 1)));
    x.cctl = reinterpret_cast<CCtl*>(take(sizeof(CCtl) * 2 * T));
    x.chdr = reinterpret_cast<CHdr*>(take(sizeof(CHdr) * 2 * T * K));
    x.cst = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * kStateWords * 2 * T * K));
    x.cdel = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * kDeltaWords * 2 * T));
    if (x.bcap > 0) x.cg = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * 64 * 2 * T * K));
    if (!combo_main(T, N, K)) {  // a chain takes at most one task per round: 1 + kSpecRounds * K + 1
      x.cq_cap = 2 * T * (kSpecRounds * (int64_t)K + 2);
      x.cq = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * x.cq_cap));
      x.cqc = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * kQWords));
      x.cpend = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 6 * T));
    }
  }
  if (w) *w = x;
  return o;
}

// ------------------------------------------------------------------ address spaces
// Kernel code reaches the workspace through explicitly global (addrspace 1)
// and LDS (addrspace 3) pointers so that every access compiles to a global_*
// or ds_* instruction rather than a flat one.
#define GMEM __attribute__((address_space(1)))
#define LMEM __attribute__((address_space(3)))

template <class T>
__device__ __forceinline__ GMEM T* gp(T* p) { return (GMEM T*)p; }
template <class T>
__device__ __forceinline__ const GMEM T* gp(const T* p) { return (const GMEM T*)p; }

struct Gw {
  GMEM int32_t* ctl;
  GMEM int64_t* tile_base;
  GMEM TilePart* tile_part;
  GMEM TileInfo* tinfo;
  GMEM uint64_t* stop_bad;
  GMEM ChainHdr* hdr;
  GMEM uint16_t* code;
  GMEM uint32_t* lx;
  const GMEM uint64_t* ev;
  GMEM Blk* mbox;
  GMEM ResRec* res;
  GMEM MfRec* mf;
  GMEM Blk* ovf;
  GMEM Blk* segs;
  GMEM uint64_t* big;
  GMEM int64_t* pblk_base;
  GMEM PlanAgg* pagg;
  GMEM int64_t* ppre;
  GMEM PlanChain* pchain;
  GMEM uint64_t* pshare;
  GMEM int32_t* cbound;
  GMEM int32_t* cnum;
  GMEM int32_t* cown;
  GMEM CCtl* cctl;
  GMEM CHdr* chdr;
  GMEM uint64_t* cst;
  GMEM uint32_t* cg;
  GMEM uint64_t* cdel;
  GMEM uint64_t* cq;
  GMEM uint32_t* cqc;
  GMEM int32_t* cpend;
  int64_t cq_cap;
  int chunks;
  GMEM uint64_t* bslot;
  GMEM uint64_t* bstate;
  int32_t bcap;
  int64_t bslot_keys, bstate_keys, bstate_words;
};
// whole-struct copies to and from global memory, 8 bytes at a time
template <class T>
__device__ __forceinline__ T gload(const GMEM T* p) {
  static_assert(sizeof(T) % 8 == 0, "8-byte multiple");
  T v;
  const GMEM uint64_t* q = (const GMEM uint64_t*)p;
  uint64_t* d = reinterpret_cast<uint64_t*>(&v);
#pragma unroll
  for (size_t i = 0; i < sizeof(T) / 8; ++i) d[i] = q[i];
  return v;
}
template <class T>
__device__ __forceinline__ void gstore(GMEM T* p, const T& v) {
  static_assert(sizeof(T) % 8 == 0, "8-byte multiple");
  GMEM uint64_t* q = (GMEM uint64_t*)p;
  const uint64_t* d = reinterpret_cast<const uint64_t*>(&v);
#pragma unroll
  for (size_t i = 0; i < sizeof(T) / 8; ++i) q[i] = d[i];
}

__device__ __forceinline__ Gw typed(const Ws& w) {
  return Gw{gp(w.ctl),  gp(w.tile_base), gp(w.tile_part), gp(w.tinfo), gp(w.stop_bad), gp(w.hdr),  gp(w.code),
            gp(w.lx),   gp(w.ev),        gp(w.mbox),      gp(w.res),       gp(w.mf),       gp(w.ovf),  gp(w.segs),
            gp(w.big),  gp(w.pblk_base), gp(w.pagg),      gp(w.ppre),     gp(w.pchain), gp(w.pshare),
            gp(w.cbound), gp(w.cnum),    gp(w.cown),      gp(w.cctl),     gp(w.chdr),
            gp(w.cst),  gp(w.cg),        gp(w.cdel),      gp(w.cq),       gp(w.cqc),  gp(w.cpend), w.cq_cap,
            w.chunks,   gp(w.bslot),     gp(w.bstate),    w.bcap,
            w.bslot_keys,
            w.bstate_keys,  w.bstate_words};
}

// ------------------------------------------------------------------ wave helpers
__device__ __forceinline__ uint32_t rl(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}
__device__ __forceinline__ uint64_t rl64(uint64_t v, int lane) {
  return (uint64_t)rl((uint32_t)v, lane) | ((uint64_t)rl((uint32_t)(v >> 32), lane) << 32);
}
// v with lane `lane` replaced by the wave-uniform value val
__device__ __forceinline__ uint64_t wl64(uint64_t val, int lane, uint64_t v) {
  return (int)threadIdx.x == lane ? val : v;
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
// Orders this wavefront's memory operations as written (single-wavefront
// workgroups: the hardware keeps a wavefront's accesses in order).
__device__ __forceinline__ void wave_order() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  const uint32_t lo = dpp<CTRL>((uint32_t)v), hi = dpp<CTRL>((uint32_t)(v >> 32));
  return (uint64_t)lo | ((uint64_t)hi << 32);
}
__device__ __forceinline__ uint64_t from_lower_lane(uint64_t v) { return dpp64<0x138>(v); }  // wave_shr:1
__device__ __forceinline__ uint64_t from_upper_lane(uint64_t v) { return dpp64<0x130>(v); }  // wave_shl:1
// v from a DPP permutation in which every lane has a source lane (no old value
// kept), so the move can fold into the instruction that uses it
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_perm(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xf, 0xf, true);
}
// minimum over all 64 lanes (all lanes active); finishing with row broadcasts
// (row_bcast:15, :31) and one read of lane 63 instead of four reads measured slower
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  v = min(v, dpp_perm<0xB1>(v));   // quad_perm [1,0,3,2]
  v = min(v, dpp_perm<0x4E>(v));   // quad_perm [2,3,0,1]
  v = min(v, dpp_perm<0x141>(v));  // row_half_mirror
  v = min(v, dpp_perm<0x140>(v));  // row_mirror
  return min(min(rl(v, 0), rl(v, 16)), min(rl(v, 32), rl(v, 48)));
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  const uint32_t hi = wave_min_u32((uint32_t)(v >> 32));
  const uint32_t lo = wave_min_u32((uint32_t)(v >> 32) == hi ? (uint32_t)v : 0xffffffffu);
  return ((uint64_t)hi << 32) | lo;
}
__device__ uint64_t wave_sum_u64(uint64_t v) {
  uint64_t s = 0;
  for (int l = 0; l < kWave; ++l) s += rl64(v, l);
  return s;
}

// ------------------------------------------------------------------ monoid of the tensor series
// (sum, max prefix, first index of the max prefix) over a run of deltas; i < 0 is
// the empty run.  Associative, so tiles reduce independently and combine in order.
__device__ __forceinline__ TilePart tp_combine(TilePart a, TilePart b) {
  if (a.i < 0) return b;
  if (b.i < 0) return a;
  TilePart r;
  r.s = (int64_t)((uint64_t)a.s + (uint64_t)b.s);
  const int64_t cand = (int64_t)((uint64_t)a.s + (uint64_t)b.m);
  if (a.m >= cand) { r.m = a.m; r.i = a.i; } else { r.m = cand; r.i = b.i; }
  return r;
}

// Workgroups are dispatched round-robin over the chip's 8 XCDs, each with its own L2.  A grid of
// 8 * per workgroups over items [0, 8 * per) maps workgroup b to item (b % 8) * per + b / 8, so
// that each XCD takes a contiguous eighth of the items, in order: a stream tile's gathers then
// find the earlier tiles of its trace in the L2 of the XCD that just read them.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_item(int64_t b, int64_t grid) {
  const int64_t per = grid / kXcds;
  return (b % kXcds) * per + b / kXcds;
}
inline int64_t xcd_grid(int64_t items) { return (items + kXcds - 1) / kXcds * kXcds; }

// ------------------------------------------------------------------ k_plan
// Block 0 plans; the other blocks zero the link words meanwhile.
__global__ __launch_bounds__(1024) void k_plan(const int64_t* off_, int64_t T, int64_t N, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  const int tid = threadIdx.x;
  if (blockIdx.x > 0) {
    for (int64_t i = (int64_t)(blockIdx.x - 1) * 1024 + tid; i < N; i += (int64_t)(gridDim.x - 1) * 1024) w.lx[i] = 0;
    return;
  }
  __shared__ int64_t part[1024];
  __shared__ int64_t ppart[1024];  // planner blocks (chunked replay)
  __shared__ int64_t wsum[16], wpsum[16];
  __shared__ int bad;
  if (tid == 0) bad = 0;
  __syncthreads();
  const int64_t per = (T + 1023) / 1024;
  const int64_t lo = min<int64_t>(T, (int64_t)tid * per), hi = min<int64_t>(T, lo + per);
  int64_t cnt = 0, pcnt = 0;
  int mybad = 0;
  for (int64_t t = lo; t < hi; ++t) {
    const int64_t len = off[t + 1] - off[t];
    if (len < 0 || len > XMEM_MAX_TRACE_EVENTS) {
      mybad = 1;
    } else {
      cnt += (len + kTile - 1) / kTile;
      pcnt += (len + kPlanBlock - 1) / kPlanBlock;
    }
    w.stop_bad[t] = kNoStop;
  }
  if (tid == 0 && (off[0] != 0 || off[T] != N)) mybad = 1;
  if (mybad) atomicOr(&bad, 1);
  // exclusive prefix sums of the per-thread counts: wavefront scans, then one over the 16 wavefront sums
  const int lane = tid & 63, wv = tid >> 6;
  int64_t x = cnt, px = pcnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o, 64), py = __shfl_up(px, o, 64);
    if (lane >= o) { x += y; px += py; }
  }
  if (lane == 63) { wsum[wv] = x; wpsum[wv] = px; }
  __syncthreads();
  if (wv == 0) {
    int64_t a = lane < 16 ? wsum[lane] : 0, pa = lane < 16 ? wpsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int64_t y = __shfl_up(a, o, 64), py = __shfl_up(pa, o, 64);
      if (lane >= o) { a += y; pa += py; }
    }
    if (lane < 16) { wsum[lane] = a; wpsum[lane] = pa; }
    if (lane == 15) {
      w.tile_base[T] = a;
      if (w.pblk_base) w.pblk_base[T] = pa;
    }
  }
  __syncthreads();
  if (tid == 0) w.ctl[0] = bad;
  int64_t acc = x - cnt + (wv > 0 ? wsum[wv - 1] : 0), pacc = px - pcnt + (wv > 0 ? wpsum[wv - 1] : 0);
  for (int64_t t = lo; t < hi; ++t) {
    w.tile_base[t] = acc;
    if (w.pblk_base) w.pblk_base[t] = pacc;
    const int64_t len = off[t + 1] - off[t];
    if (len >= 0 && len <= XMEM_MAX_TRACE_EVENTS) {
      acc += (len + kTile - 1) / kTile;
      pacc += (len + kPlanBlock - 1) / kPlanBlock;
    }
  }

}

// After k_plan: the record of each stream tile (its trace, the trace's first event, the tile's
// offset and length in it), one thread per tile, by a binary search over the tile bases.
__global__ __launch_bounds__(256) void k_tile_info(const int64_t* off_, int64_t T, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t tile = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tile >= w.tile_base[T]) return;
  int64_t lo = 0, hi = T - 1;  // the last trace whose first tile is at or before this one
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (w.tile_base[mid] <= tile) lo = mid; else hi = mid - 1;
  }
  const int64_t k = tile - w.tile_base[lo], b0 = off[lo], len = off[lo + 1] - b0;
  gstore(&w.tinfo[tile], TileInfo{b0, (int32_t)(k * kTile), (int32_t)min<int64_t>(kTile, len - k * kTile), (int32_t)lo, (int32_t)len});
}

// The largest t in [0, T) with first[t] <= x, where first is non-decreasing and first[0] = 0 <= x
// (the trace owning a tile or planner block), found by one whole wavefront: each round probes 64
// evenly spaced entries at once, so a batch of up to 4096 traces takes two rounds of loads where a
// binary search takes one dependent load per halving.
__device__ int64_t wave_find(const GMEM int64_t* first, int64_t T, int64_t x) {
  const int lane = threadIdx.x & 63;
  int64_t lo = 0, hi = T - 1;
  while (lo < hi) {
    const int64_t step = (hi - lo + 64) / 64;
    const int64_t p = lo + lane * step;
    const uint64_t m = __builtin_amdgcn_ballot_w64(p <= hi && first[p] <= x);  // lane 0: first[lo] <= x
    const int64_t nlo = lo + (63 - __builtin_clzll(m)) * step;
    hi = min<int64_t>(hi, nlo + step - 1);
    lo = nlo;
  }
  return lo;
}

// ------------------------------------------------------------------ k_stream
__device__ __forceinline__ void mark_bad(GMEM uint64_t* stop_bad, int64_t t, int64_t e, int status) {
  __hip_atomic_fetch_min(&stop_bad[t], ((uint64_t)e << 8) | (uint64_t)status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The 16-bit code k_stream writes for each event: what the replay and the planner take from it,
// beside the event word itself.
constexpr uint32_t kCodeKind = 3;    // 0: nothing to replay (no-op or malformed), 1: allocation, 2: free
constexpr uint32_t kCodeAlloc = 1, kCodeFree = 2;
constexpr uint32_t kCodePool = 4;    // the (freed) block's pool is LARGE
constexpr uint32_t kCodeInTile = 8;  // an allocation freed in its own stream tile; bits 15:4: its first such free's offset
constexpr uint32_t kNoOff = 0xffffu;
static_assert(kTile <= 4096, "an in-tile offset takes 12 bits");

// A DPP move of a 64-bit value; lanes with no source lane (a row edge, or a row the mask leaves
// out) take `old`.
template <int CTRL, int ROWS>
__device__ __forceinline__ int64_t dpp_move(int64_t old, int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)old, (int)(uint32_t)v, CTRL, ROWS, 0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)((uint64_t)old >> 32),
                                                            (int)(uint32_t)((uint64_t)v >> 32), CTRL, ROWS, 0xf, false);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ TilePart tp_scan_step(TilePart x) {
  const TilePart y{dpp_move<CTRL, ROWS>(0, x.s), dpp_move<CTRL, ROWS>(0, x.m), dpp_move<CTRL, ROWS>(-1, x.i)};
  return tp_combine(y, x);  // the earlier lanes' part first (an empty part where there is none)
}
// Inclusive scan of the monoid up the wavefront in lane order, on DPP alone: shifts by 1, 2, 4
// and 8 lanes within each row of 16, then row 0's total into row 1 and row 2's into row 3
// (row_bcast:15), then rows 0-1's total into rows 2-3 (row_bcast:31).  Lane 63 ends with the
// reduction of all 64 lanes.  All lanes active.
__device__ __forceinline__ TilePart tp_wave_scan(TilePart x) {
  x = tp_scan_step<0x111, 0xf>(x);  // row_shr:1
  x = tp_scan_step<0x112, 0xf>(x);  // row_shr:2
  x = tp_scan_step<0x114, 0xf>(x);  // row_shr:4
  x = tp_scan_step<0x118, 0xf>(x);  // row_shr:8
  x = tp_scan_step<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x = tp_scan_step<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}
__device__ __forceinline__ TilePart tp_lane(TilePart x, int lane) {
  return TilePart{(int64_t)rl64((uint64_t)x.s, lane), (int64_t)rl64((uint64_t)x.m, lane), (int64_t)rl64((uint64_t)x.i, lane)};
}

// A wavefront's reduction of non-empty parts of the monoid (the event index in 32 bits), in lane
// order, taken by the steps of the scan above.  Lane 63's result only ever combines lanes that
// have a source lane at every step, so the lanes that have none may hold anything: no empty part
// and no initial value for the moves, and one compare and three selects per step.
struct WavePart { int64_t s, m; uint32_t i; };
__device__ __forceinline__ WavePart wp_join(WavePart a, WavePart b) {  // a: the earlier run
  const int64_t cand = (int64_t)((uint64_t)a.s + (uint64_t)b.m);
  const bool keep = a.m >= cand;
  return WavePart{(int64_t)((uint64_t)a.s + (uint64_t)b.s), keep ? a.m : cand, keep ? a.i : b.i};
}
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_any(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, ROWS, 0xf, false);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ WavePart wp_step(WavePart x) {
  const WavePart y{(int64_t)(((uint64_t)dpp_any<CTRL, ROWS>((uint32_t)((uint64_t)x.s >> 32)) << 32) | dpp_any<CTRL, ROWS>((uint32_t)x.s)),
                   (int64_t)(((uint64_t)dpp_any<CTRL, ROWS>((uint32_t)((uint64_t)x.m >> 32)) << 32) | dpp_any<CTRL, ROWS>((uint32_t)x.m)),
                   dpp_any<CTRL, ROWS>(x.i)};
  return wp_join(y, x);
}
__device__ __forceinline__ WavePart wp_wave_reduce(WavePart x) {  // valid in lane 63 only
  x = wp_step<0x111, 0xf>(x);  // row_shr:1
  x = wp_step<0x112, 0xf>(x);  // row_shr:2
  x = wp_step<0x114, 0xf>(x);  // row_shr:4
  x = wp_step<0x118, 0xf>(x);  // row_shr:8
  x = wp_step<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x = wp_step<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}
// Inclusive sum of a 32-bit count up the wavefront in lane order (the same steps; lanes with no
// source lane add zero).
__device__ __forceinline__ uint32_t wave_incl_sum_u32(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);
  return x;
}

// One workgroup per 2048-event tile of one trace (a1-a3), its position from the tile record
// k_plan wrote.  Each thread loads its 8 consecutive words directly (four 16-byte loads), and for
// each free its allocation's word with one gather (from the cache when the allocation lies in
// the tile); every load is unconditional, with an address clamped into the tile where a lane has
// nothing to load, so that all of them are in flight at once.  Each event is then decoded,
// validated and rounded (Section 3.4 (i)) and its pool classified with selects.  A free links
// its allocation to itself: inside the tile by an LDS atomic minimum, so that the allocation's
// code carries its first free's offset and a repeated free stops the trace at the later of two
// (every lane issues the eight of its thread with no branch, a lane with no in-tile link on a
// spare word of its own, so that no two lanes of an instruction contend for one address); across
// tiles by a plain store of its inverted index, the free listed for k_cross_check at a position
// from a DPP sum over the wavefront and one LDS reservation per wavefront.  The tile's deltas of the tensor series reduce under the monoid (sum, max prefix,
// first argmax): each thread over its 8 events, a DPP reduction over each wavefront, then the 4
// wavefronts in order.  Out: the 16-bit codes (one 16-byte store per thread), the tile's monoid
// and its count of listed frees.
__global__ __launch_bounds__(kStreamThreads) void k_stream(const uint64_t* ev_, const int64_t* off_, int64_t T, Derived d,
                                                            Ws ws) {
  const Gw w = typed(ws);
  const GMEM uint64_t* ev = gp(ev_);
  (void)off_;
  if (w.ctl[0]) return;
  const int64_t tile = xcd_item(blockIdx.x, gridDim.x);
  if (tile >= w.tile_base[T]) return;
  __shared__ uint32_t s_first[kTile + kWave];  // per event: the offset of the first in-tile free of it (kNoOff:
                                               // none); then one spare word per lane, for lanes with no in-tile link
  __shared__ TilePart s_part[kStreamThreads / kWave];
  __shared__ uint32_t s_nx;            // frees of allocations in earlier tiles, listed
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const TileInfo ti = gload(&w.tinfo[tile]);
  const int64_t base = ti.base, t0 = ti.t0, cnt = ti.cnt, n = t0 + cnt, t = ti.t;
  const uint64_t gmask = (1ull << d.shift) - 1;
  typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
  uint64_t wd[kPerThread], wh[kPerThread];
  int32_t hh[kPerThread];  // a free's allocation (an index below the free's, so below 2^31), else -1
  {
    // this thread's 8 words; past the tile's end, zero words (a zero word is an allocation of 0
    // bytes: no code, no link, a zero delta)
    const bool live = (int64_t)tid * kPerThread < cnt;
    const int64_t i0 = live ? (int64_t)tid * kPerThread : 0;
    const GMEM u64x2* src = (const GMEM u64x2*)(ev + base + t0 + i0);
#pragma unroll
    for (int q = 0; q < kPerThread / 2; ++q) {
      const bool inb = live && i0 + 2 * q + 1 < cnt;  // the tile's last word pair may be partial
      const u64x2 v = inb ? src[q] : u64x2{0, 0};
      wd[2 * q] = v.x;
      wd[2 * q + 1] = v.y;
    }
    if ((int64_t)tid * kPerThread < cnt && cnt - (int64_t)tid * kPerThread < kPerThread) {
      // the thread holding the tile's ragged end: its words one by one
#pragma unroll
      for (int j = 0; j < kPerThread; ++j) wd[j] = (int64_t)tid * kPerThread + j < cnt ? ev[base + t0 + tid * kPerThread + j] : 0;
    }
  }
  // event indices within the trace stay below 2^31: 32-bit arithmetic; conditions as 0/1 words
  // combined with bit operations, so that the decode compiles to straight-line vector code
  const uint32_t e0 = (uint32_t)t0 + (uint32_t)tid * kPerThread;
  const uint32_t ut0 = (uint32_t)t0;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    s_first[j * kStreamThreads + tid] = kNoOff;
    const uint32_t le = e0 + j, hi = (uint32_t)(wd[j] >> 32), lo = (uint32_t)wd[j];
    // a well-formed free of an earlier event: its allocation's index, else -1
    const uint32_t ok = (hi >> 31) & ((hi & 0x7fffffffu) == 0) & (lo < le);
    hh[j] = ok ? (int32_t)lo : -1;
  }
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) wh[j] = ev[base + (hh[j] >= 0 ? (int64_t)hh[j] : t0)];  // the allocations, all at once
  if (tid == 0) s_nx = 0;
  __syncthreads();
  GMEM uint64_t* lst = (GMEM uint64_t*)w.mbox + base + t0;  // the mailbox area is free until the replay
  int64_t rs = 0, rm = 0;
  uint32_t ri = 0;                             // the running monoid: sum, max prefix, its first event
  uint32_t bad_le = 0xffffffffu, bad_st = 0;   // the thread's earliest malformed event and its status
  uint32_t anybad = 0;                         // some event of the thread is malformed
  uint32_t pk[kPerThread / 2];                 // this thread's 8 codes, two per word
  uint32_t ncross = 0, crossm = 0;             // frees of allocations in earlier tiles: count and which of the 8
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const uint32_t le = e0 + j;
    const uint64_t x = wd[j];
    const uint32_t hi = (uint32_t)(x >> 32), lo = (uint32_t)x, isfree = hi >> 31;
    const uint32_t hok = hh[j] >= 0;  // a well-formed free of an earlier event
    const uint64_t al = wh[j];        // its allocation's word (meaningful only with hok)
    const uint32_t al_free = (uint32_t)(al >> 63), al_big = al > kMaxRequest, x_big = x > kMaxRequest;
    const uint32_t linked = hok & (al_free ^ 1u) & (al_big ^ 1u);
    const uint64_t u = ((isfree ? al : x) + gmask) >> d.shift;  // Section 3.4 (i): round up to the granule
    const uint32_t sized = (isfree ? linked : x_big ^ 1u) & (u != 0);
    const uint32_t code = sized ? (isfree ? kCodeFree : kCodeAlloc) | (u > d.small_max_u ? kCodePool : 0u) : 0u;
    const int64_t r = (int64_t)(u << d.shift);
    const int64_t delta = sized ? (isfree ? -r : r) : 0;
    // malformed: a free with bits above the index, of a later event or of a free; a huge request
    // (located exactly after the loop, in the rare thread that has one)
    anybad |= isfree ? (hok ^ 1u) | al_free : x_big;
    // the tensor series: the running (sum, max prefix, first index of the max).  A thread past
    // the tile's end ends with (0, 0, its first index), which leaves every combination it enters
    // unchanged (the max prefix is never below the sum, and a tie keeps the earlier index).
    const int64_t ns = rs + delta;
    const bool take = j == 0 || ns > rm;
    rm = take ? ns : rm;
    ri = take ? le : ri;
    rs = ns;
    // in-tile link: the earliest free of each allocation of the tile; a second one stops the trace
    {
      const uint32_t intile = linked & (lo >= ut0);
      const uint32_t old = atomicMin(&s_first[intile ? lo - ut0 : (uint32_t)(kTile + lane)], le - ut0);
      if (intile && old != kNoOff) {  // the later of the two frees is malformed; keep the earliest such event
        const uint32_t second = le > ut0 + old ? le : ut0 + old;
        const uint32_t k = second < bad_le;
        bad_st = k ? XMEM_T_BAD_FREE : bad_st;
        bad_le = k ? second : bad_le;
      }
    }
    const uint32_t cross = linked & (lo < ut0);
    ncross += cross;
    crossm |= cross << j;
    if (j & 1) pk[j >> 1] |= code << 16;
    else pk[j >> 1] = code;
  }
  if (ballot(anybad)) {  // rare: the earliest malformed event of each thread that has one
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const uint32_t le = e0 + j, hi = (uint32_t)(wd[j] >> 32), isfree = hi >> 31;
      const uint32_t fbits = (hi & 0x7fffffffu) != 0, hok = hh[j] >= 0;
      const uint32_t bad_event = isfree ? fbits : (uint32_t)(wd[j] > kMaxRequest);
      const uint32_t bad_free = isfree & (fbits ^ 1u) & ((hok ^ 1u) | (hok ? (uint32_t)(wh[j] >> 63) : 0u));
      if ((bad_event | bad_free) && le < bad_le) {
        bad_le = le;
        bad_st = bad_event ? XMEM_T_BAD_EVENT : XMEM_T_BAD_FREE;
      }
    }
  }
  // cross-tile links: a plain store of the inverted free index, and the tile's list for
  // k_cross_check (one LDS reservation per wavefront, by its last lane)
  const uint32_t nx_incl = wave_incl_sum_u32(ncross);
  uint32_t wbase = 0;
  if (lane == 63 && nx_incl) wbase = atomicAdd(&s_nx, nx_incl);
  wbase = __builtin_amdgcn_readlane(wbase, 63);
  if (crossm) {
    uint32_t pos = wbase + nx_incl - ncross;
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      if (crossm & (1u << j)) {
        const uint32_t le = e0 + j;
        w.lx[base + hh[j]] = 0xffffffffu - le;
        lst[pos++] = ((uint64_t)le << 32) | (uint64_t)(uint32_t)hh[j];
      }
    }
  }
  if (ballot(bad_le != 0xffffffffu)) {  // rare: malformed events stop their trace at the earliest
    if (bad_le != 0xffffffffu) mark_bad(w.stop_bad, t, (int64_t)bad_le, (int)bad_st);
  }
  const WavePart acc = wp_wave_reduce(WavePart{rs, rm, ri});
  if (lane == 63) s_part[wv] = TilePart{acc.s, acc.m, (int64_t)acc.i};
  __syncthreads();
  // codes out: an allocation freed in the tile carries its first free's offset; one 16-byte store
  if ((int64_t)tid * kPerThread < cnt) {
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const uint32_t fo = s_first[tid * kPerThread + j];
      const uint32_t add = fo != kNoOff ? kCodeInTile | (fo << 4) : 0u;
      pk[j >> 1] |= (j & 1) ? add << 16 : add;
    }
    GMEM uint16_t* cd = w.code + base + t0 + tid * kPerThread;
    if (cnt - (int64_t)tid * kPerThread >= kPerThread && (((uintptr_t)cd) & 15) == 0) {
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      *(GMEM u32x4*)cd = u32x4{pk[0], pk[1], pk[2], pk[3]};
    } else {
#pragma unroll
      for (int j = 0; j < kPerThread; ++j)
        if ((int64_t)tid * kPerThread + j < cnt) cd[j] = (uint16_t)(pk[j >> 1] >> (16 * (j & 1)));
    }
  }
  if (tid == 0) {
    TilePart all = s_part[0];
#pragma unroll
    for (int k = 1; k < kStreamThreads / kWave; ++k) all = tp_combine(all, s_part[k]);
    gstore(&w.tile_part[tile], all);
    gp(ws.scnt)[tile] = ((uint64_t)t << 32) | s_nx;
  }
}

// After k_stream: the frees of allocations in earlier tiles, from each tile's list.  An
// allocation freed in its own tile makes any such free a repeat, which stops the trace.  Where
// several such frees name one allocation, all but the one whose plain store landed see another
// index; each of them applies an atomic max of its inverted index, so the link ends at the first
// free, and stops the trace at the later of itself and the first free the atomic had seen.  The
// earliest of those stops is the second free of that allocation: whichever of the first two
// frees comes second in atomic order (the landed store counting as the first) sees the other one
// or an earlier one, and every stop is the later of two of its frees.
__global__ __launch_bounds__(kStreamThreads) void k_cross_check(const int64_t* off_, int64_t T, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t tile = xcd_item(blockIdx.x, gridDim.x);
  if (tile >= w.tile_base[T]) return;
  const uint64_t tc = gp(ws.scnt)[tile];
  const uint32_t cnt = (uint32_t)tc;
  if (cnt == 0) return;
  const int64_t t = (int64_t)(tc >> 32), base = off[t];
  const GMEM uint64_t* lst = (const GMEM uint64_t*)w.mbox + base + (tile - w.tile_base[t]) * kTile;
  // every list entry, then every allocation's code and cross link, loaded before any is used
  uint64_t x[kPerThread];
  uint32_t cd[kPerThread], lk[kPerThread];
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const uint32_t i = j * kStreamThreads + threadIdx.x;
    x[j] = i < cnt ? lst[i] : 0;
  }
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const uint32_t i = j * kStreamThreads + threadIdx.x;
    cd[j] = i < cnt ? w.code[base + (uint32_t)x[j]] : 0;
    lk[j] = i < cnt ? w.lx[base + (uint32_t)x[j]] : 0;
  }
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const uint32_t i = j * kStreamThreads + threadIdx.x;
    const uint32_t le = (uint32_t)(x[j] >> 32), h = (uint32_t)x[j], mine = 0xffffffffu - le;
    if (i >= cnt) continue;
    if (cd[j] & kCodeInTile) {
      mark_bad(w.stop_bad, t, le, XMEM_T_BAD_FREE);  // freed first inside its own, earlier tile
    } else if (lk[j] != mine) {
      const uint32_t old = __hip_atomic_fetch_max(&w.lx[base + h], mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint32_t other = 0xffffffffu - old;
      mark_bad(w.stop_bad, t, other > le ? other : le, XMEM_T_BAD_FREE);
    }
  }
}

// The annotation the replay and the planner use for event le of a trace, rebuilt from its event
// word x, its code and its cross link lxv: the op word (kind, pool, and an allocation's units)
// and the link word (a free: the index of its allocation; an allocation: ~ the index of its first
// free, 0 if it is never freed).
__device__ __forceinline__ void annotate(uint64_t x, uint32_t c, uint32_t lxv, int64_t le, int shift, uint64_t* op,
                                         uint32_t* link) {
  const uint32_t kind = c & kCodeKind;
  const uint64_t pool = (c & kCodePool) ? kPoolBit : 0;
  const uint64_t u = (x + ((1ull << shift) - 1)) >> shift;
  *op = kind == kCodeAlloc ? (kKindAlloc << kKindShift) | pool | u : kind == kCodeFree ? (kKindFree << kKindShift) | pool : 0;
  const uint32_t first = (c & kCodeInTile) ? 0xffffffffu - (uint32_t)((le & ~(kTile - 1)) + (int64_t)(c >> 4)) : lxv;
  *link = kind == kCodeFree ? (uint32_t)x : kind == kCodeAlloc ? first : 0u;
}
// the allocated-bytes delta of event le (a free's is its allocation's rounded size, negated)
__device__ __forceinline__ int64_t event_delta(const Gw& w, int64_t base, int64_t le, int shift) {
  const uint64_t x = w.ev[base + le];
  const uint32_t kind = w.code[base + le] & kCodeKind;
  const uint64_t gm = (1ull << shift) - 1;
  if (kind == kCodeAlloc) return (int64_t)(((x + gm) >> shift) << shift);
  if (kind == kCodeFree) return -(int64_t)(((w.ev[base + (uint32_t)x] + gm) >> shift) << shift);
  return 0;
}

// ------------------------------------------------------------------ fast chain: 32-bit packed keys
// Every free block is one 64-bit key (size << 32) | address, in units, so the
// best fit of Section 3.4 (iii) -- the smallest (size, address) with size >= u
// -- is the smallest key >= (u << 32): a masked wavefront minimum.  A pool's
// keys sit unordered in the kLdsSlots slots of its LDS table.  Each event
// makes one pass over the used rows (every row load issued before the first
// use), then rewrites at most two slots from one lane.  A chain hands itself
// over when a pool would need more free blocks than its table holds (status
// kSpill, to the paged chain kernel) or when sizes or addresses reach 2^31
// units (status kRetry, to the 64-bit chain kernel); either replays it again.
constexpr int kLdsRows = 12;  // 6 KB per pool: six replay wavefronts per SIMD (80 VGPRs each)
constexpr int32_t kLdsSlots = kLdsRows * 64;
constexpr uint64_t kFastLimit = 1ull << 31;
static_assert(kStateKeys == kLdsSlots, "a chunk state holds a full LDS table");
constexpr uint64_t kNoKey = ~0ull;
constexpr int kRetry = 0x40;
constexpr int kSpill = 0x41;
constexpr int kAbandoned = 0x42;  // a speculative chunk past where its round's walk will stop

__device__ __forceinline__ uint64_t key_of(uint64_t size, uint64_t addr) { return (size << 32) | addr; }
__device__ __forceinline__ uint64_t key_size(uint64_t k) { return k >> 32; }
__device__ __forceinline__ uint64_t key_addr(uint64_t k) { return k & 0xffffffffull; }
// the same block as an address key (address << 32) | size: ordered by address
__device__ __forceinline__ uint64_t akey_of(uint64_t size, uint64_t addr) { return (addr << 32) | size; }
__device__ __forceinline__ uint64_t akey_size(uint64_t k) { return k & 0xffffffffull; }
__device__ __forceinline__ uint64_t akey_addr(uint64_t k) { return k >> 32; }

struct STab {
  LMEM uint64_t* l;  // slots [0, kLdsSlots); slots n.. hold kNoKey
  int32_t n;
};
// single writer (lane 0); v is wave-uniform
__device__ __forceinline__ void st_store(STab& t, int32_t i, uint64_t v) {
  if (threadIdx.x == 0) t.l[i] = v;
  wave_order();
}
// remove slot i; `last` is the key in slot n-1, which moves into slot i
__device__ __forceinline__ void st_remove(STab& t, int32_t i, uint64_t last) {
  const int32_t l = t.n - 1;
  if (threadIdx.x == 0) {
    if (i != l) t.l[i] = last;
    uint64_t none = kNoKey;
    asm volatile("" : "+v"(none));  // made here: a constant held through the event loop can take a spill slot
    t.l[l] = none;
  }
  wave_order();
  t.n = l;
}
// append v; false when the table is full
__device__ __forceinline__ bool st_append(STab& t, uint64_t v) {
  if (t.n == kLdsSlots) return false;
  st_store(t, t.n, v);
  t.n += 1;
  return true;
}

// this lane's keys of the rows in use (slots past the count read kNoKey).  The table
// operations take NR, the rows they cover: kLdsRows checks the count before each row;
// a smaller NR (a table of at most 64 * NR keys) covers rows 0..NR-1 with no checks,
// since the slots past the count hold kNoKey.
template <int NR>
struct Rows {
  uint64_t x[NR];
};
template <int NR>
__device__ __forceinline__ bool st_row_used(const STab& t, int r) {
  return NR < kLdsRows || 64 * r < t.n;
}
// rows r.. of the table (nested, so every row index is a constant: a loop with an early
// exit is not always unrolled, and a row array indexed at run time goes to scratch memory)
template <int NR, int r = 0>
__device__ __forceinline__ void st_rows(const STab& t, Rows<NR>& R) {
  if constexpr (r < NR) {
    if (st_row_used<NR>(t, r)) {
      R.x[r] = t.l[64 * r + (int)threadIdx.x];
      st_rows<NR, r + 1>(t, R);
    }
  }
}
// key in slot n-1 (n > 0), read from the loaded rows
template <int NR>
__device__ __forceinline__ uint64_t st_last(const STab& t, const Rows<NR>& R) {
  const int32_t i = t.n - 1;
  const int lr = i >> 6, ll = i & 63;
  uint64_t v = kNoKey;
#pragma unroll
  for (int r = 0; r < NR; ++r)
    if (NR == 1 || r == lr) v = rl64(R.x[r], ll);
  return v;
}

// wavefront minimum of 64-bit keys and a lane holding it: the size halves
// first; the address halves only when several lanes tie on the smallest size
__device__ __forceinline__ uint64_t wave_min_key(uint64_t k, int* at) {
  const uint32_t hi = wave_min_u32((uint32_t)(k >> 32));
  const uint64_t tie = ballot((uint32_t)(k >> 32) == hi);
  if (__builtin_popcountll(tie) == 1) {
    *at = __builtin_ctzll(tie);
    return ((uint64_t)hi << 32) | rl((uint32_t)k, *at);
  }
  const uint32_t lo = wave_min_u32((uint32_t)(k >> 32) == hi ? (uint32_t)k : 0xffffffffu);
  *at = __builtin_ctzll(ballot((uint32_t)(k >> 32) == hi && (uint32_t)k == lo));
  return ((uint64_t)hi << 32) | lo;
}

// smallest key >= lo and its slot (-1 if none)
template <int NR>
__device__ __forceinline__ uint64_t st_min_ge(const STab& t, const Rows<NR>& R, uint64_t lo, int32_t* slot) {
  uint64_t best = kNoKey;
  int32_t bi = -1;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    if (!st_row_used<NR>(t, r)) break;
    const uint64_t x = R.x[r];
    const bool take = x >= lo && x < best;
    best = take ? x : best;
    bi = take ? 64 * r + (int32_t)threadIdx.x : bi;
  }
  int at;
  const uint64_t m = wave_min_key(best, &at);
  if constexpr (NR == 1) *slot = m == kNoKey ? -1 : at;  // one row: the lane is the slot
  else *slot = m == kNoKey ? -1 : (int32_t)rl((uint32_t)bi, at);
  return m;
}
// slots (and keys) of the free blocks ending at a and starting at e (= a + s);
// each is unique (the pool's blocks are disjoint), so every lane keeps its own
// match through the rows and two ballots at the end find the lanes that have one
template <int NR>
__device__ __forceinline__ void st_neighbours(const STab& t, const Rows<NR>& R, uint64_t a, uint64_t e, int32_t* ls,
                                              uint64_t* lk, int32_t* rs, uint64_t* rk) {
  if constexpr (NR == 1) {  // one row: the lanes of the matches are the slots, their keys are read back
    const uint64_t x = R.x[0];
    const uint32_t xa = (uint32_t)x, xs = (uint32_t)(x >> 32);
    const uint64_t lm = ballot(xa + xs == (uint32_t)a), rm = ballot(xa == (uint32_t)e);
    *ls = -1; *lk = 0; *rs = -1; *rk = 0;
    if (lm) { *ls = __builtin_ctzll(lm); *lk = rl64(x, *ls); }
    if (rm) { *rs = __builtin_ctzll(rm); *rk = rl64(x, *rs); }
    return;
  }
  int32_t li = -1, ri = -1;
  uint64_t lv = 0, rv = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    if (!st_row_used<NR>(t, r)) break;
    const uint64_t x = R.x[r];
    const uint32_t xa = (uint32_t)x, xs = (uint32_t)(x >> 32);
    const bool lh = xa + xs == (uint32_t)a, rh = xa == (uint32_t)e;
    li = lh ? 64 * r + (int32_t)threadIdx.x : li;
    lv = lh ? x : lv;
    ri = rh ? 64 * r + (int32_t)threadIdx.x : ri;
    rv = rh ? x : rv;
  }
  const uint64_t lm = ballot(li >= 0), rm = ballot(ri >= 0);
  *ls = -1; *lk = 0; *rs = -1; *rk = 0;
  if (lm) { const int l = __builtin_ctzll(lm); *ls = (int32_t)rl((uint32_t)li, l); *lk = rl64(lv, l); }
  if (rm) { const int l = __builtin_ctzll(rm); *rs = (int32_t)rl((uint32_t)ri, l); *rk = rl64(rv, l); }
}

struct FastPool {
  STab t;
  uint64_t split_min;  // split_min of this pool, in units
  GMEM uint64_t* segs;  // keys of the segments created in this pool, slot k at segs[segdir * k]
  int segdir;
  int32_t nseg;
  uint64_t bump, created_u;
  int32_t maxfree, n_mf;
  int pool;
};
__device__ __forceinline__ int32_t pool_free_count(const FastPool& ps) { return ps.t.n; }

// A chain replays a whole trace (CH false: change points go to the trace's
// record layout) or one chunk of it (CH true: to the chunk's own record region;
// see the chunked replay below).
template <int NP, bool CH = false>
struct FastChain {
  static constexpr bool kChunk = CH;
  FastPool p[NP];
  uint64_t reserved_u;
  int32_t created, released, n_res;
  int64_t base, n;
  bool back_res;
  GMEM ChunkRes* cres;  // chunk mode: reserved change points, slot i at cres[cres_dir * i]
  int cres_dir;
  GMEM MfRec* cmf;      // chunk mode: free-count maxima, slot i at cmf[cmf_dir * i]
  int cmf_dir;
  // chunk mode, speculative rounds of the chunk scheduler: the round's bound (the walk stops at
  // or before that chunk) and this chunk's index; else null
  const GMEM int32_t* bound;
  int32_t k_self;
};

// Request-size bucket of a chunk's choice summary: two per octave of units.
__device__ __forceinline__ int gbucket(uint64_t u) {
  const int l = 63 - __builtin_clzll(u | 1);
  const int b = 2 * l + (l > 0 ? (int)((u >> (l - 1)) & 1) : 0);
  return b < 63 ? b : 63;
}
// chunk mode: block S chosen for a request of u units (summary for k_chunk_stitch)
template <class C>
__device__ __forceinline__ void note_choice(C& c, uint64_t u, uint64_t S) {
  if constexpr (C::kChunk) {
    if (S > u) {
      const int b = gbucket(u);
      c.g = ((int)threadIdx.x == b && (uint32_t)S > c.g) ? (uint32_t)S : c.g;
    }
  }
}

// change points, shared by the fast and the paged chains
template <class C>
__device__ __forceinline__ void record_reserved(C& c, const Gw& w, int64_t e, int shift) {
  if (threadIdx.x == 0) {
    if constexpr (C::kChunk) {
      gstore(&c.cres[(int64_t)c.cres_dir * c.n_res], ChunkRes{(int64_t)(c.reserved_u << shift), (int32_t)e, c.created});
    } else {
      const int64_t slot = c.back_res ? c.base + c.n - 1 - c.n_res : c.base + c.n_res;
      gstore(&w.res[slot], ResRec{(int64_t)(c.reserved_u << shift), (int32_t)e, c.created, c.released, 0});
    }
  }
  c.n_res += 1;
}
template <class C, class P>
__device__ __forceinline__ void record_free_count(C& c, P& ps, const Gw& w, int64_t e) {
  const int32_t nf = pool_free_count(ps);
  if (nf > ps.maxfree) {
    ps.maxfree = nf;
    if (threadIdx.x == 0) {
      if constexpr (C::kChunk) {
        gstore(&c.cmf[(int64_t)c.cmf_dir * ps.n_mf], MfRec{(int32_t)e, nf});
      } else {
        const int64_t slot = ps.pool == 1 ? c.base + c.n - 1 - ps.n_mf : c.base + ps.n_mf;
        gstore(&w.mf[slot], MfRec{(int32_t)e, nf});
      }
    }
    ps.n_mf += 1;
  }
}

// the free block with key x is a whole idle segment: a segment of this pool has
// the same base and size, i.e. the same key (bases ascend in creation order)
__device__ bool seg_key_idle(const GMEM uint64_t* segs, int segdir, int32_t nseg, uint64_t x) {
  int32_t lo = 0, hi = nseg - 1;
  const uint64_t a = key_addr(x);
  while (lo <= hi) {
    const int32_t mid = (lo + hi) >> 1;
    const uint64_t g = segs[(int64_t)segdir * mid];
    if (key_addr(g) == a) return g == x;
    if (key_addr(g) < a) lo = mid + 1; else hi = mid - 1;
  }
  return false;
}

// size of the segment a new block of u units opens in this pool (Section 3.4 (ii), (iv))
__device__ __forceinline__ uint64_t segment_units(const Derived& d, int pool, uint64_t u) {
  if (pool == 0) return d.small_seg_u;
  if (u < d.min_large_u) return d.mid_seg_u;
  if (d.large_round_mask) return (u + d.large_round_mask) & ~d.large_round_mask;
  return (u + d.large_round_u - 1) / d.large_round_u * d.large_round_u;
}

// Section 3.4 (iv)-(v): units held by idle segments of both pools
template <int NP, bool CH>
__device__ __forceinline__ uint64_t fast_idle_units(const FastChain<NP, CH>& c) {
  uint64_t mine = 0;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const FastPool& ps = c.p[q];
    for (int32_t i = threadIdx.x; i < ps.t.n; i += kWave) {
      const uint64_t x = ps.t.l[i];
      if (seg_key_idle(ps.segs, ps.segdir, ps.nseg, x)) mine += key_size(x);
    }
  }
  return wave_sum_u64(mine);
}

template <int NP, bool CH>
__device__ __forceinline__ void fast_release_idle(FastChain<NP, CH>& c) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    FastPool& ps = c.p[q];
    int32_t i = 0;
    while (true) {  // first idle slot at or after i; the slot refilled by the removal is examined next
      int32_t hit = -1;
      for (int32_t r = i; r < ps.t.n; r += kWave) {
        const int32_t k = r + lane;
        const bool idle = k < ps.t.n && seg_key_idle(ps.segs, ps.segdir, ps.nseg, ps.t.l[k]);
        const uint64_t m = ballot(idle);
        if (m) { hit = r + __builtin_ctzll(m); break; }
      }
      if (hit < 0) break;
      c.reserved_u -= key_size(ps.t.l[hit]);
      c.released += 1;
      st_remove(ps.t, hit, ps.t.l[ps.t.n - 1]);
      i = hit;
    }
  }
}

// The best fit of u units among the cached free blocks (Section 3.4 (iii)), split
// or taken whole; false when none fits.  NR: rows of the table covered.
template <int NR>
__device__ __forceinline__ bool fast_take(STab& t, uint64_t u, uint64_t split_min, uint64_t* blk) {
  Rows<NR> R;
  st_rows<NR>(t, R);
  int32_t slot;
  const uint64_t b = st_min_ge<NR>(t, R, u << 32, &slot);
  if (b == kNoKey) return false;
  const uint64_t S = key_size(b), A = key_addr(b), rem = S - u;
  if (rem >= split_min) { st_store(t, slot, key_of(rem, A + u)); *blk = key_of(u, A); }
  else { st_remove(t, slot, st_last<NR>(t, R)); *blk = b; }
  return true;
}

// Allocation of u units (Section 3.4 (i)-(v)); returns a status and the key of
// the block handed out in *blk.  A table of one or two rows (at most 128 free
// blocks, the usual case) is scanned with no per-row count checks.
template <int NP, bool CH>
__device__ __forceinline__ int pool_alloc(FastChain<NP, CH>& c, FastPool& ps, const Derived& d, const Gw& w, uint64_t u,
                                          int64_t e, uint64_t* blk) {
  if (u >= kFastLimit) return kRetry;
  const uint64_t split_min = ps.split_min;
  if (ps.t.n <= 64 ? fast_take<1>(ps.t, u, split_min, blk)
                    : ps.t.n <= 128 ? fast_take<2>(ps.t, u, split_min, blk) : fast_take<kLdsRows>(ps.t, u, split_min, blk))
    return XMEM_T_OK;
  // nothing cached fits: a new segment (Section 3.4 (ii), (iv))
  const uint64_t S = segment_units(d, ps.pool, u);
  if (ps.created_u + S > d.limit_u) return XMEM_T_OVERFLOW;
  if (ps.bump + S + 1 > kFastLimit) return kRetry;
  if (NP == 2 && S > d.cap_u - c.reserved_u) {  // Section 3.4 (v): reclaim idle segments, else OOM
    const uint64_t idle = fast_idle_units(c);
    if (S > d.cap_u - (c.reserved_u - idle)) return XMEM_T_OOM;
    fast_release_idle(c);
  }
  const uint64_t rem = S - u;
  // a remainder the table cannot hold: the chain is handed over before the event has changed
  // anything, so that its state is the one before the event (a chunk resumes there)
  if (rem >= split_min && ps.t.n == kLdsSlots) return kSpill;
  const uint64_t A = ps.bump;
  // the segment table serves reclamation only, which chunked (unbounded) chains never do
  if (!CH && threadIdx.x == 0) ps.segs[(int64_t)ps.segdir * ps.nseg] = key_of(S, A);
  ps.nseg += 1;
  ps.bump += S + 1;  // one-unit gap: segments are never physically adjacent
  ps.created_u += S;
  c.reserved_u += S;
  c.created += 1;
  record_reserved(c, w, e, d.shift);
  if (rem >= split_min) {
    st_append(ps.t, key_of(rem, A + u));  // room checked above
    *blk = key_of(u, A);
  } else {
    *blk = key_of(S, A);
  }
  return XMEM_T_OK;
}

// Release of the block with key b: mark it free, coalesce with its free
// physical neighbours (Section 3.4 (iii)).  NR: rows of the table covered.
template <int NR>
__device__ __forceinline__ int fast_release(STab& t, uint64_t b) {
  const uint64_t A = key_addr(b), S = key_size(b);
  Rows<NR> R;
  st_rows<NR>(t, R);
  int32_t ls, rs;
  uint64_t lk = 0, rk = 0;
  st_neighbours<NR>(t, R, A, A + S, &ls, &lk, &rs, &rk);
  uint64_t ms = S, ma = A;
  if (ls >= 0) { ms += key_size(lk); ma = key_addr(lk); }
  if (rs >= 0) ms += key_size(rk);
  const uint64_t m = key_of(ms, ma);
  if (ls >= 0 && rs >= 0) {
    st_store(t, ls, m);
    // the merged block may itself sit in the last slot
    const uint64_t last = ls == t.n - 1 ? m : st_last<NR>(t, R);
    st_remove(t, rs, last);
  } else if (ls >= 0) {
    st_store(t, ls, m);
  } else if (rs >= 0) {
    st_store(t, rs, m);
  } else if (!st_append(t, m)) {
    return kSpill;
  }
  return XMEM_T_OK;
}
template <int NP, bool CH>
__device__ __forceinline__ int pool_free(FastChain<NP, CH>&, FastPool& ps, uint64_t b) {
  return ps.t.n <= 64 ? fast_release<1>(ps.t, b) : ps.t.n <= 128 ? fast_release<2>(ps.t, b) : fast_release<kLdsRows>(ps.t, b);
}

// ------------------------------------------------------------------ the serial event loop of one chain
// Shared by the fast and the paged chain kernels.  A chain type C provides,
// for its pools P, pool_alloc(c, ps, ...), pool_free(c, ps, b) and
// pool_free_count(ps).
template <int NP, int PI, class C>
__device__ __forceinline__ int chain_step(C& c, const Derived& d, const Gw& w, GMEM uint64_t* mkey, int64_t ts, int j,
                                          uint64_t opw, uint32_t lk, uint64_t cur_mb, uint64_t& fwd_cur,
                                          const uint64_t& fwd_prev) {
  auto& ps = c.p[PI];
  const int64_t e = ts + j;
  if ((opw >> kKindShift) == kKindAlloc) {
    uint64_t b;
    const int st = pool_alloc(c, ps, d, w, opw & kUnitsMask, e, &b);
    if (st != XMEM_T_OK) return st;
    fwd_cur = wl64(b, j, fwd_cur);  // reaches its free through the lanes, or the mailbox (end of the tile)
  } else {  // lk: where the freed block is (see chain_run)
    uint64_t b;
    if (lk < kWave) b = rl64(fwd_cur, (int)lk);
    else if (lk < 2 * kWave) b = rl64(fwd_prev, (int)lk - kWave);
    else b = rl64(cur_mb, j);
    const int st = pool_free(c, ps, b);
    if (st != XMEM_T_OK) return st;
  }
  record_free_count(c, ps, w, e);
  return XMEM_T_OK;
}

// A run's lane registers of allocated blocks (this tile's and the last tile's), kept where a
// chunk on the LDS table stopped so that the paged replay can take over there: from is the
// event to resume at (-1: from the start).
struct Resume { int64_t from; uint64_t cur, prev; };

// Walks the trace's annotated stream in 64-event tiles (the next tile's op,
// link and mailbox words prefetched) and takes the chain's events with a
// ballot + s_ff1 loop.  Allocated blocks reach their frees through lane
// registers (last two tiles) or the free's mailbox slot.
// Events [lo, limit) of the trace; every free there releases an allocation
// made there.  With rs: resumes at rs->from (tiles stay aligned to lo; the
// events before it in its tile were replayed, their blocks in rs->cur and the
// last tile's in rs->prev), and leaves the registers in rs at the end.
// With ms_ticks (wall-clock ticks per millisecond; 0: off), a chunk raises its wavefront's issue
// priority as it ages (its age counted from its 64th tile and checked every 64 tiles: 1 past
// 4 ms, 2 past 8, 3 past 16), so that on a SIMD the long tasks that end a batch of few chunks
// per pool go first.
template <int NP, class C>
__device__ __forceinline__ void chain_run(C& c, const Derived& d, const Gw& w, int pool_one, int64_t lo, int64_t limit,
                                          int* status_out, int64_t* stop_out, Resume* rs = nullptr,
                                          uint64_t ms_ticks = 0) {
  GMEM uint64_t* mkey = (GMEM uint64_t*)w.mbox;  // mailbox viewed as one key per event
  const int lane = threadIdx.x;
  int status = XMEM_T_OK;
  int64_t stop = -1;
  uint64_t cur_op = 0, nxt_x = 0, cur_mb = 0, nxt_mb = 0, fwd_cur = 0, fwd_prev = 0;
  uint32_t cur_link = 0, nxt_c = 0, nxt_lx = 0;
  const bool resumed = rs && rs->from > lo;
  const int64_t skip = resumed ? rs->from : lo;                        // the first event replayed
  const int64_t first = resumed ? lo + ((skip - lo) & ~(int64_t)(kWave - 1)) : lo;  // its tile
  if (resumed) {
    fwd_cur = rs->cur;
    fwd_prev = rs->prev;
  }
  if (first + lane < limit) {
    const int64_t le = first + lane;
    annotate(w.ev[c.base + le], w.code[c.base + le], w.lx[c.base + le], le, d.shift, &cur_op, &cur_link);
    // a tile inside the run: its frees may take blocks from the mailbox (the first tile of a
    // run frees only its own allocations)
    if (resumed) cur_mb = mkey[c.base + le];
  }
  // Consume the first tile's words here: a load still outstanding at the event
  // loop would make every event wait for all earlier stores (stores and loads
  // share one counter).
  asm volatile("" ::"v"(cur_op), "v"(cur_link), "v"(cur_mb));
  uint64_t t_aged = 0;
  int prio = 0;
  for (int64_t ts = first; ts < limit; ts += kWave) {
    wave_order();
    if constexpr (C::kChunk) {
      if (ms_ticks && (((ts - first) >> 6) & 63) == 63) {
        const uint64_t now = wall_clock64();
        if (t_aged == 0) t_aged = now;
        const uint64_t age = now - t_aged;
        const int p = age > 16 * ms_ticks ? 3 : age > 8 * ms_ticks ? 2 : age > 4 * ms_ticks ? 1 : 0;
        if (p != prio) {  // the priority is an immediate operand
          prio = p;
          if (p == 1) __builtin_amdgcn_s_setprio(1);
          else if (p == 2) __builtin_amdgcn_s_setprio(2);
          else if (p == 3) __builtin_amdgcn_s_setprio(3);
        }
      }
    }
    int32_t bound = INT32_MAX;  // every fourth tile: loaded with the next tile, read after this one
    if constexpr (C::kChunk) {
      if (c.bound && (((ts - lo) >> 6) & 3) == 0)
        bound = __hip_atomic_load(c.bound, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    {  // prefetch the next tile; its mailbox slots hold the blocks of allocations two or more tiles back
      const int64_t le = ts + kWave + lane;
      nxt_x = 0; nxt_c = 0; nxt_lx = 0; nxt_mb = 0;
      if (le < limit) { nxt_x = w.ev[c.base + le]; nxt_c = w.code[c.base + le]; nxt_lx = w.lx[c.base + le]; nxt_mb = mkey[c.base + le]; }
    }
    // a free's link word (its allocation's index h) becomes where the freed block is: lane
    // h - ts of this tile's blocks, 64 + lane h - ts + 64 of the last tile's, or 128 for its
    // own mailbox slot -- one vector step per tile instead of compares per event
    {
      const int64_t hd = (int64_t)cur_link - ts;
      const uint32_t where = hd >= 0 ? (uint32_t)hd : hd >= -kWave ? (uint32_t)(hd + 2 * kWave) : 2u * kWave;
      cur_link = (cur_op >> kKindShift) == kKindFree ? where : cur_link;
    }
    const bool mine = (ts + lane < limit) && (cur_op >> kKindShift) != 0 &&
                      (NP == 2 || ((cur_op & kPoolBit) ? 1 : 0) == pool_one);
    uint64_t todo = ballot(mine && (!resumed || ts + lane >= skip));
    while (todo) {
      const int j = __builtin_ctzll(todo);
      todo &= todo - 1;
      const uint64_t opw = rl64(cur_op, j);
      const uint32_t lk = rl(cur_link, j);
      int st;
      if (NP == 1 || !(opw & kPoolBit)) st = chain_step<NP, 0>(c, d, w, mkey, ts, j, opw, lk, cur_mb, fwd_cur, fwd_prev);
      else st = chain_step<NP, NP - 1>(c, d, w, mkey, ts, j, opw, lk, cur_mb, fwd_cur, fwd_prev);
      if (st != XMEM_T_OK) { status = st; stop = ts + j; break; }
    }
    if (stop >= 0) break;
    {  // every allocation of the tile whose free lies two or more tiles ahead: its block to the
       // free's mailbox slot, all in one vector store (ordered before the next tile's loads)
      const int64_t fe = (int64_t)(0xffffffffu - cur_link);
      if (mine && (cur_op >> kKindShift) == kKindAlloc && cur_link != 0 && fe >= ts + 2 * kWave && fe < c.n)
        mkey[c.base + fe] = fwd_cur;
    }
    fwd_prev = fwd_cur;
    fwd_cur = 0;
    if constexpr (C::kChunk) {
      // another chunk of the round created segments or stopped before this one: the walk will
      // never read this chunk's results, so it ends here and writes none
      if (c.k_self > __builtin_amdgcn_readfirstlane(bound)) {
        status = kAbandoned;
        stop = ts;
        break;
      }
    }
    annotate(nxt_x, nxt_c, nxt_lx, ts + kWave + lane, d.shift, &cur_op, &cur_link);
    cur_mb = nxt_mb;
  }
  if (prio) __builtin_amdgcn_s_setprio(0);
  if (rs) {
    rs->cur = fwd_cur;
    rs->prev = fwd_prev;
  }
  *status_out = status;
  *stop_out = stop;
}

template <class C>
__device__ __forceinline__ void chain_header(const C& c, const Gw& w, int np, int64_t t, int pool_one, int status,
                                             int64_t stop, int32_t n_mf0, int32_t n_mf1) {
  if (threadIdx.x == 0) {
    if (np == 1) {
      gstore(&w.hdr[2 * t + pool_one], ChainHdr{stop, status, c.n_res, n_mf0, 0, 0});
    } else {
      gstore(&w.hdr[2 * t + 0], ChainHdr{stop, status, c.n_res, n_mf0, 0, 0});
      gstore(&w.hdr[2 * t + 1], ChainHdr{stop, status, 0, n_mf1, 0, 0});
    }
  }
}

template <int NP>
__global__ __launch_bounds__(kWave, NP == 1 ? 6 : 3) void k_replay_fast(const int64_t* off_, Derived d, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  __shared__ uint64_t s_k[NP][kLdsSlots];
  const int lane = threadIdx.x;
  const int64_t chain = blockIdx.x;
  const int64_t t = NP == 1 ? (chain >> 1) : chain;
  const int pool_one = NP == 1 ? (int)(chain & 1) : 0;  // pool of a split chain
  GMEM uint64_t* sgk = (GMEM uint64_t*)w.segs;
  FastChain<NP> c;
  c.base = off[t];
  c.n = off[t + 1] - c.base;
  const uint64_t sb = w.stop_bad[t];
  const int64_t limit = sb == kNoStop ? c.n : (int64_t)(sb >> 8);
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const int pool = NP == 1 ? pool_one : q;
    FastPool& ps = c.p[q];
    ps.t.l = (LMEM uint64_t*)s_k[q];
#pragma unroll
    for (int r = 0; r < kLdsRows; ++r) ps.t.l[64 * r + lane] = kNoKey;
    ps.t.n = 0;
    ps.segdir = pool == 0 ? 1 : -1;
    ps.segs = pool == 0 ? sgk + c.base : sgk + c.base + c.n - 1;
    ps.nseg = 0;
    ps.bump = ps.created_u = 0;
    ps.maxfree = ps.n_mf = 0;
    ps.pool = pool;
    ps.split_min = pool == 0 ? d.split_min_u[0] : d.split_min_u[1];
  }
  c.reserved_u = 0;
  c.created = c.released = c.n_res = 0;
  c.back_res = NP == 1 && pool_one == 1;
  int status;
  int64_t stop;
  chain_run<NP>(c, d, w, pool_one, 0, limit, &status, &stop);
  chain_header(c, w, NP, t, pool_one, status, stop, c.p[0].n_mf, c.p[NP - 1].n_mf);
}

// ------------------------------------------------------------------ chunked replay (unbounded capacity)
// A chain's events are cut at positions s where no allocation made before s
// is freed at or after s ("clean" positions).  Each chunk between two cuts
// then frees only blocks it allocated itself, so its replay needs nothing from
// earlier chunks but the allocator state at its start.  The cuts after the
// first all lie between two consecutive never-freed allocations, so every
// chunk but the first and the last is balanced: it leaves the set of live
// blocks as it found it.  If such a chunk also creates no segment, the state
// after it -- segments, live blocks, and hence the free blocks, which are the
// coalesced rest of the segments -- equals the state before it.
//
// So the first chunk is replayed alone; every later chunk is then replayed at
// once from the first chunk's end state, and a chunk's result is exact when no
// chunk between the frontier and it created a segment.  The first chunk that
// did ends the exact run: its end state becomes the start of the next round
// for the chunks after it.  After a fixed number of rounds the remaining
// events of a chain are replayed in one piece.  Results are exact in every
// case; the speed-up depends on segments being created early, as they are in
// training traces (memory settles after the first iterations).

// never-freed allocations in a run of events: first and last position and the
// widest gap between consecutive ones (length, left end); first < 0: none
struct NfRun { int64_t first, last, gap, gap_lo; };
__device__ __forceinline__ bool nf_better(int64_t g1, int64_t lo1, int64_t g2, int64_t lo2) {
  return g1 > g2 || (g1 == g2 && lo1 < lo2);
}
__device__ __forceinline__ NfRun nf_combine(NfRun a, NfRun b) {
  if (a.first < 0) return b;
  if (b.first < 0) return a;
  NfRun r{a.first, b.last, a.gap, a.gap_lo};
  if (nf_better(b.gap, b.gap_lo, r.gap, r.gap_lo)) { r.gap = b.gap; r.gap_lo = b.gap_lo; }
  const int64_t across = b.first - a.last;
  if (nf_better(across, a.last, r.gap, r.gap_lo)) { r.gap = across; r.gap_lo = a.last; }
  return r;
}

// What event e contributes to the plans of the trace's two pool chains: a
// 4-bit code per pool (pool 0 in bits 0-3, pool 1 in bits 4-7).  kOwn: an
// event of that pool before the limit; kUp: it opens a block freed before the
// limit; kDown: it frees one; kNf: an allocation never freed before the limit.
constexpr uint32_t kOwn = 1, kUp = 2, kDown = 4, kNf = 8;

// The code of event le, from its 16-bit stream code and cross link alone (the parts of its op
// and link words the plan needs: kind, pool, and an allocation's first free)
__device__ __forceinline__ uint32_t plan_code_of(uint32_t c, uint32_t lxv, int64_t le, int64_t limit) {
  const uint32_t kind = c & kCodeKind;
  if (kind == 0) return 0;
  uint32_t r = kOwn | kDown;
  if (kind == kCodeAlloc) {
    const uint32_t lk = (c & kCodeInTile) ? 0xffffffffu - (uint32_t)((le & ~(int64_t)(kTile - 1)) + (int64_t)(c >> 4)) : lxv;
    const bool freed = lk != 0 && (int64_t)(0xffffffffu - lk) < limit;
    r = kOwn | (freed ? kUp : kNf);
  }
  return (c & kCodePool) ? r << 4 : r;
}

// wavefront reduction of never-freed runs in lane order; the result is in lane 0
__device__ __forceinline__ NfRun nf_wave_reduce(NfRun r) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    NfRun x;
    x.first = __shfl_down(r.first, o, 64);
    x.last = __shfl_down(r.last, o, 64);
    x.gap = __shfl_down(r.gap, o, 64);
    x.gap_lo = __shfl_down(r.gap_lo, o, 64);
    if ((threadIdx.x & 63) + o < 64) r = nf_combine(r, x);
  }
  return r;
}

// exclusive scan over the workgroup in thread order; *total gets the sum
__device__ uint64_t plan_excl_scan(uint64_t v, uint64_t* s_w, uint64_t* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  // inclusive scan up the wavefront on DPP alone (the steps of tp_wave_scan)
  uint64_t x = v;
  x += (uint64_t)dpp_move<0x111, 0xf>(0, (int64_t)x);  // row_shr:1
  x += (uint64_t)dpp_move<0x112, 0xf>(0, (int64_t)x);  // row_shr:2
  x += (uint64_t)dpp_move<0x114, 0xf>(0, (int64_t)x);  // row_shr:4
  x += (uint64_t)dpp_move<0x118, 0xf>(0, (int64_t)x);  // row_shr:8
  x += (uint64_t)dpp_move<0x142, 0xa>(0, (int64_t)x);  // row_bcast:15 into rows 1 and 3
  x += (uint64_t)dpp_move<0x143, 0xc>(0, (int64_t)x);  // row_bcast:31 into rows 2 and 3
  if (lane == 63) s_w[wv] = x;
  __syncthreads();
  uint64_t before = 0, tot = 0;
  for (int i = 0; i < kPlanThreads / 64; ++i) {
    const uint64_t t = s_w[i];
    if (i < wv) before += t;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

// The planner runs over 2048-event blocks of all traces at once, in four steps:
//   k_plan_blocks  per block: each event's code byte, and per pool the block's
//                  own-event count, coverage sum (blocks opened - closed) and
//                  never-freed run;
//   k_plan_chains  per trace: the blocks' prefixes, and per pool chain the
//                  widest never-freed gap [amin, amax] and the chunk count;
//   k_plan_cuts    per block: every clean position in a chain's gap offered to
//                  the share it reaches (share = floor(before * kc / own));
//                  the smallest key wins each share; the largest key short of
//                  the first chunk's target is kept apart;
//   k_plan_final   per chain: the first cut takes the clean position nearest
//                  to the first chunk's target, before or after it (the first
//                  chunk is replayed alone, so it should not run a whole
//                  iteration long for want of a few events); every later cut
//                  is the first clean position of a share past it (a suffix
//                  minimum).
// A chain of more than target own events has kFineShares times as many shares
// as target-sized chunks (at most the chunk count; all of them when target is
// 0); in the large pool its first chunk still aims at one target-sized chunk.  Clean positions
// can be as sparse as iteration boundaries; a share narrower than the spacing
// puts a cut at each of them, where shares a little wider than one iteration
// would leave some chunks two iterations long, and those set the round's end.
constexpr int64_t kFineShares = 2;
struct PlanAgg { int64_t own[2], cov[2]; NfRun run[2]; };

// One planner thread's part of a block, for both pools: own events, coverage, and the
// never-freed run with 32-bit positions (a trace's events lie below 2^31); first < 0: no run.
struct NfRun32 { int32_t first, last, gap, gap_lo; };
struct PlanPart { int32_t own0, own1, cov0, cov1; NfRun32 run0, run1; };
// a then b, in event order (nf_combine with selects)
__device__ __forceinline__ NfRun32 nf_join(NfRun32 a, NfRun32 b) {
  int32_t gap = a.gap, lo = a.gap_lo;
  if (b.gap > gap || (b.gap == gap && b.gap_lo < lo)) { gap = b.gap; lo = b.gap_lo; }
  const int32_t across = b.first - a.last;
  if (across > gap || (across == gap && a.last < lo)) { gap = across; lo = a.last; }
  // field by field: a select of whole structs goes through scratch memory
  const bool ea = a.first < 0, eb = b.first < 0;
  return NfRun32{eb ? a.first : ea ? b.first : a.first, eb ? a.last : b.last, eb ? a.gap : ea ? b.gap : gap,
                 eb ? a.gap_lo : ea ? b.gap_lo : lo};
}
__device__ __forceinline__ PlanPart pp_join(const PlanPart& a, const PlanPart& b) {
  return PlanPart{a.own0 + b.own0, a.own1 + b.own1, a.cov0 + b.cov0, a.cov1 + b.cov1, nf_join(a.run0, b.run0),
                  nf_join(a.run1, b.run1)};
}
template <int CTRL, int ROWS>
__device__ __forceinline__ int32_t dpp32(int32_t old, int32_t v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWS, 0xf, false);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ NfRun32 nf_dpp(NfRun32 r) {
  return NfRun32{dpp32<CTRL, ROWS>(-1, r.first), dpp32<CTRL, ROWS>(-1, r.last), dpp32<CTRL, ROWS>(-1, r.gap),
                 dpp32<CTRL, ROWS>(-1, r.gap_lo)};
}
template <int CTRL, int ROWS>
__device__ __forceinline__ PlanPart pp_scan_step(const PlanPart& x) {
  // the earlier lanes' part (an empty one where there is none)
  const PlanPart y{dpp32<CTRL, ROWS>(0, x.own0), dpp32<CTRL, ROWS>(0, x.own1), dpp32<CTRL, ROWS>(0, x.cov0),
                   dpp32<CTRL, ROWS>(0, x.cov1), nf_dpp<CTRL, ROWS>(x.run0), nf_dpp<CTRL, ROWS>(x.run1)};
  return pp_join(y, x);
}
// inclusive scan up the wavefront in lane order on DPP alone, as tp_wave_scan: lane 63 ends
// with the wavefront's part.  All lanes active.
__device__ __forceinline__ PlanPart pp_wave_scan(PlanPart x) {
  x = pp_scan_step<0x111, 0xf>(x);  // row_shr:1
  x = pp_scan_step<0x112, 0xf>(x);  // row_shr:2
  x = pp_scan_step<0x114, 0xf>(x);  // row_shr:4
  x = pp_scan_step<0x118, 0xf>(x);  // row_shr:8
  x = pp_scan_step<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x = pp_scan_step<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}
struct PlanChain { int64_t own, amin, amax; int32_t kc, first; };
static_assert(sizeof(PlanAgg) == 96 && sizeof(PlanChain) == 32, "sizes the workspace carving assumes");

// the trace of planner block b, found by wave 0 and shared through LDS (call from every thread)
// A planner block is the stream tile of the same index: both cut each trace into kTile-event
// units from its start (kPlanBlock == kTile), so the tile's record names the block's trace.
static_assert(kPlanBlock == kTile, "planner blocks are the stream tiles");
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int64_t plan_limit(const Gw& w, int64_t t, int64_t n) {
  const uint64_t sb = w.stop_bad[t];
  return sb == kNoStop ? n : (int64_t)(sb >> 8);
}

__global__ __launch_bounds__(kPlanThreads) void k_plan_blocks(const int64_t* off_, int64_t T, Derived d, Ws ws) {
  const Gw w = typed(ws);
  const int64_t b = blockIdx.x;
  // the grid is the tile capacity, so every block's tile record lies in the workspace
  const int32_t bad = w.ctl[0];
  const int64_t nb = w.pblk_base[T];
  const TileInfo ti = gload(&w.tinfo[b]);
  if (bad || b >= nb) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t t = ti.t, b0 = ti.t0, base = ti.base, limit = plan_limit(w, t, ti.len);
  GMEM uint8_t* codes = (GMEM uint8_t*)w.mbox + base;  // the mailbox area is free until the replay
  __shared__ PlanPart s_pp[kPlanThreads / 64];
  // this thread's 8 consecutive events: their words loaded beside the trace's limit (the events
  // at or past it count as none), 16 bytes at a time when the trace starts on an 8-event boundary
  // (then every thread's words and code bytes are aligned), else one by one
  uint64_t cw = 0;  // byte j: the code of event e0 + j
  {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const int32_t i0 = tid * kPlanPer;
    const int64_t lim = limit - b0;
    const GMEM uint16_t* cdb = w.code + base + b0 + i0;
    const GMEM uint32_t* lxb = w.lx + base + b0 + i0;
    const bool vec = (base & 7) == 0 && i0 + kPlanPer <= ti.cnt;
    uint32_t cw8[kPlanPer], lx8[kPlanPer];
    if (vec) {
      const u32x4 c4 = *(const GMEM u32x4*)cdb;
      const u32x4 l0 = *(const GMEM u32x4*)lxb, l1 = *(const GMEM u32x4*)(lxb + 4);
      const uint32_t cv[4] = {c4.x, c4.y, c4.z, c4.w}, lv[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
#pragma unroll
      for (int j = 0; j < kPlanPer; ++j) {
        cw8[j] = (cv[j >> 1] >> (16 * (j & 1))) & 0xffffu;
        lx8[j] = lv[j];
      }
    } else {
#pragma unroll
      for (int j = 0; j < kPlanPer; ++j) {
        cw8[j] = i0 + j < ti.cnt ? cdb[j] : 0;
        lx8[j] = i0 + j < ti.cnt ? lxb[j] : 0;
      }
    }
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j)
      cw |= (uint64_t)plan_code_of(i0 + j < lim ? cw8[j] : 0u, lx8[j], b0 + i0 + j, limit) << (8 * j);
    GMEM uint8_t* cd = codes + b0 + i0;
    if (vec && i0 + kPlanPer <= lim) {
      *(GMEM uint64_t*)cd = cw;
    } else {
#pragma unroll
      for (int j = 0; j < kPlanPer; ++j)
        if (i0 + j < lim) cd[j] = (uint8_t)(cw >> (8 * j));
    }
  }
  const int32_t e0 = (int32_t)(b0 + (int64_t)tid * kPlanPer);  // positions stay below 2^31
  int32_t own_q[2], cov_q[2];
  NfRun32 run_q[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    // this thread's 8 events in order: never-freed positions (first, last, widest gap), counts
    int32_t first = -1, last = -1, gap = -1, gap_lo = -1, own = 0, cov = 0;
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) {
      const uint32_t c = ((uint32_t)(cw >> (8 * j)) >> (4 * q)) & 0xfu;
      own += (c & kOwn) ? 1 : 0;
      cov += ((c & kUp) ? 1 : 0) - ((c & kDown) ? 1 : 0);
      if (c & kNf) {
        if (first < 0) {
          first = e0 + j;
        } else if (e0 + j - last > gap) {  // ties keep the earlier gap
          gap = e0 + j - last;
          gap_lo = last;
        }
        last = e0 + j;
      }
    }
    own_q[q] = own;
    cov_q[q] = cov;
    run_q[q] = NfRun32{first, last, gap, gap_lo};
  }
  const PlanPart part = pp_wave_scan(PlanPart{own_q[0], own_q[1], cov_q[0], cov_q[1], run_q[0], run_q[1]});
  if (lane == kWave - 1) s_pp[wv] = part;
  __syncthreads();
  if (tid == 0) {  // the wavefronts' parts in order
    PlanPart a = s_pp[0];
#pragma unroll
    for (int i = 1; i < kPlanThreads / 64; ++i) a = pp_join(a, s_pp[i]);
    GMEM int64_t* agg = (GMEM int64_t*)(w.pagg + b);  // own[2], cov[2], run[2] (4 words each)
    const int32_t v[12] = {a.own0, a.own1, a.cov0, a.cov1, a.run0.first, a.run0.last, a.run0.gap, a.run0.gap_lo,
                           a.run1.first, a.run1.last, a.run1.gap, a.run1.gap_lo};
#pragma unroll
    for (int i = 0; i < 12; ++i) agg[i] = v[i];
  }
}

// one wavefront per trace
__global__ __launch_bounds__(64) void k_plan_chains(const int64_t* off_, int64_t T, int64_t target, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t t = blockIdx.x;
  const int lane = threadIdx.x;
  const int K = w.chunks;
  const int64_t bb = w.pblk_base[t], nb = w.pblk_base[t + 1] - bb;
  const int64_t n = off[t + 1] - off[t], limit = plan_limit(w, t, n);
  int64_t carry[4] = {0, 0, 0, 0};  // own 0, own 1, cov 0, cov 1 before the group
  NfRun tot[2] = {{-1, -1, -1, -1}, {-1, -1, -1, -1}};
  for (int64_t i0 = 0; i0 < nb; i0 += 64) {
    const int64_t i = i0 + lane;
    PlanAgg a{{0, 0}, {0, 0}, {{-1, -1, -1, -1}, {-1, -1, -1, -1}}};
    if (i < nb) a = gload(&w.pagg[bb + i]);
    int64_t v[4] = {a.own[0], a.own[1], a.cov[0], a.cov[1]}, x[4];
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      x[f] = v[f];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(x[f], o, 64);
        if (lane >= o) x[f] += y;
      }
    }
    if (i < nb) {
      GMEM int64_t* pre = w.ppre + 4 * (bb + i);
#pragma unroll
      for (int f = 0; f < 4; ++f) pre[f] = carry[f] + x[f] - v[f];
    }
#pragma unroll
    for (int f = 0; f < 4; ++f) carry[f] += __shfl(x[f], 63, 64);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const NfRun r = nf_wave_reduce(a.run[q]);
      NfRun r0;
      r0.first = __shfl(r.first, 0, 64);
      r0.last = __shfl(r.last, 0, 64);
      r0.gap = __shfl(r.gap, 0, 64);
      r0.gap_lo = __shfl(r.gap_lo, 0, 64);
      tot[q] = nf_combine(tot[q], r0);
    }
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int64_t own = carry[q];
    int64_t glo = -1, glen = limit + 1;  // no never-freed allocation: the whole chain
    if (tot[q].first >= 0) {
      glo = -1;
      glen = tot[q].first + 1;
      if (nf_better(tot[q].gap, tot[q].gap_lo, glen, glo)) { glen = tot[q].gap; glo = tot[q].gap_lo; }
      if (nf_better(limit - tot[q].last, tot[q].last, glen, glo)) { glen = limit - tot[q].last; glo = tot[q].last; }
    }
    PlanChain pc;
    pc.own = own;
    pc.amin = max<int64_t>(glo + 1, 1);
    pc.amax = min<int64_t>(glo + glen, limit - 1);
    int64_t kc0 = own > 0 ? K : 1, kc = kc0;  // target-sized chunks; shares
    if (target > 0) {
      kc0 = max<int64_t>(1, min<int64_t>(K, (own + target - 1) / target));
      kc = kc0 > 1 ? min<int64_t>(K, (own * kFineShares + target - 1) / target) : 1;
    }
    if (pc.amin > pc.amax) kc0 = kc = 1;
    pc.kc = (int32_t)kc;
    // the first chunk's target own events: one target-sized chunk in the large pool, whose
    // later chunks are replayed again after a chunk that creates a segment; one share in the
    // small pool, where such chunks are certified instead
    pc.first = (int32_t)((own + (q == 0 ? kc : kc0) - 1) / (q == 0 ? kc : kc0));
    const int64_t chain = 2 * t + q;
    if (lane == 0) gstore(&w.pchain[chain], pc);
    GMEM uint64_t* sh = w.pshare + chain * (K + 1);
    for (int k = lane; k <= K; k += 64) sh[k] = k < K ? ~0ull : 0ull;
  }
}

__global__ __launch_bounds__(kPlanThreads) void k_plan_cuts(const int64_t* off_, int64_t T, Ws ws) {
  const Gw w = typed(ws);
  const int64_t b = blockIdx.x;
  // the grid is the tile capacity, so every block's tile record lies in the workspace
  const int32_t bad = w.ctl[0];
  const int64_t nb = w.pblk_base[T];
  const TileInfo ti = gload(&w.tinfo[b]);
  const GMEM int64_t* pre = w.ppre + 4 * b;  // the block's prefix counts, loaded early
  int64_t pre4[4];
#pragma unroll
  for (int f = 0; f < 4; ++f) pre4[f] = pre[f];
  if (bad || b >= nb) return;
  const int tid = threadIdx.x;
  const int K = w.chunks;
  const int64_t t = ti.t, b0 = ti.t0, b1 = b0 + kPlanBlock - 1, base = ti.base;
  // this thread's 8 consecutive code bytes, loaded beside the trace's limit and the chains' plans:
  // one 8-byte load when the trace starts on an 8-event boundary, else one by one
  const int32_t i0 = tid * kPlanPer;
  const GMEM uint8_t* cd = (const GMEM uint8_t*)w.mbox + base + b0 + i0;
  uint64_t cw = 0;
  if ((base & 7) == 0 && i0 + kPlanPer <= ti.cnt) {
    cw = *(const GMEM uint64_t*)cd;
  } else {
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) cw |= (uint64_t)(i0 + j < ti.cnt ? cd[j] : (uint8_t)0) << (8 * j);
  }
  const int64_t limit = plan_limit(w, t, ti.len);
  PlanChain pc[2];
  bool any = false;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    pc[q] = gload(&w.pchain[2 * t + q]);
    any = any || (pc[q].kc > 1 && b0 <= pc[q].amax && b1 >= pc[q].amin);
  }
  if (!any) return;
  __shared__ uint64_t s_w[kPlanThreads / 64];
  static_assert(2 * kCutSlots <= kPlanThreads, "one thread per share slot");
  __shared__ uint64_t s_min[2][kCutSlots];
  if (tid < 2 * kCutSlots) s_min[tid / kCutSlots][tid % kCutSlots] = tid % kCutSlots == 0 ? 0ull : ~0ull;
  // past the limit the mailbox holds no code
  const int64_t below = limit - b0 - i0;
  if (below < kPlanPer) cw = below <= 0 ? 0 : cw & ((1ull << (8 * below)) - 1);
  __syncthreads();  // s_min ready
  // within the block, 16-bit fields: opens - closes + 8 per thread, own events; pool 0 then pool 1
  // (every field's partial sums stay in [0, 2^16))
  uint64_t v = 0;
#pragma unroll
  for (int j = 0; j < kPlanPer; ++j) {
    const uint32_t c = (uint32_t)(cw >> (8 * j)) & 0xffu;
    v += ((c & kUp) ? 1u : 0u) + ((c & kOwn) ? 1ull << 16 : 0u) + ((c & (kUp << 4)) ? 1ull << 32 : 0u) +
         ((c & (kOwn << 4)) ? 1ull << 48 : 0u);
    v -= ((c & kDown) ? 1u : 0u) + ((c & (kDown << 4)) ? 1ull << 32 : 0u);
  }
  v += 8ull + (8ull << 32);
  uint64_t btot;
  const uint64_t ex = plan_excl_scan(v, s_w, &btot);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    if (pc[q].kc <= 1) continue;
    int64_t cov = pre4[2 + q] + (int64_t)((ex >> (32 * q)) & 0xffffu) - 8 * tid;
    int64_t before = pre4[q] + (int64_t)((ex >> (32 * q + 16)) & 0xffffu);
    const int64_t own = pc[q].own, kc = pc[q].kc;
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) {
      const uint32_t c = ((uint32_t)(cw >> (8 * j)) >> (4 * q)) & 0xfu;
      const int64_t e = b0 + (int64_t)tid * kPlanPer + j;
      if (cov == 0 && e >= pc[q].amin && e <= pc[q].amax) {
        const uint64_t key = ((uint64_t)e << 32) | (uint64_t)before;
        // short of the first chunk's target, else the share reached (>= 1: the target is at least one share)
        if (before < pc[q].first) atomicMax((unsigned long long*)&s_min[q][0], key);
        else atomicMin((unsigned long long*)&s_min[q][min<int64_t>(kc - 1, before * kc / own)], key);
      }
      cov += ((c & kUp) ? 1 : 0) - ((c & kDown) ? 1 : 0);
      before += (c & kOwn) ? 1 : 0;
    }
  }
  __syncthreads();
  if (tid < 2 * kCutSlots) {
    const int q = tid / kCutSlots, k = tid % kCutSlots;
    const uint64_t key = s_min[q][k];
    GMEM unsigned long long* sh = (GMEM unsigned long long*)w.pshare + (2 * t + q) * (K + 1);
    // the share table: [0, K) smallest key per share (entry 0 unused), [K] the last key short of share 1
    if (k == 0 && key != 0) __hip_atomic_fetch_max(sh + K, (unsigned long long)key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (k > 0 && k < K && key != ~0ull)
      __hip_atomic_fetch_min(sh + k, (unsigned long long)key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// one wavefront per chain: the cuts (lane k of group g: cut 64 g + k; two groups for up to 127 chunks)
__global__ __launch_bounds__(64) void k_plan_final(const int64_t* off_, int64_t T, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t chain = blockIdx.x;
  const int lane = threadIdx.x;
  const int K = w.chunks;
  const int64_t t = chain >> 1;
  const int64_t n = off[t + 1] - off[t], limit = plan_limit(w, t, n);
  const PlanChain pc = gload(&w.pchain[chain]);
  const int kcq = (int)pc.kc;
  const GMEM uint64_t* sh = w.pshare + chain * (K + 1);
  GMEM int32_t* bnd = w.cbound + chain * (K + 1);
  GMEM int32_t* own_before = w.cown + chain * (K + 1);
  // cut j >= 1 takes share s1 + j - 1, where s1 is the share holding the first chunk's target;
  // cut j: the smallest key of the shares >= s1 + j - 1, i.e. of the first such share that has one
  // (a later share's keys lie after an earlier share's).  The second group first: its first key
  // ends the first group's search.
  const int s1 = kcq > 1 ? (int)min<int64_t>(kcq - 1, (int64_t)pc.first * kcq / pc.own) : kcq;
  const bool mine1 = s1 + 64 + lane - 1 < kcq;
  const uint64_t v1 = mine1 ? sh[s1 + 64 + lane - 1] : ~0ull;
  const uint64_t has1 = ballot(mine1 && v1 != ~0ull);
  const uint64_t at1 = has1 & (~0ull << lane);
  uint64_t key1 = __shfl(v1, at1 ? __builtin_ctzll(at1) : 0, 64);
  if (!mine1 || at1 == 0) key1 = ~0ull;
  const uint64_t next1 = __shfl(v1, has1 ? __builtin_ctzll(has1) : 0, 64);  // the second group's first key
  const bool mine = lane >= 1 && s1 + lane - 1 < kcq;
  const uint64_t v = mine ? sh[s1 + lane - 1] : ~0ull;
  const uint64_t has = ballot(mine && v != ~0ull);
  const uint64_t at = has & (~0ull << lane);
  uint64_t key = __shfl(v, at ? __builtin_ctzll(at) : 0, 64);
  if (at == 0) key = has1 ? next1 : ~0ull;
  if (!mine) key = ~0ull;
  if (lane == 1) {  // the first cut: the clean position nearest to the first chunk's target, before or after it
    const uint64_t alt = sh[K];
    const int64_t tgt = pc.first;
    if (alt != 0 && (key == ~0ull || tgt - (int64_t)(uint32_t)alt < (int64_t)(uint32_t)key - tgt)) key = alt;
  }
  // keep a cut past the one before it (the keys do not decrease with the cut index)
  const uint64_t prev = __shfl_up(key, 1, 64);
  const bool keep = mine && key != ~0ull && (lane == 1 || (key >> 32) > (prev >> 32));
  const uint64_t kept = ballot(keep);
  const uint64_t last0 = __shfl(key, 63, 64);
  const uint64_t prev1 = lane == 0 ? last0 : __shfl_up(key1, 1, 64);
  const bool keep1 = mine1 && key1 != ~0ull && (key1 >> 32) > (prev1 >> 32);
  const uint64_t kept1 = ballot(keep1);
  const int idx = 1 + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(kept >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)kept, 0u));
  const int idx1 = 1 + __builtin_popcountll(kept) +
                   (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(kept1 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)kept1, 0u));
  if (keep) {
    bnd[idx] = (int32_t)(key >> 32);
    own_before[idx] = (int32_t)(uint32_t)key;
  }
  if (keep1) {
    bnd[idx1] = (int32_t)(key1 >> 32);
    own_before[idx1] = (int32_t)(uint32_t)key1;
  }
  if (lane == 0) {
    const int nk = 1 + __builtin_popcountll(kept) + __builtin_popcountll(kept1);
    bnd[0] = 0;
    own_before[0] = 0;
    bnd[nk] = (int32_t)limit;
    own_before[nk] = (int32_t)pc.own;
    w.cnum[chain] = nk;
    gstore(&w.cctl[chain], CCtl{0, 0, 0, 0, 0, 0});
  }
}

// the chunk's choice summary, made cumulative over buckets: entry b is the
// largest block chosen for any request of bucket b or below
__device__ __forceinline__ void store_choices(const Gw& w, int64_t slot, uint32_t g) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(g, o, 64);
    if (lane >= o) g = y > g ? y : g;
  }
  w.cg[slot * 64 + lane] = g;
}

// A round replays, per chain, in MODE 0 the frontier chunk alone; in MODE 1
// every chunk from the frontier on, each from the frontier's state; in MODE 2
// the frontier chunk extended to the end of the chain.
// One chunk on the LDS table: events [lo, hi) of the chain from the frontier's state.
// Returns kChunkGrew when the chunk created segments, kChunkStopped when it stopped.
constexpr int kChunkGrew = 1, kChunkStopped = 2;
template <bool KEEP = false>  // KEEP: a first chunk that spills keeps its lane registers (the paged rounds resume there)
__device__ __forceinline__ int fast_chunk(const Gw& w, const GMEM int64_t* off, const Derived& d, int64_t chain, int k,
                                           int64_t lo, int64_t hi, const CCtl& ctl, LMEM uint64_t* s_k,
                                           const GMEM int32_t* bound = nullptr, uint64_t ms_ticks = 0) {
  const int lane = threadIdx.x;
  const int K = w.chunks;
  const int64_t t = chain >> 1;
  const int pool_one = (int)(chain & 1);
  FastChain<1, true> c;
  c.base = off[t];
  c.n = off[t + 1] - c.base;
  FastPool& ps = c.p[0];
  ps.t.l = s_k;
  ps.segdir = 1;
  ps.segs = (GMEM uint64_t*)w.segs + c.base;  // not written in chunk mode
  ps.nseg = 0;
  ps.pool = pool_one;
  ps.split_min = pool_one == 0 ? d.split_min_u[0] : d.split_min_u[1];
  // a small-pool chunk may be certified, with its counts shifted by a delta: it
  // records every new maximum of its own from its first event on
  ps.maxfree = pool_one == 0 ? -1 : ctl.runmax;
  ps.n_mf = 0;
  if (ctl.f == 0) {
#pragma unroll
    for (int r = 0; r < kLdsRows; ++r) ps.t.l[64 * r + lane] = kNoKey;
    ps.t.n = 0;
    ps.bump = ps.created_u = 0;
    c.reserved_u = 0;
    c.created = 0;
  } else {  // the frontier's state: the end state of the chunk before it
    const GMEM uint64_t* src = w.cst + (chain * K + ctl.f - 1) * kStateWords;
    const uint64_t cw = src[kStateKeys + 3];
    const int32_t cnt = (int32_t)(uint32_t)cw;
    uint64_t none = kNoKey;
    asm volatile("" : "+v"(none));  // made here: a constant held through the task loop can take a spill slot
#pragma unroll
    for (int r = 0; r < kLdsRows; ++r) {
      const int32_t i = 64 * r + lane;
      ps.t.l[i] = i < cnt ? src[i] : none;
    }
    ps.t.n = cnt;
    ps.bump = src[kStateKeys];
    ps.created_u = src[kStateKeys + 1];
    c.reserved_u = src[kStateKeys + 2];
    c.created = (int32_t)(cw >> 32);
    if (ctl.nd > 0) {  // plus the delta keys (certification left room for them) and the counters after them
      const GMEM uint64_t* del = w.cdel + chain * kDeltaWords;
      if (lane < ctl.nd && cnt + lane < kLdsSlots) ps.t.l[cnt + lane] = del[lane];
      ps.t.n = cnt + ctl.nd;
      ps.bump = del[kMaxDelta];
      ps.created_u = del[kMaxDelta + 1];
      c.reserved_u = del[kMaxDelta + 2];
      c.created = (int32_t)del[kMaxDelta + 3];
    }
  }
  wave_order();
  const int32_t n0 = ps.t.n;
  c.released = c.n_res = 0;
  c.back_res = false;
  // the chunk's records sit at the chain's own-event positions: pool 0 from the
  // front of the trace's slots, pool 1 from the back (the pools' events are disjoint)
  const int64_t olo = w.cown[chain * (K + 1) + k];
  c.cres = (GMEM ChunkRes*)w.ovf + c.base + (pool_one ? c.n - 1 - olo : olo);
  c.cres_dir = pool_one ? -1 : 1;
  c.cmf = (GMEM MfRec*)w.segs + c.base + (pool_one ? c.n - 1 - olo : olo);
  c.cmf_dir = pool_one ? -1 : 1;
  c.bound = bound;
  c.k_self = k;
  const int32_t created0 = c.created;
  int status;
  int64_t stop;
  Resume rs{-1, 0, 0};
  chain_run<1>(c, d, w, pool_one, lo, hi, &status, &stop, KEEP ? &rs : nullptr, ms_ticks);
  if (status == kAbandoned) return 0;
  if (KEEP && status == kSpill && ctl.mode == 0 && ctl.f == 0) {
    // the first chunk outgrew the table (its state below is the one before the stopping event):
    // the lane registers go with it, to the paged state slot of chunk 1, which no chunk writes
    // before the paged replay has resumed from them
    GMEM uint64_t* fw = w.bstate + (chain * K + 1) * w.bstate_words;
    fw[lane] = rs.cur;
    fw[kWave + lane] = rs.prev;
  }
  GMEM uint64_t* dst = w.cst + (chain * K + k) * kStateWords;
#pragma unroll
  for (int r = 0; r < kLdsRows; ++r) {
    const int32_t i = 64 * r + lane;
    if (i < ps.t.n) dst[i] = ps.t.l[i];
  }
  if (lane == 0) {
    dst[kStateKeys] = ps.bump;
    dst[kStateKeys + 1] = ps.created_u;
    dst[kStateKeys + 2] = c.reserved_u;
    dst[kStateKeys + 3] = (uint64_t)(uint32_t)ps.t.n | ((uint64_t)(uint32_t)c.created << 32);
    gstore(&w.chdr[chain * K + k],
           CHdr{stop, status, c.n_res, ps.n_mf, c.created - created0, ps.maxfree > n0 ? ps.maxfree : n0, 0});
  }
  return (c.created != created0 ? kChunkGrew : 0) | (status != XMEM_T_OK ? kChunkStopped : 0);
}

// One wavefront per chain, after each of its rounds (BIG: a round on the paged
// sets): walks the chunks whose results are exact, moves their change
// points into the chain's record layout (free-count maxima only where they pass
// the running maximum), and advances the frontier; a finished chain gets its
// header.
//
// Certification (paged chains, and small-pool chains on the LDS table; for a
// large pool on the LDS table the choice summary per allocation did not repay
// its cost).  A chunk that created segments is exact when it ran from the
// right state, and since it frees what it allocates, its end state is the
// frontier's state plus its new segments, each one whole free block above every
// older address (the delta).  A later chunk that created no segment ran from
// the frontier's state without the delta; its run is still the true one when
// no allocation in it would have preferred a delta block, i.e. no delta size s
// has u <= s < S for a request u served by a block of size S (equal sizes go to
// the lower, older address), and the delta blocks fit in its table beside its
// largest free count.  The first condition holds by itself in the small pool
// (no small block is larger than a new small segment); elsewhere it is checked
// against the chunk's choice summary: per request bucket, the largest block
// chosen for that bucket or below, an upper bound of every S with u <= s.  A
// certified chunk's free counts are its own plus the delta's size, and it has
// no reserved change.  The first chunk not certified becomes the frontier,
// starting from the end state of the chunk before it plus the delta.
// The walk for one chain after a round of mode MODE.
// The n (<= 64) distinct keys of lanes [0, n) in descending order over the same lanes (each key's
// rank: the keys above it), through LDS; lanes past n get kNoKey.
__device__ __forceinline__ uint64_t wave_sort_desc(uint64_t v, int n, LMEM uint64_t* s) {
  const int lane = threadIdx.x;
  int rank = 0;
  for (int j = 0; j < n; ++j) rank += __shfl(v, j, 64) > v ? 1 : 0;
  wave_order();
  if (lane < n) s[rank] = v;
  wave_order();
  const uint64_t r = lane < n ? s[lane] : kNoKey;
  wave_order();
  return r;
}
// RENAME: small-pool chunks on the LDS table may be certified past later growers (below); only
// where every chunk of the round ran, i.e. no bound gave up the chunks past a second grower
// (chunks on the paged sets always run).
__device__ __forceinline__ void stitch_walk(const Gw& w, const GMEM int64_t* off, int64_t chain, const int MODE,
                                            const bool BIG, CCtl& ctl, int64_t* stop_out, int* status_out,
                                            LMEM uint64_t* s_del, const bool RENAME = true) {
  const int lane = threadIdx.x;
  const int K = w.chunks;
  const int64_t t = chain >> 1;
  const int pool_one = (int)(chain & 1);
  const int nk = w.cnum[chain];
  const int64_t base = off[t], n = off[t + 1] - base;
  // certification: paged chunks, and small-pool chunks on the LDS table, which need no choice
  // summary (a small request never prefers a whole new small segment: no small block is larger,
  // and an equal one sits at a lower address)
  const bool CERT = BIG || pool_one == 0;
  // the frontier state's bump: segments created by chunks replayed from it lie at or above it
  GMEM uint64_t* del = w.cdel + chain * kDeltaWords;
  uint64_t sf_bump = 0;
  if (CERT && ctl.nd > 0) sf_bump = del[kMaxDelta];
  else if (BIG && ctl.f > 0) sf_bump = w.bstate[(chain * K + ctl.f - 1) * w.bstate_words];
  else if (CERT && ctl.f > 0) sf_bump = w.cst[(chain * K + ctl.f - 1) * kStateWords + kStateKeys];
  const int32_t room = BIG ? 32 * w.bcap : kLdsSlots;  // free blocks a state certainly holds
  int nd = 0;              // delta keys of this walk (new segments of chunk jd)
  int jd = -1;
  uint64_t dkey = kNoKey;  // lane i < nd: delta key i, in descending address order
  uint64_t dc0 = 0, dc1 = 0, dc2 = 0, dc3 = 0;  // end-state counters of chunk jd
  int have = 0;            // delta segments the last walked chunk's end state holds (the lowest ones)
  int64_t stop = -1;
  int status = XMEM_T_OK;
  for (int k = ctl.f;; ++k) {
    const CHdr h = gload(&w.chdr[chain * K + k]);
    // A small-pool chunk on the paged sets that created segments although a delta was pending
    // ran from the state without the delta, and its new segments are the delta's lowest ones
    // (every small segment has one size, and both runs create them at the same bump, in the
    // same order): with the delta present, each of those requests takes the delta segment of
    // that address instead, and nothing else changes (no small request prefers a whole free
    // segment to a block it fits, and delta segments sit above every older block).  Its first
    // `renamed` records are no growth, and its free count lacks the delta segments it has not
    // yet taken; creations past the delta are true growth and extend it.
    int renamed = 0, kfound = 0;
    uint64_t kgot = kNoKey, kc0 = 0, kc1 = 0, kc2 = 0, kc3 = 0;
    if (nd > 0) {
      bool ok = h.status == XMEM_T_OK && h.maxc + nd <= room;
      if (ok && h.changed != 0) {
        ok = false;
        if (pool_one == 0 && (BIG || RENAME)) {
          bool over;
          if (BIG) {
            const GMEM uint64_t* st = w.bstate + (chain * K + k) * w.bstate_words;
            const int32_t cnt = (int32_t)(st[3] >> 32);
            const int32_t i = cnt - 1 - lane;
            const uint64_t a = i >= 0 ? st[8 + w.bstate_keys + i] : 0;
            const bool is_new = i >= 0 && akey_addr(a) >= sf_bump;
            kfound = __builtin_popcountll(ballot(is_new));
            over = kfound == kWave && cnt > kWave && akey_addr(st[8 + w.bstate_keys + cnt - 1 - kWave]) >= sf_bump;
            kgot = is_new ? key_of(akey_size(a), akey_addr(a)) : kNoKey;  // lane i < kfound: new key i, descending
            kc0 = st[0]; kc1 = st[1]; kc2 = st[2]; kc3 = st[4];
          } else {  // the saved table, unordered: its keys at or above the bump, then sorted
            const GMEM uint64_t* st = w.cst + (chain * K + k) * kStateWords;
            const uint64_t cw = st[kStateKeys + 3];
            const int32_t cnt = (int32_t)(uint32_t)cw;
            kc0 = st[kStateKeys]; kc1 = st[kStateKeys + 1]; kc2 = st[kStateKeys + 2]; kc3 = cw >> 32;
            for (int32_t r0 = 0; r0 < cnt; r0 += kWave) {
              const int32_t i = r0 + lane;
              const uint64_t x = i < cnt ? st[i] : kNoKey;
              const bool is_new = i < cnt && key_addr(x) >= sf_bump;
              const uint64_t m = ballot(is_new);
              const int pos = kfound + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
              if (is_new && pos < kMaxDelta) s_del[pos] = x;
              kfound += __builtin_popcountll(m);
            }
            wave_order();
            over = kfound > kMaxDelta;
            const uint64_t g = lane < kfound && !over ? s_del[lane] : kNoKey;
            wave_order();
            kgot = over ? kNoKey : wave_sort_desc(g, kfound, s_del);
          }
          if (k == nk - 1 && h.n_res == h.changed) {
            // the chain's last chunk ends where the trace does, not at a clean position, so its
            // new segments need not be whole free blocks at its end, and no later chunk starts
            // from its end state: its new segments are the delta's by construction alone
            ok = true;
            renamed = h.changed < nd ? h.changed : nd;
          } else if (!over && kfound == h.changed) {
            const int r = kfound < nd ? kfound : nd;
            // lane i < r: the (i+1)-th lowest new segment and the (i+1)-th lowest delta segment
            const uint64_t ak = __shfl(kgot, lane < kfound ? kfound - 1 - lane : 0, 64);
            const uint64_t ad = __shfl(dkey, lane < nd ? nd - 1 - lane : 0, 64);
            if (ballot(lane < r && ak != ad) == 0) {
              ok = true;
              renamed = r;
            }
          }
        }
      }
      if (ok && BIG) {
        const uint64_t sz = key_size(dkey);
        const uint32_t g = lane < nd ? w.cg[(chain * K + k) * 64 + gbucket(sz)] : 0u;
        ok = ballot(lane < nd && (uint64_t)g > sz) == 0;
      }
      if (!ok) {  // chunk k becomes the frontier
        ctl.f = k;
        ctl.nd = nd - have;  // the end state of chunk k - 1 holds the lowest `have` delta segments already
        if (ctl.nd > 0) {
          if (lane < ctl.nd) del[lane] = dkey;
          if (lane == 0) {
            del[kMaxDelta] = dc0;
            del[kMaxDelta + 1] = dc1;
            del[kMaxDelta + 2] = dc2;
            del[kMaxDelta + 3] = dc3;
          }
        }
        break;
      }
    }
    const int64_t olo = w.cown[chain * (K + 1) + k];
    const GMEM ChunkRes* cr = (const GMEM ChunkRes*)w.ovf + base + (pool_one ? n - 1 - olo : olo);
    const GMEM MfRec* cm = (const GMEM MfRec*)w.segs + base + (pool_one ? n - 1 - olo : olo);
    const int dir = pool_one ? -1 : 1;
    for (int32_t i = renamed + lane; i < h.n_res; i += kWave) {
      const ChunkRes r = gload(&cr[(int64_t)dir * i]);
      const int64_t j = ctl.n_res + (i - renamed);
      gstore(&w.res[pool_one ? base + n - 1 - j : base + j], ResRec{r.reserved, r.event, r.created, 0, 0});
    }
    ctl.n_res += h.n_res - renamed;
    if (renamed > 0) {
      // true count = own count + nd - (renamed creations so far): a shift that only falls, so every
      // true new maximum is one of the chunk's own; each is kept if above everything before it
      const int32_t cev = lane < renamed ? gload(&cr[(int64_t)dir * lane]).event : INT32_MAX;
      int32_t run = ctl.runmax;
      for (int32_t i0 = 0; i0 < h.n_mf; i0 += kWave) {
        const int32_t i = i0 + lane;
        const MfRec r = i < h.n_mf ? gload(&cm[(int64_t)dir * i]) : MfRec{INT32_MAX, INT32_MIN};
        int c = 0;
        for (int j = 0; j < renamed; ++j) c += __shfl(cev, j, 64) <= r.event ? 1 : 0;
        const int32_t tv = i < h.n_mf ? r.value + (nd - c) : INT32_MIN;
        int32_t pm = tv;  // inclusive prefix maximum up the lanes
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const int32_t y = __shfl_up(pm, o, 64);
          if (lane >= o) pm = y > pm ? y : pm;
        }
        const int32_t ex = __shfl_up(pm, 1, 64);
        const int32_t before = lane == 0 ? run : (ex > run ? ex : run);
        const bool keep = i < h.n_mf && tv > before;
        const uint64_t km = ballot(keep);
        const int pos = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(km >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)km, 0u));
        if (keep) {
          const int64_t j = ctl.n_mf + pos;
          gstore(&w.mf[pool_one ? base + n - 1 - j : base + j], MfRec{r.event, tv});
        }
        ctl.n_mf += __builtin_popcountll(km);
        const int32_t gm = __shfl(pm, 63, 64);
        run = gm > run ? gm : run;
      }
      ctl.runmax = run;
    }
    // the chunk's maxima (of its own counts, plus the delta) increase: keep those above the running maximum
    int32_t first = h.n_mf;
    for (int32_t i0 = 0; renamed == 0 && i0 < h.n_mf; i0 += kWave) {
      const int32_t i = i0 + lane;
      const uint64_t m = ballot(i < h.n_mf && cm[(int64_t)dir * i].value + nd > ctl.runmax);
      if (m) {
        first = i0 + __builtin_ctzll(m);
        break;
      }
    }
    for (int32_t i = first + lane; i < h.n_mf; i += kWave) {
      const int64_t j = ctl.n_mf + (i - first);
      const MfRec r = gload(&cm[(int64_t)dir * i]);
      gstore(&w.mf[pool_one ? base + n - 1 - j : base + j], MfRec{r.event, r.value + nd});
    }
    if (first < h.n_mf) {
      ctl.runmax = cm[(int64_t)dir * (h.n_mf - 1)].value + nd;
      ctl.n_mf += h.n_mf - first;
    }
    if (h.status != XMEM_T_OK) {
      ctl.done = 1;
      stop = h.stop;
      status = h.status;
      break;
    }
    if (MODE == 2 || k == nk - 1) {
      ctl.done = 1;
      break;
    }
    if (MODE == 0) {
      ctl.f = k + 1;
      ctl.nd = 0;
      break;
    }
    if (h.changed != 0 && !CERT) {  // the chunks after it ran from a stale state
      ctl.f = k + 1;
      ctl.nd = 0;
      break;
    }
    if (renamed > 0) {
      if (kfound > nd) {  // growth past the delta: its end state holds the whole, larger delta
        dkey = kgot;
        nd = kfound;
        jd = k;
        dc0 = kc0; dc1 = kc1; dc2 = kc2; dc3 = kc3;
      }
      have = kfound;
      continue;
    }
    have = 0;
    if (h.changed != 0) {  // exact (nd == 0 here): its new segments become the delta
      uint64_t c0, c1, c2, c3, got;
      int found = 0;
      bool over = false;
      if (BIG) {
        // the end state's keys in address order: the new segments are the last entries
        const GMEM uint64_t* st = w.bstate + (chain * K + k) * w.bstate_words;
        const int32_t cnt = (int32_t)(st[3] >> 32);
        c0 = st[0]; c1 = st[1]; c2 = st[2]; c3 = st[4];
        const int32_t i = cnt - 1 - lane;
        const uint64_t a = i >= 0 ? st[8 + w.bstate_keys + i] : 0;
        const bool is_new = i >= 0 && akey_addr(a) >= sf_bump;
        found = __builtin_popcountll(ballot(is_new));
        over = found == kWave && cnt > kWave && akey_addr(st[8 + w.bstate_keys + cnt - 1 - kWave]) >= sf_bump;
        got = is_new ? key_of(akey_size(a), akey_addr(a)) : kNoKey;  // lane i < found: new key i
      } else {
        // the end state's table, unordered: gather the keys at or above the bump in LDS
        const GMEM uint64_t* st = w.cst + (chain * K + k) * kStateWords;
        const uint64_t cw = st[kStateKeys + 3];
        const int32_t cnt = (int32_t)(uint32_t)cw;
        c0 = st[kStateKeys]; c1 = st[kStateKeys + 1]; c2 = st[kStateKeys + 2]; c3 = cw >> 32;
        for (int32_t r0 = 0; r0 < cnt; r0 += kWave) {
          const int32_t i = r0 + lane;
          const uint64_t x = i < cnt ? st[i] : kNoKey;
          const bool is_new = i < cnt && key_addr(x) >= sf_bump;
          const uint64_t m = ballot(is_new);
          const int pos = found + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
          if (is_new && pos < kMaxDelta) s_del[pos] = x;
          found += __builtin_popcountll(m);
        }
        wave_order();
        over = found > kMaxDelta || found != h.changed;
        got = lane < found && !over ? s_del[lane] : kNoKey;
        wave_order();
        if (!over) got = wave_sort_desc(got, found, s_del);  // descending, as from the paged state
      }
      if (over || found == 0) {  // too many new segments to track: chunk k + 1 is the frontier
        ctl.f = k + 1;
        ctl.nd = 0;
        break;
      }
      dkey = got;
      nd = found;
      jd = k;
      dc0 = c0; dc1 = c1; dc2 = c2; dc3 = c3;
      have = nd;
    }
  }
  *stop_out = stop;
  *status_out = status;
}

// ------------------------------------------------------------------ chunk scheduler (many traces)
// One persistent grid of replay wavefronts takes chunk tasks from a queue
// instead of one launch per round, so a chain's next round starts as soon as
// the last chunk of its current round is done: one chain's second round runs
// beside other chains' first, and no round waits for the slowest chain of the
// batch.  The wavefront that finishes a chain's last pending chunk walks the
// chain and queues the chunks of its next round.
// The queue is a ticket FIFO: a wavefront draws the next ticket (one atomic
// add, so wavefronts never retry against each other) and waits for the task of
// that slot; a producer reserves its slots with another atomic add and writes
// the task words.  Tickets drawn past the last task wait until every chain is
// done.  Every wavefront leaves once all chains are done, or after a safety
// time limit (then the chains not done are reported as aborted).
constexpr uint64_t kTaskValid = 1ull << 63;
__device__ __forceinline__ uint64_t task_word(int64_t chain, int k, int mode) {
  return kTaskValid | ((uint64_t)chain << 16) | ((uint64_t)k << 2) | (uint64_t)mode;
}
__device__ __forceinline__ uint32_t q_load(const GMEM uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void q_abort(const Gw& w) {
  __hip_atomic_store(w.cqc + kQAbort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t rfl64(uint64_t v) {
  return (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v) |
         ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32)) << 32);
}

// lane 0 only: the task of ticket t, or 0 once every chain is done (or the
// safety limit has passed).  The limit counts from the last sign of progress
// seen while waiting: a task queued, finished or still running (tickets below
// the reservations not all finished), or a chain done; a task that runs long
// therefore never trips it.  The wait between looks grows from about 0.1 us
// to 14 us.
__device__ uint64_t q_wait(const Gw& w, uint32_t t, int64_t nchains, uint64_t limit) {
  const GMEM uint64_t* slot = w.cq + t;
  uint64_t since = wall_clock64();
  uint32_t seen_resv = 0, seen_fin = 0, seen_done = 0;
  for (int idle = 0;; idle = idle < 8 ? idle + 1 : 8) {
    if (t < (uint64_t)w.cq_cap) {
      const uint64_t x = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (x != 0) return x;
    }
    const uint32_t done = q_load(w.cqc + kQDone);
    if (done >= (uint64_t)nchains || q_load(w.cqc + kQAbort) != 0) return 0;
    const uint32_t resv = q_load(w.cqc + kQResv), fin = q_load(w.cqc + kQFin), head = q_load(w.cqc + kQHead);
    const uint64_t now = wall_clock64();
    if (resv != seen_resv || fin != seen_fin || done != seen_done || fin < (head < resv ? head : resv)) {
      since = now;
      seen_resv = resv;
      seen_fin = fin;
      seen_done = done;
    } else if (now - since > limit) {
      q_abort(w);
      return 0;
    }
    if (idle < 5) {
      for (int i = 0; i < (4 << idle); ++i) __builtin_amdgcn_s_sleep(1);
    } else {
      for (int i = 0; i < (1 << (idle - 5)); ++i) __builtin_amdgcn_s_sleep(127);
    }
  }
}

// A speculative round keeps at most kWindow of its chunks queued or running: the walk queues
// the first kWindow, and each finished chunk queues the round's next one, unless the walk is
// already known to stop before it, in which case that chunk and every later one are never run.
// A large pool's walk (such a chain is not certified: the chunks after one that created segments
// ran from a stale state) stops at the first chunk that created segments or stopped; a small
// pool's walk certifies past the first chunk that created segments, but stops at the second one,
// or at a chunk that stopped.  The window trades a chain's round latency for fewer stale chunks,
// which pays when the chains' windows alone keep the chip busy (a chain per 4 scheduler
// wavefronts or more: 1.5 windowed tasks per wavefront).
//
// A batch of fewer chains queues a large pool's round all at once, and half of a small pool's
// first speculative round, each of those queuing one more when it is done.  Small-pool chunks
// are the short ones (the large pool's chunks hold whole iterations), and a chain's small-pool
// round ends before its large-pool round starts; queued all at once they would take the
// wavefronts first and leave the long large-pool tasks for the end of the queue, where the last
// of them run on an emptying chip.  Half of them queued at once, the other half behind whatever
// was queued meanwhile, the short tasks fill the end instead.
//
// Once the queue holds fewer tasks not yet taken than a third of the scheduler's wavefronts
// (wavefronts about to wait, near the end of the batch), a round starts, and a finished chunk
// continues, by queuing all of its round's remaining chunks up to where the walk would stop:
// chunks that may turn out stale then run on wavefronts that would otherwise wait, and the
// chains at the end of the batch are not held to their windows' latency.
constexpr int kWindow = 6;
__device__ __forceinline__ bool sched_starved(const Gw& w) {
  const uint32_t resv = q_load(w.cqc + kQResv), head = q_load(w.cqc + kQHead);
  return (int32_t)(resv - head) < (int32_t)(gridDim.x / 3);
}
// whether a batch's rounds are windowed (the scheduler's instance is chosen on the host by it)
__host__ __device__ inline bool sched_windowed(int64_t waves, int64_t nchains) { return 4 * nchains >= waves; }
// the tasks of a round queued by the walk; the rest are queued by finished chunks
__device__ __forceinline__ int sched_first_tasks(int64_t chain, int mode, int rounds, int n, int win) {
  if (mode != 1) return n;
  if (win < n) return win;
  return (chain & 1) || rounds ? n : (n + 1) / 2;
}

// After the last chunk of a chain's round: the walk, then the next round's tasks.
__device__ void sched_walk(const Gw& w, const GMEM int64_t* off, int64_t chain, int64_t nchains, int win,
                           LMEM uint64_t* s_del, bool rename) {
  const int lane = threadIdx.x;
  CCtl ctl = gload(&w.cctl[chain]);
  const int mode = ctl.mode;
  int64_t stop;
  int status;
  stitch_walk(w, off, chain, mode, false, ctl, &stop, &status, s_del, rename);
  if (!ctl.done) {
    if (mode == 0) {
      ctl.mode = 1;
      ctl.rounds = 0;
    } else if (mode == 1 && ++ctl.rounds >= kSpecRounds) {
      ctl.mode = 2;
    }
  }
  const int nk = w.cnum[chain];
  const int n = ctl.done ? 0 : ctl.mode == 1 ? nk - ctl.f : 1;  // at most kMaxChunks
  int nq = sched_first_tasks(chain, ctl.mode, ctl.rounds, n, win);  // queued now; the rest by finished chunks
  if (nq < n && __builtin_amdgcn_readfirstlane((int)(lane == 0 && sched_starved(w)))) nq = n;
  if (lane == 0) {
    gstore(&w.cctl[chain], ctl);
    if (ctl.done) gstore(&w.hdr[chain], ChainHdr{stop, status, ctl.n_res, ctl.n_mf, 0, 0});
    else w.cpend[chain] = n;
    w.cpend[nchains + chain] = nk;  // no chunk of the new round has created segments or stopped yet
    w.cpend[2 * nchains + chain] = ctl.f + nq;
    w.cdel[chain * kDeltaWords + kRoundMask] = 0;
  }
  // release: the walk's results before the chain counts as done or its next tasks appear (a
  // one-way fence: a full one would also invalidate this XCD's L2 for every wavefront on it)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  if (ctl.done) {
    if (lane == 0) __hip_atomic_fetch_add(w.cqc + kQDone, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  uint32_t base = 0;
  if (lane == 0) base = __hip_atomic_fetch_add(w.cqc + kQResv, (uint32_t)nq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  base = (uint32_t)__builtin_amdgcn_readfirstlane((int)base);
  if ((int64_t)base + nq > w.cq_cap) {  // cannot happen: a chain queues at most one task per chunk and round
    if (lane == 0) q_abort(w);
    return;
  }
  if (lane < nq)
    __hip_atomic_store(w.cq + base + lane, task_word(chain, ctl.mode == 1 ? ctl.f + lane : ctl.f, ctl.mode),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// lane 0: after task k of a speculative round, the round's next chunk not yet queued (all of
// them up to the bound when the queue is short; none once the walk is known to stop before it).
// out: what task k reported (kChunkGrew, kChunkStopped).  Returns the chunks of the round given
// up here, which will never run.  Every chunk past the round's first tasks is claimed once, by
// one atomic add (or the final maximum) on the chain's next-chunk word, and then either queued
// or given up.
__device__ __forceinline__ int sched_successor(const Gw& w, int64_t chain, int64_t nchains, int k, int mode, int nk,
                                               int out, bool rename) {
  if (mode != 1) return 0;
  // the round's bound (the walk stops at or before that chunk): a large pool's first chunk that
  // created segments or stopped; a small pool's first chunk that stopped, and, unless its walk
  // certifies later growing chunks too (rename), its second that created segments.  Whichever of
  // two growing chunks reports second sees both bits, so the word settles on the true second one
  // and never drops below it.
  GMEM int32_t* first_end = w.cpend + nchains + chain;
  if ((chain & 1) ? out != 0 : (out & kChunkStopped) != 0)
    __hip_atomic_fetch_min(first_end, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (!rename && !(chain & 1) && (out & kChunkGrew)) {
    GMEM uint64_t* grew = w.cdel + chain * kDeltaWords + kRoundMask;
    const uint64_t m =
        __hip_atomic_fetch_or(grew, 1ull << k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) | (1ull << k);
    const uint64_t m2 = m & (m - 1);  // without the first chunk that grew: the second is its lowest bit
    if (m2) __hip_atomic_fetch_min(first_end, (int32_t)__builtin_ctzll(m2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  GMEM int32_t* next = w.cpend + 2 * nchains + chain;
  if (__hip_atomic_load(next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= nk) return 0;  // all claimed
  const int bound = __hip_atomic_load(first_end, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // a bound read late only lets a stale chunk run, which the walk never reads
  const int want = sched_starved(w) ? kMaxChunks : 1;
  const int c = __hip_atomic_fetch_add(next, want, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (c >= nk) return 0;
  const int e = c + want < nk ? c + want : nk;     // claimed: chunks c .. e - 1
  const int qe = bound + 1 < e ? bound + 1 : e;    // of which these are queued: c .. qe - 1
  const int nq = qe > c ? qe - c : 0;
  int given_up = e - c - nq;
  if (e < nk && bound < e) {  // the rest lies past the bound as well: claimed and given up now
    const int o = __hip_atomic_fetch_max(next, nk, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (o < nk) given_up += nk - o;
  }
  if (nq > 0) {
    const uint32_t slot = __hip_atomic_fetch_add(w.cqc + kQResv, (uint32_t)nq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((int64_t)slot + nq > w.cq_cap) {  // cannot happen: the round's tasks are counted in the queue's size
      q_abort(w);
      return 0;
    }
    for (int i = 0; i < nq; ++i)
      __hip_atomic_store(w.cq + slot + i, task_word(chain, c + i, mode), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return given_up;
}

// The scheduler's arguments, read through the kernel-argument pointer afresh in
// each phase of a task (taking it, replaying the chunk, the walk), so that the
// workspace pointers a phase needs are not held in registers through the
// others' loops.
struct SchedArgs {
  Ws ws;
  Derived d;
  const int64_t* off;
  int64_t nchains;
  uint64_t limit;
};
#define KARG __attribute__((address_space(4)))
__device__ __forceinline__ const KARG SchedArgs* sched_args() {
  uint64_t p = (uint64_t)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(p));
  return (const KARG SchedArgs*)p;
}
// whole-struct copy out of the kernel-argument segment, 8 bytes at a time
template <class T>
__device__ __forceinline__ T kload(const KARG T* p) {
  static_assert(sizeof(T) % 8 == 0, "8-byte multiple");
  T v;
  const KARG uint64_t* q = (const KARG uint64_t*)p;
  uint64_t* d = reinterpret_cast<uint64_t*>(&v);
#pragma unroll
  for (size_t i = 0; i < sizeof(T) / 8; ++i) d[i] = q[i];
  return v;
}

// WIN: the batch's rounds are windowed, and a running chunk past its round's bound is abandoned
// (a batch of fewer chains runs the instance with no such check in its event loop, which it
// would pay for without gaining)
template <bool WIN, bool AGED>
__device__ __forceinline__ void sched_run(LMEM uint64_t* s_k) {
  const int lane = threadIdx.x;
  for (;;) {
    uint64_t task = 0;
    {
      const KARG SchedArgs* A = sched_args();
      const Ws ws = kload(&A->ws);
      const Gw w = typed(ws);
      if (w.ctl[0]) return;
      if (lane == 0) {
        const uint32_t t = __hip_atomic_fetch_add(w.cqc + kQHead, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        task = q_wait(w, t, A->nchains, A->limit);
      }
      task = rfl64(task);
    }
    if (task == 0) return;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // the frontier the chain's last walk wrote
    const int64_t chain = (int64_t)((task >> 16) & 0x7fffffffffffull);
    const int k = (int)((task >> 2) & 63);
    const int mode = (int)(task & 3);
    int nk;
    int out;
    {
      const KARG SchedArgs* A = sched_args();
      const Ws ws = kload(&A->ws);
      const Gw w = typed(ws);
      const Derived d = kload(&A->d);
      const int K = w.chunks;
      const CCtl ctl = gload(&w.cctl[chain]);
      nk = w.cnum[chain];
      const GMEM int32_t* bnd = w.cbound + chain * (K + 1);
      // without windows (a batch of fewer chains): a chunk of a chain's later round, which the
      // chain waits for, issues before first-round chunks on its SIMD (its priority: the round,
      // at most 3; the rest in one piece: 3).  With windows the rounds interleave, and it costs.
      const int tp = WIN ? 0 : mode == 2 ? 3 : ctl.rounds > 2 ? 3 : ctl.rounds;
      if (tp == 1) __builtin_amdgcn_s_setprio(1);
      else if (tp == 2) __builtin_amdgcn_s_setprio(2);
      else if (tp >= 3) __builtin_amdgcn_s_setprio(3);
      out = fast_chunk(w, gp(A->off), d, chain, k, bnd[k], mode == 2 ? bnd[nk] : bnd[k + 1], ctl, s_k,
                       WIN && mode == 1 ? w.cpend + A->nchains + chain : nullptr,
                       AGED ? A->limit / (kSchedLimitSeconds * 1000) : 0);
      if (tp) __builtin_amdgcn_s_setprio(0);
    }
    // release: this chunk's state, records and header before it counts as done; and, for a
    // successor task queued below, what this task acquired (the walk's frontier), so that the
    // successor's taker, which acquires after reading its task word, sees it too
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    {
      const KARG SchedArgs* A = sched_args();
      const Ws ws = kload(&A->ws);
      const Gw w = typed(ws);
      int last = 0;
      if (lane == 0) {
        // this task and the tasks of the round that will never run
        const int done = 1 + sched_successor(w, chain, A->nchains, k, mode, nk, out, WIN && !AGED);
        last = __hip_atomic_fetch_add(w.cpend + chain, -done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == done;
      }
      if (__builtin_amdgcn_readfirstlane(last)) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // the other chunks of the round
        sched_walk(w, gp(A->off), chain, A->nchains, WIN ? kWindow : kMaxChunks, s_k, WIN && !AGED);
      }
      // counted after the walk queued the next round, so that a waiting wavefront sees either
      // this task in flight or the new reservations
      if (lane == 0) __hip_atomic_fetch_add(w.cqc + kQFin, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}
template <bool WIN>
__global__ __launch_bounds__(kWave, 6) void k_chunk_sched(SchedArgs args) {
  (void)args;  // the first argument: at the start of the kernel-argument segment
  __shared__ uint64_t s_k[kLdsSlots];  // the chunk's table; then the walk's delta keys
  sched_run<WIN, false>((LMEM uint64_t*)s_k);
}
// Batches of few chunks per pool (fewer than 16): every task is a long part of its chain, and
// the batch ends with its slowest chains.  Windowed rounds, and each chunk raises its
// wavefront's issue priority as it ages (chain_run), so that a SIMD's oldest tasks go first.
// Short tasks never reach an age check, but the loop state costs the kernels of finer batches
// about 1-2%, so they run the instances above.
__global__ __launch_bounds__(kWave, 6) void k_chunk_sched_aged(SchedArgs args) {
  (void)args;
  __shared__ uint64_t s_k[kLdsSlots];
  sched_run<true, true>((LMEM uint64_t*)s_k);
}

// Before k_chunk_sched: an empty queue, then every chain's first chunk (large pools first).
__global__ void k_chunk_qinit(int64_t T, Ws ws) {
  const Gw w = typed(ws);
  const int64_t nchains = 2 * T, nslots = w.cq_cap;
  int64_t n = nslots > nchains ? nslots : nchains;
  if (n < kQWords) n = kQWords;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    if (i < nslots) w.cq[i] = i < nchains ? task_word(i < T ? 2 * i + 1 : 2 * (i - T), 0, 0) : 0;
    if (i < nchains) {
      w.cpend[i] = 1;
      w.cpend[nchains + i] = kMaxChunks;
      w.cpend[2 * nchains + i] = kMaxChunks;
    }
    if (i < kQWords) w.cqc[i] = i == kQResv ? (uint32_t)nchains : 0u;
  }
}

// After k_chunk_sched: a chain it left unfinished (safety time limit) is reported as aborted.
__global__ void k_chunk_sched_end(int64_t nchains, Ws ws) {
  const Gw w = typed(ws);
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (w.ctl[0] || i >= nchains || w.cqc[kQAbort] == 0) return;
  if (!w.cctl[i].done) gstore(&w.hdr[i], ChainHdr{0, XMEM_T_ABORTED, 0, 0, 0, 0});
}
// After the scheduler, where the batch has paged slots: a pool that spilled (its chain done with
// kSpill) starts the paged-set rounds from the beginning of its chain; every other chain counts
// as done for them (its header stays as the scheduler left it).
__global__ void k_combo_adopt(int64_t nchains, Ws ws) {
  const Gw w = typed(ws);
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (w.ctl[0] || i >= nchains) return;
  const CCtl c = gload(&w.cctl[i]);
  if (c.done && w.hdr[i].status == kSpill) gstore(&w.cctl[i], CCtl{0, 0, 0, 0, 0, 0, 0, 1, 0, 0});
  else if (!c.done) w.cctl[i].done = 1;
}

// ------------------------------------------------------------------ paged chain: sorted key pages
// A chain whose pool outgrows its LDS table is replayed again by k_replay_big,
// with each pool's free blocks held twice, in paged sorted sets: by key (size,
// address), where best fit (Section 3.4 (iii)) is the first key >= (u << 32),
// and by address key (address, size), where a block's free physical neighbours
// are the entries just before and after its own address (Section 3.4 (iii),
// coalescing).  A set is a sequence of pages of at most kPage sorted keys in
// this workgroup's slot of the workspace.  An LDS directory holds each page's
// first key, id and count in key order, and one register per lane holds the
// first key of every 64th directory entry, so a key is located with two
// ballots.  A full page splits; a page that falls below half merges with a
// neighbour or takes keys from it, so every page but a lone one is at least
// half full.  A set that would need more pages than its directory holds hands
// the chain to the 64-bit kernel (status kRetry).
constexpr int kPage = 64;
constexpr int32_t kBigDir1 = 4096;  // directory entries per set: chains of one pool (two sets)
constexpr int32_t kBigDir2 = 2048;  // directory entries per set: chains of both pools (four sets)
constexpr int kBigSlots = 64;       // chains the paged kernel replays at once
constexpr int64_t kBigSlotKeys = 4 * (int64_t)(kBigDir2 + 2) * kPage;
static_assert(2 * (int64_t)(kBigDir1 + 2) * kPage <= kBigSlotKeys, "slot holds both layouts");
static_assert(kBigDir1 <= 64 * kWave, "one summary register covers the directory");
static_assert(kBigSlotKeys == kBigSlotKeysHost && kBigSlots == 64, "the workspace carving matches this layout");

__device__ __forceinline__ uint32_t uni(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t uni64(uint64_t v) {
  return (uint64_t)uni((uint32_t)v) | ((uint64_t)uni((uint32_t)(v >> 32)) << 32);
}
__device__ __forceinline__ int msb64(uint64_t m) { return 63 - __builtin_clzll(m); }

struct Pss {
  LMEM uint64_t* dkey;   // first key of directory entry i < np, ascending
  LMEM uint32_t* dpg;    // entry i < np: page id | count << 16; the last nfree words: free page ids
  GMEM uint64_t* pages;  // page p: key l at pages[kPage * p + l], ascending, kNoKey past the count
  uint64_t S;            // lane r: dkey[64 r] (kNoKey past the directory)
  uint64_t cv;           // keys of page cpid: the last page loaded or stored
  int32_t cpid, np, nfree, bump, cap, nkeys;
};

__device__ __forceinline__ void pss_init(Pss& P, LMEM uint64_t* dkey, LMEM uint32_t* dpg, GMEM uint64_t* pages,
                                         int32_t cap) {
  P.dkey = dkey; P.dpg = dpg; P.pages = pages;
  P.S = kNoKey; P.cv = kNoKey; P.cpid = -1;
  P.np = P.nfree = P.bump = P.nkeys = 0;
  P.cap = cap;
}
__device__ __forceinline__ void pss_summary(Pss& P) {
  const int32_t k = 64 * (int32_t)threadIdx.x;
  P.S = k < P.np ? P.dkey[k] : kNoKey;
}
struct Ent { int32_t pid, cnt; };
__device__ __forceinline__ Ent pss_decode(const Pss& P, uint32_t e) {
  const int32_t pid = (int32_t)(e & 0xffffu);
  return Ent{pid <= P.cap + 1 ? pid : P.cap + 1, (int32_t)(e >> 16)};  // ids stay inside the set's pages
}
__device__ __forceinline__ Ent pss_ent(const Pss& P, int32_t i) { return pss_decode(P, uni(P.dpg[i])); }
// last directory entry whose first key is <= x (-1 if none), and that entry: the row's first keys
// and page words are read together, so the entry costs no second LDS round trip
__device__ __forceinline__ int32_t pss_locate(const Pss& P, uint64_t x, Ent* en) {
  const uint64_t m = ballot(P.S <= x);
  if (!m) return -1;
  const int32_t r0 = 64 * msb64(m);
  const int32_t k = r0 + (int32_t)threadIdx.x;
  const uint64_t dk = k < P.np ? P.dkey[k] : kNoKey;
  const uint32_t dp = k < P.np ? P.dpg[k] : 0u;
  const int l = msb64(ballot(dk <= x));
  *en = pss_decode(P, rl(dp, l));
  return r0 + l;
}
__device__ __forceinline__ void pss_set(Pss& P, int32_t i, uint64_t first, int32_t pid, int32_t cnt) {
  if (threadIdx.x == 0) { P.dkey[i] = first; P.dpg[i] = (uint32_t)pid | ((uint32_t)cnt << 16); }
  if ((i & 63) == 0) P.S = (int)threadIdx.x == (i >> 6) ? first : P.S;
  wave_order();
}
__device__ __forceinline__ uint64_t page_get(Pss& P, int32_t pid) {
  if (pid != P.cpid) {
    P.cv = P.pages[(int64_t)kPage * pid + threadIdx.x];
    P.cpid = pid;
  }
  return P.cv;
}
__device__ __forceinline__ void page_put(Pss& P, int32_t pid, uint64_t v) {
  P.pages[(int64_t)kPage * pid + threadIdx.x] = v;
  P.cv = v;
  P.cpid = pid;
}
__device__ __forceinline__ int32_t page_new(Pss& P) {
  if (P.nfree > 0) {
    const int32_t pid = (int32_t)uni(P.dpg[P.cap + 2 - P.nfree]);
    P.nfree -= 1;
    return pid;
  }
  return P.bump++;  // at most cap + 1 pages are ever in use
}
__device__ __forceinline__ void page_drop(Pss& P, int32_t pid) {
  P.nfree += 1;
  if (threadIdx.x == 0) P.dpg[P.cap + 2 - P.nfree] = (uint32_t)pid;
  wave_order();
  if (P.cpid == pid) P.cpid = -1;
}
// the page with key v at lane pos removed; lane 63 becomes empty
__device__ __forceinline__ uint64_t page_del(uint64_t v, int pos) {
  const int lane = threadIdx.x;
  uint64_t up = from_upper_lane(v);
  up = lane == 63 ? kNoKey : up;
  return lane >= pos ? up : v;
}
// the page (fewer than kPage keys) with x inserted at lane pos
__device__ __forceinline__ uint64_t page_ins(uint64_t v, int pos, uint64_t x) {
  const int lane = threadIdx.x;
  const uint64_t dn = from_lower_lane(v);
  return lane > pos ? dn : (lane == pos ? x : v);
}
// entries [i, np) move up one (rows from the last, each read before it is written)
__device__ __forceinline__ void dir_shift_up(LMEM uint64_t* dkey, LMEM uint32_t* dpg, int32_t np, int32_t i) {
  const int32_t lane = threadIdx.x;
  for (int32_t r0 = ((np - 1) >> 6) << 6; r0 >= (i & ~63); r0 -= 64) {
    const int32_t k = r0 + lane;
    const bool mv = k >= i && k < np;
    const uint64_t a = mv ? dkey[k] : 0;
    const uint32_t b = mv ? dpg[k] : 0;
    wave_order();
    if (mv) { dkey[k + 1] = a; dpg[k + 1] = b; }
    wave_order();
  }
}
// entries [i + 1, np) move down one (rows from the first)
__device__ __forceinline__ void dir_shift_down(LMEM uint64_t* dkey, LMEM uint32_t* dpg, int32_t np, int32_t i) {
  const int32_t lane = threadIdx.x;
  for (int32_t r0 = (i + 1) & ~63; r0 < np; r0 += 64) {
    const int32_t k = r0 + lane;
    const bool mv = k > i && k < np;
    const uint64_t a = mv ? dkey[k] : 0;
    const uint32_t b = mv ? dpg[k] : 0;
    wave_order();
    if (mv) { dkey[k - 1] = a; dpg[k - 1] = b; }
    wave_order();
  }
}
__device__ __forceinline__ void pss_dir_insert(Pss& P, int32_t i, uint64_t first, int32_t pid, int32_t cnt) {
  dir_shift_up(P.dkey, P.dpg, P.np, i);
  P.np += 1;
  if (threadIdx.x == 0) { P.dkey[i] = first; P.dpg[i] = (uint32_t)pid | ((uint32_t)cnt << 16); }
  wave_order();
  pss_summary(P);
}
__device__ __forceinline__ void pss_dir_remove(Pss& P, int32_t i) {
  dir_shift_down(P.dkey, P.dpg, P.np, i);
  P.np -= 1;
  wave_order();
  pss_summary(P);
}

// first key >= x (kNoKey if none)
__device__ __forceinline__ uint64_t pss_first_ge(Pss& P, uint64_t x) {
  if (P.np == 0) return kNoKey;
  Ent en;
  const int32_t i = pss_locate(P, x, &en);
  if (i < 0) return rl64(P.S, 0);  // x is below every key
  const uint64_t v = page_get(P, en.pid);
  const uint64_t m = ballot(v >= x);
  const int pos = m ? __builtin_ctzll(m) : kPage;
  if (pos < en.cnt) return rl64(v, pos);
  return i + 1 < P.np ? uni64(P.dkey[i + 1]) : kNoKey;
}
// last key <= x (kNoKey if none)
__device__ __forceinline__ uint64_t pss_last_le(Pss& P, uint64_t x) {
  if (P.np == 0) return kNoKey;
  Ent en;
  const int32_t i = pss_locate(P, x, &en);
  if (i < 0) return kNoKey;
  const uint64_t v = page_get(P, en.pid);
  return rl64(v, msb64(ballot(v <= x)));  // the page's first key is <= x
}

constexpr int kOpErase = 0, kOpInsert = 1, kOpRekey = 2;

// Page i (keys w, count cnt) fell below half: merge it with a neighbour, or even
// the two out when together they fill more than a page.
__device__ __forceinline__ void pss_rebalance(Pss& P, LMEM uint64_t* stage, int32_t i, uint64_t w, int32_t pid,
                                              int32_t cnt) {
  const int lane = threadIdx.x;
  const int32_t j = i + 1 < P.np ? i + 1 : i - 1;
  const Ent ej = pss_ent(P, j);
  const uint64_t vj = page_get(P, ej.pid);
  const bool il = i < j;
  const int32_t l = il ? i : j, r = il ? j : i;
  const uint64_t vl = il ? w : vj, vr = il ? vj : w;
  const int32_t cl = il ? cnt : ej.cnt, cr = il ? ej.cnt : cnt;
  const int32_t pl = il ? pid : ej.pid, pr = il ? ej.pid : pid;
  const int32_t tot = cl + cr;
  if (lane < cl) stage[lane] = vl;
  if (lane < cr) stage[cl + lane] = vr;
  wave_order();
  if (tot <= kPage) {
    const uint64_t m = lane < tot ? stage[lane] : kNoKey;
    wave_order();
    page_put(P, pl, m);
    pss_set(P, l, rl64(m, 0), pl, tot);
    page_drop(P, pr);
    pss_dir_remove(P, r);
  } else {
    const int32_t h = tot / 2;
    const uint64_t a = lane < h ? stage[lane] : kNoKey;
    const uint64_t b = lane < tot - h ? stage[h + lane] : kNoKey;
    wave_order();
    page_put(P, pl, a);
    page_put(P, pr, b);
    pss_set(P, l, rl64(a, 0), pl, h);
    pss_set(P, r, rl64(b, 0), pr, tot - h);
  }
}

// One update of a set: erase x, insert x, or replace x by y (y sorts where x
// did).  Erased and replaced keys are present; inserted keys are not.  False
// when an insert needs a page the directory has no entry for.
__device__ __forceinline__ bool pss_op(Pss& P, LMEM uint64_t* stage, int kind, uint64_t x, uint64_t y) {
  const int lane = threadIdx.x;
  if (P.np == 0) {  // only an insert reaches an empty set
    const int32_t pid = page_new(P);
    page_put(P, pid, lane == 0 ? x : kNoKey);
    pss_dir_insert(P, 0, x, pid, 1);
    P.nkeys += 1;
    return true;
  }
  Ent en;
  int32_t i = pss_locate(P, x, &en);
  if (i < 0) {  // an insert below every key
    i = 0;
    en = pss_ent(P, 0);
  }
  const uint64_t v = page_get(P, en.pid);
  if (kind != kOpInsert) {
    const uint64_t hit = ballot(v == x);
    const int pos = hit ? __builtin_ctzll(hit) : kPage - 1;
    if (kind == kOpRekey) {
      const uint64_t nv = lane == pos ? y : v;
      page_put(P, en.pid, nv);
      if (pos == 0) pss_set(P, i, y, en.pid, en.cnt);
      return true;
    }
    const uint64_t nv = page_del(v, pos);
    const int32_t cnt = en.cnt - 1;
    P.nkeys -= 1;
    if (cnt == 0) {  // a lone page emptied
      page_drop(P, en.pid);
      pss_dir_remove(P, i);
      return true;
    }
    page_put(P, en.pid, nv);
    pss_set(P, i, rl64(nv, 0), en.pid, cnt);
    if (cnt < kPage / 2 && P.np > 1) pss_rebalance(P, stage, i, nv, en.pid, cnt);
    return true;
  }
  const int pos = __builtin_popcountll(ballot(v < x));
  if (en.cnt < kPage) {
    const uint64_t nv = page_ins(v, pos, x);
    page_put(P, en.pid, nv);
    pss_set(P, i, rl64(nv, 0), en.pid, en.cnt + 1);
    P.nkeys += 1;
    return true;
  }
  if (P.np >= P.cap) return false;
  const int32_t pid2 = page_new(P);
  stage[lane + (lane >= pos ? 1 : 0)] = v;  // the kPage + 1 keys in order, split 33 | 32
  if (lane == 0) stage[pos] = x;
  wave_order();
  const uint64_t a = lane < kPage / 2 + 1 ? stage[lane] : kNoKey;
  const uint64_t b = lane < kPage / 2 ? stage[kPage / 2 + 1 + lane] : kNoKey;
  wave_order();
  page_put(P, en.pid, a);
  page_put(P, pid2, b);
  pss_set(P, i, rl64(a, 0), en.pid, kPage / 2 + 1);
  pss_dir_insert(P, i + 1, rl64(b, 0), pid2, kPage / 2);
  P.nkeys += 1;
  return true;
}

// the updates one event makes to one set (at most three), in order
struct SetOps {
  int k, kind0, kind1, kind2;
  uint64_t x0, x1, x2, y0, y1, y2;
};
// (selects, not branches: the fields stay in registers)
__device__ __forceinline__ void ops_add(SetOps& o, int kind, uint64_t x, uint64_t y) {
  const bool a0 = o.k == 0, a1 = o.k == 1, a2 = o.k == 2;
  o.kind0 = a0 ? kind : o.kind0; o.x0 = a0 ? x : o.x0; o.y0 = a0 ? y : o.y0;
  o.kind1 = a1 ? kind : o.kind1; o.x1 = a1 ? x : o.x1; o.y1 = a1 ? y : o.y1;
  o.kind2 = a2 ? kind : o.kind2; o.x2 = a2 ? x : o.x2; o.y2 = a2 ? y : o.y2;
  o.k += 1;
}
__device__ __forceinline__ bool ops_run(Pss& P, LMEM uint64_t* stage, const SetOps& o) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (k >= o.k) break;
    const int kind = k == 0 ? o.kind0 : (k == 1 ? o.kind1 : o.kind2);
    const uint64_t x = k == 0 ? o.x0 : (k == 1 ? o.x1 : o.x2);
    const uint64_t y = k == 0 ? o.y0 : (k == 1 ? o.y1 : o.y2);
    if (!pss_op(P, stage, kind, x, y)) return false;
  }
  return true;
}

struct BigPool {
  Pss sz, ad;           // free blocks by key (size, address) and by address key (address, size)
  SetOps osz, oad;      // this event's updates of each
  uint64_t split_min;   // split_min of this pool, in units
  GMEM uint64_t* segs;  // keys of the segments created in this pool, slot k at segs[segdir * k]
  int segdir;
  int32_t nseg;
  uint64_t bump, created_u;
  int32_t maxfree, n_mf;
  int pool;
};
__device__ __forceinline__ int32_t pool_free_count(const BigPool& ps) { return ps.sz.nkeys; }

template <int NP, bool CH = false>
struct BigChain {
  static constexpr bool kChunk = CH;
  BigPool p[NP];
  uint64_t reserved_u;
  int32_t created, released, n_res;
  int64_t base, n;
  bool back_res;
  LMEM uint64_t* stage;  // 2 kPage + 2 keys of LDS for page merges and splits
  GMEM ChunkRes* cres;   // chunk mode, as for FastChain
  int cres_dir;
  GMEM MfRec* cmf;
  int cmf_dir;
  uint32_t g;            // chunk mode: lane b, the largest block chosen for a request of bucket b (gbucket)
  const GMEM int32_t* bound;  // as for FastChain; the paged chunks' rounds never set it
  int32_t k_self;
};

// Section 3.4 (iv)-(v) on the paged sets: units held by idle segments of both pools
template <int NP, bool CH>
__device__ __forceinline__ uint64_t big_idle_units(BigChain<NP, CH>& c) {
  uint64_t mine = 0;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    BigPool& ps = c.p[q];
    for (int32_t i = 0; i < ps.sz.np; ++i) {
      const Ent en = pss_ent(ps.sz, i);
      const uint64_t x = page_get(ps.sz, en.pid);
      if ((int32_t)threadIdx.x < en.cnt && seg_key_idle(ps.segs, ps.segdir, ps.nseg, x)) mine += key_size(x);
    }
  }
  return wave_sum_u64(mine);
}
// release every idle segment of both pools; false if a set update failed
template <int NP, bool CH>
__device__ __forceinline__ bool big_release_idle(BigChain<NP, CH>& c) {
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    BigPool& ps = c.p[q];
    int32_t i = 0;
    while (i < ps.sz.np) {  // pages before i hold no idle segment
      const Ent en = pss_ent(ps.sz, i);
      const uint64_t x = page_get(ps.sz, en.pid);
      const uint64_t m = ballot((int32_t)threadIdx.x < en.cnt && seg_key_idle(ps.segs, ps.segdir, ps.nseg, x));
      if (!m) { ++i; continue; }
      const uint64_t k = rl64(x, __builtin_ctzll(m));
      c.reserved_u -= key_size(k);
      c.released += 1;
      if (!pss_op(ps.sz, c.stage, kOpErase, k, 0)) return false;
      if (!pss_op(ps.ad, c.stage, kOpErase, akey_of(key_size(k), key_addr(k)), 0)) return false;
      i = i > 0 ? i - 1 : 0;  // a merge may have moved keys into the page before
    }
  }
  return true;
}

template <int NP, bool CH>
__device__ __forceinline__ int pool_alloc(BigChain<NP, CH>& c, BigPool& ps, const Derived& d, const Gw& w, uint64_t u,
                                          int64_t e, uint64_t* blk) {
  if (u >= kFastLimit) return kRetry;
  ps.osz.k = ps.oad.k = 0;
  const uint64_t b = pss_first_ge(ps.sz, u << 32);
  const uint64_t split_min = ps.split_min;
  if (b != kNoKey) {
    const uint64_t S = key_size(b), A = key_addr(b), rem = S - u;
    note_choice(c, u, S);
    ops_add(ps.osz, kOpErase, b, 0);
    if (rem >= split_min) {  // the remainder keeps the block's place in address order
      ops_add(ps.oad, kOpRekey, akey_of(S, A), akey_of(rem, A + u));
      ops_add(ps.osz, kOpInsert, key_of(rem, A + u), 0);
      *blk = key_of(u, A);
    } else {
      ops_add(ps.oad, kOpErase, akey_of(S, A), 0);
      *blk = b;
    }
  } else {
    // nothing cached fits: a new segment (Section 3.4 (ii), (iv))
    const uint64_t S = segment_units(d, ps.pool, u);
    if (ps.created_u + S > d.limit_u) return XMEM_T_OVERFLOW;
    if (ps.bump + S + 1 > kFastLimit) return kRetry;
    if (NP == 2 && S > d.cap_u - c.reserved_u) {  // Section 3.4 (v): reclaim idle segments, else OOM
      const uint64_t idle = big_idle_units(c);
      if (S > d.cap_u - (c.reserved_u - idle)) return XMEM_T_OOM;
      if (!big_release_idle(c)) return kRetry;
    }
    const uint64_t A = ps.bump;
    if (!CH && threadIdx.x == 0) ps.segs[(int64_t)ps.segdir * ps.nseg] = key_of(S, A);
    ps.nseg += 1;
    ps.bump += S + 1;  // one-unit gap: segments are never physically adjacent
    ps.created_u += S;
    c.reserved_u += S;
    c.created += 1;
    record_reserved(c, w, e, d.shift);
    const uint64_t rem = S - u;
    if (rem >= split_min) {
      ops_add(ps.osz, kOpInsert, key_of(rem, A + u), 0);
      ops_add(ps.oad, kOpInsert, akey_of(rem, A + u), 0);
      *blk = key_of(u, A);
    } else {
      *blk = key_of(S, A);
    }
  }
  return ops_run(ps.sz, c.stage, ps.osz) && ops_run(ps.ad, c.stage, ps.oad) ? XMEM_T_OK : kRetry;
}

template <int NP, bool CH>
__device__ __forceinline__ int pool_free(BigChain<NP, CH>& c, BigPool& ps, uint64_t b) {
  const uint64_t A = key_addr(b), S = key_size(b), E = A + S;
  ps.osz.k = ps.oad.k = 0;
  // the free blocks just before and just after [A, E) in address order
  const uint64_t la = A > 0 ? pss_last_le(ps.ad, (A << 32) - 1) : kNoKey;
  const uint64_t ra = pss_first_ge(ps.ad, E << 32);
  const bool hl = la != kNoKey && akey_addr(la) + akey_size(la) == A;
  const bool hr = ra != kNoKey && akey_addr(ra) == E;
  uint64_t ms = S, ma = A;
  if (hl) { ms += akey_size(la); ma = akey_addr(la); }
  if (hr) ms += akey_size(ra);
  if (hr) ops_add(ps.oad, kOpErase, ra, 0);
  if (hl) ops_add(ps.oad, kOpRekey, la, akey_of(ms, ma));  // the merged block starts where the left one did
  else ops_add(ps.oad, kOpInsert, akey_of(ms, ma), 0);
  if (hl) ops_add(ps.osz, kOpErase, key_of(akey_size(la), akey_addr(la)), 0);
  if (hr) ops_add(ps.osz, kOpErase, key_of(akey_size(ra), akey_addr(ra)), 0);
  ops_add(ps.osz, kOpInsert, key_of(ms, ma), 0);
  return ops_run(ps.sz, c.stage, ps.osz) && ops_run(ps.ad, c.stage, ps.oad) ? XMEM_T_OK : kRetry;
}

template <int NP>
__global__ __launch_bounds__(kWave) void k_replay_big(const int64_t* off_, int64_t nchains, Derived d, Ws ws) {
  constexpr int32_t cap = NP == 1 ? kBigDir1 : kBigDir2;
  __shared__ uint64_t s_dkey[2 * NP][cap + 2];
  __shared__ uint32_t s_dpg[2 * NP][cap + 2];
  __shared__ uint64_t s_stage[2 * kPage + 2];
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  GMEM uint64_t* slot = (GMEM uint64_t*)w.big + (int64_t)blockIdx.x * kBigSlotKeys;
  GMEM uint64_t* sgk = (GMEM uint64_t*)w.segs;
  for (int64_t chain = blockIdx.x; chain < nchains; chain += gridDim.x) {
    const int64_t t = NP == 1 ? (chain >> 1) : chain;
    const int pool_one = NP == 1 ? (int)(chain & 1) : 0;
    if (w.hdr[2 * t + pool_one].status != kSpill) continue;  // finished by the fast kernel
    BigChain<NP> c;
    c.base = off[t];
    c.n = off[t + 1] - c.base;
    c.stage = (LMEM uint64_t*)s_stage;
    const uint64_t sb = w.stop_bad[t];
    const int64_t limit = sb == kNoStop ? c.n : (int64_t)(sb >> 8);
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int pool = NP == 1 ? pool_one : q;
      BigPool& ps = c.p[q];
      pss_init(ps.sz, (LMEM uint64_t*)s_dkey[2 * q], (LMEM uint32_t*)s_dpg[2 * q],
               slot + (int64_t)(2 * q) * (cap + 2) * kPage, cap);
      pss_init(ps.ad, (LMEM uint64_t*)s_dkey[2 * q + 1], (LMEM uint32_t*)s_dpg[2 * q + 1],
               slot + (int64_t)(2 * q + 1) * (cap + 2) * kPage, cap);
      ps.osz.k = ps.oad.k = 0;
      ps.segdir = pool == 0 ? 1 : -1;
      ps.segs = pool == 0 ? sgk + c.base : sgk + c.base + c.n - 1;
      ps.nseg = 0;
      ps.bump = ps.created_u = 0;
      ps.maxfree = ps.n_mf = 0;
      ps.pool = pool;
      ps.split_min = pool == 0 ? d.split_min_u[0] : d.split_min_u[1];
    }
    c.reserved_u = 0;
    c.created = c.released = c.n_res = 0;
    c.back_res = NP == 1 && pool_one == 1;
    int status;
    int64_t stop;
    chain_run<NP>(c, d, w, pool_one, 0, limit, &status, &stop);
    chain_header(c, w, NP, t, pool_one, status, stop, c.p[0].n_mf, c.p[NP - 1].n_mf);
    wave_order();
  }
}

// ------------------------------------------------------------------ chunked replay on the paged sets
// A chain whose pool outgrew the LDS table during the chunked replay is
// replayed again, in the same chunks and rounds, on the paged sets -- when the
// batch is small enough for every (chain, chunk) to have its own page slot (a
// few long traces, the case with no parallelism across chains).  A chunk state
// is the pool's scalars and both sets' keys in order; a chunk starts by packing
// them into fresh pages.
static_assert(kBigDir1 == kBigDirMaxHost, "the chunked paged slots match the directory size");

// the set's keys in order into dst; returns their count
__device__ __forceinline__ int32_t pss_dump(Pss& P, GMEM uint64_t* dst) {
  int32_t pos = 0;
  for (int32_t i = 0; i < P.np; ++i) {
    const Ent en = pss_ent(P, i);
    const uint64_t x = page_get(P, en.pid);
    if ((int32_t)threadIdx.x < en.cnt) dst[pos + (int32_t)threadIdx.x] = x;
    pos += en.cnt;
  }
  wave_order();
  return pos;
}
// an empty set (pss_init) filled with cnt ascending keys, about 48 to a page
__device__ __forceinline__ void pss_load(Pss& P, const GMEM uint64_t* src, int32_t cnt) {
  const int32_t per = (int64_t)cnt > 48 * (int64_t)P.cap ? kPage : 48;
  const int32_t np = (cnt + per - 1) / per;
  for (int32_t i = 0; i < np; ++i) {
    const int32_t a = (int32_t)((int64_t)i * cnt / np), b = (int32_t)((int64_t)(i + 1) * cnt / np);
    const uint64_t x = (int32_t)threadIdx.x < b - a ? src[a + (int32_t)threadIdx.x] : kNoKey;
    P.pages[(int64_t)kPage * i + threadIdx.x] = x;
    if (threadIdx.x == 0) {
      P.dkey[i] = x;
      P.dpg[i] = (uint32_t)i | ((uint32_t)(b - a) << 16);
    }
  }
  wave_order();
  P.np = np;
  P.bump = np;
  P.nfree = 0;
  P.nkeys = cnt;
  P.cpid = -1;
  P.cv = kNoKey;
  pss_summary(P);
}


// One chunk on the paged sets: events [lo, hi) of the chain from the frontier's state.
__device__ __forceinline__ void big_chunk(const Gw& w, const GMEM int64_t* off, const Derived& d, int64_t chain, int k,
                                          int64_t lo, int64_t hi, const CCtl& ctl, LMEM uint64_t* dkey0,
                                          LMEM uint64_t* dkey1, LMEM uint32_t* dpg0, LMEM uint32_t* dpg1,
                                          LMEM uint64_t* s_stage) {
  const int lane = threadIdx.x;
  const int K = w.chunks;
  const int64_t t = chain >> 1;
  const int pool_one = (int)(chain & 1);
  const int32_t cap = w.bcap;
  GMEM uint64_t* slot = w.bslot + (chain * K + k) * w.bslot_keys;
  BigChain<1, true> c;
  c.base = off[t];
  c.n = off[t + 1] - c.base;
  c.stage = s_stage;
  BigPool& ps = c.p[0];
  pss_init(ps.sz, dkey0, dpg0, slot, cap);
  pss_init(ps.ad, dkey1, dpg1, slot + (int64_t)(cap + 2) * kPage, cap);
  ps.osz.k = ps.oad.k = 0;
  ps.segdir = 1;
  ps.segs = (GMEM uint64_t*)w.segs + c.base;  // not written in chunk mode
  ps.nseg = 0;
  ps.pool = pool_one;
  ps.split_min = pool_one == 0 ? d.split_min_u[0] : d.split_min_u[1];
  ps.maxfree = -1;  // the chunk records every new maximum from its first event on
  ps.n_mf = 0;
  c.g = 0;
  bool loaded = true;
  ps.bump = ps.created_u = 0;
  c.reserved_u = 0;
  c.created = 0;
  if (ctl.f > 0) {  // the frontier's state: the end state of the chunk before it, plus the delta keys
    const GMEM uint64_t* src = w.bstate + (chain * K + ctl.f - 1) * w.bstate_words;
    const uint64_t cnts = src[3];
    ps.bump = src[0];
    ps.created_u = src[1];
    c.reserved_u = src[2];
    c.created = (int32_t)src[4];
    pss_load(ps.sz, src + 8, (int32_t)(uint32_t)cnts);
    pss_load(ps.ad, src + 8 + w.bstate_keys, (int32_t)(cnts >> 32));
  }
  if (ctl.nd > 0) {
    const GMEM uint64_t* del = w.cdel + chain * kDeltaWords;
    ps.bump = del[kMaxDelta];
    ps.created_u = del[kMaxDelta + 1];
    c.reserved_u = del[kMaxDelta + 2];
    c.created = (int32_t)del[kMaxDelta + 3];
    for (int i = 0; i < ctl.nd && loaded; ++i) {
      const uint64_t x = del[i];
      loaded = pss_op(ps.sz, c.stage, kOpInsert, x, 0) &&
               pss_op(ps.ad, c.stage, kOpInsert, akey_of(key_size(x), key_addr(x)), 0);
    }
  }
  c.released = c.n_res = 0;
  int32_t created0 = c.created;
  Resume rs{-1, 0, 0};
  if (ctl.resume > 0) {
    // the first chunk resumes where it outgrew the LDS table: that run's state (table keys and
    // counters), records, free-count maximum and lane registers; its records stay in place
    const GMEM uint64_t* src = w.cst + (chain * K + k) * kStateWords;
    const uint64_t cw = src[kStateKeys + 3];
    const int32_t cnt = (int32_t)(uint32_t)cw;
    ps.bump = src[kStateKeys];
    ps.created_u = src[kStateKeys + 1];
    c.reserved_u = src[kStateKeys + 2];
    c.created = (int32_t)(cw >> 32);
    for (int32_t i = 0; i < cnt && loaded; ++i) {
      const uint64_t x = src[i];
      loaded = pss_op(ps.sz, c.stage, kOpInsert, x, 0) &&
               pss_op(ps.ad, c.stage, kOpInsert, akey_of(key_size(x), key_addr(x)), 0);
    }
    const CHdr h = gload(&w.chdr[chain * K + k]);
    c.n_res = h.n_res;
    ps.n_mf = h.n_mf;
    ps.maxfree = h.maxc;
    created0 = 0;  // the chunk's start: the empty state
    const GMEM uint64_t* fw = w.bstate + (chain * K + 1) * w.bstate_words;
    rs = Resume{(int64_t)ctl.resume - 1, fw[lane], fw[kWave + lane]};
  }
  const int32_t n0 = ps.sz.nkeys;
  c.back_res = false;
  const int64_t olo = w.cown[chain * (K + 1) + k];
  c.cres = (GMEM ChunkRes*)w.ovf + c.base + (pool_one ? c.n - 1 - olo : olo);
  c.cres_dir = pool_one ? -1 : 1;
  c.cmf = (GMEM MfRec*)w.segs + c.base + (pool_one ? c.n - 1 - olo : olo);
  c.cmf_dir = pool_one ? -1 : 1;
  c.bound = nullptr;
  c.k_self = k;
  int status = kRetry;
  int64_t stop = lo;
  if (loaded) chain_run<1>(c, d, w, pool_one, lo, hi, &status, &stop, &rs);
  GMEM uint64_t* dst = w.bstate + (chain * K + k) * w.bstate_words;
  const int32_t nsz = pss_dump(ps.sz, dst + 8);
  const int32_t nad = pss_dump(ps.ad, dst + 8 + w.bstate_keys);
  if (lane == 0) {
    dst[0] = ps.bump;
    dst[1] = ps.created_u;
    dst[2] = c.reserved_u;
    dst[3] = (uint64_t)(uint32_t)nsz | ((uint64_t)(uint32_t)nad << 32);
    dst[4] = (uint64_t)(uint32_t)c.created;
    gstore(&w.chdr[chain * K + k],
           CHdr{stop, status, c.n_res, ps.n_mf, c.created - created0, ps.maxfree > n0 ? ps.maxfree : n0, 0});
  }
  store_choices(w, chain * K + k, c.g);
}

// Few traces (every (chain, chunk) has its own paged slot, one wavefront per
// CU): one round of the chunked replay for every chain, each in its own mode
// and on its own path, so a pool moved to the paged sets runs its rounds beside
// the other pools' rounds on the LDS table.
__global__ __launch_bounds__(kWave) void k_replay_combo(const int64_t* off_, int64_t nchains, Derived d, Ws ws) {
  __shared__ uint64_t s_dkey[2][kBigDir1 + 2];
  __shared__ uint32_t s_dpg[2][kBigDir1 + 2];
  __shared__ uint64_t s_stage[2 * kPage + 2];
  static_assert(sizeof(s_dkey[0]) >= sizeof(uint64_t) * kLdsRows * 64, "the LDS table fits in a directory");
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t chain = blockIdx.x % nchains;
  const int K = w.chunks;
  const CCtl ctl = gload(&w.cctl[chain]);
  if (ctl.done) return;
  const int nk = w.cnum[chain];
  const int kk = (int)(blockIdx.x / nchains);
  if (ctl.mode != 1 && kk != 0) return;
  const int k = ctl.mode == 1 ? kk : ctl.f;
  if (k < ctl.f || k >= nk) return;
  const GMEM int32_t* bnd = w.cbound + chain * (K + 1);
  const int64_t lo = bnd[k], hi = ctl.mode == 2 ? bnd[nk] : bnd[k + 1];
  if (ctl.big)
    big_chunk(w, off, d, chain, k, lo, hi, ctl, (LMEM uint64_t*)s_dkey[0], (LMEM uint64_t*)s_dkey[1],
              (LMEM uint32_t*)s_dpg[0], (LMEM uint32_t*)s_dpg[1], (LMEM uint64_t*)s_stage);
  else
    fast_chunk<true>(w, off, d, chain, k, lo, hi, ctl, (LMEM uint64_t*)s_dkey[0]);
}

// After each k_replay_combo round: the walk of k_chunk_stitch in each chain's
// own mode and path, then the chain's next mode: a pool that outgrew the LDS
// table starts over on the paged sets; after the first chunk come the
// speculative rounds, and after kSpecRounds of them the rest in one piece.
__global__ __launch_bounds__(kWave) void k_chunk_stitch_combo(const int64_t* off_, int64_t nchains, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  const int64_t chain = blockIdx.x;
  CCtl ctl = gload(&w.cctl[chain]);
  if (ctl.done) return;
  __shared__ uint64_t s_del[kMaxDelta];
  int64_t stop;
  int status;
  const int mode = ctl.mode, f0 = ctl.f;
  stitch_walk(w, off, chain, mode, ctl.big != 0, ctl, &stop, &status, (LMEM uint64_t*)s_del);
  if (ctl.done && status == kSpill && !ctl.big) {
    // the paged sets from the start; where the first chunk spilled in its own round, its paged
    // round resumes at the spill from the state the LDS run left
    const int32_t resume = mode == 0 && f0 == 0 && stop > 0 ? (int32_t)stop + 1 : 0;
    ctl = CCtl{0, 0, 0, 0, 0, 0, 0, 1, 0, resume};
  } else if (!ctl.done) {
    if (mode == 0) {
      ctl.mode = 1;
      ctl.rounds = 0;
      ctl.resume = 0;
    } else if (mode == 1 && ++ctl.rounds >= kSpecRounds) {
      ctl.mode = 2;
    }
  }
  if (threadIdx.x == 0) {
    gstore(&w.cctl[chain], ctl);
    if (ctl.done) gstore(&w.hdr[chain], ChainHdr{stop, status, ctl.n_res, ctl.n_mf, 0, 0});
  }
}

// ------------------------------------------------------------------ wide chain: 64-bit fields
// The same replay with 64-bit sizes and addresses and a table kept sorted by
// (size, address); it replays only the chains the fast kernel handed over.
// free blocks of one pool
// A pool's free blocks live in two places.
//  * A table sorted by (size, address), held in VGPRs: entry k sits in lane
//    k % 64 of row k / 64.  Best fit (Section 3.4 (iii)) is the first entry
//    with size >= u: one 64-bit compare and a ballot per row.  Insertions,
//    removals and re-keyed entries move a window of entries by one slot with
//    DPP whole-wavefront shifts.  Slots past the count hold size 0 and address
//    ~0, which no search matches.
//  * Past kRows * 64 entries, an unordered overflow: LDS first, then this
//    pool's region of the workspace (searched by a wavefront argmin).
constexpr int kRows = 12;
constexpr int32_t kTableCap = kRows * 64;
constexpr uint64_t kNoAddr = ~0ull;

template <int R>
struct VTable {
  uint64_t sz[R], ad[R];
  int32_t n;
};

template <int R>
__device__ __forceinline__ void vt_init(VTable<R>& t) {
#pragma unroll
  for (int r = 0; r < R; ++r) { t.sz[r] = 0; t.ad[r] = kNoAddr; }
  t.n = 0;
}

// Remove the entry at `from` and put (S, A) at `to` (indices of the final
// order).  from == n inserts (n < capacity); to == n-1 with (0, ~0) deletes.
template <int R>
__device__ __forceinline__ void vt_place(VTable<R>& t, int32_t from, int32_t to, uint64_t S, uint64_t A) {
  const int lane = threadIdx.x;
  if (to <= from) {  // [to, from) move up one slot
    const int rlo = to >> 6, rhi = from >> 6;
#pragma unroll
    for (int r = R - 1; r >= 0; --r) {
      if (r < rlo || r > rhi) continue;
      const int32_t idx = 64 * r + lane;
      uint64_t ns = from_lower_lane(t.sz[r]), na = from_lower_lane(t.ad[r]);
      if (r > 0) {  // lane 0 takes the last lane of the row below, not yet moved
        const uint64_t cs = rl64(t.sz[r - 1], 63), ca = rl64(t.ad[r - 1], 63);
        if (lane == 0) { ns = cs; na = ca; }
      }
      const bool put = idx == to, mv = idx > to && idx <= from;
      t.sz[r] = put ? S : (mv ? ns : t.sz[r]);
      t.ad[r] = put ? A : (mv ? na : t.ad[r]);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {  // (from, to] move down one slot
    const int rlo = from >> 6, rhi = to >> 6;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r < rlo || r > rhi) continue;
      const int32_t idx = 64 * r + lane;
      uint64_t ns = from_upper_lane(t.sz[r]), na = from_upper_lane(t.ad[r]);
      if (r + 1 < R) {  // lane 63 takes the first lane of the row above, not yet moved
        const uint64_t cs = rl64(t.sz[r + 1], 0), ca = rl64(t.ad[r + 1], 0);
        if (lane == 63) { ns = cs; na = ca; }
      }
      const bool put = idx == to, mv = idx >= from && idx < to;
      t.sz[r] = put ? S : (mv ? ns : t.sz[r]);
      t.ad[r] = put ? A : (mv ? na : t.ad[r]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// first entry with size >= u, or -1
template <int R>
__device__ __forceinline__ int32_t vt_first_ge(const VTable<R>& t, uint64_t u) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (64 * r >= t.n) break;
    const uint64_t m = ballot(t.sz[r] >= u);
    if (m) return 64 * r + __builtin_ctzll(m);
  }
  return -1;
}
// number of entries with key < (S, A): the sorted position of (S, A)
template <int R>
__device__ __forceinline__ int32_t vt_rank(const VTable<R>& t, uint64_t S, uint64_t A) {
  int32_t c = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (64 * r >= t.n) break;
    uint64_t m = ballot(t.sz[r] < S || (t.sz[r] == S && t.ad[r] < A));
    const int32_t valid = t.n - 64 * r;
    if (valid < 64) m &= (1ull << valid) - 1;
    c += __builtin_popcountll(m);
  }
  return c;
}
// entry whose address is x, or -1
template <int R>
__device__ __forceinline__ int32_t vt_find_addr(const VTable<R>& t, uint64_t x) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (64 * r >= t.n) break;
    const uint64_t m = ballot(t.ad[r] == x);
    if (m) return 64 * r + __builtin_ctzll(m);
  }
  return -1;
}
// entry ending at x (address + size == x), or -1
template <int R>
__device__ __forceinline__ int32_t vt_find_end(const VTable<R>& t, uint64_t x) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (64 * r >= t.n) break;
    const uint64_t m = ballot(t.ad[r] + t.sz[r] == x);
    if (m) return 64 * r + __builtin_ctzll(m);
  }
  return -1;
}
template <int R>
__device__ __forceinline__ void vt_get(const VTable<R>& t, int32_t k, uint64_t* S, uint64_t* A) {
  const int kr = k >> 6, kl = k & 63;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (r == kr) { *S = rl64(t.sz[r], kl); *A = rl64(t.ad[r], kl); }
}

// ---- unordered overflow (LDS, then HBM)
struct FreeSet {
  LMEM uint64_t* la;  // addresses
  LMEM uint64_t* ls;  // sizes
  GMEM Blk* g;        // overflow slot k at g[dir * k]
  int dir;
  int32_t n;
};

__device__ __forceinline__ Blk fs_load(const FreeSet& f, int32_t i) {
  if (i < kLdsEntries) return Blk{f.la[i], f.ls[i]};
  return gload(&f.g[(int64_t)f.dir * (i - kLdsEntries)]);
}
// single writer (lane 0); b is wave-uniform
__device__ __forceinline__ void fs_store(FreeSet& f, int32_t i, Blk b) {
  if (threadIdx.x == 0) {
    if (i < kLdsEntries) { f.la[i] = b.a; f.ls[i] = b.s; }
    else gstore(&f.g[(int64_t)f.dir * (i - kLdsEntries)], b);
  }
  wave_order();
}
__device__ __forceinline__ void fs_append(FreeSet& f, Blk b) { fs_store(f, f.n, b); f.n += 1; }
__device__ __forceinline__ void fs_remove(FreeSet& f, int32_t i) {
  const int32_t last = f.n - 1;
  if (i != last) fs_store(f, i, fs_load(f, last));
  f.n = last;
}
// the overflow block minimising (size, address) with size >= u; -1 if none
__device__ int32_t fs_best_fit(const FreeSet& f, uint64_t u, Blk* out) {
  const int lane = threadIdx.x;
  uint64_t bs = ~0ull, ba = ~0ull;
  int32_t bi = -1;
  for (int32_t i = lane; i < f.n; i += kWave) {
    const Blk b = fs_load(f, i);
    if (b.s >= u && (b.s < bs || (b.s == bs && b.a < ba))) { bs = b.s; ba = b.a; bi = i; }
  }
  const uint64_t ms = wave_min_u64(bs);
  if (ms == ~0ull) return -1;
  const uint64_t ma = wave_min_u64(bs == ms ? ba : ~0ull);
  const uint64_t who = ballot(bs == ms && ba == ma);  // addresses are unique: one lane
  const int32_t idx = (int32_t)rl((uint32_t)bi, __builtin_ctzll(who));
  *out = fs_load(f, idx);
  return idx;
}
// overflow blocks ending at a / starting at a + s
__device__ void fs_neighbours(const FreeSet& f, uint64_t a, uint64_t s, int32_t* left, int32_t* right) {
  const int lane = threadIdx.x;
  int32_t li = -1, ri = -1;
  for (int32_t i = lane; i < f.n; i += kWave) {
    const Blk b = fs_load(f, i);
    if (b.a + b.s == a) li = i;
    if (b.a == a + s) ri = i;
  }
  const uint64_t lm = ballot(li >= 0), rm = ballot(ri >= 0);
  *left = lm ? (int32_t)rl((uint32_t)li, __builtin_ctzll(lm)) : -1;
  *right = rm ? (int32_t)rl((uint32_t)ri, __builtin_ctzll(rm)) : -1;
}

// ------------------------------------------------------------------ allocator chain
struct PoolState {
  VTable<kRows> vt;
  FreeSet ov;
  GMEM Blk* segs;  // segments created in this pool (base, size), slot k at segs[segdir * k]
  int segdir;
  int32_t nseg;
  uint64_t bump, created_u;
  int32_t maxfree, n_mf;
  int pool;  // 0 SMALL, 1 LARGE
};

template <int NP>
struct Chain {
  PoolState p[NP];
  uint64_t reserved_u;
  int32_t created, released, n_res;
  int64_t base, n;  // trace range
  bool back_res;    // reserved records fill from the back (LARGE split chain)
};

template <int NP>
__device__ __forceinline__ void record_reserved(Chain<NP>& c, const Gw& w, int64_t e, int shift) {
  if (threadIdx.x == 0) {
    const int64_t slot = c.back_res ? c.base + c.n - 1 - c.n_res : c.base + c.n_res;
    gstore(&w.res[slot], ResRec{(int64_t)(c.reserved_u << shift), (int32_t)e, c.created, c.released, 0});
  }
  c.n_res += 1;
}

template <int NP>
__device__ __forceinline__ void record_free_count(Chain<NP>& c, PoolState& ps, const Gw& w, int64_t e) {
  const int32_t nf = ps.vt.n + ps.ov.n;
  if (nf > ps.maxfree) {
    ps.maxfree = nf;
    if (threadIdx.x == 0) {
      const int64_t slot = ps.pool == 1 ? c.base + c.n - 1 - ps.n_mf : c.base + ps.n_mf;
      gstore(&w.mf[slot], MfRec{(int32_t)e, nf});
    }
    ps.n_mf += 1;
  }
}

// a free block is an idle segment when a segment of this pool starts at its
// address with its size (segment bases ascend in creation order)
__device__ bool seg_idle(const PoolState& ps, uint64_t a, uint64_t s) {
  int32_t lo = 0, hi = ps.nseg - 1;
  while (lo <= hi) {
    const int32_t mid = (lo + hi) >> 1;
    const Blk g = gload(&ps.segs[(int64_t)ps.segdir * mid]);
    if (g.a == a) return g.s == s;
    if (g.a < a) lo = mid + 1; else hi = mid - 1;
  }
  return false;
}

// Section 3.4 (iv)-(v): units held by segments that are one idle free block
template <int NP>
__device__ uint64_t idle_units(const Chain<NP>& c) {
  uint64_t mine = 0;
  const int lane = threadIdx.x;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const PoolState& ps = c.p[q];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
      if (64 * r + lane < ps.vt.n && seg_idle(ps, ps.vt.ad[r], ps.vt.sz[r])) mine += ps.vt.sz[r];
    for (int32_t i = lane; i < ps.ov.n; i += kWave) {
      const Blk x = fs_load(ps.ov, i);
      if (seg_idle(ps, x.a, x.s)) mine += x.s;
    }
  }
  return wave_sum_u64(mine);
}

template <int NP>
__device__ void release_idle(Chain<NP>& c) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    PoolState& ps = c.p[q];
    while (true) {  // highest idle table entry first, so lower indices stay valid
      int32_t hit = -1;
#pragma unroll
      for (int r = kRows - 1; r >= 0; --r) {
        if (hit >= 0 || 64 * r >= ps.vt.n) continue;
        const uint64_t m = ballot(64 * r + lane < ps.vt.n && seg_idle(ps, ps.vt.ad[r], ps.vt.sz[r]));
        if (m) hit = 64 * r + 63 - __builtin_clzll(m);
      }
      if (hit < 0) break;
      uint64_t S, A;
      vt_get(ps.vt, hit, &S, &A);
      c.reserved_u -= S;
      c.released += 1;
      vt_place(ps.vt, hit, ps.vt.n - 1, 0, kNoAddr);
      ps.vt.n -= 1;
    }
    int32_t i = 0;
    while (true) {
      int32_t hit = -1;
      for (int32_t r = i; r < ps.ov.n; r += kWave) {
        const int32_t k = r + lane;
        bool idle = false;
        if (k < ps.ov.n) { const Blk x = fs_load(ps.ov, k); idle = seg_idle(ps, x.a, x.s); }
        const uint64_t m = ballot(idle);
        if (m) { hit = r + __builtin_ctzll(m); break; }
      }
      if (hit < 0) break;
      c.reserved_u -= fs_load(ps.ov, hit).s;
      c.released += 1;
      fs_remove(ps.ov, hit);
      i = hit;  // the entry moved into `hit` is examined next
    }
  }
}

// Up to two table moves per event, executed at one place per pool (scalar
// fields, so nothing is indexed at run time).
struct Moves {
  int32_t f0, t0, d0, f1, t1, d1;
  uint64_t S0, A0, S1, A1;
  int k;
  __device__ __forceinline__ void add(int32_t f, int32_t t, uint64_t s, uint64_t a, int32_t d) {
    if (k == 0) { f0 = f; t0 = t; S0 = s; A0 = a; d0 = d; }
    else { f1 = f; t1 = t; S1 = s; A1 = a; d1 = d; }
    ++k;
  }
};

// Allocation of u units (Section 3.4 (i)-(v)): plans the table moves, returns a
// status and the block handed out in *blk.
template <int NP>
__device__ __forceinline__ int chain_alloc(Chain<NP>& c, PoolState& ps, const Derived& d, const Gw& w, uint64_t u,
                                           int64_t e, Blk* blk, Moves& mv) {
  const int32_t pos = vt_first_ge(ps.vt, u);
  uint64_t S1 = 0, A1 = 0;
  if (pos >= 0) vt_get(ps.vt, pos, &S1, &A1);
  int32_t opos = -1;
  Blk ob{0, 0};
  if (ps.ov.n > 0) opos = fs_best_fit(ps.ov, u, &ob);
  const uint64_t split_min = d.split_min_u[ps.pool];
  if (opos >= 0 && (pos < 0 || ob.s < S1 || (ob.s == S1 && ob.a < A1))) {
    const uint64_t rem = ob.s - u;
    if (rem >= split_min) { fs_store(ps.ov, opos, Blk{ob.a + u, rem}); *blk = Blk{ob.a, u}; }
    else { fs_remove(ps.ov, opos); *blk = ob; }
    return XMEM_T_OK;
  }
  if (pos >= 0) {
    const uint64_t rem = S1 - u;
    if (rem >= split_min) { mv.add(pos, vt_rank(ps.vt, rem, A1 + u), rem, A1 + u, 0); *blk = Blk{A1, u}; }
    else { mv.add(pos, ps.vt.n - 1, 0, kNoAddr, -1); *blk = Blk{A1, S1}; }
    return XMEM_T_OK;
  }
  // nothing cached fits: a new segment (Section 3.4 (ii), (iv))
  uint64_t S;
  if (ps.pool == 0) S = d.small_seg_u;
  else if (u < d.min_large_u) S = d.mid_seg_u;
  else S = (u + d.large_round_u - 1) / d.large_round_u * d.large_round_u;
  if (ps.created_u + S > d.limit_u) return XMEM_T_OVERFLOW;
  // Section 3.4 (v): reclaim idle segments, else OOM.  A split chain runs only
  // when the capacity can never be reached.
  if (NP == 2 && S > d.cap_u - c.reserved_u) {
    const uint64_t idle = idle_units(c);
    if (S > d.cap_u - (c.reserved_u - idle)) return XMEM_T_OOM;
    release_idle(c);
  }
  const uint64_t base = ps.bump;
  if (threadIdx.x == 0) gstore(&ps.segs[(int64_t)ps.segdir * ps.nseg], Blk{base, S});
  ps.nseg += 1;
  ps.bump += S + 1;  // one-unit gap: segments are never physically adjacent
  ps.created_u += S;
  c.reserved_u += S;
  c.created += 1;
  record_reserved(c, w, e, d.shift);
  const uint64_t rem = S - u;
  if (rem >= split_min) {
    if (ps.vt.n < kTableCap) mv.add(ps.vt.n, vt_rank(ps.vt, rem, base + u), rem, base + u, 1);
    else fs_append(ps.ov, Blk{base + u, rem});
    *blk = Blk{base, u};
  } else {
    *blk = Blk{base, S};
  }
  return XMEM_T_OK;
}

// Release of block b: mark it free and coalesce with its free physical
// neighbours (Section 3.4 (iii)); plans the table moves.
__device__ __forceinline__ void chain_free(PoolState& ps, Blk b, Moves& mv) {
  const int32_t lpos = vt_find_end(ps.vt, b.a), rpos = vt_find_addr(ps.vt, b.a + b.s);
  int32_t lo = -1, ro = -1;
  if (ps.ov.n > 0 && (lpos < 0 || rpos < 0)) {
    fs_neighbours(ps.ov, b.a, b.s, &lo, &ro);
    if (lpos >= 0) lo = -1;
    if (rpos >= 0) ro = -1;
  }
  uint64_t ms = b.s, ma = b.a;
  if (lpos >= 0) { uint64_t s, a; vt_get(ps.vt, lpos, &s, &a); ms += s; ma = a; }
  else if (lo >= 0) { const Blk L = fs_load(ps.ov, lo); ms += L.s; ma = L.a; }
  if (rpos >= 0) { uint64_t s, a; vt_get(ps.vt, rpos, &s, &a); ms += s; }
  else if (ro >= 0) { ms += fs_load(ps.ov, ro).s; }
  if (lo >= 0 && ro >= 0) { fs_remove(ps.ov, lo > ro ? lo : ro); fs_remove(ps.ov, lo > ro ? ro : lo); }
  else if (lo >= 0) fs_remove(ps.ov, lo);
  else if (ro >= 0) fs_remove(ps.ov, ro);
  // the merged key is larger than either table neighbour's (its size is larger)
  if (lpos >= 0 && rpos >= 0) {
    const int32_t rank = vt_rank(ps.vt, ms, ma);  // counts both neighbours
    mv.add(rpos, ps.vt.n - 1, 0, kNoAddr, -1);
    mv.add(lpos - (rpos < lpos ? 1 : 0), rank - 2, ms, ma, 0);
  } else if (lpos >= 0 || rpos >= 0) {
    mv.add(lpos >= 0 ? lpos : rpos, vt_rank(ps.vt, ms, ma) - 1, ms, ma, 0);
  } else if (ps.vt.n < kTableCap) {
    mv.add(ps.vt.n, vt_rank(ps.vt, ms, ma), ms, ma, 1);
  } else {
    fs_append(ps.ov, Blk{ma, ms});
  }
}

struct Tile {
  uint64_t op;
  uint32_t link;
  Blk mb;
};

// one annotated event of this chain in pool state PI; returns a status
template <int NP, int PI>
__device__ __forceinline__ int chain_event(Chain<NP>& c, const Derived& d, const Gw& w, int64_t ts, int j,
                                           uint64_t opw, uint32_t lk, const Tile& cur, Blk& fwd_cur, const Blk& fwd_prev) {
  PoolState& ps = c.p[PI];
  const int64_t e = ts + j;
  Moves mv{};
  if ((opw >> kKindShift) == kKindAlloc) {
    Blk b;
    const int st = chain_alloc(c, ps, d, w, opw & kUnitsMask, e, &b, mv);
    if (st != XMEM_T_OK) return st;
    fwd_cur.a = wl64(b.a, j, fwd_cur.a);
    fwd_cur.s = wl64(b.s, j, fwd_cur.s);
    if (lk != 0) {  // deliver the block to the slot of its free, unless lane registers will
      const int64_t fe = (int64_t)(0xffffffffu - lk);
      if (fe >= ts + 2 * kWave && fe < c.n && threadIdx.x == 0) gstore(&w.mbox[c.base + fe], b);
    }
  } else {
    const int64_t h = (int64_t)lk;
    Blk b;
    if (h >= ts) { b.a = rl64(fwd_cur.a, (int)(h - ts)); b.s = rl64(fwd_cur.s, (int)(h - ts)); }
    else if (h >= ts - kWave) { b.a = rl64(fwd_prev.a, (int)(h - ts + kWave)); b.s = rl64(fwd_prev.s, (int)(h - ts + kWave)); }
    else { b.a = rl64(cur.mb.a, j); b.s = rl64(cur.mb.s, j); }
    chain_free(ps, b, mv);
  }
#pragma unroll 1
  for (int k = 0; k < mv.k; ++k) {
    const bool z = k == 0;
    vt_place(ps.vt, z ? mv.f0 : mv.f1, z ? mv.t0 : mv.t1, z ? mv.S0 : mv.S1, z ? mv.A0 : mv.A1);
    ps.vt.n += z ? mv.d0 : mv.d1;
  }
  record_free_count(c, ps, w, e);
  return XMEM_T_OK;
}

template <int NP>
__global__ __launch_bounds__(kWave) void k_replay_wide(const int64_t* off_, Derived d, Ws ws) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  if (w.ctl[0]) return;
  __shared__ uint64_t s_a[NP][kLdsEntries], s_s[NP][kLdsEntries];
  const int lane = threadIdx.x;
  const int64_t chain = blockIdx.x;
  const int64_t t = NP == 1 ? (chain >> 1) : chain;
  const int pool_one = NP == 1 ? (int)(chain & 1) : 0;  // pool of a split chain
  if (w.hdr[2 * t + pool_one].status != kRetry) return;  // the fast kernel finished this chain
  Chain<NP> c;
  c.base = off[t];
  c.n = off[t + 1] - c.base;
  const uint64_t sb = w.stop_bad[t];
  const int64_t limit = sb == kNoStop ? c.n : (int64_t)(sb >> 8);
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const int pool = NP == 1 ? pool_one : q;
    PoolState& ps = c.p[q];
    vt_init(ps.vt);
    ps.ov.la = (LMEM uint64_t*)s_a[q];
    ps.ov.ls = (LMEM uint64_t*)s_s[q];
    ps.ov.dir = pool == 0 ? 1 : -1;
    ps.ov.g = pool == 0 ? w.ovf + c.base : w.ovf + c.base + c.n - 1;
    ps.ov.n = 0;
    ps.segdir = pool == 0 ? 1 : -1;
    ps.segs = pool == 0 ? w.segs + c.base : w.segs + c.base + c.n - 1;
    ps.nseg = 0;
    ps.bump = ps.created_u = 0;
    ps.maxfree = ps.n_mf = 0;
    ps.pool = pool;
  }
  c.reserved_u = 0;
  c.created = c.released = c.n_res = 0;
  c.back_res = NP == 1 && pool_one == 1;

  int status = XMEM_T_OK;
  int64_t stop = -1;
  Tile cur{0, 0, Blk{0, 0}}, nxt{0, 0, Blk{0, 0}};
  Blk fwd_cur{0, 0}, fwd_prev{0, 0};
  if (lane < limit) annotate(w.ev[c.base + lane], w.code[c.base + lane], w.lx[c.base + lane], lane, d.shift, &cur.op, &cur.link);
  for (int64_t ts = 0; ts < limit; ts += kWave) {
    wave_order();
    {  // prefetch the next tile; its mailbox slots hold the blocks of allocations two or more tiles back
      const int64_t le = ts + kWave + lane;
      nxt = Tile{0, 0, Blk{0, 0}};
      if (le < limit) {
        annotate(w.ev[c.base + le], w.code[c.base + le], w.lx[c.base + le], le, d.shift, &nxt.op, &nxt.link);
        nxt.mb = gload(&w.mbox[c.base + le]);
      }
    }
    const bool mine = (ts + lane < limit) && (cur.op >> kKindShift) != 0 &&
                      (NP == 2 || ((cur.op & kPoolBit) ? 1 : 0) == pool_one);
    uint64_t todo = ballot(mine);
    while (todo) {
      const int j = __builtin_ctzll(todo);
      todo &= todo - 1;
      const uint64_t opw = rl64(cur.op, j);
      const uint32_t lk = rl(cur.link, j);
      int st;
      if (NP == 1 || !(opw & kPoolBit)) st = chain_event<NP, 0>(c, d, w, ts, j, opw, lk, cur, fwd_cur, fwd_prev);
      else st = chain_event<NP, NP - 1>(c, d, w, ts, j, opw, lk, cur, fwd_cur, fwd_prev);
      if (st != XMEM_T_OK) { status = st; stop = ts + j; break; }
    }
    if (stop >= 0) break;
    fwd_prev = fwd_cur;
    fwd_cur = Blk{0, 0};
    cur = nxt;
  }
  if (lane == 0) {
    if (NP == 1) {
      gstore(&w.hdr[2 * t + pool_one], ChainHdr{stop, status, c.n_res, c.p[0].n_mf, 0, 0});
    } else {
      gstore(&w.hdr[2 * t + 0], ChainHdr{stop, status, c.n_res, c.p[0].n_mf, 0, 0});
      gstore(&w.hdr[2 * t + 1], ChainHdr{stop, status, 0, c.p[NP - 1].n_mf, 0, 0});
    }
  }
}

// ------------------------------------------------------------------ k_finalize
// number of records (front: first + k, back: first - k) with event < stop, minus one
template <class R>
__device__ int64_t last_before(const GMEM R* r, int64_t first, int dir, int32_t k, int64_t stop) {
  int64_t lo = 0, hi = k;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (r[first + dir * mid].event < stop) lo = mid + 1; else hi = mid;
  }
  return lo - 1;
}

__global__ __launch_bounds__(kWave) void k_finalize(const int64_t* off_, int64_t T, Derived d, Ws ws,
                                                    xmem_trace_result* out_) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  GMEM xmem_trace_result* out = gp(out_);
  const int64_t t = blockIdx.x;
  const int lane = threadIdx.x;
  if (w.ctl[0]) {
    if (lane == 0) {
      xmem_trace_result r{};
      r.peak_allocated_event = r.peak_reserved_event = -1;
      r.stop_event = 0;
      r.status = XMEM_T_BAD_BATCH;
      gstore(&out[t], r);
    }
    return;
  }
  const int64_t base = off[t], n = off[t + 1] - base;
  int64_t stop = n;
  int status = XMEM_T_OK;
  const uint64_t sb = w.stop_bad[t];
  if (sb != kNoStop) { stop = (int64_t)(sb >> 8); status = (int)(sb & 0xff); }
  for (int p = 0; p < 2; ++p) {
    const ChainHdr h = gload(&w.hdr[2 * t + p]);
    if (h.stop >= 0 && h.stop < stop) { stop = h.stop; status = h.status; }
  }
  // tensor series up to the stop: whole tiles from k_stream, then a re-reduced partial tile
  const int64_t t0 = w.tile_base[t], nt = w.tile_base[t + 1] - t0;
  const int64_t whole = stop == n ? nt : stop / kTile;
  const int64_t tail_lo = whole * kTile, tail_hi = stop == n ? tail_lo : stop;
  TilePart acc{0, 0, -1};
  {
    const int64_t per = (whole + kWave - 1) / kWave;
    for (int64_t k = lane * per; k < min<int64_t>(whole, (lane + 1) * per); ++k) acc = tp_combine(acc, gload(&w.tile_part[t0 + k]));
    TilePart tail{0, 0, -1};
    const int64_t tper = (tail_hi - tail_lo + kWave - 1) / kWave;
    for (int64_t le = tail_lo + lane * tper; le < min<int64_t>(tail_hi, tail_lo + (lane + 1) * tper); ++le) {
      const int64_t dl = event_delta(w, base, le, d.shift);
      tail = tp_combine(tail, TilePart{dl, dl, le});
    }
    // the lanes' parts in lane order (lane 63 of each DPP scan holds the whole wavefront's), whole
    // tiles before the tail
    acc = tp_combine(tp_lane(tp_wave_scan(acc), kWave - 1), tp_lane(tp_wave_scan(tail), kWave - 1));
  }
  // finite capacity: the reserved series' maximum and its first event, each lane over every 64th
  // change point up to the stop, then the first maximum across the lanes
  int64_t rpeak = 0, rpev = -1, rk = -1;
  if (!d.split_pools) {
    const ChainHdr h = gload(&w.hdr[2 * t]);
    rk = last_before(w.res, base, 1, h.n_res, stop);
    int64_t ri = INT64_MAX;
    for (int64_t i = lane; i <= rk; i += kWave) {
      const ResRec rr = gload(&w.res[base + i]);
      if (rr.reserved > rpeak) { rpeak = rr.reserved; rpev = rr.event; ri = i; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const int64_t p2 = __shfl_xor(rpeak, o, kWave), e2 = __shfl_xor(rpev, o, kWave), i2 = __shfl_xor(ri, o, kWave);
      const bool take = p2 > rpeak || (p2 == rpeak && i2 < ri);
      rpeak = take ? p2 : rpeak;
      rpev = take ? e2 : rpev;
      ri = take ? i2 : ri;
    }
  }
  if (lane != 0) return;
  xmem_trace_result r{};
  r.peak_allocated = (acc.i >= 0 && acc.m > 0) ? acc.m : 0;
  r.peak_allocated_event = (acc.i >= 0 && acc.m > 0) ? acc.i : -1;
  r.final_allocated = acc.i >= 0 ? acc.s : 0;
  // segment series
  if (d.split_pools) {
    // unbounded capacity: reserved never decreases, so its peak is its value at the
    // stop, first reached at the later of the two pools' last changes
    int64_t total = 0, last_ev = -1, created = 0, released = 0;
    for (int p = 0; p < 2; ++p) {
      const ChainHdr h = gload(&w.hdr[2 * t + p]);
      const int64_t first = p == 0 ? base : base + n - 1;
      const int dir = p == 0 ? 1 : -1;
      const int64_t k = last_before(w.res, first, dir, h.n_res, stop);
      if (k >= 0) {
        const ResRec rr = gload(&w.res[first + dir * k]);
        total += rr.reserved;
        created += rr.created;
        released += rr.released;
        if (rr.event > last_ev) last_ev = rr.event;
      }
    }
    r.peak_reserved = total;
    r.peak_reserved_event = total > 0 ? last_ev : -1;
    r.final_reserved = total;
    r.segments_created = created;
    r.segments_released = released;
  } else {
    r.peak_reserved = rpeak;
    r.peak_reserved_event = rpev;
    if (rk >= 0) {
      const ResRec rr = gload(&w.res[base + rk]);
      r.final_reserved = rr.reserved;
      r.segments_created = rr.created;
      r.segments_released = rr.released;
    }
  }
  for (int p = 0; p < 2; ++p) {
    const ChainHdr h = gload(&w.hdr[2 * t + p]);
    const int64_t first = p == 0 ? base : base + n - 1;
    const int dir = p == 0 ? 1 : -1;
    const int64_t k = last_before(w.mf, first, dir, h.n_mf, stop);
    const int64_t v = k >= 0 ? w.mf[first + dir * k].value : 0;
    if (p == 0) r.max_free_blocks_small = v; else r.max_free_blocks_large = v;
  }
  r.stop_event = stop < n ? stop : -1;
  r.status = status;
  gstore(&out[t], r);
}

// ------------------------------------------------------------------ k_series
__device__ int64_t reserved_at(const GMEM ResRec* r, int64_t first, int dir, int32_t k, int64_t e) {
  int64_t lo = 0, hi = k;  // number of records with event <= e
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (r[first + dir * mid].event <= e) lo = mid + 1; else hi = mid;
  }
  return lo > 0 ? r[first + dir * (lo - 1)].reserved : 0;
}

__global__ __launch_bounds__(kStreamThreads) void k_series(const int64_t* off_, int64_t T, Derived d, Ws ws,
                                                            const xmem_trace_result* res_, int64_t* series_) {
  const Gw w = typed(ws);
  const GMEM int64_t* off = gp(off_);
  const GMEM xmem_trace_result* res = gp(res_);
  GMEM int64_t* series = gp(series_);
  if (w.ctl[0]) return;
  const int64_t tile = blockIdx.x;
  if (tile >= w.tile_base[T]) return;
  __shared__ int64_t s_t;
  if (threadIdx.x < 64) {
    const int64_t tt = wave_find(w.tile_base, T, tile);
    if (threadIdx.x == 0) s_t = tt;
  }
  __syncthreads();
  const int64_t t = s_t;
  const int64_t base = off[t], n = off[t + 1] - base;
  const int64_t stop = res[t].stop_event < 0 ? n : res[t].stop_event;
  const ChainHdr h0 = gload(&w.hdr[2 * t]), h1 = gload(&w.hdr[2 * t + 1]);
  const int64_t lo = (tile - w.tile_base[t]) * kTile;
  for (int64_t le = lo + threadIdx.x; le < min<int64_t>(n, lo + kTile); le += kStreamThreads) {
    int64_t v = -1;
    if (le < stop) {
      v = reserved_at(w.res, base, 1, h0.n_res, le);
      if (d.split_pools) v += reserved_at(w.res, base + n - 1, -1, h1.n_res, le);
    }
    series[base + le] = v;
  }
}

// ------------------------------------------------------------------ k_oom_predicted
// Section 4.1, Eq. (1) per trace: 1 when the estimated peak (peak reserved) exceeds m_max or the
// simulated allocator stopped with OOM, 0 when it does not, -1 when the replay gave no estimate.
__global__ void k_oom_predicted(const xmem_trace_result* res_, int64_t n, int64_t m_max, int32_t* flags_) {
  const GMEM xmem_trace_result* res = gp(res_);
  GMEM int32_t* flags = gp(flags_);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
    const int32_t st = res[t].status;
    flags[t] = st == XMEM_T_OOM ? 1 : st != XMEM_T_OK ? -1 : (res[t].peak_reserved > m_max ? 1 : 0);
  }
}

// ------------------------------------------------------------------ host side
bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int derive(const xmem_allocator_params* p, Derived* d) {
  if (xmem_validate_params(p) != XMEM_OK) return XMEM_EINVAL;
  int shift = 0;
  while ((int64_t(1) << shift) < p->round_bytes) ++shift;
  d->shift = shift;
  d->small_max_u = (uint64_t)p->small_max_bytes >> shift;
  d->small_seg_u = (uint64_t)p->small_segment_bytes >> shift;
  d->mid_seg_u = (uint64_t)p->mid_segment_bytes >> shift;
  d->min_large_u = (uint64_t)p->min_large_alloc_bytes >> shift;
  d->large_round_u = (uint64_t)p->large_round_bytes >> shift;
  d->large_round_mask = (d->large_round_u & (d->large_round_u - 1)) == 0 ? d->large_round_u - 1 : 0;
  d->split_min_u[0] = ((uint64_t)p->split_min_small_bytes + (uint64_t)p->round_bytes - 1) >> shift;
  d->split_min_u[1] = ((uint64_t)p->split_min_large_bytes + (uint64_t)p->round_bytes - 1) >> shift;
  d->cap_u = (uint64_t)p->device_capacity_bytes >> shift;
  d->limit_u = (uint64_t(1) << 61) >> shift;
  // reserved never passes 2^62 (2^61 per pool) plus one segment (< 2^49): a larger
  // capacity can never be reached, so the pools cannot interact
  d->split_pools = p->device_capacity_bytes > (int64_t(1) << 62) + (int64_t(1) << 50);
  return XMEM_OK;
}

// Chunk grain of the chunked replay: the flags' request, else kChunkWaves per
// trace, capped.  Speculation pays only with a fine grain (each speculative
// round costs one chunk); below kMinAutoChunks a batch has chains enough to
// fill the chip, and two chunks per chain -- replayed one after the other, no
// speculation -- only even out the load of the scheduler's wavefronts; past
// kSerialTraces the serial replay, one chain per wavefront.  1: serial.
constexpr int64_t kChunkWaves = 64512;
constexpr int kAutoChunks = 63;
constexpr int kMinAutoChunks = 16;
constexpr int64_t kSerialTraces = 16384;
// a single trace this short replays serially: the chunked rounds' fixed cost (about 1.5 ms of
// launches) is more than its serial replay (about 0.27 us per event)
constexpr int64_t kShortEvents = 4096;
inline int chunk_count(const xmem_allocator_params* p, const Derived& d, int64_t T, int64_t N) {
  if (!d.split_pools || T <= 0) return 1;
  int k = (int)(p->flags & XMEM_FLAGS_CHUNKS_MASK);
  if (k == 0 && long_few(T, N)) {  // the paged-set rounds, 2 x traces x chunks <= 254 CUs
    const int64_t c = kMaxComboChunks / T;
    return (int)(T == 1 ? c : c < kMaxChunks ? c : kMaxChunks);
  }
  if (k == 0 && T == 1 && N <= kShortEvents) return 1;
  if (k == 0) {
    const int64_t want = kChunkWaves / T;
    k = want > kAutoChunks ? kAutoChunks : want >= kMinAutoChunks ? (int)want : T < kSerialTraces ? 2 : 1;
  }
  if (k > kMaxChunks) k = kMaxChunks;
  while (k > 1 && 2 * T * k > INT32_MAX) --k;
  return k;
}

// Host-side argument checks shared by every replay entry point; *d receives the derived
// parameters.  XMEM_OK, or the code to return.
int check_replay_args(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces, int64_t total_events,
                      const xmem_allocator_params* params, const xmem_trace_result* d_out, Derived* d) {
  if (n_traces < 0 || total_events < 0 || !d_offsets) return XMEM_EINVAL;
  if (n_traces > 0 && !d_out) return XMEM_EINVAL;
  if (total_events > 0 && !d_events) return XMEM_EINVAL;
  if (derive(params, d) != XMEM_OK) return XMEM_EINVAL;
  if (n_traces == 0 && total_events != 0) return XMEM_EOFFSETS;
  const int64_t max_tiles = n_traces + total_events / kTile + 1;
  if (max_tiles > INT32_MAX || 2 * n_traces > INT32_MAX) return XMEM_EINVAL;
  return XMEM_OK;
}

// Every kernel of one replay on stream st, with the workspace carved for grain K and nbig
// paged-chain slots.
int replay_launch(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces, int64_t total_events,
                  const Derived& d, int K, int64_t nbig, xmem_trace_result* d_out, int64_t* d_reserved_series,
                  void* d_workspace, hipStream_t st, void* const* phase_events) {
  const int64_t max_tiles = n_traces + total_events / kTile + 1;
  Ws w;
  carve(d_workspace, n_traces, total_events, K, &w, nbig);
  w.ev = d_events;
  auto mark = [&](int i) -> bool {
    return !phase_events || hipEventRecord(static_cast<hipEvent_t>(phase_events[i]), st) == hipSuccess;
  };
  bool ok = mark(0);
  {
    const int64_t clear = (total_events + 1023) / 1024 < 4096 ? (total_events + 1023) / 1024 : 4096;
    k_plan<<<(unsigned)(1 + clear), 1024, 0, st>>>(d_offsets, n_traces, total_events, w);
    k_tile_info<<<(unsigned)((max_tiles + 255) / 256), 256, 0, st>>>(d_offsets, n_traces, w);
  }
  ok = ok && mark(1);
  k_stream<<<(unsigned)xcd_grid(max_tiles), kStreamThreads, 0, st>>>(d_events, d_offsets, n_traces, d, w);
  k_cross_check<<<(unsigned)xcd_grid(max_tiles), kStreamThreads, 0, st>>>(d_offsets, n_traces, w);
  ok = ok && mark(2);
  bool marked = false;  // the replay kernel's own boundaries, [3] and [4]
  if (d.split_pools) {
    const int64_t chains = 2 * n_traces;
    if (K > 1) {
      // chunks of about equal own-event counts across the batch (K for a chain holding a whole
      // mean-length trace); with a few traces only, K chunks for every chain
      int64_t target = (total_events + n_traces * K - 1) / (n_traces * K);
      if (target < 1) target = 1;
      if (w.bcap > 0) target = 0;
      const int64_t pblocks = n_traces + total_events / kPlanBlock + 1;
      k_plan_blocks<<<(unsigned)pblocks, kPlanThreads, 0, st>>>(d_offsets, n_traces, d, w);
      k_plan_chains<<<(unsigned)n_traces, 64, 0, st>>>(d_offsets, n_traces, target, w);
      k_plan_cuts<<<(unsigned)pblocks, kPlanThreads, 0, st>>>(d_offsets, n_traces, w);
      k_plan_final<<<(unsigned)chains, 64, 0, st>>>(d_offsets, n_traces, w);
      if (combo_main(n_traces, total_events, K)) {  // a few traces: every chain in its own mode, on the LDS table or the paged sets
        ok = ok && mark(3);
        for (int r = 0; r < 2 * (kSpecRounds + 2); ++r) {
          k_replay_combo<<<(unsigned)(chains * K), kWave, 0, st>>>(d_offsets, chains, d, w);
          k_chunk_stitch_combo<<<(unsigned)chains, kWave, 0, st>>>(d_offsets, chains, w);
        }
        ok = ok && mark(4);
        marked = true;
      } else {  // many traces: the persistent chunk scheduler, as many wavefronts as fit at once
        int dev = 0, cus = 0, per = 0, per_w = 0, per_a = 0, rate_khz = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_w, k_chunk_sched<true>, kWave, 0) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, k_chunk_sched<false>, kWave, 0) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_a, k_chunk_sched_aged, kWave, 0) != hipSuccess)
          return XMEM_EHIP;
        const bool windowed = sched_windowed((int64_t)(cus > 0 ? cus : 1) * (per_w > 0 ? per_w : 1), chains);
        const bool aged = windowed && K < kMinAutoChunks && per_a == per_w;
        if (windowed) per = per_w;
        const int64_t waves = (int64_t)(cus > 0 ? cus : 1) * (per > 0 ? per : 1);
        const uint64_t limit = (uint64_t)(rate_khz > 0 ? rate_khz : 100000) * 1000ull * kSchedLimitSeconds;
        const int64_t qn = w.cq_cap > chains ? w.cq_cap : chains;
        k_chunk_qinit<<<(unsigned)((qn + 255) / 256 < 4096 ? (qn + 255) / 256 : 4096), 256, 0, st>>>(n_traces, w);
        ok = ok && mark(3);
        if (aged) k_chunk_sched_aged<<<(unsigned)waves, kWave, 0, st>>>(SchedArgs{w, d, d_offsets, chains, limit});
        else if (windowed) k_chunk_sched<true><<<(unsigned)waves, kWave, 0, st>>>(SchedArgs{w, d, d_offsets, chains, limit});
        else k_chunk_sched<false><<<(unsigned)waves, kWave, 0, st>>>(SchedArgs{w, d, d_offsets, chains, limit});
        k_chunk_sched_end<<<(unsigned)((chains + 255) / 256), 256, 0, st>>>(chains, w);
        if (w.bcap > 0) {  // the pools that spilled: the paged-set rounds (empty launches when none did)
          k_combo_adopt<<<(unsigned)((chains + 255) / 256), 256, 0, st>>>(chains, w);
          for (int r = 0; r < 2 * (kSpecRounds + 2); ++r) {
            k_replay_combo<<<(unsigned)(chains * K), kWave, 0, st>>>(d_offsets, chains, d, w);
            k_chunk_stitch_combo<<<(unsigned)chains, kWave, 0, st>>>(d_offsets, chains, w);
          }
        }
        ok = ok && mark(4);
        marked = true;
      }
    } else {
      ok = ok && mark(3);
      k_replay_fast<1><<<(unsigned)chains, kWave, 0, st>>>(d_offsets, d, w);
      ok = ok && mark(4);
      marked = true;
    }
    k_replay_big<1><<<(unsigned)w.nbig, kWave, 0, st>>>(d_offsets, chains, d, w);
    k_replay_wide<1><<<(unsigned)chains, kWave, 0, st>>>(d_offsets, d, w);
  } else {
    ok = ok && mark(3);
    k_replay_fast<2><<<(unsigned)n_traces, kWave, 0, st>>>(d_offsets, d, w);
    ok = ok && mark(4);
    marked = true;
    k_replay_big<2><<<(unsigned)w.nbig, kWave, 0, st>>>(d_offsets, n_traces, d, w);
    k_replay_wide<2><<<(unsigned)n_traces, kWave, 0, st>>>(d_offsets, d, w);
  }
  if (!marked) return XMEM_EINVAL;  // every path above records [3] and [4]
  ok = ok && mark(5);
  k_finalize<<<(unsigned)n_traces, kWave, 0, st>>>(d_offsets, n_traces, d, w, d_out);
  ok = ok && mark(6);
  if (d_reserved_series && total_events > 0)
    k_series<<<(unsigned)max_tiles, kStreamThreads, 0, st>>>(d_offsets, n_traces, d, w, d_out, d_reserved_series);
  ok = ok && mark(7);
  return (ok && hipGetLastError() == hipSuccess) ? XMEM_OK : XMEM_EHIP;
}

// ------------------------------------------------------------------ the no-allocation entry point
// Its workspace: a fixed area of device memory that every GPU the library runs on holds from the
// first call on it until the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: the device address of each GPU's copy comes from hipGetSymbolAddress.
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return XMEM_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return XMEM_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return XMEM_OK;
}

// The grain and paged-slot count of a batch replayed in at most `cap` bytes of workspace: the
// library's own choice when it fits, else the serial replay (no chunk state) with as many paged
// slots as fit, at least one (k_replay_big then takes the spilled chains one after another).
// Results are the same for every choice.  False when even that does not fit.
bool fit_workspace(const xmem_allocator_params* p, const Derived& d, int64_t T, int64_t N, size_t cap, int* K,
                   int64_t* nbig) {
  *K = chunk_count(p, d, T, N);
  *nbig = big_slots(T);
  if (carve(nullptr, T, N, *K, nullptr, *nbig) <= cap) return true;
  *K = 1;
  for (int64_t b = big_slots(T); b >= 1; b = b > 8 ? 8 : b - 1) {
    *nbig = b;
    if (carve(nullptr, T, N, 1, nullptr, b) <= cap) return true;
  }
  return false;
}

}  // namespace

extern "C" {

int xmem_default_params(xmem_allocator_params* p, int preset) {
  if (!p || (preset != XMEM_PRESET_PAPER && preset != XMEM_PRESET_PYTORCH_LIKE)) return XMEM_EINVAL;
  const int64_t MiB = int64_t(1) << 20;
  p->abi_version = XMEM_ABI_VERSION;
  p->flags = 0;
  p->round_bytes = 512;
  p->small_max_bytes = MiB;
  p->small_segment_bytes = 2 * MiB;
  p->mid_segment_bytes = 20 * MiB;
  p->min_large_alloc_bytes = 10 * MiB;
  p->large_round_bytes = 2 * MiB;
  p->split_min_small_bytes = 512;
  p->split_min_large_bytes = preset == XMEM_PRESET_PYTORCH_LIKE ? MiB + 1 : 512;
  p->device_capacity_bytes = INT64_MAX;
  return XMEM_OK;
}

int xmem_validate_params(const xmem_allocator_params* p) {
  if (!p || p->abi_version != XMEM_ABI_VERSION || (p->flags & ~XMEM_FLAGS_CHUNKS_MASK) != 0 ||
      (p->flags & XMEM_FLAGS_CHUNKS_MASK) > (uint32_t)kMaxChunks)
    return XMEM_EINVAL;
  const int64_t lim = int64_t(1) << 40;
  if (!pow2(p->round_bytes) || p->round_bytes > (int64_t(1) << 30)) return XMEM_EINVAL;
  const int64_t mult[] = {p->small_max_bytes, p->small_segment_bytes, p->mid_segment_bytes, p->min_large_alloc_bytes,
                          p->large_round_bytes};
  for (int64_t v : mult)
    if (v < 1 || v > lim || v % p->round_bytes != 0) return XMEM_EINVAL;
  if (p->small_max_bytes > p->small_segment_bytes || p->min_large_alloc_bytes > p->mid_segment_bytes) return XMEM_EINVAL;
  if (p->split_min_small_bytes < 1 || p->split_min_small_bytes > lim) return XMEM_EINVAL;
  if (p->split_min_large_bytes < 1 || p->split_min_large_bytes > lim) return XMEM_EINVAL;
  if (p->device_capacity_bytes < 1) return XMEM_EINVAL;
  return XMEM_OK;
}

size_t xmem_workspace_bytes(int64_t n_traces, int64_t total_events, const xmem_allocator_params* params) {
  if (n_traces < 0 || total_events < 0 || xmem_validate_params(params) != XMEM_OK) return 0;
  Derived d;
  derive(params, &d);
  return carve(nullptr, n_traces, total_events, chunk_count(params, d, n_traces, total_events), nullptr);
}

int xmem_replay_batch_ex_timed(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                               int64_t total_events, const xmem_allocator_params* params, xmem_trace_result* d_out,
                               int64_t* d_reserved_series, void* d_workspace, size_t workspace_bytes,
                               void* hip_stream, void* const* phase_events, int n_phase_events) {
  Derived d;
  const int rc = check_replay_args(d_events, d_offsets, n_traces, total_events, params, d_out, &d);
  if (rc != XMEM_OK) return rc;
  if (phase_events && n_phase_events < XMEM_PHASE_EVENTS) return XMEM_EINVAL;
  if (n_traces == 0) return XMEM_OK;
  const int K = chunk_count(params, d, n_traces, total_events);
  const size_t need = carve(nullptr, n_traces, total_events, K, nullptr);
  if (!d_workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(d_workspace) & 255)) return XMEM_EWORKSPACE;
  return replay_launch(d_events, d_offsets, n_traces, total_events, d, K, big_slots(n_traces), d_out,
                       d_reserved_series, d_workspace, static_cast<hipStream_t>(hip_stream), phase_events);
}

int xmem_replay_batch_noalloc(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                              int64_t total_events, const xmem_allocator_params* params, xmem_trace_result* d_out,
                              int64_t* d_reserved_series, void* hip_stream) {
  Derived d;
  const int rc = check_replay_args(d_events, d_offsets, n_traces, total_events, params, d_out, &d);
  if (rc != XMEM_OK) return rc;
  if (n_traces == 0) return XMEM_OK;
  int K = 1;
  int64_t nbig = 1;
  if (!fit_workspace(params, d, n_traces, total_events, XMEM_NOALLOC_SCRATCH_BYTES, &K, &nbig)) return XMEM_ESCRATCH;
  void* ws = nullptr;
  const int sr = scratch_address(&ws);
  if (sr != XMEM_OK) return sr;
  return replay_launch(d_events, d_offsets, n_traces, total_events, d, K, nbig, d_out, d_reserved_series, ws,
                       static_cast<hipStream_t>(hip_stream), nullptr);
}

int xmem_replay_batch_ex(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces, int64_t total_events,
                         const xmem_allocator_params* params, xmem_trace_result* d_out, int64_t* d_reserved_series,
                         void* d_workspace, size_t workspace_bytes, void* hip_stream) {
  return xmem_replay_batch_ex_timed(d_events, d_offsets, n_traces, total_events, params, d_out, d_reserved_series,
                                    d_workspace, workspace_bytes, hip_stream, nullptr, 0);
}

int xmem_replay_batch(const uint64_t* d_events, const int64_t* d_offsets, int64_t n_traces,
                      const xmem_allocator_params* params, xmem_trace_result* d_out) {
  if (n_traces < 0 || !d_offsets || (n_traces > 0 && !d_out)) return XMEM_EINVAL;
  if (xmem_validate_params(params) != XMEM_OK) return XMEM_EINVAL;
  if (n_traces == 0) return XMEM_OK;
  int64_t* h = static_cast<int64_t*>(malloc(sizeof(int64_t) * (n_traces + 1)));
  if (!h) return XMEM_ENOMEM;
  if (hipMemcpy(h, d_offsets, sizeof(int64_t) * (n_traces + 1), hipMemcpyDeviceToHost) != hipSuccess) {
    free(h);
    return XMEM_EHIP;
  }
  int rc = h[0] == 0 ? XMEM_OK : XMEM_EOFFSETS;
  for (int64_t t = 0; rc == XMEM_OK && t < n_traces; ++t) {
    const int64_t len = h[t + 1] - h[t];
    if (len < 0 || len > XMEM_MAX_TRACE_EVENTS) rc = XMEM_EOFFSETS;
  }
  const int64_t N = h[n_traces];
  free(h);
  if (rc != XMEM_OK) return rc;
  if (N > 0 && !d_events) return XMEM_EINVAL;
  Derived d;
  derive(params, &d);
  const size_t need = carve(nullptr, n_traces, N, chunk_count(params, d, n_traces, N), nullptr);
  void* ws = nullptr;
  if (hipMalloc(&ws, need) != hipSuccess) return XMEM_ENOMEM;
  rc = xmem_replay_batch_ex(d_events, d_offsets, n_traces, N, params, d_out, nullptr, ws, need, nullptr);
  if (rc == XMEM_OK && hipStreamSynchronize(nullptr) != hipSuccess) rc = XMEM_EHIP;
  if (hipFree(ws) != hipSuccess && rc == XMEM_OK) rc = XMEM_EHIP;
  return rc;
}

int xmem_oom_predicted(const xmem_trace_result* d_results, int64_t n_traces, int64_t m_max_bytes, int32_t* d_flags,
                       void* hip_stream) {
  if (n_traces < 0 || m_max_bytes < 0 || (n_traces > 0 && (!d_results || !d_flags))) return XMEM_EINVAL;
  if (n_traces == 0) return XMEM_OK;
  const int64_t blocks = (n_traces + 255) / 256 < 65536 ? (n_traces + 255) / 256 : 65536;
  k_oom_predicted<<<(unsigned)blocks, 256, 0, static_cast<hipStream_t>(hip_stream)>>>(d_results, n_traces,
                                                                                      m_max_bytes, d_flags);
  return hipGetLastError() == hipSuccess ? XMEM_OK : XMEM_EHIP;
}

const char* xmem_strerror(int code) {
  switch (code) {
    case XMEM_OK: return "ok";
    case XMEM_EINVAL: return "invalid argument or allocator parameters";
    case XMEM_EOFFSETS: return "invalid trace offsets";
    case XMEM_EHIP: return "HIP runtime error";
    case XMEM_ENOMEM: return "device allocation failed";
    case XMEM_EWORKSPACE: return "workspace missing, misaligned or too small";
    case XMEM_ESCRATCH: return "batch needs more workspace than the no-allocation entry point's fixed area holds";
    case XMEM_T_OOM: return "trace stopped: out of device capacity after reclaiming idle segments";
    case XMEM_T_BAD_FREE: return "trace stopped: free of a non-allocation, a later event, or a freed block";
    case XMEM_T_BAD_EVENT: return "trace stopped: undecodable event word";
    case XMEM_T_OVERFLOW: return "trace stopped: segment bytes of a pool would pass 2^61";
    case XMEM_T_BAD_BATCH: return "offsets rejected on the device";
    case XMEM_T_ABORTED: return "trace not finished: the chunked replay stopped at its safety time limit";
  }
  return "unknown error code";
}

}  // extern "C"
