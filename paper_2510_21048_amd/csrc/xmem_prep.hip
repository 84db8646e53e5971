// xmem_prep.hip -- trace preparation upstream of the Memory Simulator, on MI355X (gfx950).
//
//   xmem_lifecycles   Section 3.2: pair raw allocator events by address into
//                     memory blocks.  A stable sort by (trace, address) puts
//                     every address's events next to each other in stream
//                     order; an allocation is closed by the event right after
//                     it when that is a free at the same address.
//   xmem_attribute    Section 3.2: link each block to the operator window it
//                     belongs to.  Per block: a binary search for the last
//                     window of its trace that starts no later than the
//                     allocation, a climb to the innermost window containing
//                     it, then the two rules tried outward.  Section 3.3 item
//                     5: the sizes of each trace's parameter blocks go into a
//                     per-trace open-addressing hash set, and a product
//                     allocated in an optimizer.step() phase whose size is in
//                     it becomes an optimizer state.  Kept blocks are
//                     compacted by a scan.
//   xmem_orchestrate  Section 3.3: retime each block's free by category, then
//                     a stable sort of the allocations and frees by (trace,
//                     time, rank) gives the Simulator's event order, and a
//                     scatter writes the event words.
//
// Both are HBM-bound.  The sort is an LSD radix sort of (64-bit key, 32-bit
// value) pairs, 8 bits a pass, in three kernels per pass; an address or time key
// is first rebased to its batch's minimum (and shifted past the trailing zero
// bits its values share), so that it takes only the passes its span needs:
//   k_rs_hist     digit histogram of each 4096-element tile;
//   k_scan_*      exclusive scan of the digit-major histogram (tile offsets);
//   k_rs_scatter  each wavefront ranks its 64-element steps with eight
//                 ballots (lanes with the same digit; stable by lane order),
//                 the tile is reordered by digit in LDS, and each digit's run
//                 is written to consecutive addresses.
// Keys are rebuilt between key groups from the values (record indices), so
// a composite key (trace, time, rank) costs one pass per 8 bits it uses.
#include <hip/hip_runtime.h>
#include <algorithm>
#include <stddef.h>
#include <stdint.h>

#include "xmem.h"
#include "xmem_prep.h"

namespace {

constexpr int kThreads = 256;             // 4 wavefronts
constexpr int kItems = 16;                // elements per lane per tile
constexpr int kTileN = kThreads * kItems;  // 4096
constexpr int kBins = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kScanThreads = 1024;
constexpr int64_t kPersist = INT64_MAX;
constexpr uint64_t kFree = 1ull << 63;

__host__ __device__ inline size_t al256(size_t x) { return (x + 255) & ~size_t(255); }
__host__ __device__ inline int64_t tiles_of(int64_t n) { return (n + kTileN - 1) / kTileN; }

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
// a sort pass over bits [sh, sh + 8) runs only below the key width found on the device (*gate)
__device__ __forceinline__ bool gated(const int32_t* gate, int sh) { return gate && sh >= *gate; }

// ---------------------------------------------------------------- generic exclusive scan of uint32
// in[0..m) -> out[0..m) (may alias); part: tiles_of(m) words.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xf, false);
}
// inclusive scan up the wavefront in lane order on DPP alone: shifts by 1, 2, 4 and 8 lanes within
// each row of 16, then row 0's total into row 1 and row 2's into row 3 (row_bcast:15), then rows
// 0-1's total into rows 2-3 (row_bcast:31).  All lanes active.
__device__ __forceinline__ uint32_t wave_scan_u32(uint32_t x) {
  x += dpp_u32<0x111, 0xf>(0, x);
  x += dpp_u32<0x112, 0xf>(0, x);
  x += dpp_u32<0x114, 0xf>(0, x);
  x += dpp_u32<0x118, 0xf>(0, x);
  x += dpp_u32<0x142, 0xa>(0, x);
  x += dpp_u32<0x143, 0xc>(0, x);
  return x;
}
// A lane's kItems consecutive elements from base: four 16-byte loads where they all lie below m
// (the scans' buffers are workspace buffers, 256-byte aligned, and base is a multiple of kItems).
__device__ __forceinline__ void scan_load(const uint32_t* in, int64_t base, int64_t m, uint32_t (&v)[kItems]) {
  if (base + kItems <= m) {
    const u32x4* p = reinterpret_cast<const u32x4*>(in + base);
#pragma unroll
    for (int q = 0; q < kItems / 4; ++q) {
      const u32x4 x = p[q];
      v[4 * q] = x.x;
      v[4 * q + 1] = x.y;
      v[4 * q + 2] = x.z;
      v[4 * q + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kItems; ++i) v[i] = base + i < m ? in[base + i] : 0u;
  }
}
__global__ __launch_bounds__(kThreads) void k_scan_reduce(const uint32_t* in, int64_t m, uint32_t* part,
                                                          const int32_t* gate, int sh) {
  if (gated(gate, sh)) return;
  __shared__ uint32_t s[kWaves];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t v[kItems];
  scan_load(in, (int64_t)blockIdx.x * kTileN + (int64_t)threadIdx.x * kItems, m, v);
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) acc += v[i];
  acc = wave_scan_u32(acc);
  if (lane == 63) s[wv] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
#pragma unroll
    for (int k = 0; k < kWaves; ++k) t += s[k];
    part[blockIdx.x] = t;
  }
}
// exclusive scan of part[0..np) in place, one workgroup; total to *total
__global__ __launch_bounds__(kScanThreads) void k_scan_top(uint32_t* part, int64_t np, uint32_t* total,
                                                           const int32_t* gate, int sh) {
  if (gated(gate, sh)) return;
  __shared__ uint32_t s[kScanThreads];
  const int64_t per = (np + kScanThreads - 1) / kScanThreads;
  const int64_t lo = (int64_t)threadIdx.x * per;
  uint32_t acc = 0;
  for (int64_t i = lo; i < lo + per && i < np; ++i) acc += part[i];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int st = 1; st < kScanThreads; st <<= 1) {  // inclusive Hillis-Steele
    const uint32_t v = (int)threadIdx.x >= st ? s[threadIdx.x - st] : 0u;
    __syncthreads();
    s[threadIdx.x] += v;
    __syncthreads();
  }
  uint32_t run = threadIdx.x ? s[threadIdx.x - 1] : 0u;
  for (int64_t i = lo; i < lo + per && i < np; ++i) {
    const uint32_t v = part[i];
    part[i] = run;
    run += v;
  }
  if (threadIdx.x == kScanThreads - 1 && total) *total = s[kScanThreads - 1];
}
__global__ __launch_bounds__(kThreads) void k_scan_down(const uint32_t* in, int64_t m, const uint32_t* part,
                                                        uint32_t* out, const int32_t* gate, int sh) {
  if (gated(gate, sh)) return;
  __shared__ uint32_t s[kWaves];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t base = (int64_t)blockIdx.x * kTileN + (int64_t)threadIdx.x * kItems;
  uint32_t v[kItems];
  scan_load(in, base, m, v);
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) acc += v[i];
  const uint32_t x = wave_scan_u32(acc);
  if (lane == 63) s[wv] = x;
  __syncthreads();
  uint32_t run = part[blockIdx.x] + x - acc;
#pragma unroll
  for (int k = 0; k < kWaves - 1; ++k) run += k < wv ? s[k] : 0u;
  uint32_t o[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    o[i] = run;
    run += v[i];
  }
  if (base + kItems <= m) {  // in place too: every lane reads its elements before it writes them
    u32x4* p = reinterpret_cast<u32x4*>(out + base);
#pragma unroll
    for (int q = 0; q < kItems / 4; ++q) p[q] = u32x4{o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
  } else {
#pragma unroll
    for (int i = 0; i < kItems; ++i)
      if (base + i < m) out[base + i] = o[i];
  }
}

struct ScanWs { uint32_t* part; uint32_t* total; };

void scan_u32(const uint32_t* in, uint32_t* out, int64_t m, const ScanWs& w, hipStream_t st,
              const int32_t* gate = nullptr, int sh = 0) {
  if (m <= 0) return;
  const int64_t nt = tiles_of(m);
  k_scan_reduce<<<(unsigned)nt, kThreads, 0, st>>>(in, m, w.part, gate, sh);
  k_scan_top<<<1, kScanThreads, 0, st>>>(w.part, nt, w.total, gate, sh);
  k_scan_down<<<(unsigned)nt, kThreads, 0, st>>>(in, m, w.part, out, gate, sh);
}

// ---------------------------------------------------------------- LSD radix sort
// digit histogram of each tile, digit-major: hist[d * ntiles + tile]
__global__ __launch_bounds__(kThreads) void k_rs_hist(const uint64_t* keys, int64_t n, int shift, uint32_t* hist,
                                                      int64_t ntiles, const int32_t* gate) {
  if (gated(gate, shift)) return;
  __shared__ uint32_t h[kBins];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTileN;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t k = base + (int64_t)i * kThreads + threadIdx.x;
    const bool ok = k < n;
    const uint32_t d = ok ? (uint32_t)(keys[k] >> shift) & (kBins - 1) : 0u;
    // a wavefront whose elements share one digit (the high digits of keys sorted by the low ones)
    // adds once: 64 atomics on one LDS word would be serialized
    const uint64_t act = ballot(ok);
    const uint32_t d0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)d);
    const uint64_t same = ballot(ok && d == d0);
    if (same == act) {
      if (act && (threadIdx.x & 63) == (uint32_t)__builtin_ctzll(act)) atomicAdd(&h[d0], (uint32_t)__builtin_popcountll(act));
    } else if (ok) {
      atomicAdd(&h[d], 1u);
    }
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one tile by one digit.  off[d * ntiles + tile]: where this
// tile's elements of digit d start in the output.
__global__ __launch_bounds__(kThreads, 4) void k_rs_scatter(const uint64_t* kin, const uint32_t* vin, uint64_t* kout,
                                                         uint32_t* vout, int64_t n, int shift, const uint32_t* off,
                                                         int64_t ntiles, const int32_t* gate) {
  if (gated(gate, shift)) return;
  __shared__ uint32_t wcnt[kWaves][kBins];  // per-wavefront digit counts, then their exclusive scan
  __shared__ uint32_t tbase[kBins];         // start of each digit in the tile's local order
  __shared__ uint32_t gbase[kBins];         // start of each digit's run in the output
  __shared__ uint64_t sk[kTileN];           // the tile in output order: keys, then values (two phases, so
                                            // that the block's LDS allows four workgroups per CU)
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint64_t below = (1ull << lane) - 1;
  for (int d = lane; d < kBins; d += 64) wcnt[wv][d] = 0;
  const int64_t base = (int64_t)blockIdx.x * kTileN + (int64_t)wv * (kTileN / kWaves);
  uint64_t key[kItems];
  uint32_t val[kItems], rd[kItems];  // rank in the wavefront's digit run | digit << 16 (kBins: no element)
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t k = base + (int64_t)i * 64 + lane;
    const bool ok = k < n;
    key[i] = ok ? kin[k] : 0;
    val[i] = ok ? vin[k] : 0;
    const uint32_t d = (uint32_t)(key[i] >> shift) & (kBins - 1);
    uint64_t peers = ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t bb = ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? bb : ~bb;
    }
    const uint32_t before = (uint32_t)__builtin_popcountll(peers & below);
    const uint32_t c = wcnt[wv][d];
    rd[i] = (c + before) | ((ok ? d : (uint32_t)kBins) << 16);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    if (ok && before == 0) wcnt[wv][d] = c + (uint32_t)__builtin_popcountll(peers);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  }
  __syncthreads();
  {  // thread tid owns digit tid: exclusive scan over the wavefronts, tile total
    uint32_t s = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = wcnt[w][tid];
      wcnt[w][tid] = s;
      s += c;
    }
    tbase[tid] = s;  // tile count of digit tid, scanned below
    gbase[tid] = off[(int64_t)tid * ntiles + blockIdx.x];
  }
  __syncthreads();
  if (tid < 64) {  // exclusive scan of the 256 tile counts by one wavefront (4 per lane)
    uint32_t c[4], s = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) { c[j] = tbase[4 * tid + j]; s += c[j]; }
    uint32_t incl = s;
#pragma unroll
    for (int st = 1; st < 64; st <<= 1) {
      const uint32_t o = __shfl_up(incl, st, 64);
      if (lane >= st) incl += o;
    }
    uint32_t run = incl - s;
#pragma unroll
    for (int j = 0; j < 4; ++j) { tbase[4 * tid + j] = run; run += c[j]; }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {  // rd becomes the element's place in the tile (all ones: no element)
    const uint32_t d = rd[i] >> 16;
    rd[i] = d < kBins ? tbase[d] + wcnt[wv][d] + (rd[i] & 0xffffu) : 0xffffffffu;
    if (rd[i] != 0xffffffffu) sk[rd[i]] = key[i];
  }
  __syncthreads();
  const int64_t cnt = n - (int64_t)blockIdx.x * kTileN < kTileN ? n - (int64_t)blockIdx.x * kTileN : kTileN;
  // sorted place tid + kThreads j of the tile: its output index (below XMEM_PREP_MAX_RECORDS)
  uint32_t out_at[kItems];
#pragma unroll
  for (int j = 0; j < kItems; ++j) {  // digit runs go to consecutive output addresses
    const int i = tid + j * kThreads;
    out_at[j] = 0xffffffffu;
    if (i < cnt) {
      const uint64_t k = sk[i];
      const uint32_t d = (uint32_t)(k >> shift) & (kBins - 1);
      out_at[j] = gbase[d] + ((uint32_t)i - tbase[d]);
      kout[out_at[j]] = k;
    }
  }
  __syncthreads();
  uint32_t* sv = reinterpret_cast<uint32_t*>(sk);
#pragma unroll
  for (int i = 0; i < kItems; ++i)
    if (rd[i] != 0xffffffffu) sv[rd[i]] = val[i];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kItems; ++j)
    if (out_at[j] != 0xffffffffu) vout[out_at[j]] = sv[tid + j * kThreads];
}

struct SortWs {
  uint64_t *ka, *kb;
  uint32_t *va, *vb;
  uint32_t* hist;
  ScanWs scan;
};

// Sorts (ka, va)[0..n) by key bits [lo, hi), stably; returns true when the
// result is in (kb, vb), false when in (ka, va).  With a gate, the passes at and
// above bit *gate (found on the device: an even number of passes below it) exit
// at once; hi - lo must then span an even number of passes, so that the result
// lands where the host expects it.
bool sort_bits(SortWs& w, int64_t n, int lo, int hi, bool in_b, hipStream_t st, const int32_t* gate = nullptr) {
  const int64_t nt = tiles_of(n);
  for (int sh = lo; sh < hi; sh += 8) {
    uint64_t* kin = in_b ? w.kb : w.ka;
    uint32_t* vin = in_b ? w.vb : w.va;
    uint64_t* kout = in_b ? w.ka : w.kb;
    uint32_t* vout = in_b ? w.va : w.vb;
    k_rs_hist<<<(unsigned)nt, kThreads, 0, st>>>(kin, n, sh, w.hist, nt, gate);
    scan_u32(w.hist, w.hist, (int64_t)kBins * nt, w.scan, st, gate, sh);
    k_rs_scatter<<<(unsigned)nt, kThreads, 0, st>>>(kin, vin, kout, vout, n, sh, w.hist, nt, gate);
    in_b = !in_b;
  }
  return in_b;
}

int bits_for(int64_t maxval) {  // bits needed for values 0..maxval, rounded up to a pass
  int b = 0;
  while (b < 64 && (maxval >> b) != 0) ++b;
  return (b + 7) / 8 * 8;
}

// ---------------------------------------------------------------- workspace
struct PrepWs {
  SortWs s;
  uint32_t* tid;     // n: trace of each record
  uint32_t* u;       // n: flags, then their exclusive scan
  int64_t* t64;      // n: per-record int64 scratch (free time of an allocation / retimed free of a block),
                     // or the attribution's parameter-size hash sets (2 u32 slots per parameter block)
  uint32_t* apos;    // n: position of an allocation word within its trace
  int32_t* bad;      // 1
  uint64_t* kr;      // 8: a sort key's range on the device (min, max, OR of its values XOR a reference, gate),
                     // then the lifecycle sort's second gate and its layout (kr[5], see k_life_keys)
};

size_t carve(void* base, int64_t T, int64_t n, PrepWs* w) {
  size_t o = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) { char* p = b ? b + o : nullptr; o += al256(bytes); return p; };
  const int64_t nt = tiles_of(n > 0 ? n : 1);
  const int64_t hist_n = (int64_t)kBins * nt;
  PrepWs x;
  x.s.ka = reinterpret_cast<uint64_t*>(take(8 * n));
  x.s.kb = reinterpret_cast<uint64_t*>(take(8 * n));
  x.s.va = reinterpret_cast<uint32_t*>(take(4 * n));
  x.s.vb = reinterpret_cast<uint32_t*>(take(4 * n));
  x.s.hist = reinterpret_cast<uint32_t*>(take(4 * hist_n));
  x.s.scan.part = reinterpret_cast<uint32_t*>(take(4 * (tiles_of(hist_n > n ? hist_n : n) + 1)));
  x.s.scan.total = reinterpret_cast<uint32_t*>(take(4));
  x.tid = reinterpret_cast<uint32_t*>(take(4 * n));
  x.u = reinterpret_cast<uint32_t*>(take(4 * (n + 1)));
  x.t64 = reinterpret_cast<int64_t*>(take(8 * n));
  x.apos = reinterpret_cast<uint32_t*>(take(4 * n));
  x.bad = reinterpret_cast<int32_t*>(take(4));
  x.kr = reinterpret_cast<uint64_t*>(take(64));
  (void)T;
  if (w) *w = x;
  return o;
}

// ---------------------------------------------------------------- shared small kernels
// offsets valid: off[0] == 0, non-decreasing, off[T] == n (n < 0: any end)
__global__ void k_check_offsets(const int64_t* off, int64_t T, int64_t n, int32_t* bad) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0 && (off[0] != 0 || (n >= 0 && off[T] != n))) atomicOr(bad, 1);
  if (i < T && off[i + 1] < off[i]) atomicOr(bad, 1);
}
__global__ void k_zero_i32(int32_t* p) { *p = 0; }
// trace of each of n records (binary search in off[0..T])
// The trace of each record: per workgroup of kThreads, kTileN consecutive records (coalesced,
// record base + kThreads i + thread); one binary search for the trace of the first, then each
// thread steps over the trace boundaries its records pass (the next trace's offset in a register).
__global__ __launch_bounds__(kThreads) void k_trace_of(const int64_t* off, int64_t T, int64_t n, const int32_t* bad,
                                                       uint32_t* tid) {
  __shared__ int64_t s_t;
  const int64_t base = (int64_t)blockIdx.x * kTileN;
  if (base >= n || *bad) return;
  if (threadIdx.x == 0) {
    int64_t lo = 0, hi = T - 1;
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (off[mid] <= base) lo = mid; else hi = mid - 1;
    }
    s_t = lo;
  }
  __syncthreads();
  int64_t t = s_t, next = t + 1 < T ? off[t + 1] : INT64_MAX;
#pragma unroll 4
  for (int i = 0; i < kItems; ++i) {
    const int64_t k = base + (int64_t)i * kThreads + threadIdx.x;
    if (k >= n) break;
    while (k >= next) {  // empty traces included: the last trace whose first record is at or before k
      ++t;
      next = t + 1 < T ? off[t + 1] : INT64_MAX;
    }
    tid[k] = (uint32_t)t;
  }
}
__global__ void k_fill_offsets_zero(int64_t* off, int64_t T, const int32_t* bad, int32_t* status) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) *status = *bad ? XMEM_T_BAD_BATCH : 0;
  if (*bad && i <= T) off[i] = 0;
}

unsigned grid_of(int64_t n, int t) { return (unsigned)((n + t - 1) / t > 0 ? (n + t - 1) / t : 1); }

// ---------------------------------------------------------------- lifecycles (Section 3.2)
// keys: address for every record, value = record index
// ---------------------------------------------------------------- key ranges
// A sort key spans fewer bits than its 64: kr receives the minimum and maximum of the keys that
// take part, and the OR of each XOR a reference value, whose trailing zeros all differences share.
// The key then sorts as (key - min) >> trailing zeros, over the passes its width needs.
__global__ void k_range_init(uint64_t* kr) {
  kr[0] = ~0ull;
  kr[1] = 0;
  kr[2] = 0;
  kr[3] = 0;
}
// a thread's running part of a range
struct RangePart {
  uint64_t mn = ~0ull, mx = 0, ox = 0;
  __device__ void add(bool in, uint64_t v, uint64_t ref) {
    mn = in && v < mn ? v : mn;
    mx = in && v > mx ? v : mx;
    ox |= in ? v ^ ref : 0;
  }
};
constexpr int kRangeBlocks = 1024;  // workgroups of a range kernel (grid-stride; one set of atomics each)
constexpr int kRangeUnroll = 8;     // records a range kernel's thread loads at once
// the workgroup's parts combined (wavefront butterflies, then LDS), then one atomic per word
__device__ __forceinline__ void range_commit(uint64_t* kr, RangePart p) {
  __shared__ uint64_t s[3][kThreads / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t a = __shfl_xor(p.mn, o, 64), b = __shfl_xor(p.mx, o, 64), c = __shfl_xor(p.ox, o, 64);
    p.mn = a < p.mn ? a : p.mn;
    p.mx = b > p.mx ? b : p.mx;
    p.ox |= c;
  }
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { s[0][wv] = p.mn; s[1][wv] = p.mx; s[2][wv] = p.ox; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / 64; ++k) {
      p.mn = s[0][k] < p.mn ? s[0][k] : p.mn;
      p.mx = s[1][k] > p.mx ? s[1][k] : p.mx;
      p.ox |= s[2][k];
    }
    if (p.mn <= p.mx) {
      atomicMin((unsigned long long*)&kr[0], (unsigned long long)p.mn);
      atomicMax((unsigned long long*)&kr[1], (unsigned long long)p.mx);
      atomicOr((unsigned long long*)&kr[2], (unsigned long long)p.ox);
    }
  }
}
// the shift and the pass gate of a range: bits of (max - min) >> shift, as an even number of
// 8-bit passes (so that a gated sort ends in the buffer it started from)
__device__ __forceinline__ int range_shift(const uint64_t* kr, bool use_tz) {
  return use_tz && kr[2] != 0 ? __builtin_ctzll(kr[2]) : 0;
}
// bits of (max - min) >> shift
__device__ __forceinline__ int range_bits(const uint64_t* kr, int shift) {
  const uint64_t span = kr[0] <= kr[1] ? (kr[1] - kr[0]) >> shift : 0;
  return span ? 64 - __builtin_clzll(span) : 0;
}
__device__ __forceinline__ int32_t range_gate(const uint64_t* kr, int shift) {
  const int passes = (range_bits(kr, shift) + 7) / 8;
  return 8 * (passes + (passes & 1));
}

// addresses of the allocation and free records (0-byte events take no part)
__global__ __launch_bounds__(kThreads) void k_life_range(const xmem_raw_event* raw, int64_t n, const int32_t* bad,
                                                         uint64_t* kr) {
  if (*bad) return;
  RangePart p;
  const uint64_t ref = raw[0].addr;
  // kRangeUnroll records per step, their loads all issued before any is used
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k0 < n; k0 += kRangeUnroll * stride) {
    uint64_t a[kRangeUnroll];
    int64_t by[kRangeUnroll];
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) {
      const int64_t k = k0 + u * stride;
      a[u] = k < n ? raw[k].addr : 0;
      by[u] = k < n ? raw[k].bytes : 0;
    }
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) p.add(by[u] != 0, a[u], ref);
  }
  range_commit(kr, p);
}
// The lifecycle sort's layout, chosen on the device from the address range (kr[5]: bit 0 set
// for the joint key, bit 1 the buffer that ends up holding the sorted pairs, bits 8.. the
// address bits b).  Joint key, when the trace and the address fit in 64 bits together and
// record indices in 31: (trace << b) | address, rebased and shifted, with 0-byte records last
// (T << b); one sort of b + trace bits, and the value carries the record index with bit 31 set
// for a free.  Otherwise the address alone (0 for 0-byte records), sorted in an even number of
// passes, then again by trace (k_life_trace_keys); the value is the record index.
constexpr uint64_t kJoint = 1, kJointBuf = 2;
// Also each record's allocation flag (bytes > 0), scanned after the pairing to number the blocks.
__global__ void k_life_keys(const xmem_raw_event* raw, const uint32_t* tid, int64_t n, int64_t T, int tbits,
                            bool second_odd, const int32_t* bad, uint64_t* kr, uint64_t* key, uint32_t* val,
                            int32_t* gate, int32_t* gate2, uint32_t* flag) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= n || *bad) return;
  const int sh = range_shift(kr, true), b = range_bits(kr, sh);
  const bool joint = n <= INT32_MAX && b + tbits <= 64;
  if (k == 0) {
    const int jp = (b + tbits + 7) / 8;  // passes of the joint sort
    *gate = joint ? 8 * jp : range_gate(kr, sh);
    *gate2 = joint ? 0 : 64;
    kr[5] = (joint ? kJoint : 0) | ((joint ? (jp & 1) : second_odd) ? kJointBuf : 0) | ((uint64_t)b << 8);
  }
  const xmem_raw_event r = raw[k];
  const uint64_t a = (r.addr - kr[0]) >> sh;
  flag[k] = r.bytes > 0 ? 1u : 0u;
  if (joint) {
    key[k] = r.bytes != 0 ? ((uint64_t)tid[k] << b) | a : (uint64_t)T << b;
    val[k] = (uint32_t)k | (r.bytes < 0 ? 0x80000000u : 0u);
  } else {
    key[k] = r.bytes != 0 ? a : 0;
    val[k] = (uint32_t)k;
  }
}
// keys after the address sort: trace of the record (T for 0-byte events, which sort last)
__global__ void k_life_trace_keys(const xmem_raw_event* raw, const uint32_t* tid, int64_t n, int64_t T,
                                  const int32_t* bad, const uint64_t* kr, const uint32_t* val, uint64_t* key) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n || *bad || (kr[5] & kJoint)) return;
  const uint32_t k = val[p];
  key[p] = raw[k].bytes == 0 ? (uint64_t)T : (uint64_t)tid[k];
}
// in (trace, address, stream) order: an allocation is closed by the next
// record when it is a free of the same trace and address.  With the joint key both
// come from the sorted keys and values, and only a closing free's time is read.
__global__ void k_life_pair(const xmem_raw_event* raw, const uint32_t* tid, const uint64_t* kr, const uint64_t* ka,
                            const uint32_t* va, const uint64_t* kb, const uint32_t* vb, int64_t n, int64_t T,
                            const int32_t* bad, int64_t* tfree, int64_t* unmatched) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n || *bad) return;
  const uint64_t meta = kr[5];
  const uint32_t* val = (meta & kJointBuf) ? vb : va;
  if (meta & kJoint) {
    const uint64_t* key = (meta & kJointBuf) ? kb : ka;
    const int b = (int)(meta >> 8);
    const uint64_t x = key[p];
    const uint64_t t = x >> b;
    if (t >= (uint64_t)T) return;  // 0-byte records
    const uint32_t v = val[p];
    const uint32_t k = v & 0x7fffffffu;
    if (!(v >> 31)) {
      int64_t f = kPersist;
      if (p + 1 < n && key[p + 1] == x) {
        const uint32_t vn = val[p + 1];
        if (vn >> 31) f = raw[vn & 0x7fffffffu].ts;
      }
      tfree[k] = f;
    } else if (unmatched) {
      const bool closes = p > 0 && key[p - 1] == x && !(val[p - 1] >> 31);
      if (!closes) atomicAdd((unsigned long long*)&unmatched[t], 1ull);
    }
    return;
  }
  const uint32_t k = val[p];
  const xmem_raw_event r = raw[k];
  if (r.bytes == 0) return;
  const bool has_next = p + 1 < n, has_prev = p > 0;
  const uint32_t kn = has_next ? val[p + 1] : 0, kp = has_prev ? val[p - 1] : 0;
  if (r.bytes > 0) {
    int64_t f = kPersist;
    if (has_next) {
      const xmem_raw_event q = raw[kn];
      if (q.bytes < 0 && q.addr == r.addr && tid[kn] == tid[k]) f = q.ts;
    }
    tfree[k] = f;
  } else if (unmatched) {
    bool closes = false;
    if (has_prev) {
      const xmem_raw_event q = raw[kp];
      closes = q.bytes > 0 && q.addr == r.addr && tid[kp] == tid[k];
    }
    if (!closes) atomicAdd((unsigned long long*)&unmatched[tid[k]], 1ull);
  }
}
__global__ void k_life_emit(const xmem_raw_event* raw, const int32_t* cat, int64_t n, const int32_t* bad,
                            const uint32_t* bidx, const int64_t* tfree, xmem_block* blocks) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= n || *bad) return;
  const xmem_raw_event r = raw[k];
  if (r.bytes <= 0) return;
  xmem_block b;
  b.size = r.bytes;
  b.t_alloc = r.ts;
  b.t_free = tfree[k];
  b.category = cat ? cat[k] : XMEM_CAT_OTHER;
  b.pad = 0;
  blocks[bidx[k]] = b;
}
// block offsets: allocations before each trace start (exclusive scan of the flags)
__global__ void k_life_offsets(const int64_t* off, int64_t T, int64_t n, const int32_t* bad, const uint32_t* scan,
                               const uint32_t* total, int64_t* boff) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t > T || *bad) return;
  boff[t] = off[t] < n ? (int64_t)scan[off[t]] : (int64_t)*total;
}
__global__ void k_zero_i64(int64_t* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// ---------------------------------------------------------------- attribution (Section 3.2)
// the enclosing window of window i of a trace whose windows start at w (-1: a root)
__device__ __forceinline__ int64_t win_parent(const xmem_window* w, int64_t i) {
  const int64_t p = w[i].parent;
  return (p >= 0 && p < i) ? p : -1;
}
// per window: the end of its nearest enclosing component (kPersist: none), and whether it lies in
// an optimizer.step() phase (itself or an enclosing window is a component of category optimizer)
__global__ void k_att_comp_end(const xmem_window* win, const int64_t* woff, int64_t T, int64_t nw, const int32_t* bad,
                               int64_t* comp_end, uint32_t* in_step) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= nw || *bad) return;
  int64_t lo = 0, hi = T - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (woff[mid] <= g) lo = mid; else hi = mid - 1;
  }
  const xmem_window* w = win + woff[lo];
  int64_t c = win_parent(w, g - woff[lo]);
  while (c >= 0 && w[c].kind != XMEM_WIN_COMPONENT) c = win_parent(w, c);
  comp_end[g] = c >= 0 ? w[c].end : kPersist;
  uint32_t step = 0;
  for (int64_t a = g - woff[lo]; a >= 0 && !step; a = win_parent(w, a))
    step = w[a].kind == XMEM_WIN_COMPONENT && w[a].category == XMEM_CAT_OPTIMIZER;
  in_step[g] = step;
}
constexpr int64_t kStepCandidate = int64_t(1) << 32;  // role bit: a product allocated in an optimizer.step() phase
// the window each block links to (index in its trace, -1 if none), its role by the operator rule
// (with kStepCandidate for a product in an optimizer.step() phase), and whether it is a product of
// a parameter operator (pflag)
__global__ void k_att_blocks(const xmem_block* blocks, const uint32_t* btid, int64_t nb, const xmem_window* win,
                             const int64_t* woff, const int64_t* comp_end, const uint32_t* in_step,
                             const int32_t* bad, int32_t* bwin, uint32_t* flag, int64_t* role, uint32_t* pflag) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad) return;
  const uint32_t t = btid[b];
  const int64_t base = woff[t], n = woff[t + 1] - base;
  const xmem_window* w = win + base;
  const int64_t ta = blocks[b].t_alloc, tf = blocks[b].t_free;
  int64_t lo = 0, hi = n;  // last window that starts no later than the allocation
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (w[mid].start <= ta) lo = mid + 1; else hi = mid;
  }
  int64_t i = lo - 1;
  while (i >= 0 && w[i].end < ta) i = win_parent(w, i);  // up to the innermost window containing it
  const bool step = i >= 0 && in_step[base + i];
  int32_t link = -1;
  int64_t cat = XMEM_CAT_OTHER;
  bool product = false;
  for (; i >= 0; i = win_parent(w, i)) {
    const xmem_window x = w[i];
    if (x.kind != XMEM_WIN_OPERATOR) continue;
    if (x.start < ta && tf < x.end) { link = (int32_t)i; break; }  // (i) a temporary: strictly inside the window
    if (tf > comp_end[base + i]) {                                   // (ii) a product
      link = (int32_t)i;
      cat = x.category;
      product = true;
      break;
    }
  }
  if (bwin) bwin[b] = link;
  flag[b] = link >= 0 ? 1u : 0u;
  role[b] = cat | (product && step ? kStepCandidate : 0);
  pflag[b] = product && cat == XMEM_CAT_PARAMETER ? 1u : 0u;
}
// Section 3.3 item 5: the parameter sizes of each trace as an open-addressing hash set of block
// indices + 1 (0: empty), two slots per parameter block at [2 * first, 2 * end) of the trace's
// parameters in the exclusive scan pscan of pflag.  At most half full, so every probe sequence
// reaches an empty slot.
struct ParamSet { int64_t base, cap; };
__device__ __forceinline__ ParamSet param_set(const int64_t* boff, int64_t nb, const uint32_t* pscan,
                                              const uint32_t* total, uint32_t t) {
  const int64_t lo = boff[t], hi = boff[t + 1];
  const int64_t ps = lo < nb ? pscan[lo] : *total, pe = hi < nb ? pscan[hi] : *total;
  return ParamSet{2 * ps, 2 * (pe - ps)};
}
__device__ __forceinline__ uint64_t size_hash(int64_t size) {
  return ((uint64_t)size * 0x9E3779B97F4A7C15ull) >> 32;
}
__global__ void k_opt_flags_keep(const uint32_t* pflag, int64_t nb, const int32_t* bad, uint32_t* copy) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad) return;
  copy[b] = pflag[b];
}
// each parameter block clears its two slots of its trace's set
__global__ void k_opt_clear(const uint32_t* pflag_scan, const uint32_t* pflag, int64_t nb, const int32_t* bad,
                            uint32_t* tab) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad || !pflag[b]) return;
  tab[2 * (int64_t)pflag_scan[b]] = 0;
  tab[2 * (int64_t)pflag_scan[b] + 1] = 0;
}
__global__ void k_opt_insert(const xmem_block* blocks, const uint32_t* btid, const int64_t* boff, int64_t nb,
                             const uint32_t* pflag, const uint32_t* pscan, const uint32_t* total, const int32_t* bad,
                             uint32_t* tab) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad || !pflag[b]) return;
  const ParamSet ps = param_set(boff, nb, pscan, total, btid[b]);
  const int64_t size = blocks[b].size;
  for (int64_t s = (int64_t)(size_hash(size) % (uint64_t)ps.cap);; s = s + 1 == ps.cap ? 0 : s + 1) {
    const uint32_t old = atomicCAS(&tab[ps.base + s], 0u, (uint32_t)(b + 1));
    if (old == 0 || blocks[old - 1].size == size) return;  // inserted, or the size is there already
  }
}
// a product in an optimizer.step() phase whose size is a parameter's becomes an optimizer state
__global__ void k_opt_mark(const xmem_block* blocks, const uint32_t* btid, const int64_t* boff, int64_t nb,
                           const uint32_t* pscan, const uint32_t* total, const int32_t* bad, const uint32_t* tab,
                           int64_t* role) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad) return;
  const int64_t r = role[b];
  if (!(r & kStepCandidate)) return;
  int64_t out = r & ~kStepCandidate;
  const ParamSet ps = param_set(boff, nb, pscan, total, btid[b]);
  if (ps.cap > 0) {
    const int64_t size = blocks[b].size;
    for (int64_t s = (int64_t)(size_hash(size) % (uint64_t)ps.cap);; s = s + 1 == ps.cap ? 0 : s + 1) {
      const uint32_t v = tab[ps.base + s];
      if (v == 0) break;
      if (blocks[v - 1].size == size) { out = XMEM_CAT_OPTIMIZER; break; }
    }
  }
  role[b] = out;
}
__global__ void k_att_emit(const xmem_block* blocks, int64_t nb, const int32_t* bad, const uint32_t* flag,
                           const uint32_t* idx, const int64_t* role, xmem_block* kept) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad || !flag[b]) return;
  xmem_block x = blocks[b];
  x.category = (int32_t)(role[b] & ~kStepCandidate);
  kept[idx[b]] = x;
}

// ---------------------------------------------------------------- orchestration (Section 3.3)
// first value > t in the ascending v[lo, hi), or kPersist
__device__ __forceinline__ int64_t next_marker(const int64_t* v, int64_t lo, int64_t hi, int64_t t) {
  int64_t a = lo, b = hi;
  while (a < b) {
    const int64_t mid = (a + b) >> 1;
    if (v[mid] > t) b = mid; else a = mid + 1;
  }
  return a < hi ? v[a] : kPersist;
}
// retimed free of each block, and the two sort records of each block
// (2b: allocation, 2b+1: free); first key group: the rank at equal times
__global__ void k_orch_retime(const xmem_block* blocks, const uint32_t* btid, int64_t nb, const int64_t* steps,
                              const int64_t* soff, const int64_t* zg, const int64_t* zoff, const int32_t* bad,
                              int64_t* tfr, uint64_t* key, uint32_t* val) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad) return;
  const xmem_block x = blocks[b];
  const uint32_t t = btid[b];
  int64_t f = x.t_free;
  switch (x.category) {
    case XMEM_CAT_PARAMETER:
    case XMEM_CAT_OPTIMIZER:
      f = kPersist;
      break;
    case XMEM_CAT_BATCH: {
      const int64_t e = next_marker(steps, soff[t], soff[t + 1], x.t_alloc);
      f = f < e ? f : e;
      break;
    }
    case XMEM_CAT_GRADIENT:
      f = next_marker(zg, zoff[t], zoff[t + 1], x.t_alloc);
      break;
    default:
      break;
  }
  if (f != kPersist && f < x.t_alloc) f = x.t_alloc;
  tfr[b] = f;
  key[2 * b] = 1;                          // allocation
  key[2 * b + 1] = f == x.t_alloc ? 2 : 0;  // free of a block allocated at that time, or of an earlier one
  val[2 * b] = (uint32_t)(2 * b);
  val[2 * b + 1] = (uint32_t)(2 * b + 1);
}
// the times of the allocation and free records (sign bit flipped: signed order as unsigned); a
// persistent block's free takes no part (it sorts last by its trace key)
__global__ __launch_bounds__(kThreads) void k_orch_range(const xmem_block* blocks, const int64_t* tfr, int64_t nb,
                                                         const int32_t* bad, uint64_t* kr) {
  if (*bad) return;
  RangePart p;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b0 < nb; b0 += kRangeUnroll * stride) {
    int64_t ta[kRangeUnroll], tf[kRangeUnroll];
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) {
      const int64_t b = b0 + u * stride;
      ta[u] = b < nb ? blocks[b].t_alloc : 0;
      tf[u] = b < nb ? tfr[b] : kPersist;
    }
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) {
      p.add(b0 + u * stride < nb, (uint64_t)ta[u] ^ (1ull << 63), 0);
      p.add(tf[u] != kPersist, (uint64_t)tf[u] ^ (1ull << 63), 0);
    }
  }
  range_commit(kr, p);
}
// The orchestration sort's layout, chosen on the device from the time range (kr[5]: bit 0 set
// for the joint key, bit 1 when the sorted records end in the second buffer, bits 8.. the time
// bits tb).  Joint key, when trace, time and rank fit in 64 bits together:
// (trace << (tb + 2)) | (time << 2) | rank, the free of a persistent block last (T << (tb + 2));
// one sort of tbits + tb + 2 bits.  Otherwise three key groups as separate sorts: the rank
// (k_orch_retime), the time in an even number of passes, then the trace.  The host launches
// the same kernels either way; the gates skip the passes a layout does not take: gate[0] the
// time sort (or the joint sort), gate[1] the rank sort, gate[2] the trace sort.
__global__ void k_orch_mode(uint64_t* kr, int tbits, bool trace_odd, int32_t* gate) {
  const int tb = range_bits(kr, 0);
  const bool joint = tbits + tb + 2 <= 64;
  const int jp = (tbits + tb + 2 + 7) / 8;
  gate[0] = joint ? 8 * jp : range_gate(kr, 0);
  gate[1] = joint ? 0 : 64;
  gate[2] = joint ? 0 : 64;
  // the time sort starts in the second buffer; the separate layout then takes the trace passes
  const bool in_b = joint ? !(jp & 1) : !trace_odd;
  kr[5] = (joint ? kJoint : 0) | (in_b ? kJointBuf : 0) | ((uint64_t)tb << 8);
}
// second key group: the time, rebased to the batch's earliest; with the joint key, the whole key
// of every record (in record order, into the buffer the time sort starts from)
__global__ void k_orch_time_keys(const xmem_block* blocks, const uint32_t* btid, const int64_t* tfr, int64_t n,
                                 int64_t T, const int32_t* bad, const uint64_t* kr, uint32_t* val, uint64_t* key) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n || *bad) return;
  const uint64_t meta = kr[5];
  if (meta & kJoint) {
    const int tb = (int)(meta >> 8);
    const int64_t b = p >> 1;
    const int64_t ta = blocks[b].t_alloc, f = tfr[b];
    uint64_t k;
    if (p & 1) {
      k = f == kPersist ? (uint64_t)T << (tb + 2)
                        : ((uint64_t)btid[b] << (tb + 2)) | ((((uint64_t)f ^ (1ull << 63)) - kr[0]) << 2) |
                              (f == ta ? 2u : 0u);
    } else {
      k = ((uint64_t)btid[b] << (tb + 2)) | ((((uint64_t)ta ^ (1ull << 63)) - kr[0]) << 2) | 1u;
    }
    key[p] = k;
    val[p] = (uint32_t)p;
    return;
  }
  const uint32_t r = val[p];
  const int64_t tm = (r & 1) ? tfr[r >> 1] : blocks[r >> 1].t_alloc;
  key[p] = ((r & 1) && tm == kPersist) ? 0 : ((uint64_t)tm ^ (1ull << 63)) - kr[0];
}
// third key group: the trace, T for the free of a persistent block (sorts last)
__global__ void k_orch_trace_keys(const uint32_t* btid, const int64_t* tfr, int64_t n, int64_t T, const int32_t* bad,
                                  const uint64_t* kr, const uint32_t* val, uint64_t* key) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n || *bad || (kr[5] & kJoint)) return;
  const uint32_t r = val[p];
  key[p] = ((r & 1) && tfr[r >> 1] == kPersist) ? (uint64_t)T : (uint64_t)btid[r >> 1];
}
// words per block: 1 + (a free after retiming)
__global__ void k_orch_counts(const int64_t* tfr, int64_t nb, const int32_t* bad, uint32_t* cnt) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb || *bad) return;
  cnt[b] = tfr[b] == kPersist ? 1u : 2u;
}
__global__ void k_orch_offsets(const int64_t* boff, int64_t T, int64_t nb, const int32_t* bad, const uint32_t* scan,
                               const uint32_t* total, int64_t* eoff) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t > T || *bad) return;
  eoff[t] = boff[t] < nb ? (int64_t)scan[boff[t]] : (int64_t)*total;
}
// position of each allocation's word within its trace (the joint key holds the trace)
__global__ void k_orch_apos(const uint32_t* btid, const int64_t* eoff, const uint32_t* total, const int32_t* bad,
                            const uint64_t* kr, const uint64_t* ka, const uint32_t* va, const uint64_t* kb,
                            const uint32_t* vb, uint32_t* apos) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (*bad || p >= (int64_t)*total) return;
  const uint64_t meta = kr[5];
  const uint32_t r = ((meta & kJointBuf) ? vb : va)[p];
  if (r & 1) return;
  const uint64_t t = (meta & kJoint) ? ((meta & kJointBuf) ? kb : ka)[p] >> ((int)(meta >> 8) + 2) : btid[r >> 1];
  apos[r >> 1] = (uint32_t)(p - eoff[t]);
}
__global__ void k_orch_words(const xmem_block* blocks, const uint32_t* total, const int32_t* bad, const uint64_t* kr,
                             const uint32_t* va, const uint32_t* vb, const uint32_t* apos, uint64_t* events) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (*bad || p >= (int64_t)*total) return;
  const uint32_t r = ((kr[5] & kJointBuf) ? vb : va)[p];
  events[p] = (r & 1) ? (kFree | (uint64_t)apos[r >> 1]) : (uint64_t)blocks[r >> 1].size;
}

bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255) == 0; }

}  // namespace

extern "C" {

size_t xmem_prep_workspace_bytes(int64_t n_traces, int64_t n_records) {
  if (n_traces < 0 || n_records < 0 || n_records > XMEM_PREP_MAX_RECORDS || n_traces > INT32_MAX - 1) return 0;
  return carve(nullptr, n_traces, n_records, nullptr);
}

int xmem_lifecycles(const xmem_raw_event* d_raw, const int32_t* d_category, const int64_t* d_raw_offsets,
                    int64_t n_traces, int64_t total_raw, xmem_block* d_blocks, int64_t* d_block_offsets,
                    int64_t* d_unmatched_frees, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                    void* hip_stream) {
  if (n_traces < 0 || total_raw < 0 || total_raw > XMEM_PREP_MAX_RECORDS || n_traces > INT32_MAX - 1) return XMEM_EINVAL;
  if (!d_raw_offsets || !d_block_offsets || !d_status || (total_raw > 0 && (!d_raw || !d_blocks))) return XMEM_EINVAL;
  const size_t need = carve(nullptr, n_traces, total_raw, nullptr);
  if (!d_workspace || workspace_bytes < need || !aligned256(d_workspace)) return XMEM_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  PrepWs w;
  carve(d_workspace, n_traces, total_raw, &w);
  const int64_t T = n_traces, n = total_raw;
  k_zero_i32<<<1, 1, 0, st>>>(w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_raw_offsets, T, n, w.bad);
  if (d_unmatched_frees && T > 0) k_zero_i64<<<grid_of(T, 256), 256, 0, st>>>(d_unmatched_frees, T);
  if (n > 0 && T > 0) {
    k_trace_of<<<(unsigned)tiles_of(n), kThreads, 0, st>>>(d_raw_offsets, T, n, w.bad, w.tid);
    int32_t* gate = reinterpret_cast<int32_t*>(w.kr + 3);
    int32_t* gate2 = reinterpret_cast<int32_t*>(w.kr + 4);
    int tbits = 0;
    while (tbits < 63 && (T >> tbits) != 0) ++tbits;  // bits of the trace field (0..T)
    const bool second_odd = (bits_for(T) / 8) & 1;
    k_range_init<<<1, 1, 0, st>>>(w.kr);
    k_life_range<<<(unsigned)std::min<int64_t>(kRangeBlocks, grid_of(n, kThreads)), kThreads, 0, st>>>(d_raw, n, w.bad, w.kr);
    k_life_keys<<<grid_of(n, 256), 256, 0, st>>>(d_raw, w.tid, n, T, tbits, second_odd, w.bad, w.kr, w.s.ka, w.s.va,
                                                 gate, gate2, w.u);
    // by (trace, address), or by address in an even number of passes; stream order kept
    sort_bits(w.s, n, 0, 64, false, st, gate);
    // the separate layout only: then by trace (from the buffer the even passes end in)
    k_life_trace_keys<<<grid_of(n, 256), 256, 0, st>>>(d_raw, w.tid, n, T, w.bad, w.kr, w.s.va, w.s.ka);
    sort_bits(w.s, n, 0, bits_for(T), false, st, gate2);
    k_life_pair<<<grid_of(n, 256), 256, 0, st>>>(d_raw, w.tid, w.kr, w.s.ka, w.s.va, w.s.kb, w.s.vb, n, T, w.bad,
                                                 w.t64, d_unmatched_frees);
    ScanWs sw{w.s.scan.part, w.s.scan.total};
    scan_u32(w.u, w.u, n, sw, st);
    k_life_emit<<<grid_of(n, 256), 256, 0, st>>>(d_raw, d_category, n, w.bad, w.u, w.t64, d_blocks);
    k_life_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_raw_offsets, T, n, w.bad, w.u, w.s.scan.total,
                                                        d_block_offsets);
  } else {
    k_zero_i64<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T + 1);
  }
  k_fill_offsets_zero<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T, w.bad, d_status);
  return hipGetLastError() == hipSuccess ? XMEM_OK : XMEM_EHIP;
}

int xmem_attribute(const xmem_block* d_blocks, const int64_t* d_block_offsets, int64_t n_traces,
                   int64_t total_blocks, const xmem_window* d_windows, const int64_t* d_window_offsets,
                   int64_t total_windows, xmem_block* d_kept, int64_t* d_kept_offsets, int32_t* d_block_window,
                   int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* hip_stream) {
  if (n_traces < 0 || total_blocks < 0 || total_windows < 0 || n_traces > INT32_MAX - 1) return XMEM_EINVAL;
  const int64_t n = total_blocks > total_windows ? total_blocks : total_windows;
  if (n > XMEM_PREP_MAX_RECORDS) return XMEM_EINVAL;
  if (!d_block_offsets || !d_window_offsets || !d_kept_offsets || !d_status) return XMEM_EINVAL;
  if ((total_blocks > 0 && (!d_blocks || !d_kept)) || (total_windows > 0 && !d_windows)) return XMEM_EINVAL;
  const int64_t T = n_traces, nb = total_blocks, nw = total_windows;
  const size_t need = carve(nullptr, T, n, nullptr);
  if (!d_workspace || workspace_bytes < need || !aligned256(d_workspace)) return XMEM_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  PrepWs w;
  carve(d_workspace, T, n, &w);
  int64_t* comp_end = reinterpret_cast<int64_t*>(w.s.ka);  // n words each: the sort buffers are free here
  int64_t* role = reinterpret_cast<int64_t*>(w.s.kb);
  uint32_t* in_step = w.apos;                                  // per window
  uint32_t* pflag = w.s.vb;                                    // per block, then its exclusive scan
  uint32_t* tab = reinterpret_cast<uint32_t*>(w.t64);          // 2n slots: the parameter-size sets
  k_zero_i32<<<1, 1, 0, st>>>(w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T, nb, w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_window_offsets, T, nw, w.bad);
  if (nb > 0 && T > 0) {
    if (nw > 0)
      k_att_comp_end<<<grid_of(nw, 256), 256, 0, st>>>(d_windows, d_window_offsets, T, nw, w.bad, comp_end, in_step);
    k_trace_of<<<(unsigned)tiles_of(nb), kThreads, 0, st>>>(d_block_offsets, T, nb, w.bad, w.tid);
    k_att_blocks<<<grid_of(nb, 256), 256, 0, st>>>(d_blocks, w.tid, nb, d_windows, d_window_offsets, comp_end, in_step,
                                                   w.bad, d_block_window, w.u, role, pflag);
    ScanWs sw{w.s.scan.part, w.s.scan.total};
    // Section 3.3 item 5: parameter sizes per trace, then the products of the optimizer.step() phases
    k_opt_flags_keep<<<grid_of(nb, 256), 256, 0, st>>>(pflag, nb, w.bad, w.s.va);
    scan_u32(pflag, pflag, nb, sw, st);
    k_opt_clear<<<grid_of(nb, 256), 256, 0, st>>>(pflag, w.s.va, nb, w.bad, tab);
    k_opt_insert<<<grid_of(nb, 256), 256, 0, st>>>(d_blocks, w.tid, d_block_offsets, nb, w.s.va, pflag,
                                                   w.s.scan.total, w.bad, tab);
    k_opt_mark<<<grid_of(nb, 256), 256, 0, st>>>(d_blocks, w.tid, d_block_offsets, nb, pflag, w.s.scan.total, w.bad,
                                                 tab, role);
    scan_u32(w.u, w.s.va, nb, sw, st);
    k_att_emit<<<grid_of(nb, 256), 256, 0, st>>>(d_blocks, nb, w.bad, w.u, w.s.va, role, d_kept);
    k_life_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T, nb, w.bad, w.s.va, w.s.scan.total,
                                                        d_kept_offsets);
  } else {
    k_zero_i64<<<grid_of(T + 1, 256), 256, 0, st>>>(d_kept_offsets, T + 1);
  }
  k_fill_offsets_zero<<<grid_of(T + 1, 256), 256, 0, st>>>(d_kept_offsets, T, w.bad, d_status);
  return hipGetLastError() == hipSuccess ? XMEM_OK : XMEM_EHIP;
}

int xmem_orchestrate(const xmem_block* d_blocks, const int64_t* d_block_offsets, int64_t n_traces,
                     int64_t total_blocks, const int64_t* d_step_ts, const int64_t* d_step_offsets,
                     const int64_t* d_zero_grad_ts, const int64_t* d_zero_grad_offsets, uint64_t* d_events,
                     int64_t* d_event_offsets, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                     void* hip_stream) {
  if (n_traces < 0 || total_blocks < 0 || 2 * total_blocks > XMEM_PREP_MAX_RECORDS || n_traces > INT32_MAX - 1)
    return XMEM_EINVAL;
  if (!d_block_offsets || !d_step_offsets || !d_zero_grad_offsets || !d_event_offsets || !d_status) return XMEM_EINVAL;
  if (total_blocks > 0 && (!d_blocks || !d_events)) return XMEM_EINVAL;
  const int64_t T = n_traces, nb = total_blocks, n = 2 * total_blocks;
  const size_t need = carve(nullptr, T, n, nullptr);
  if (!d_workspace || workspace_bytes < need || !aligned256(d_workspace)) return XMEM_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  PrepWs w;
  carve(d_workspace, T, n, &w);
  k_zero_i32<<<1, 1, 0, st>>>(w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T, nb, w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_step_offsets, T, -1, w.bad);
  k_check_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_zero_grad_offsets, T, -1, w.bad);
  if (nb > 0 && T > 0) {
    k_trace_of<<<(unsigned)tiles_of(nb), kThreads, 0, st>>>(d_block_offsets, T, nb, w.bad, w.tid);
    k_orch_retime<<<grid_of(nb, 256), 256, 0, st>>>(d_blocks, w.tid, nb, d_step_ts, d_step_offsets, d_zero_grad_ts,
                                                    d_zero_grad_offsets, w.bad, w.t64, w.s.ka, w.s.va);
    // gate[0]: the time (or joint) sort, gate[1]: the rank sort, gate[2]: the trace sort
    int32_t* gate = reinterpret_cast<int32_t*>(w.kr + 3);
    int tbits = 0;
    while (tbits < 63 && (T >> tbits) != 0) ++tbits;  // bits of the trace field (0..T)
    k_range_init<<<1, 1, 0, st>>>(w.kr);
    k_orch_range<<<(unsigned)std::min<int64_t>(kRangeBlocks, grid_of(nb, kThreads)), kThreads, 0, st>>>(d_blocks, w.t64, nb,
                                                                                                  w.bad, w.kr);
    k_orch_mode<<<1, 1, 0, st>>>(w.kr, tbits, (bits_for(T) / 8) & 1, gate);
    sort_bits(w.s, n, 0, 8, false, st, gate + 1);  // rank at equal times (separate layout)
    k_orch_time_keys<<<grid_of(n, 256), 256, 0, st>>>(d_blocks, w.tid, w.t64, n, T, w.bad, w.kr, w.s.vb, w.s.kb);
    sort_bits(w.s, n, 0, 64, true, st, gate);  // time (its span only), or the joint key
    k_orch_trace_keys<<<grid_of(n, 256), 256, 0, st>>>(w.tid, w.t64, n, T, w.bad, w.kr, w.s.vb, w.s.kb);
    sort_bits(w.s, n, 0, bits_for(T), true, st, gate + 2);  // trace; persistent blocks' frees last
    k_orch_counts<<<grid_of(nb, 256), 256, 0, st>>>(w.t64, nb, w.bad, w.u);
    ScanWs sw{w.s.scan.part, w.s.scan.total};
    scan_u32(w.u, w.u, nb, sw, st);
    k_orch_offsets<<<grid_of(T + 1, 256), 256, 0, st>>>(d_block_offsets, T, nb, w.bad, w.u, w.s.scan.total,
                                                        d_event_offsets);
    k_orch_apos<<<grid_of(n, 256), 256, 0, st>>>(w.tid, d_event_offsets, w.s.scan.total, w.bad, w.kr, w.s.ka, w.s.va,
                                                 w.s.kb, w.s.vb, w.apos);
    k_orch_words<<<grid_of(n, 256), 256, 0, st>>>(d_blocks, w.s.scan.total, w.bad, w.kr, w.s.va, w.s.vb, w.apos,
                                                  d_events);
  } else {
    k_zero_i64<<<grid_of(T + 1, 256), 256, 0, st>>>(d_event_offsets, T + 1);
  }
  k_fill_offsets_zero<<<grid_of(T + 1, 256), 256, 0, st>>>(d_event_offsets, T, w.bad, d_status);
  return hipGetLastError() == hipSuccess ? XMEM_OK : XMEM_EHIP;
}

}  // extern "C"
