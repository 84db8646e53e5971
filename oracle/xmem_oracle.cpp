// xmem_oracle.cpp -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT PATH.
//
// Plain, slow-on-purpose CPU reference of the xMem Memory Simulator
// (Section 3.4): every trace is replayed chronologically through a caching
// allocator model with (i) size round-up, (ii) segment requests, (iii) best fit
// with coalescing (search, split, merge), (iv) caching of freed blocks and
// (v) OOM after reclaiming cached segments.  Only tests, the smoke check and
// the benchmark's CPU-baseline leg may load this library.
//
// It shares no code with the GPU library: its own structs (same byte layout as
// the public ABI, by construction, checked field by field in the tests), its
// own validation, its own data structures (explicit segments, physically
// linked blocks, an ordered std::set per pool as the best-fit index).
//
// Readings of the paper that this file fixes (the paper is silent on them):
//  * two pools, classified by the ROUNDED size: SMALL iff r <= small_max;
//    a pool only searches its own segments;
//  * best fit = minimum (size, address) among free blocks with size >= r;
//  * address model: one bump pointer per trace, segments laid out in creation
//    order, never reused;
//  * the front r bytes of the chosen block are used; the remainder becomes a
//    free block iff it is >= split_min of the pool;
//  * coalescing is immediate, with both physical neighbours, within a segment;
//  * segments are released only under capacity pressure: all segments that are
//    one whole free block, in both pools, then one retry;
//  * a zero-byte request is a no-op allocation (its free is a no-op);
//  * allocated = sum of rounded sizes of live handles; reserved = sum of live
//    segment sizes; both are sampled after every event, peaks take the first
//    event that reaches the maximum, -1 if the maximum is 0;
//  * a malformed event, an overflow or an OOM stops the trace; the state
//    reported is the one after the previous event, the series holds -1 from
//    the stopping event on.
#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstring>
#include <limits>
#include <set>
#include <thread>
#include <tuple>
#include <vector>

namespace {

struct OracleParams {  // field order of the public parameter struct
  uint32_t abi_version, flags;
  int64_t round_bytes, small_max, small_segment, mid_segment, min_large_alloc,
      large_round, split_min_small, split_min_large, capacity;
};

struct OracleResult {  // field order of the public result struct
  int64_t peak_allocated, peak_reserved, peak_allocated_event, peak_reserved_event;
  int64_t final_allocated, final_reserved, segments_created, segments_released;
  int64_t max_free_small, max_free_large, stop_event;
  int32_t status, pad;
};

constexpr uint64_t kFreeBit = 1ull << 63;
constexpr int64_t kMaxRequest = int64_t(1) << 48;
constexpr int64_t kPoolCreatedLimit = int64_t(1) << 61;
constexpr int64_t kMaxTraceEvents = 0x7fffffff;

enum { ST_OK = 0, ST_OOM = 1, ST_BAD_FREE = 2, ST_BAD_EVENT = 3, ST_OVERFLOW = 4 };
enum { E_OK = 0, E_INVAL = -1, E_OFFSETS = -2 };
enum { SMALL = 0, LARGE = 1 };

bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int validate(const OracleParams* p) {
  if (!p) return E_INVAL;
  const int64_t lim = int64_t(1) << 40;
  if (p->abi_version != 1u || p->flags != 0) return E_INVAL;
  if (!pow2(p->round_bytes) || p->round_bytes > (int64_t(1) << 30)) return E_INVAL;
  const int64_t multiples[] = {p->small_max, p->small_segment, p->mid_segment, p->min_large_alloc,
                               p->large_round};
  for (int64_t v : multiples)
    if (v < 1 || v > lim || v % p->round_bytes != 0) return E_INVAL;
  if (p->small_max > p->small_segment) return E_INVAL;
  if (p->min_large_alloc > p->mid_segment) return E_INVAL;
  if (p->split_min_small < 1 || p->split_min_small > lim) return E_INVAL;
  if (p->split_min_large < 1 || p->split_min_large > lim) return E_INVAL;
  if (p->capacity < 1) return E_INVAL;
  return E_OK;
}

// A block is a contiguous byte range of one segment, either handed out or free.
struct Block {
  int64_t addr, size;
  int64_t seg;
  int64_t prev, next;  // physical neighbours inside the segment, -1 at the ends
  bool free;
};

struct Segment {
  int64_t base, size;
  int pool;
  bool live;
  int64_t first;  // block at the segment base (never changes: merges keep the lower block)
};

class Replay {
 public:
  Replay(const OracleParams& p, const uint64_t* ev, int64_t n, int64_t* series)
      : P(p), ev_(ev), n_(n), series_(series) {}

  OracleResult run() {
    OracleResult R{};
    R.peak_allocated_event = -1;
    R.peak_reserved_event = -1;
    R.stop_event = -1;
    kind_.assign(n_, 0);      // 0 = not an alloc, 1 = alloc
    freed_.assign(n_, 0);
    handle_.assign(n_, -1);   // block of the allocation, -1 for a no-op allocation
    req_.assign(n_, 0);       // rounded request of the allocation
    for (int64_t e = 0; e < n_; ++e) {
      const int status = step(e);
      if (status != ST_OK) {
        R.status = status;
        R.stop_event = e;
        if (series_)
          for (int64_t k = e; k < n_; ++k) series_[k] = -1;
        break;
      }
      if (series_) series_[e] = reserved_;
      if (allocated_ > R.peak_allocated) { R.peak_allocated = allocated_; R.peak_allocated_event = e; }
      if (reserved_ > R.peak_reserved) { R.peak_reserved = reserved_; R.peak_reserved_event = e; }
      R.max_free_small = std::max<int64_t>(R.max_free_small, (int64_t)index_[SMALL].size());
      R.max_free_large = std::max<int64_t>(R.max_free_large, (int64_t)index_[LARGE].size());
    }
    R.final_allocated = allocated_;
    R.final_reserved = reserved_;
    R.segments_created = created_;
    R.segments_released = released_;
    return R;
  }

 private:
  // Section 3.4 (i): round the request up to a multiple of the granule.
  int64_t round_up(int64_t s) const { return (s + P.round_bytes - 1) / P.round_bytes * P.round_bytes; }

  // Section 3.4 (ii) with Section 2.2.2 and 6.4 (iii): size of a new segment.
  int64_t segment_size(int pool, int64_t r) const {
    if (pool == SMALL) return P.small_segment;
    if (r < P.min_large_alloc) return P.mid_segment;
    return (r + P.large_round - 1) / P.large_round * P.large_round;
  }

  void index_insert(int64_t b) { index_[segs_[blocks_[b].seg].pool].insert({blocks_[b].size, blocks_[b].addr, b}); }
  void index_erase(int64_t b) { index_[segs_[blocks_[b].seg].pool].erase({blocks_[b].size, blocks_[b].addr, b}); }

  // Section 3.4 (iii): best fit -- smallest free block that can hold r, lowest address on ties.
  int64_t best_fit(int pool, int64_t r) const {
    auto it = index_[pool].lower_bound({r, std::numeric_limits<int64_t>::min(), std::numeric_limits<int64_t>::min()});
    return it == index_[pool].end() ? -1 : std::get<2>(*it);
  }

  // Section 3.4 (iv)-(v): bytes held by segments that are one whole free block.
  bool segment_idle(const Segment& s) const {
    const Block& b = blocks_[s.first];
    return s.live && b.free && b.size == s.size;
  }

  int64_t new_segment(int pool, int64_t S) {
    Segment s{bump_, S, pool, true, (int64_t)blocks_.size()};
    segs_.push_back(s);
    blocks_.push_back(Block{bump_, S, (int64_t)segs_.size() - 1, -1, -1, true});
    index_insert(s.first);
    bump_ += S;
    reserved_ += S;
    created_bytes_[pool] += S;
    ++created_;
    return s.first;
  }

  int alloc(int64_t e, int64_t s) {
    if (s > kMaxRequest) return ST_BAD_EVENT;
    kind_[e] = 1;
    const int64_t r = s == 0 ? 0 : round_up(s);
    if (r == 0) return ST_OK;  // no-op allocation
    const int pool = r <= P.small_max ? SMALL : LARGE;
    int64_t b = best_fit(pool, r);
    if (b < 0) {
      const int64_t S = segment_size(pool, r);
      if (created_bytes_[pool] > kPoolCreatedLimit - S) return ST_OVERFLOW;
      if (S > P.capacity - reserved_) {
        int64_t idle = 0;
        for (const Segment& g : segs_)
          if (segment_idle(g)) idle += g.size;
        if (S > P.capacity - (reserved_ - idle)) return ST_OOM;
        for (Segment& g : segs_)
          if (segment_idle(g)) {
            index_erase(g.first);
            g.live = false;
            reserved_ -= g.size;
            ++released_;
          }
      }
      b = new_segment(pool, S);
    }
    index_erase(b);
    const int64_t rem = blocks_[b].size - r;
    if (rem >= (pool == SMALL ? P.split_min_small : P.split_min_large)) {
      Block tail{blocks_[b].addr + r, rem, blocks_[b].seg, b, blocks_[b].next, true};
      const int64_t t = (int64_t)blocks_.size();
      blocks_.push_back(tail);
      if (tail.next >= 0) blocks_[tail.next].prev = t;
      blocks_[b].next = t;
      blocks_[b].size = r;
      index_insert(t);
    }
    blocks_[b].free = false;
    handle_[e] = b;
    req_[e] = r;
    allocated_ += r;
    return ST_OK;
  }

  int release(int64_t e, uint64_t w) {
    if (((w >> 32) & 0x7fffffffull) != 0) return ST_BAD_EVENT;
    const int64_t h = (int64_t)(w & 0xffffffffull);
    if (h >= e || kind_[h] != 1 || freed_[h]) return ST_BAD_FREE;
    freed_[h] = 1;
    int64_t b = handle_[h];
    if (b < 0) return ST_OK;  // free of a no-op allocation
    allocated_ -= req_[h];
    blocks_[b].free = true;
    const int64_t p = blocks_[b].prev;
    if (p >= 0 && blocks_[p].free) {  // merge into the lower neighbour
      index_erase(p);
      blocks_[p].size += blocks_[b].size;
      blocks_[p].next = blocks_[b].next;
      if (blocks_[b].next >= 0) blocks_[blocks_[b].next].prev = p;
      b = p;
    }
    const int64_t q = blocks_[b].next;
    if (q >= 0 && blocks_[q].free) {  // absorb the upper neighbour
      index_erase(q);
      blocks_[b].size += blocks_[q].size;
      blocks_[b].next = blocks_[q].next;
      if (blocks_[q].next >= 0) blocks_[blocks_[q].next].prev = b;
    }
    index_insert(b);
    return ST_OK;
  }

  int step(int64_t e) {
    const uint64_t w = ev_[e];
    return (w & kFreeBit) ? release(e, w) : alloc(e, (int64_t)w);
  }

  const OracleParams& P;
  const uint64_t* ev_;
  int64_t n_;
  int64_t* series_;
  std::vector<Block> blocks_;
  std::vector<Segment> segs_;
  std::set<std::tuple<int64_t, int64_t, int64_t>> index_[2];
  std::vector<uint8_t> kind_, freed_;
  std::vector<int64_t> handle_, req_;
  int64_t allocated_ = 0, reserved_ = 0, bump_ = 0;
  int64_t created_bytes_[2] = {0, 0};
  int64_t created_ = 0, released_ = 0;
};

}  // namespace

extern "C" {

int xmem_oracle_validate_params(const OracleParams* p) { return validate(p); }

// Host pointers throughout.  out_series may be NULL.  n_threads <= 0 means 1.
int xmem_oracle_replay_batch(const uint64_t* events, const int64_t* offsets, int64_t n_traces,
                             const OracleParams* params, OracleResult* out, int64_t* out_series,
                             int n_threads) {
  if (n_traces < 0 || !offsets || (n_traces > 0 && !out)) return E_INVAL;
  if (n_traces > 0 && !events && offsets[n_traces] > 0) return E_INVAL;
  if (validate(params) != E_OK) return E_INVAL;
  if (offsets[0] != 0) return E_OFFSETS;
  for (int64_t t = 0; t < n_traces; ++t) {
    const int64_t len = offsets[t + 1] - offsets[t];
    if (len < 0 || len > kMaxTraceEvents) return E_OFFSETS;
  }
  if (n_threads <= 0) n_threads = 1;
  std::atomic<int64_t> next{0};
  auto worker = [&]() {
    for (int64_t t; (t = next.fetch_add(1)) < n_traces;) {
      const int64_t b = offsets[t], n = offsets[t + 1] - offsets[t];
      Replay rp(*params, events + b, n, out_series ? out_series + b : nullptr);
      out[t] = rp.run();
    }
  };
  if (n_threads == 1) {
    worker();
  } else {
    std::vector<std::thread> pool;
    for (int i = 0; i < n_threads; ++i) pool.emplace_back(worker);
    for (auto& th : pool) th.join();
  }
  return E_OK;
}

// Section 4.1, Eq. (1): an estimate predicts an out-of-memory failure on a device whose maximum
// memory is m_max when the estimated peak exceeds it.  The estimated peak is the peak of the
// segment series (Section 3.4: the maximum of the series is the estimated peak memory).  A
// replay that the simulated allocator itself stopped with OOM (Section 3.4 (v)) predicts OOM; a
// replay stopped for any other reason gives no estimate (-1).
int xmem_oracle_oom_predicted(const OracleResult* results, int64_t n_traces, int64_t m_max, int32_t* flags) {
  if (n_traces < 0 || m_max < 0 || (n_traces > 0 && (!results || !flags))) return E_INVAL;
  for (int64_t t = 0; t < n_traces; ++t) {
    const OracleResult& r = results[t];
    if (r.status == ST_OOM)
      flags[t] = 1;
    else if (r.status != ST_OK)
      flags[t] = -1;
    else
      flags[t] = r.peak_reserved > m_max ? 1 : 0;
  }
  return E_OK;
}

}  // extern "C"
