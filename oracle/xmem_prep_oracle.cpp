// CPU oracle of the trace-preparation steps upstream of the Memory Simulator
// -- TEST INFRASTRUCTURE.  Only the tests, the smoke check and the CPU leg of
// the benchmark load it; the HIP library never includes, links or calls it.
//
// Plain sequential code that follows the paper's description step by step:
//
//   lifecycles   Section 3.2 (Analyzer): the raw allocator events of a trace
//                are read in stream order and paired by address -- an
//                allocation opens a block at its address, the next
//                deallocation at that address closes it -- with addresses
//                reused after a close.  A block never closed is persistent.
//   attribute    Section 3.2 (time-based attribution): each block is linked to
//                an operator execution window that contains its allocation
//                time, if (i) its whole lifespan lies strictly inside that
//                window or (ii) it outlives the operator's high-level
//                component; blocks with no such operator are filtered out of
//                the sequence.  Then Section 3.3 item 5 (Optimizer): among the
//                blocks allocated during the optimizer.step() phase, those
//                whose size equals the size of one of the trace's parameter
//                blocks are its optimizer states.
//   orchestrate  Section 3.3 (Memory Orchestrator): each block's lifetime is
//                adjusted by category (parameters and optimizer states
//                persistent, batch data bounded by the iteration, gradients
//                freed at the zero_grad that follows them, activations and
//                everything else unchanged), then the allocations and frees
//                are put in time order and written as the Simulator's event
//                words.
//
// Readings where the paper is silent (stated once here, used below):
//   * a second allocation at an address whose block is still open leaves that
//     block without a deallocation, i.e. persistent;
//   * a deallocation at an address with no open block is dropped and counted;
//   * an event of 0 bytes is ignored; the size of a block is its allocation's;
//   * a batch-data block is freed at the first iteration boundary after its
//     allocation, or at its own free if that comes first;
//   * a gradient is freed at the first zero_grad strictly after its
//     allocation; with none, it stays to the end of the trace (persistent);
//   * a free earlier than its allocation is moved to the allocation time;
//   * at equal times: frees of blocks allocated earlier, then allocations,
//     then frees of blocks allocated at that same time; within each, the
//     blocks' allocation order;
//   * attribution looks at the operators whose window contains the allocation
//     time, end points included ("allocated during" the window), innermost
//     first (windows are properly nested; a window's parent encloses it);
//     rule (i) asks for start < t_alloc and t_free < end (the lifespan lies
//     strictly inside the window: a block allocated at the window's start or
//     freed at its end does not satisfy it); the component of an operator is
//     its nearest enclosing component window;
//   * a block linked by (ii) is a product of the operator and takes its role
//     (parameter, batch data, gradient); a block linked by (i) is a
//     temporary of the operator and takes the role "other";
//   * the optimizer.step() phase is a component window whose category is
//     "optimizer"; a product (rule (ii)) allocated inside such a window, end
//     points included, is an optimizer state when its size equals the size
//     of a block of the same trace whose role from the operator rule is
//     "parameter"; other blocks keep the role the operator rule gave them.
//     Only products qualify: the paper describes optimizer states as
//     persistent, and a temporary is freed inside its operator.
#include <stdint.h>

#include <algorithm>
#include <set>
#include <unordered_map>
#include <vector>

namespace {

struct RawEvent { int64_t ts; uint64_t addr; int64_t bytes; };
struct Block { int64_t size, t_alloc, t_free; int32_t category, pad; };
struct Window { int64_t start, end; int32_t parent, kind, category, pad; };
enum { WIN_COMPONENT = 0, WIN_OPERATOR = 1 };

constexpr int64_t kPersistent = INT64_MAX;
constexpr uint64_t kFreeBit = 1ull << 63;
enum { CAT_OTHER = 0, CAT_PARAMETER = 1, CAT_BATCH = 2, CAT_GRADIENT = 3, CAT_OPTIMIZER = 4 };

// Section 3.2: one trace's raw events -> its blocks in allocation order
int64_t lifecycles_one(const RawEvent* raw, const int32_t* cat, int64_t n, std::vector<Block>& out) {
  std::unordered_map<uint64_t, int64_t> open;  // address -> index in out of the open block
  int64_t unmatched = 0;
  for (int64_t k = 0; k < n; ++k) {
    const RawEvent& r = raw[k];
    if (r.bytes > 0) {
      out.push_back(Block{r.bytes, r.ts, kPersistent, cat ? cat[k] : CAT_OTHER, 0});
      open[r.addr] = (int64_t)out.size() - 1;  // a block still open there is never closed
    } else if (r.bytes < 0) {
      auto it = open.find(r.addr);
      if (it == open.end()) { ++unmatched; continue; }
      out[it->second].t_free = r.ts;
      open.erase(it);
    }
  }
  return unmatched;
}

// first value in the ascending list v[0..n) that is > t, or kPersistent
int64_t first_after(const int64_t* v, int64_t n, int64_t t) {
  for (int64_t i = 0; i < n; ++i)
    if (v[i] > t) return v[i];
  return kPersistent;
}

// Section 3.3: the lifetime of one block after the category rule
int64_t retimed_free(const Block& b, const int64_t* steps, int64_t ns, const int64_t* zg, int64_t nz) {
  int64_t f = b.t_free;
  switch (b.category) {
    case CAT_PARAMETER:
    case CAT_OPTIMIZER:
      f = kPersistent;
      break;
    case CAT_BATCH: {
      const int64_t end = first_after(steps, ns, b.t_alloc);
      f = std::min(f, end);
      break;
    }
    case CAT_GRADIENT:
      f = first_after(zg, nz, b.t_alloc);
      break;
    default:
      break;
  }
  if (f != kPersistent && f < b.t_alloc) f = b.t_alloc;
  return f;
}

struct Ev {
  int64_t time;
  int rank;       // 0 free of an earlier block, 1 allocation, 2 free of a block allocated at that time
  int64_t block;  // allocation order
  bool alloc;
};

void orchestrate_one(const Block* blocks, int64_t nb, const int64_t* steps, int64_t ns, const int64_t* zg, int64_t nz,
                     std::vector<uint64_t>& words) {
  std::vector<Ev> ev;
  for (int64_t b = 0; b < nb; ++b) {
    ev.push_back(Ev{blocks[b].t_alloc, 1, b, true});
    const int64_t f = retimed_free(blocks[b], steps, ns, zg, nz);
    if (f != kPersistent) ev.push_back(Ev{f, f == blocks[b].t_alloc ? 2 : 0, b, false});
  }
  std::stable_sort(ev.begin(), ev.end(), [](const Ev& a, const Ev& b) {
    if (a.time != b.time) return a.time < b.time;
    if (a.rank != b.rank) return a.rank < b.rank;
    return a.block < b.block;
  });
  std::vector<int64_t> pos(nb, -1);  // output index of each block's allocation
  for (size_t i = 0; i < ev.size(); ++i) {
    if (ev[i].alloc) {
      pos[ev[i].block] = (int64_t)i;
      words.push_back((uint64_t)blocks[ev[i].block].size);
    } else {
      words.push_back(kFreeBit | (uint64_t)pos[ev[i].block]);
    }
  }
}

// the enclosing window of window i, -1 for a root (a parent must come before its child)
int64_t parent_of(const Window* w, int64_t i) {
  const int64_t p = w[i].parent;
  return (p >= 0 && p < i) ? p : -1;
}

// Section 3.2: the window (index within the trace) a block is attributed to, or -1;
// *product is true when the link is rule (ii)
int64_t attribute_one(const Block& b, const Window* w, int64_t nw, bool* product) {
  int64_t inner = -1;  // innermost window containing the allocation time: the one that started last
  for (int64_t i = 0; i < nw; ++i)
    if (w[i].start <= b.t_alloc && b.t_alloc <= w[i].end && (inner < 0 || w[i].start >= w[inner].start)) inner = i;
  for (int64_t i = inner; i >= 0; i = parent_of(w, i)) {
    if (w[i].kind != WIN_OPERATOR) continue;
    if (w[i].start < b.t_alloc && b.t_free < w[i].end) {  // (i): the lifespan strictly inside the window
      *product = false;
      return i;
    }
    int64_t c = parent_of(w, i);  // (ii): outlives the operator's component
    while (c >= 0 && w[c].kind != WIN_COMPONENT) c = parent_of(w, c);
    if (c >= 0 && b.t_free > w[c].end) {
      *product = true;
      return i;
    }
  }
  return -1;
}

// Section 3.3 item 5: is the allocation time inside an optimizer.step() phase (a component
// window of category "optimizer", end points included)?
bool in_optimizer_step(const Block& b, const Window* w, int64_t nw) {
  for (int64_t i = 0; i < nw; ++i)
    if (w[i].kind == WIN_COMPONENT && w[i].category == CAT_OPTIMIZER && w[i].start <= b.t_alloc &&
        b.t_alloc <= w[i].end)
      return true;
  return false;
}

bool offsets_ok(const int64_t* off, int64_t T) {
  if (off[0] != 0) return false;
  for (int64_t t = 0; t < T; ++t)
    if (off[t + 1] < off[t]) return false;
  return true;
}

}  // namespace

extern "C" {

// cat: category of each raw event, given to the block its allocation opens (nullable: all 0).
// blocks: capacity raw_off[T]; block_off: T + 1; unmatched: T (nullable).  0, or -2 for bad offsets.
int xmem_oracle_lifecycles(const RawEvent* raw, const int32_t* cat, const int64_t* raw_off, int64_t T, Block* blocks,
                           int64_t* block_off, int64_t* unmatched) {
  if (!offsets_ok(raw_off, T)) return -2;
  block_off[0] = 0;
  for (int64_t t = 0; t < T; ++t) {
    std::vector<Block> out;
    const int64_t u = lifecycles_one(raw + raw_off[t], cat ? cat + raw_off[t] : nullptr, raw_off[t + 1] - raw_off[t], out);
    std::copy(out.begin(), out.end(), blocks + block_off[t]);
    block_off[t + 1] = block_off[t] + (int64_t)out.size();
    if (unmatched) unmatched[t] = u;
  }
  return 0;
}

// kept: capacity block_off[T]; kept_off: T + 1; block_window: block_off[T] (nullable).
// 0, or -2 for bad offsets.
int xmem_oracle_attribute(const Block* blocks, const int64_t* block_off, int64_t T, const Window* win,
                          const int64_t* win_off, Block* kept, int64_t* kept_off, int32_t* block_window) {
  if (!offsets_ok(block_off, T) || !offsets_ok(win_off, T)) return -2;
  kept_off[0] = 0;
  for (int64_t t = 0; t < T; ++t) {
    const Window* w = win + win_off[t];
    const int64_t nw = win_off[t + 1] - win_off[t];
    // the operator rule for every block of the trace
    std::vector<int64_t> link;
    std::vector<int32_t> role;
    std::vector<bool> product;
    std::set<int64_t> param_sizes;
    for (int64_t b = block_off[t]; b < block_off[t + 1]; ++b) {
      bool prod = false;
      const int64_t i = attribute_one(blocks[b], w, nw, &prod);
      link.push_back(i);
      product.push_back(i >= 0 && prod);
      role.push_back(i >= 0 && prod ? w[i].category : CAT_OTHER);
      if (i >= 0 && prod && w[i].category == CAT_PARAMETER) param_sizes.insert(blocks[b].size);
    }
    // then the optimizer rule, against the trace's parameter sizes
    int64_t k = kept_off[t];
    for (int64_t b = block_off[t]; b < block_off[t + 1]; ++b) {
      const int64_t j = b - block_off[t];
      if (block_window) block_window[b] = (int32_t)link[j];
      if (link[j] < 0) continue;
      kept[k] = blocks[b];
      kept[k].category = role[j];
      if (product[j] && in_optimizer_step(blocks[b], w, nw) && param_sizes.count(blocks[b].size))
        kept[k].category = CAT_OPTIMIZER;
      ++k;
    }
    kept_off[t + 1] = k;
  }
  return 0;
}

// events: capacity 2 * block_off[T]; event_off: T + 1.  0, or -2 for bad offsets.
int xmem_oracle_orchestrate(const Block* blocks, const int64_t* block_off, int64_t T, const int64_t* steps,
                            const int64_t* step_off, const int64_t* zg, const int64_t* zg_off, uint64_t* events,
                            int64_t* event_off) {
  if (!offsets_ok(block_off, T) || !offsets_ok(step_off, T) || !offsets_ok(zg_off, T)) return -2;
  event_off[0] = 0;
  for (int64_t t = 0; t < T; ++t) {
    std::vector<uint64_t> words;
    orchestrate_one(blocks + block_off[t], block_off[t + 1] - block_off[t], steps + step_off[t],
                    step_off[t + 1] - step_off[t], zg + zg_off[t], zg_off[t + 1] - zg_off[t], words);
    std::copy(words.begin(), words.end(), events + event_off[t]);
    event_off[t + 1] = event_off[t] + (int64_t)words.size();
  }
  return 0;
}

}  // extern "C"
