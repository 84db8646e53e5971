// Sanitizer driver for the CPU oracle and the trace generators -- TEST
// INFRASTRUCTURE.  Built with AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_sanitizers.py and run on the CPU: it generates traces of every
// workload configuration (short lengths), replays them through the oracle under
// several parameter sets and thread counts with the series, runs the OOM
// prediction, and runs the trace-preparation oracle on a synthetic profile with
// nested windows.  Any sanitizer report fails the run (-fno-sanitize-recover).
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

extern "C" {
int tg_trace(int config, int64_t trace_index, uint64_t seed, int64_t frag_pairs, uint64_t* out, int64_t n_events);
struct Params { uint32_t abi_version, flags; int64_t v[9]; };
struct Result { int64_t f[11]; int32_t status, pad; };
int xmem_oracle_replay_batch(const uint64_t*, const int64_t*, int64_t, const Params*, Result*, int64_t*, int);
int xmem_oracle_oom_predicted(const Result*, int64_t, int64_t, int32_t*);
struct Raw { int64_t ts; uint64_t addr; int64_t bytes; };
struct Block { int64_t size, t_alloc, t_free; int32_t category, pad; };
struct Window { int64_t start, end; int32_t parent, kind, category, pad; };
int xmem_oracle_lifecycles(const Raw*, const int32_t*, const int64_t*, int64_t, Block*, int64_t*, int64_t*);
int xmem_oracle_attribute(const Block*, const int64_t*, int64_t, const Window*, const int64_t*, Block*, int64_t*,
                          int32_t*);
int xmem_oracle_orchestrate(const Block*, const int64_t*, int64_t, const int64_t*, const int64_t*, const int64_t*,
                            const int64_t*, uint64_t*, int64_t*);
}

static Params paper(int64_t cap, int64_t split_large) {
  const int64_t MiB = int64_t(1) << 20;
  Params p;
  p.abi_version = 1;
  p.flags = 0;
  const int64_t v[9] = {512, MiB, 2 * MiB, 20 * MiB, 10 * MiB, 2 * MiB, 512, split_large, cap};
  std::memcpy(p.v, v, sizeof v);
  return p;
}

static int fail(const char* what) {
  std::fprintf(stderr, "driver: %s\n", what);
  return 1;
}

int main() {
  // every configuration, a few traces each, ragged lengths; one batch
  std::vector<uint64_t> ev;
  std::vector<int64_t> off{0};
  const int64_t lens[5] = {4096, 20000, 30001, 9999, 120000};
  for (int c = 1; c <= 5; ++c) {
    for (int64_t t = 0; t < (c == 5 ? 1 : 3); ++t) {
      std::vector<uint64_t> tr(lens[c - 1]);
      if (tg_trace(c, t, 0, c == 5 ? 2000 : -1, tr.data(), (int64_t)tr.size()) != 0) return fail("tg_trace");
      ev.insert(ev.end(), tr.begin(), tr.end());
      off.push_back((int64_t)ev.size());
    }
  }
  // malformed words: an oversized request, a free of a later event, a double free
  const uint64_t bad[] = {uint64_t(1) << 50, (uint64_t(1) << 63) | 5, 8, (uint64_t(1) << 63) | 2,
                          (uint64_t(1) << 63) | 2};
  ev.insert(ev.end(), bad, bad + 5);
  off.push_back((int64_t)ev.size());
  off.push_back((int64_t)ev.size());  // an empty trace
  const int64_t T = (int64_t)off.size() - 1;
  std::vector<Result> res(T);
  std::vector<int64_t> ser(ev.size());
  const int64_t MiB = int64_t(1) << 20;
  const Params ps[] = {paper(INT64_MAX, 512), paper(INT64_MAX, MiB + 1), paper(40 * MiB, 512), paper(3 * MiB, 512)};
  for (const Params& p : ps) {
    for (int th : {1, 4}) {
      if (xmem_oracle_replay_batch(ev.data(), off.data(), T, &p, res.data(), ser.data(), th) != 0)
        return fail("replay");
    }
    std::vector<int32_t> flags(T);
    if (xmem_oracle_oom_predicted(res.data(), T, 64 * MiB, flags.data()) != 0) return fail("oom");
  }
  // trace preparation: a synthetic profile (address reuse, nested windows, markers)
  std::vector<Raw> raw;
  std::vector<Window> win;
  int64_t ts = 0;
  for (int it = 0; it < 50; ++it) {
    win.push_back(Window{ts, ts + 100, -1, 0, it % 5 == 4 ? 4 : 0, 0});
    const int32_t comp = (int32_t)win.size() - 1;
    win.push_back(Window{ts + 1, ts + 90, comp, 1, it % 4, 0});
    for (int k = 0; k < 20; ++k) {
      raw.push_back(Raw{ts + 2 + k, 0x1000u + 64u * (uint64_t)(k % 7), 100 + (it * 7 + k) % 13});
      if (k % 3 == 0) raw.push_back(Raw{ts + 3 + k, 0x1000u + 64u * (uint64_t)(k % 7), -1});
    }
    ts += 120;
  }
  const int64_t roff[3] = {0, (int64_t)raw.size() / 2, (int64_t)raw.size()};
  const int64_t woff[3] = {0, (int64_t)win.size(), (int64_t)win.size()};
  std::vector<Block> blocks(raw.size()), kept(raw.size());
  std::vector<int64_t> boff(3), koff(3), unm(2);
  std::vector<int32_t> bw(raw.size());
  if (xmem_oracle_lifecycles(raw.data(), nullptr, roff, 2, blocks.data(), boff.data(), unm.data()) != 0)
    return fail("lifecycles");
  if (xmem_oracle_attribute(blocks.data(), boff.data(), 2, win.data(), woff, kept.data(), koff.data(), bw.data()) != 0)
    return fail("attribute");
  const int64_t steps[4] = {0, 500, 2000, 4000}, soff[3] = {0, 2, 4};
  const int64_t zg[2] = {700, 3000}, zoff[3] = {0, 1, 2};
  std::vector<uint64_t> words(2 * raw.size());
  std::vector<int64_t> eoff(3);
  if (xmem_oracle_orchestrate(kept.data(), koff.data(), 2, steps, soff, zg, zoff, words.data(), eoff.data()) != 0)
    return fail("orchestrate");
  std::printf("driver ok: %lld traces, %zu events, %lld attributed blocks, %lld words\n", (long long)T, ev.size(),
              (long long)koff[2], (long long)eoff[2]);
  return 0;
}
