"""Parity of the HIP path (through the C ABI) with the CPU oracle: every result
field and every entry of the per-event reserved series must be identical
(integer work: bit-exact).

Sizes: the reduced cases span several 2048-event stream tiles and 64-event
replay tiles with ragged tails; the full-size cases are the five workload
configurations at their full shapes, in the launch configuration the benchmark
times (xmem_replay_batch_ex on the torch stream)."""
import numpy as np
import pytest

import oracle
import tracegen
from bf_traces import enumerate_traces, to_csr
from evw import A, F, MiB
from gpu_util import check, compare, compare_series, gpu_replay, log
from pin_traces import catalogue
from spill_traces import batch, churn, fragment

pytestmark = pytest.mark.gpu

P = oracle.paper_params()
PT = oracle.pytorch_like_params()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2510_21048_amd as xm
    xm.load()
    yield


def test_pin_catalogue():
    cat = catalogue()
    groups = {}
    for name, tr, p in cat:
        groups.setdefault(tuple(sorted(p.items())), []).append((name, tr))
    for key, items in groups.items():
        traces = [tr for _, tr in items]
        ev, off = to_csr(traces)
        check(ev, off, dict(key), what="pins " + ",".join(n for n, _ in items), traces=traces)


@pytest.mark.parametrize("pname,pdict", [
    ("paper", P), ("pytorch_like", PT),
    ("cap20", oracle.paper_params(device_capacity_bytes=20 * MiB)),
    ("cap14", oracle.paper_params(device_capacity_bytes=14 * MiB)),
    ("cap4", oracle.paper_params(device_capacity_bytes=4 * MiB)),
])
def test_bruteforce_batch(pname, pdict):
    """Every <=3-block trace over the boundary alphabet, as one batch."""
    traces = enumerate_traces(3)
    ev, off = to_csr(traces)
    check(ev, off, pdict, what=f"bruteforce[{pname}]", traces=traces)


REDUCED = {  # config: (traces, events per trace, frag pairs)
    1: (1, 4096, -1),
    2: (6, 20001, -1),
    3: (5, 40003, -1),
    4: (40, 9999, -1),
    5: (1, 400000, 3000),
}


@pytest.mark.parametrize("cfg", sorted(REDUCED))
def test_configs_reduced(cfg):
    nt, ne, fp = REDUCED[cfg]
    ev, off = tracegen.generate(cfg, nt, ne, frag_pairs=fp)
    gres, ores = check(ev, off, P, what=f"C{cfg} reduced")
    if cfg == 5:
        assert ores["max_free_blocks_small"][0] > 2000  # the LDS table spills to HBM


def test_ragged_batch_with_empty_traces():
    ev3, off3 = tracegen.generate(3, 12, 30000)
    rng = np.random.default_rng(7)
    traces = []
    for t in range(12):
        k = int(rng.integers(0, 30000))
        traces.append(ev3[off3[t]:off3[t] + k])
        if t % 3 == 0:
            traces.append(ev3[:0])
    off = np.zeros(len(traces) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in traces])
    ev = np.concatenate(traces).astype(np.uint64)
    check(ev, off, P, what="ragged")


PARAM_VARIANTS = {
    "round1": oracle.paper_params(round_bytes=1),
    "round4096": oracle.paper_params(round_bytes=4096),
    "small256k": oracle.paper_params(small_max_bytes=256 << 10, small_segment_bytes=1 << 20),
    "mid8": oracle.paper_params(mid_segment_bytes=8 << 20, min_large_alloc_bytes=4 << 20, large_round_bytes=1 << 20),
    # a large-segment granule that is not a power of two of the rounding granule (the kernels divide)
    "large3m": oracle.paper_params(large_round_bytes=3 << 20),
    "split64k": oracle.paper_params(split_min_small_bytes=64 << 10, split_min_large_bytes=(4 << 20) + 1),
    "pytorch_like": PT,
}


@pytest.mark.parametrize("name", sorted(PARAM_VARIANTS))
def test_param_variants(name):
    ev, off = tracegen.generate(4, 24, 12000)
    check(ev, off, PARAM_VARIANTS[name], what=f"params[{name}]")


@pytest.mark.parametrize("cfg,frac", [(2, 0.6), (3, 0.5), (4, 0.8)])
def test_capacity_reclaim_and_oom(cfg, frac):
    """A finite capacity: one chain per trace, reclaim and OOM both happen."""
    nt, ne = {2: (8, 20000), 3: (6, 30000), 4: (32, 8000)}[cfg]
    ev, off = tracegen.generate(cfg, nt, ne)
    _, free_res, _ = oracle.replay(ev, off, P, threads=16)
    cap = int(np.median(free_res["peak_reserved"]) * frac)
    gres, ores = check(ev, off, oracle.paper_params(device_capacity_bytes=cap), what=f"C{cfg} cap={cap}")
    assert (ores["status"] == 1).any() or (ores["segments_released"] > 0).any()


def test_malformed_traces_are_isolated():
    """A bad event stops only its own trace; neighbours are unaffected."""
    ev, off = tracegen.generate(3, 8, 20000)
    ev = ev.copy()
    bad_at = {}
    # trace 1: double free of an earlier freed allocation
    t = 1
    seg = ev[off[t]:off[t + 1]]
    frees = np.flatnonzero(seg >> np.uint64(63))
    e = int(frees[len(frees) // 2])
    victim_free = int(frees[10])
    seg[e] = seg[victim_free]
    bad_at[t] = (e, 2)
    # trace 3: undecodable size
    seg = ev[off[3]:off[4]]
    allocs = np.flatnonzero((seg >> np.uint64(63)) == 0)
    seg[int(allocs[5000])] = np.uint64((1 << 48) + 7)
    bad_at[3] = (int(allocs[5000]), 3)
    # trace 5: free bits set
    seg = ev[off[5]:off[6]]
    frees = np.flatnonzero(seg >> np.uint64(63))
    seg[int(frees[3000])] |= np.uint64(1 << 45)
    bad_at[5] = (int(frees[3000]), 3)
    gres, ores = check(ev, off, P, what="malformed")
    for t, (e, st) in bad_at.items():
        assert int(ores["stop_event"][t]) <= e and int(ores["status"][t]) != 0


@pytest.mark.parametrize("n_events", [4096, 1000])
def test_malformed_event_after_a_repeated_free_in_one_thread(n_events):
    """One stream thread holds 8 consecutive events.  Allocation X (event 2) is freed at event 13
    and again at event 96; event 14, a free word with bits set above the index, is malformed.
    Event 96's thread links its free in the same wavefront before event 13's thread does, so the
    thread of events 8-15 first learns of a stop at 96 (the second free of X), and only then reaches
    its own malformed event 14.  The trace must stop at event 14 as in the oracle: the earliest
    malformed event counts, whatever was found before it.  4096 events: whole tiles; 1000: one
    partial tile."""
    free_bit = np.uint64(1) << np.uint64(63)
    ev = np.full(n_events, 1024, np.uint64)  # allocations that stay live
    ev[2] = 4096
    ev[13] = free_bit | np.uint64(2)
    ev[14] = free_bit | (np.uint64(1) << np.uint64(45))
    ev[96] = free_bit | np.uint64(2)
    off = np.array([0, n_events], np.int64)
    gres, ores = check(ev, off, P, what=f"malformed after a repeated free, {n_events} events")
    assert int(ores["stop_event"][0]) == 14 and int(ores["status"][0]) == 3


def test_repeated_frees_of_one_allocation():
    """Several frees naming one allocation, in one stream tile and across tiles, in either order
    relative to the true free: the first free stands and the trace stops at the second, exactly as
    in the oracle (the links are stored plainly, then checked and repaired with atomics)."""
    rng = np.random.default_rng(7)
    ev, off = tracegen.generate(3, 8, 20000)
    ev = ev.copy()
    free_bit = np.uint64(1) << np.uint64(63)

    def frees_of(t):
        seg = ev[off[t]:off[t + 1]]
        fr = np.flatnonzero(seg >> np.uint64(63))
        return seg, fr, (seg[fr] & np.uint64(0xffffffff)).astype(np.int64)

    # trace 0: two extra frees of one allocation, several stream tiles after its true free
    seg, fr, h = frees_of(0)
    i = len(fr) // 4
    for k in (fr[i] + 5000, fr[i] + 9000):
        j = fr[np.searchsorted(fr, k)]
        seg[j] = free_bit | np.uint64(h[i])
    # trace 2: three frees of one allocation inside one tile (the true one and the next two frees)
    seg, fr, h = frees_of(2)
    i = len(fr) // 3
    seg[fr[i + 1]] = free_bit | np.uint64(h[i])
    seg[fr[i + 2]] = free_bit | np.uint64(h[i])
    # trace 4: an extra free before the true one (the true free becomes the second)
    seg, fr, h = frees_of(4)
    i = len(fr) // 2
    j = int(np.searchsorted(fr, h[i] + 1))  # the first free after the allocation
    if fr[j] != fr[i]:
        seg[fr[j]] = free_bit | np.uint64(h[i])
    # trace 6: many random frees redirected to earlier allocations
    seg, fr, h = frees_of(6)
    for j in rng.choice(len(fr), 40, replace=False):
        seg[fr[j]] = free_bit | np.uint64(h[rng.integers(0, j + 1)])  # freed by a free at or before j
    gres, ores = check(ev, off, P, what="repeated frees")
    for t in (0, 2, 4, 6):
        assert int(ores["status"][t]) == 2, (t, int(ores["status"][t]))
    for t in (1, 3, 5, 7):
        assert int(ores["status"][t]) == 0


def test_pool_overflow_gpu():
    n = 8193
    ev = np.array([A(1 << 48)] * n, dtype=np.uint64)
    off = np.array([0, n], np.int64)
    gres, ores = check(ev, off, P, what="overflow")
    assert int(gres["status"][0]) == 4 and int(gres["stop_event"][0]) == n - 1


def test_determinism():
    ev, off = tracegen.generate(4, 64, 8192)
    a, sa = gpu_replay(ev, off, P)
    b, sb = gpu_replay(ev, off, P)
    assert a.tobytes() == b.tobytes() and (sa == sb).all()


def test_bad_offsets_reported_on_device():
    import torch
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding
    dev = torch.device("cuda:0")
    ev = torch.zeros(10, dtype=torch.int64, device=dev)
    off = torch.tensor([0, 6, 4, 10], dtype=torch.int64, device=dev)  # decreasing
    out, _ = binding.replay(ev, off, xm.params())
    r = binding.to_numpy(out)
    assert (r["status"] == 5).all() and (r["stop_event"] == 0).all()
    # the synchronous form checks on the host
    res = torch.empty((3, 96), dtype=torch.uint8, device=dev)
    assert xm.xmem_replay_batch(ev, off, 3, xm.params(), res) == -2


def test_sync_entry_point():
    import torch
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding
    ev, off = tracegen.generate(2, 4, 10000)
    dev = torch.device("cuda:0")
    e = torch.from_numpy(ev.view(np.int64)).to(dev)
    o = torch.from_numpy(off).to(dev)
    res = torch.empty((4, 96), dtype=torch.uint8, device=dev)
    assert xm.xmem_replay_batch(e, o, 4, xm.params(), res) == 0
    _, ores, _ = oracle.replay(ev, off, P)
    compare(binding.to_numpy(res), ores, what="sync")


# ---------------------------------------------------------------- full sizes
_FULL = {}


def _full(cfg):
    """The full-size batch of a workload configuration, generated once per test session."""
    if cfg not in _FULL:
        _FULL[cfg] = tracegen.generate(cfg, *tracegen.default_shape(cfg))
    return _FULL[cfg]


def _check_full(cfg, pdict, what):
    """GPU against oracle on a full-size batch: every result field of every trace and the whole
    per-event reserved series (every event of every trace)."""
    ev, off = _full(cfg)
    log(f"[gpu-parity] {what}: {len(off) - 1} x {len(ev) // (len(off) - 1)}")
    gres, gser = gpu_replay(ev, off, pdict, series=True)
    rc, ores, oser = oracle.replay(ev, off, pdict, series=True, threads=16)
    assert rc == 0
    compare(gres, ores, what=what)
    compare_series(gser, oser, off, what=what)
    return ores


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_full_size_configs(cfg):
    ores = _check_full(cfg, P, f"C{cfg} full")
    assert (ores["status"] == 0).all()


@pytest.mark.parametrize("cfg,frac", [(2, 0.9), (3, 0.8), (4, 0.8)])
def test_full_size_capacity(cfg, frac):
    """Full-size batches under a device capacity below many traces' unbounded peaks: one chain
    per trace (the pools interact), idle segments released (Section 3.4 (v)) and OOM stops."""
    ev, off = _full(cfg)
    rc, free_res, _ = oracle.replay(ev, off, P, threads=16)
    assert rc == 0
    cap = int(np.median(free_res["peak_reserved"]) * frac)
    ores = _check_full(cfg, oracle.paper_params(device_capacity_bytes=cap), f"C{cfg} full, capacity {cap}")
    assert (ores["status"] == 1).any() and (ores["status"] == 0).any()
    assert (ores["segments_released"] > 0).any()


def test_full_size_c3_pytorch_like():
    """Full GPT-style batch under the split preset that keeps large remainders below 1 MiB + 1
    inside the allocated block."""
    _check_full(3, PT, "C3 full, PYTORCH_LIKE")


def test_oom_predicted():
    """Eq. (1) of Section 4.1 over GPU replay results, against the oracle's predicate over the
    oracle's results: thresholds at, just below and just above every trace's estimated peak,
    0 and a huge one; the batch holds OOM stops, a malformed trace and an empty one."""
    import torch
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding
    ev3, off3 = tracegen.generate(3, 6, 30000)
    traces = [ev3[off3[t]:off3[t + 1]] for t in range(6)]
    traces += [np.array([A(1 << 49)], np.uint64), np.zeros(0, np.uint64), np.array([A(10_000_000)], np.uint64)]
    off = np.zeros(len(traces) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in traces])
    ev = np.concatenate(traces)
    _, free_res, _ = oracle.replay(ev, off, P, threads=16)
    cap = int(np.median(free_res["peak_reserved"][:6]))
    pd = oracle.paper_params(device_capacity_bytes=cap)
    gres_t = binding.replay(torch.from_numpy(ev.view(np.int64)).cuda(), torch.from_numpy(off).cuda(),
                            xm.params(**pd))[0]
    rc, ores, _ = oracle.replay(ev, off, pd, threads=16)
    assert rc == 0
    compare(binding.to_numpy(gres_t), ores, what="OOM predicate batch")
    assert set(ores["status"].tolist()) >= {0, 1, 3}
    peaks = sorted(set(int(x) for x in ores["peak_reserved"]))
    for m_max in [0, 1 << 62, cap] + [p + d for p in peaks for d in (-1, 0, 1) if p + d >= 0]:
        got = xm.oom_predicted(gres_t, m_max).cpu().numpy()
        rc, want = oracle.oom_predicted(ores, m_max)
        assert rc == 0 and np.array_equal(got, want), (m_max, got, want)
    assert xm.oom_predicted(gres_t[:0], 5).numel() == 0


def test_c5_full_fragmentation_prefix():
    """The long GPT trace through its whole fragmentation phase (~62K simultaneously free
    small blocks, the table spilled to HBM) and ~330K events after it."""
    ev, off = tracegen.generate(5, 1, 600000)
    gres, ores = check(ev, off, P, what="C5 600K-event prefix")
    assert int(ores["max_free_blocks_small"][0]) >= 60000


def test_full_size_c5():
    """One 16,777,216-event trace with ~62K simultaneously free small blocks: its small pool is
    replayed on the paged sets."""
    ev, off = tracegen.generate(5)
    log("[gpu-parity] C5 full: 1 x 16777216")
    gres, gser = gpu_replay(ev, off, P, series=True)
    rc, ores, oser = oracle.replay(ev, off, P, series=True)
    assert rc == 0
    compare(gres, ores, what="C5 full")
    compare_series(gser, oser, off, what="C5 full")
    assert 60000 <= int(ores["max_free_blocks_small"][0]) <= 65536


def test_wide_fallback_chains():
    """Chains whose sizes or addresses pass 2^31 granules are replayed again with 64-bit
    fields; mixed with ordinary chains in one batch."""
    GiB = 1 << 30
    big = [
        [A(1 << 40), F(0), A(1 << 40), A(5)],                         # a request of 2^31 granules
        [A(400 * GiB), A(400 * GiB), F(0), A(300 * GiB), A(200 * GiB), F(1), A(100)],  # > 2^31 granules of segments
        [A(MiB)] * 3 + [A(600 * GiB), F(3), A(600 * GiB), A(600 * GiB), A(1 << 20)],
    ]
    ev3, off3 = tracegen.generate(3, 4, 9000)
    traces = [list(ev3[off3[t]:off3[t + 1]]) for t in range(4)]
    traces = [traces[0], big[0], traces[1], big[1], big[2], traces[2], traces[3]]
    ev, off = to_csr(traces)
    check(ev, off, P, what="wide fallback")
    check(ev, off, oracle.paper_params(device_capacity_bytes=1900 * GiB), what="wide fallback, capacity")
    # granule of one byte: every GPT chain's addresses pass 2^31 units
    ev4, off4 = tracegen.generate(3, 6, 20000)
    check(ev4, off4, oracle.paper_params(round_bytes=1), what="round 1 B")


# ---------------------------------------------------------------- paged free-block sets
def _spill_traces():
    return [churn(1, 150000, 12000, 512, 64 << 10), churn(2, 150000, 6000, 512, 512 << 10, waves=3),
            churn(3, 120000, 5000, (1 << 20) + 1, 8 << 20), churn(4, 60000, 3000, 512, 2 << 20, waves=1),
            fragment(5, 30000, 40000), fragment(6, 9000, 20000, (1 << 20) + 1, 4 << 20)]


def test_paged_sets():
    """Pools with more free blocks than the LDS table holds are replayed with the paged sets:
    pages split, merge, even out and empty as the free set rises and falls (up to ~15K free
    blocks, several summary rows of the directory), in both pools."""
    ev, off = batch(_spill_traces())
    gres, ores = check(ev, off, P, what="paged sets")
    big = (ores["max_free_blocks_small"] > 1024) | (ores["max_free_blocks_large"] > 1024)
    assert big.sum() >= 5 and ores["max_free_blocks_small"].max() > 10000


@pytest.mark.parametrize("frac", [0.6, 0.9])
def test_paged_sets_capacity(frac):
    """The same traces under a capacity below each one's unbounded peak: one chain per trace
    (both pools) on the paged sets, stopping with OOM."""
    for k, tr in enumerate(_spill_traces()):
        ev, off = batch([tr])
        _, free_res, _ = oracle.replay(ev, off, P)
        cap = int(int(free_res["peak_reserved"][0]) * frac)
        check(ev, off, oracle.paper_params(device_capacity_bytes=cap), what=f"paged trace {k} cap={cap}")


def test_paged_sets_reclaim():
    """~15K free small blocks coalesce back into idle segments; then mid-size allocations need
    new large-pool segments past the capacity, so the paged chain releases the idle small
    segments (Section 3.4 (v)) and finally stops with OOM."""
    fr = fragment(7, 30000, 20000)
    ev0, off0 = batch([fr])
    _, r0, _ = oracle.replay(ev0, off0, P)
    cap = int(r0["final_reserved"][0]) + (500 << 20)
    ev, off = batch([np.concatenate([fr, np.full(120, 8 << 20, dtype=np.uint64)])])
    gres, ores = check(ev, off, oracle.paper_params(device_capacity_bytes=cap), what=f"paged reclaim cap={cap}")
    assert int(ores["segments_released"][0]) > 100 and int(ores["status"][0]) == 1
