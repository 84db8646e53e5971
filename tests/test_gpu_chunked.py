"""Parity of the chunked replay (unbounded capacity: each pool of a trace cut at clean
positions and its chunks replayed at once from a speculated start state, verified and
re-run) with the CPU oracle, bit-exact, for explicit chunk counts (flags bits [5:0]).

chunks=1 is the one-wavefront-per-pool serial replay; the counts above it cover one
speculative round, several rounds, the final in-one-piece completion, hand-overs to the
paged and 64-bit chain kernels from inside a chunk, stops inside a chunk, and traces with
no clean position at all."""
import numpy as np
import pytest

import oracle
import tracegen
from bf_traces import enumerate_traces, to_csr
from evw import A, F, KiB, MiB
from gpu_util import check, compare, gpu_replay
from spill_traces import batch, churn, fragment, spill_mix

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


def growing(n_iter: int, step_mib: int, steady_after: int | None = None, persistent: int = 3) -> np.ndarray:
    """A few never-freed blocks, then iterations that each allocate one large block (and a few
    temporaries) and free everything again.  The large block grows by step_mib every iteration
    (a new segment each time) until steady_after iterations, then keeps its size."""
    ev = [A(4 * KiB * (p + 1)) for p in range(persistent)]
    for i in range(n_iter):
        g = i if steady_after is None else min(i, steady_after)
        s0 = len(ev)
        ev.append(A((21 + step_mib * g) * MiB))
        ev += [A(100 * KiB), A(3 * MiB), A(700)]
        ev += [F(s0 + 2), F(s0 + 1), F(s0 + 3), F(s0)]
    return np.array(ev, dtype=np.uint64)


def fragmenting(n_iter: int, blocks: int = 400) -> np.ndarray:
    """Iterations that fill one small segment with 4 KiB blocks and free them; iteration i frees
    every other block of its first i*8 first, so the free-block count peaks higher and higher
    in later iterations while no segment is ever added."""
    ev = [A(64)]  # never freed
    for i in range(n_iter):
        s0 = len(ev)
        ev += [A(4 * KiB)] * blocks
        k = min(2 * (i * 4), blocks)
        order = list(range(0, k, 2)) + [j for j in range(blocks) if not (j < k and j % 2 == 0)]
        ev += [F(s0 + j) for j in order]
    return np.array(ev, dtype=np.uint64)


@pytest.mark.parametrize("chunks", [1, 2, 3, 8, 16, 32])
@pytest.mark.parametrize("cfg,nt,ne", [(2, 6, 20001), (3, 3, 40003), (4, 24, 9999)])
def test_chunk_counts(cfg, nt, ne, chunks):
    ev, off = tracegen.generate(cfg, nt, ne)
    check(ev, off, P, what=f"C{cfg} chunks={chunks}", chunks=chunks)


@pytest.mark.parametrize("chunks", [4, 16])
def test_chunked_pytorch_like_split(chunks):
    ev, off = tracegen.generate(3, 4, 30000)
    check(ev, off, PT, what=f"C3 pytorch-like chunks={chunks}", chunks=chunks)


@pytest.mark.parametrize("chunks", [4, 8, 32])
def test_rounds_and_completion(chunks):
    """Segments created in every chunk (the frontier moves one chunk per round and the rest is
    replayed in one piece), created in the first few chunks only (resolved by the speculative
    rounds), and free-count maxima reached only in late chunks."""
    traces = [growing(300, 2), growing(300, 2, steady_after=40), growing(300, 2, steady_after=120),
              fragmenting(60), growing(300, 2, steady_after=0, persistent=0)]
    ev, off = batch(traces)
    gres, ores = check(ev, off, P, what=f"rounds chunks={chunks}", chunks=chunks)
    assert int(ores["segments_created"][0]) > 300 and int(ores["max_free_blocks_small"][3]) > 100


@pytest.mark.parametrize("chunks", [8, 63])
def test_windowed_rounds(chunks):
    """A batch with a chain per 4 scheduler wavefronts or more (800 traces, 1,600 chains): a
    speculative round keeps at most 6 of its chunks queued or running, each finished chunk claims
    the round's next one, the chunks past where the walk will stop are given up, and the rounds
    open up once the queue runs short.  GPT shapes, plus traces that create segments in every
    chunk, in the first chunks only or after a while, and fragmenting ones (several rounds, and
    small-pool walks that stop at their second growing chunk)."""
    ev3, off3 = tracegen.generate(3, 640, 3000)
    kinds = [growing(60, 2), growing(60, 2, steady_after=8), growing(60, 2, steady_after=25), fragmenting(16)]
    traces = [ev3[off3[i]:off3[i + 1]] for i in range(640)] + [kinds[i % 4] for i in range(160)]
    ev, off = batch(traces)
    check(ev, off, P, what=f"windowed rounds chunks={chunks}", chunks=chunks)


def test_no_clean_position():
    """Every block stays live until the very end (strict LIFO): one chunk, whatever is asked."""
    n = 3000
    ev = [A(512 * (1 + (i % 7))) for i in range(n)] + [F(n - 1 - i) for i in range(n)]
    ev, off = batch([np.array(ev, dtype=np.uint64)])
    check(ev, off, P, what="no clean position", chunks=32)


def test_chunked_spill_to_paged_sets():
    """A chunk whose pool outgrows the LDS table hands its whole chain to the paged kernel."""
    traces = [churn(1, 60000, 3000, 512, 64 << 10), fragment(5, 12000, 20000), growing(200, 1)]
    ev, off = batch(traces)
    gres, ores = check(ev, off, P, what="chunked spill", chunks=8)
    assert int(ores["max_free_blocks_small"].max()) > 1024


def test_chunked_wide_fallback():
    GiB = 1 << 30
    big = [A(1 << 40), F(0), A(1 << 40), A(5)] + [A(MiB), F(4)] * 50
    ev3, off3 = tracegen.generate(3, 3, 9000)
    traces = [ev3[off3[t]:off3[t + 1]] for t in range(3)]
    traces.insert(1, np.array(big, dtype=np.uint64))
    traces.append(np.array([A(600 * GiB), F(0)] * 40 + [A(600 * GiB)] * 5, dtype=np.uint64))
    ev, off = batch(traces)
    check(ev, off, P, what="chunked wide", chunks=8)
    ev4, off4 = tracegen.generate(3, 3, 20000)
    check(ev4, off4, oracle.paper_params(round_bytes=1), what="chunked round 1 B", chunks=8)


def test_chunked_malformed_and_overflow():
    ev, off = tracegen.generate(3, 6, 20000)
    ev = ev.copy()
    seg = ev[off[1]:off[2]]
    frees = np.flatnonzero(seg >> np.uint64(63))
    seg[int(frees[len(frees) // 2])] = seg[int(frees[10])]  # double free midway
    seg = ev[off[3]:off[4]]
    allocs = np.flatnonzero((seg >> np.uint64(63)) == 0)
    seg[int(allocs[len(allocs) - 50])] = np.uint64((1 << 48) + 7)  # bad word near the end
    check(ev, off, P, what="chunked malformed", chunks=8)
    n = 8193
    ov = [A(1 << 48)] * n
    tr = [np.array(ov, dtype=np.uint64), growing(100, 2, steady_after=5)]
    ev2, off2 = batch(tr)
    gres, _ = check(ev2, off2, P, what="chunked overflow", chunks=8)
    assert int(gres["status"][0]) == 4


def test_chunked_empty_and_tiny_traces():
    traces = [np.zeros(0, np.uint64), np.array([A(5)], np.uint64), np.array([A(0), F(0)], np.uint64),
              np.array([A(MiB), F(0), A(MiB)], np.uint64), np.zeros(0, np.uint64), growing(50, 1)]
    ev, off = batch(traces)
    check(ev, off, P, what="chunked tiny", chunks=32)
    bf = enumerate_traces(3)
    ev2, off2 = to_csr(bf)
    check(ev2, off2, P, what="bruteforce chunked", traces=bf, chunks=4)


def test_chunk_counts_agree_bitwise():
    """Every chunk count gives the same bytes as the serial replay, series included."""
    ev, off = tracegen.generate(2, 4, 30000)
    base, sbase = gpu_replay(ev, off, P, chunks=1)
    for k in (2, 5, 8, 13, 32):
        r, s = gpu_replay(ev, off, P, chunks=k)
        assert r.tobytes() == base.tobytes() and (s == sbase).all(), k


@pytest.mark.parametrize("chunks", [2, 8, 63])
def test_chunked_paged_sets(chunks):
    """A pool past the LDS table in a batch of one or two traces: its chunks are replayed again
    on the paged sets, each from the packed key lists of the chunk before (the frontier)."""
    spill = churn(11, 90000, 8000, 512, 64 << 10, waves=3)
    for traces in ([spill], [fragment(12, 30000, 40000)], [growing(100, 1), spill]):
        ev, off = batch(traces)
        gres, ores = check(ev, off, P, what=f"chunked paged chunks={chunks}", chunks=chunks)
        assert int(max(ores["max_free_blocks_small"].max(), ores["max_free_blocks_large"].max())) > 1024


@pytest.mark.parametrize("chunks", [2, 8, 32, 63])
def test_paged_resume_after_spill(chunks):
    """A first chunk that outgrows the LDS table hands over to the paged sets at the event where
    it did, from the state it left there; temporaries freed within 150 events, at seeded points
    of the 64-event tile, reach the resumed run through both tiles' lane registers and the
    mailbox, in either pool.  One trace per batch, and two (chunks <= 32) with the few-trace
    rounds."""
    for seed in range(4):
        ev, off = batch([spill_mix(seed)])
        gres, ores = check(ev, off, P, what=f"resume seed={seed} chunks={chunks}", chunks=chunks)
        assert int(ores["max_free_blocks_small"][0]) > 768
    ev, off = batch([spill_mix(20, large=True)])
    gres, ores = check(ev, off, P, what=f"resume large pool chunks={chunks}", chunks=chunks)
    assert int(ores["max_free_blocks_large"][0]) > 768
    if chunks <= 32:
        ev, off = batch([spill_mix(10), spill_mix(11, large=True)])
        check(ev, off, P, what=f"resume two traces chunks={chunks}", chunks=chunks)


def test_one_long_trace_fine_grain():
    """A single trace of 2^20 events or more is cut into up to 127 chunks per pool (the automatic
    grain; the cut planner takes the second group of 64 cuts), replayed in the paged-set rounds:
    a GPT-style trace that stays on the LDS table, and a fragmented one that spills."""
    for cfg, fp in ((3, -1), (5, 3000)):
        ev, off = tracegen.generate(cfg, 1, 1 << 20, frag_pairs=fp)
        gres, ores = check(ev, off, P, what=f"C{cfg} 1 x 2^20, automatic grain")
        if cfg == 5:
            assert int(ores["max_free_blocks_small"][0]) > 768


def test_two_long_traces_paged_rounds():
    """Two traces of 2^20 events or more on average take the paged-set rounds at 63 chunks per
    pool (automatic grain) instead of the scheduler: one GPT-style trace that stays on the LDS
    table beside a fragmented one whose small pool spills and resumes on the paged sets."""
    ev3, off3 = tracegen.generate(3, 1, 1 << 20)
    ev5, off5 = tracegen.generate(5, 1, (1 << 20) + 4097, frag_pairs=3000)
    ev, off = batch([ev3, ev5])
    gres, ores = check(ev, off, P, what="two long traces, automatic grain")
    assert int(ores["max_free_blocks_small"][1]) > 768


def test_long_traces_spill_after_scheduler():
    """Three traces averaging 2^20 events or more run the chunk scheduler; the pool that outgrows
    the LDS table there is replayed by the paged-set rounds afterwards (not the serial paged
    kernel), beside two that finish under the scheduler."""
    ev3, off3 = tracegen.generate(3, 2, 1 << 20)
    ev5, off5 = tracegen.generate(5, 1, (1 << 20) + 4097, frag_pairs=3000)
    ev, off = batch([ev3[off3[0]:off3[1]], ev5, ev3[off3[1]:off3[2]]])
    gres, ores = check(ev, off, P, what="three long traces, a spill under the scheduler")
    assert int(ores["max_free_blocks_small"][1]) > 768


def spill_late(seed: int, n_iter: int, spill_at: int, blocks: int = 2600) -> np.ndarray:
    """Balanced iterations of small temporaries; from iteration spill_at on, each iteration first
    frees every other block of its 2600, so the small pool passes 1024 free blocks only in later
    chunks."""
    rng = np.random.default_rng(seed)
    ev = [A(64)]
    for i in range(n_iter):
        s0 = len(ev)
        sizes = rng.integers(1, 8, size=blocks) * 512
        ev += [A(int(x)) for x in sizes]
        order = list(range(blocks)) if i < spill_at else list(range(0, blocks, 2)) + list(range(1, blocks, 2))
        ev += [F(s0 + j) for j in order]
    return np.array(ev, dtype=np.uint64)


@pytest.mark.parametrize("chunks", [4, 16])
def test_chunked_spill_in_late_chunk(chunks):
    ev, off = batch([spill_late(13, 40, 25)])
    gres, ores = check(ev, off, P, what=f"late spill chunks={chunks}", chunks=chunks)
    assert int(ores["max_free_blocks_small"][0]) > 1024



def small_growth(n_iter: int, grow_at: tuple, frag_at: tuple = (), m: int = 40, size: int = 64 * KiB,
                 frag_m: int | None = None, gstep: int = 4) -> np.ndarray:
    """Small-pool iterations of m blocks of `size` plus g blocks of 512 KiB, all freed again; g grows
    by gstep at the iterations in grow_at (new 2 MiB segments in a middle chunk), and the
    iterations in frag_at allocate frag_m blocks of `size` and free every other one first
    (free-count maxima in later chunks, to be shifted by the new segments)."""
    ev = [A(64)]
    g = 0
    for i in range(n_iter):
        if i in grow_at:
            g += gstep
        s0 = len(ev)
        k = frag_m if (i in frag_at and frag_m) else m
        ev += [A(size)] * k + [A(512 * KiB)] * g
        order = list(range(0, k, 2)) + list(range(1, k, 2)) if i in frag_at else list(range(k))
        ev += [F(s0 + j) for j in order + list(range(k, k + g))]
    return np.array(ev, dtype=np.uint64)


def _concat(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Trace a followed by trace b, b's frees renumbered past a."""
    b = b.copy()
    fr = (b >> np.uint64(63)) == 1
    b[fr] = b[fr] + np.uint64(len(a))
    return np.concatenate([a, b])


@pytest.mark.parametrize("chunks", [8, 32, 63])
def test_paged_chunks_past_later_growers(chunks):
    """A small pool on the paged sets (its first chunk spills) whose later iterations grow twice:
    speculative chunks after the first growing one ran without its segments and created them
    again; they are certified with those segments standing for the delta's (no growth recorded,
    free-count maxima shifted by the delta segments not yet taken), and one growing further
    extends the delta.  Fragmenting iterations put free-count maxima inside such chunks."""
    for seed in (3, 4):
        tail = small_growth(60, grow_at=(10, 30), frag_at=(20, 31, 45), m=40, size=64 * KiB, frag_m=300,
                            gstep=4 + seed)
        ev, off = batch([_concat(spill_mix(seed, iters=0), tail)])
        gres, ores = check(ev, off, P, what=f"paged chunks past growers seed={seed} chunks={chunks}", chunks=chunks)
        assert int(ores["max_free_blocks_small"][0]) > 768


# 1 KiB blocks freed every other: the oracle's largest small-pool free count is 766 (766 - 2 on the
# chunk's speculative run, without the two new segments) -- certified within the 768-slot table;
# with 8 more blocks it is 769, so that chunk is not certified and its true run spills
FRAG_NEAR = 1528


@pytest.mark.parametrize("chunks", [4, 8, 32])
def test_small_pool_certification(chunks):
    """Small-pool chunks after one that created segments are certified instead of replayed again:
    the new segments join the next frontier's table, later maxima shift by their count, a later
    segment-creating chunk ends the certified run, and a chunk whose free count with the delta
    would pass the LDS table is not certified (the last trace: the true run spills)."""
    traces = [small_growth(120, (30,), frag_at=(60, 100)),
              small_growth(120, (10, 50, 90), frag_at=(20, 70, 110)),
              small_growth(60, (20,), frag_at=(40,), m=100, size=KiB, frag_m=FRAG_NEAR, gstep=8),
              growing(150, 2, steady_after=40),
              small_growth(60, (20,), frag_at=(40,), m=100, size=KiB, frag_m=FRAG_NEAR + 8, gstep=8)]
    ev, off = batch(traces)
    gres, ores = check(ev, off, P, what=f"small-pool certification chunks={chunks}", chunks=chunks)
    mf = ores["max_free_blocks_small"]
    assert int(mf[2]) <= 768 < int(mf[4]) and int(ores["segments_created"][1]) >= 5
    for t in range(2):  # a batch of one trace: the rounds of the few-traces kernels
        ev1, off1 = batch([traces[t]])
        check(ev1, off1, P, what=f"small-pool certification, one trace, chunks={chunks}", chunks=chunks)
