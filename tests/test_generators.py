"""The seeded workload generators (tracegen): exact event counts, the shapes the workloads
promise, and stable output per seed.  Format checks only: the generators hold no allocator
logic, and these tests use none beyond the oracle's status for validity and, for the long
fragmented trace, its free-block diagnostic."""
import hashlib

import numpy as np
import pytest

import oracle
import tracegen

FREE = np.uint64(1) << np.uint64(63)


def _frees(e):
    isf = (e & FREE) != 0
    return isf, (e & np.uint64(0xffffffff)).astype(np.int64)


@pytest.mark.parametrize("cfg,n,m", [(1, 1, 4096), (2, 3, 7001), (3, 3, 12345), (4, 5, 3000), (5, 1, 50000)])
def test_exact_event_counts_and_validity(cfg, n, m):
    ev, off = tracegen.generate(cfg, n, m)
    assert len(ev) == n * m and list(np.diff(off)) == [m] * n
    rc, res, _ = oracle.replay(ev, off, oracle.paper_params())
    assert rc == 0 and (res["status"] == 0).all()  # every free names an earlier, unfreed allocation


def test_default_shapes():
    assert [tracegen.default_shape(c) for c in range(1, 6)] == [
        (1, 4096), (256, 65536), (1024, 262144), (4096, 65536), (1, 16777216)]


def test_c1_balanced_and_strictly_lifo():
    ev, _ = tracegen.generate(1)
    isf, h = _frees(ev)
    assert isf.sum() == 2048
    stack = []
    for e in range(len(ev)):
        if isf[e]:
            assert stack and stack[-1] == h[e], f"event {e} does not free the most recent live block"
            stack.pop()
        else:
            stack.append(e)
    assert stack == []  # balanced
    sizes = ev[~isf]
    assert sizes.min() >= 1024 and sizes.max() <= 8 << 20 and (sizes % 4 == 0).all()


def test_c2_batch_sweep():
    """Trace t's input batch x is b x 3 x 224 x 224 fp32 and its labels b x 8 bytes, with
    b = 16 + floor(496 t / 255): 16 for the first trace, 512 for the last."""
    for t in (0, 1, 100, 254, 255):
        e = tracegen.generate(2, 1, 3000, first_trace=t)[0]
        b = 16 + (496 * t) // 255
        x = np.flatnonzero(e == np.uint64(b * 3 * 224 * 224 * 4))
        assert len(x) and e[x[0] + 1] == np.uint64(8 * b), t
    assert 16 + (496 * 0) // 255 == 16 and 16 + (496 * 255) // 255 == 512


@pytest.mark.parametrize("t", [0, 7, 143, 144, 4095])
def test_c4_jitter_bounds_and_shuffle_windows(t):
    m = 20000
    base = tracegen.trace_stage(4, t, m, 0)
    jit = tracegen.trace_stage(4, t, m, 1)
    fin = tracegen.trace_stage(4, t, m, 2)
    assert np.array_equal(fin, tracegen.generate(4, 1, m, first_trace=t)[0])
    isf_b, _ = _frees(base)
    # jitter: only the allocation sizes move, each by at most 10% (floor), then up to 4 B, at least 4
    assert np.array_equal(base[isf_b], jit[isf_b])
    s, s2 = base[~isf_b].astype(np.int64), jit[~isf_b].astype(np.int64)
    assert (s2 % 4 == 0).all() and (s2 >= 4).all()
    assert (s2 >= s - s // 10 - 1).all() and (s2 <= s + s // 10 + 4).all()
    assert (s2 != s).mean() > 0.9
    # shuffle: allocations stay; each maximal run of frees is permuted within chunks of 8 from its start
    isf_j, _ = _frees(jit)
    assert np.array_equal(isf_j, (fin & FREE) != 0)
    assert np.array_equal(jit[~isf_j], fin[~isf_j])
    moved = 0
    i = 0
    while i < m:
        if not isf_j[i]:
            i += 1
            continue
        j = i
        while j < m and isf_j[j]:
            j += 1
        for c in range(i, j, 8):
            a, b = jit[c:min(c + 8, j)], fin[c:min(c + 8, j)]
            assert sorted(a.tolist()) == sorted(b.tolist())
            moved += int((a != b).any())
        i = j
    assert moved > 0


def test_c5_fragmentation_band():
    """The long trace's fragmentation phase leaves between 60,000 and 65,536 free small blocks."""
    ev, off = tracegen.generate(5)
    rc, res, _ = oracle.replay(ev, off, oracle.paper_params())
    assert rc == 0 and res["status"][0] == 0
    assert 60000 <= int(res["max_free_blocks_small"][0]) <= 65536


def test_stable_per_seed():
    """The same seed gives the same bytes (regression pins), another seed other bytes."""
    want = {1: "0a74b1883bc6e54b6bc22f2bbd40101efb6e2d4b9dc90feea0990cfa33ed5a7c",
            2: "0fc9832a2c269056cde76f643f5f56f87f05ad411aba9ea5d2c042cbdb9aaa0d",
            3: "24eb7720918ef9490e960e04ddc0aa20480ad85a1b1771fd885895fd3776c197",
            4: "95f6dec8517dd9c04928c6fd125fc4a6ed155ae3b0bfead1ac6e0d2d4a1fb071",
            5: "8e2c4147b5dcdaaa5ccd97a62d8de5c03e43e381d2986be322a02baa6b48f213"}
    shapes = {1: (1, 4096), 2: (2, 5000), 3: (2, 5000), 4: (2, 5000), 5: (1, 20000)}
    for c, (n, m) in shapes.items():
        ev, _ = tracegen.generate(c, n, m)
        assert hashlib.sha256(ev.tobytes()).hexdigest() == want[c], c
        ev2, _ = tracegen.generate(c, n, m, seed=1)
        assert not np.array_equal(ev, ev2) or c == 1


def test_spill_mix_passes_the_table_early():
    """The resume traces pass 768 free blocks (the LDS table's slots) of their pool in their
    fragmentation phase, with every temporary freed and no free of a free."""
    import oracle
    from spill_traces import spill_mix, batch
    for seed in range(3):
        tr = spill_mix(seed)
        frees = tr[(tr >> np.uint64(63)) == 1] & np.uint64((1 << 63) - 1)
        assert len(np.unique(frees)) == len(frees)
        assert 2 * len(frees) == len(tr)  # every allocation freed exactly once
        ev, off = batch([tr])
        rc, res, _ = oracle.replay(ev, off, oracle.paper_params(), series=False)
        assert rc == 0 and int(res["status"][0]) == 0
        assert int(res["max_free_blocks_small"][0]) > 768
    ev, off = batch([spill_mix(20, large=True)])
    rc, res, _ = oracle.replay(ev, off, oracle.paper_params(), series=False)
    assert rc == 0 and int(res["status"][0]) == 0 and int(res["max_free_blocks_large"][0]) > 768
