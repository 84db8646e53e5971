"""Properties the oracle must satisfy on random valid traces (hypothesis).

* I1  reserved >= allocated after every event (blocks are disjoint inside live
      segments), so peak_reserved >= peak_allocated;
* I2  peak_allocated is the maximum prefix sum of the +r / -r deltas (its plain
      definition, computed here with numpy), first index on ties;
* I3  with the paper parameters every segment is a multiple of 2 MiB;
* I4  with unbounded capacity nothing is released: reserved never decreases and
      peak = final = the sum of created segments;
* I7  with unbounded capacity the two pools never interact: the reserved series
      is the sum of the series of the SMALL-only and LARGE-only sub-traces;
* I8  a balanced trace ends with allocated 0 and reserved unchanged;
* I9  determinism: 1 thread and 8 threads give identical bytes;
* capacity: a cap equal to the unbounded peak changes nothing; a smaller cap
  either releases segments or stops with OOM;
* scaling: doubling every size and every size parameter doubles every byte count.
"""
import numpy as np
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
from evw import A, F, MiB

P = oracle.paper_params()
FREE_BIT = 1 << 63


@st.composite
def traces(draw, max_len=120, balanced=None):
    n_alloc = draw(st.integers(1, max_len // 2))
    lifo = draw(st.booleans())
    sizes = draw(st.lists(st.one_of(
        st.integers(0, 4096), st.integers(4096, 2 * MiB), st.integers(2 * MiB, 64 * MiB),
        st.sampled_from([MiB, MiB + 1, 10 * MiB, 10 * MiB - 512, 512])), min_size=n_alloc, max_size=n_alloc))
    rnd = np.random.default_rng(draw(st.integers(0, 2**32 - 1)))
    bal = draw(st.booleans()) if balanced is None else balanced
    ev, live, k = [], [], 0
    while k < n_alloc or (bal and live):
        if k < n_alloc and (not live or rnd.random() < 0.55):
            live.append(len(ev))
            ev.append(A(sizes[k]))
            k += 1
        else:
            i = len(live) - 1 if lifo else int(rnd.integers(len(live)))
            ev.append(F(live.pop(i)))
    return ev


def rounded(ev, g=512):
    """Rounded request of each alloc (0 for frees): a plain formula, not the oracle."""
    out = np.zeros(len(ev), dtype=np.int64)
    for i, w in enumerate(ev):
        if not w & FREE_BIT:
            out[i] = -(-w // g) * g
    return out


def deltas(ev, g=512):
    r = rounded(ev, g)
    d = r.copy()
    for i, w in enumerate(ev):
        if w & FREE_BIT:
            d[i] = -r[w & 0xFFFFFFFF]
    return d


def run(ev, params=P, threads=1):
    e = np.array(ev, dtype=np.uint64)
    rc, out, ser = oracle.replay(e, np.array([0, len(e)], np.int64), params, series=True, threads=threads)
    assert rc == 0
    return out[0], ser


SET = settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@SET
@given(traces())
def test_i1_i2_i3_i4(ev):
    res, ser = run(ev)
    alloc_series = np.cumsum(deltas(ev))
    assert res["status"] == 0
    assert (ser >= alloc_series).all()                                  # I1
    peak = alloc_series.max(initial=0)
    assert res["peak_allocated"] == peak                                # I2
    assert res["peak_allocated_event"] == (int(np.argmax(alloc_series)) if peak > 0 else -1)
    assert res["final_allocated"] == alloc_series[-1]
    assert (ser % (2 * MiB) == 0).all()                                 # I3
    assert (np.diff(ser) >= 0).all()                                    # I4
    assert res["peak_reserved"] == res["final_reserved"] == ser[-1]
    assert res["segments_released"] == 0
    assert res["peak_reserved_event"] == (int(np.argmax(ser)) if ser[-1] > 0 else -1)


def sub_trace(ev, keep):
    """Events of one pool only, with handles renumbered."""
    new_index, out = {}, []
    for i, w in enumerate(ev):
        if not keep[i]:
            continue
        if w & FREE_BIT:
            out.append(F(new_index[w & 0xFFFFFFFF]))
        else:
            new_index[i] = len(out)
            out.append(w)
    return out


@SET
@given(traces(), st.sampled_from([oracle.paper_params(), oracle.pytorch_like_params()]))
def test_i7_pool_independence(ev, params):
    r = rounded(ev)
    pool = np.zeros(len(ev), dtype=np.int64)  # 0 none, 1 small, 2 large
    for i, w in enumerate(ev):
        src = (w & 0xFFFFFFFF) if w & FREE_BIT else i
        pool[i] = 0 if r[src] == 0 else (1 if r[src] <= MiB else 2)
    _, full = run(ev, params)
    total = np.zeros(len(ev), dtype=np.int64)
    for p in (1, 2):
        keep = pool == p
        if not keep.any():
            continue
        _, part = run(sub_trace(ev, keep), params)
        # expand the sub-series back to the full event axis (step function)
        idx = np.flatnonzero(keep)
        expanded = np.zeros(len(ev), dtype=np.int64)
        expanded[idx] = part
        expanded = np.maximum.accumulate(expanded)
        total += expanded
    assert (full == total).all()


@SET
@given(traces(balanced=True))
def test_i8_balanced_end(ev):
    res, ser = run(ev)
    assert res["final_allocated"] == 0
    assert res["final_reserved"] == res["peak_reserved"]


@settings(max_examples=20, deadline=None)
@given(st.lists(traces(max_len=200), min_size=1, max_size=40))
def test_i9_determinism_threads(trs):
    off = np.zeros(len(trs) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in trs])
    ev = np.array([w for t in trs for w in t], dtype=np.uint64)
    a = oracle.replay(ev, off, P, series=True, threads=1)
    b = oracle.replay(ev, off, P, series=True, threads=8)
    assert a[1].tobytes() == b[1].tobytes() and (a[2] == b[2]).all()


@SET
@given(traces(), st.floats(0.05, 1.0))
def test_capacity(ev, frac):
    res, ser = run(ev)
    peak = int(res["peak_reserved"])
    if peak == 0:
        return
    same, sser = run(ev, oracle.paper_params(device_capacity_bytes=peak))
    assert same.tobytes() == res.tobytes() and (sser == ser).all()
    cap = max(1, int(peak * frac) - 1)
    low, lser = run(ev, oracle.paper_params(device_capacity_bytes=cap))
    assert (lser[lser >= 0] <= cap).all()
    assert low["status"] == 1 or low["segments_released"] > 0 or low["peak_reserved"] <= cap
    if low["status"] == 1:
        e = int(low["stop_event"])
        assert (lser[e:] == -1).all() and (lser[:e] >= 0).all()


@SET
@given(traces())
def test_scaling(ev):
    res, ser = run(ev)
    ev2 = [w if w & FREE_BIT else 2 * w for w in ev]
    p2 = {k: (2 * v if k != "device_capacity_bytes" else v) for k, v in P.items()}
    res2, ser2 = run(ev2, p2)
    assert (ser2 == 2 * ser).all()
    for k in ("peak_allocated", "peak_reserved", "final_allocated", "final_reserved"):
        assert res2[k] == 2 * res[k]
    for k in ("peak_allocated_event", "peak_reserved_event", "segments_created",
              "max_free_blocks_small", "max_free_blocks_large"):
        assert res2[k] == res[k]
