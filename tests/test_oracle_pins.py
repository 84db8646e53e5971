"""Pins of the CPU oracle: values the paper states, hand-derived worked examples
and edge cases, each checked on the C++ oracle AND on the brute-force model.

Every expected number below is derived by hand from the rules of Section 3.4
(round up, segment, best fit with coalescing, caching, OOM after reclaim); the
derivation is in the comment next to it.  A mistake in the oracle such as
first fit instead of best fit, highest-address ties, no coalescing, splitting
the wrong side, or reclaiming before the check fails at least one of them.
"""
import json
import os

import numpy as np
import pytest

import oracle
from bf_model import run as bf_run
from evw import A, F, KiB, MiB

pytestmark = pytest.mark.filterwarnings("ignore")
HERE = os.path.dirname(os.path.abspath(__file__))
P = oracle.paper_params()
PT = oracle.pytorch_like_params()
OK, OOM, BAD_FREE, BAD_EVENT, OVERFLOW = 0, 1, 2, 3, 4


def both(trace, params=P):
    """Run oracle and brute force, assert they agree everywhere, return (result, series)."""
    res, ser = oracle.replay_one(trace, params)
    bres, bser = bf_run(trace, params)
    for k, v in bres.items():
        assert int(res[k]) == v, (k, int(res[k]), v)
    assert [int(x) for x in ser] == bser
    return {k: int(res[k]) for k in oracle.RESULT_FIELDS}, [int(x) for x in ser]


def test_paper_examples_golden():
    with open(os.path.join(HERE, "golden", "paper_examples.json")) as f:
        ex = {e["id"]: e for e in json.load(f)["examples"]}
    for s, r in zip(ex["round_up_512"]["trace_bytes"], ex["round_up_512"]["expected_rounded"]):
        res, _ = both([A(s)])
        assert res["peak_allocated"] == r and res["final_allocated"] == r
    for k in ("segment_2mb_for_1mb", "segment_2mb_for_1mib", "segment_20mb_for_10mb"):
        res, ser = both([A(b) for b in ex[k]["trace_bytes"]])
        assert res["peak_reserved"] == ex[k]["expected_reserved"], k
        assert res["peak_allocated"] == ex[k]["expected_allocated"], k
        assert ser == [ex[k]["expected_reserved"]]


def test_w2_min_large_boundary():
    # r = 10 MiB is not < min_large (10 MiB): segment = ceil(r / 2 MiB) * 2 MiB = 10 MiB
    res, _ = both([A(10 * MiB)])
    assert res["peak_reserved"] == 10 * MiB
    # one granule below: r = 10 MiB - 512 < 10 MiB -> 20 MiB segment
    res, _ = both([A(10 * MiB - 512)])
    assert res["peak_reserved"] == 20 * MiB


def test_w3_pool_boundary_and_noop():
    res, _ = both([A(MiB)])          # r = 1 MiB <= small_max -> SMALL, 2 MiB segment
    assert res["peak_reserved"] == 2 * MiB and res["max_free_blocks_small"] == 1
    res, _ = both([A(MiB + 1)])      # r = 1 MiB + 512 -> LARGE, < 10 MiB -> 20 MiB
    assert res["peak_reserved"] == 20 * MiB and res["max_free_blocks_large"] == 1
    res, ser = both([A(0), F(0)])    # no-op allocation and its free
    assert res == dict(res, peak_allocated=0, peak_reserved=0, peak_allocated_event=-1,
                       peak_reserved_event=-1, status=OK, stop_event=-1, segments_created=0)
    assert ser == [0, 0]


def test_w4_coalesce():
    # four 512 KiB blocks fill one 2 MiB segment; freeing e1 and e2 merges them into
    # one 1 MiB hole that the 1 MiB request fits exactly (no coalescing -> 4 MiB)
    t = [A(512 * KiB)] * 4 + [F(1), F(2), A(MiB)]
    res, ser = both(t)
    assert ser == [2 * MiB] * 7
    assert res["peak_allocated"] == 2 * MiB and res["peak_allocated_event"] == 3
    assert res["segments_created"] == 1 and res["final_allocated"] == 2 * MiB


def test_w5_best_fit_not_first_fit():
    # holes: 768K@0 and 512K@1M; A512K takes the exact 512K hole (first fit would
    # split the 768K hole and A768K would then need a second segment)
    t = [A(768 * KiB), A(256 * KiB), A(512 * KiB), A(512 * KiB), F(0), F(2), A(512 * KiB), A(768 * KiB)]
    res, ser = both(t)
    assert ser == [2 * MiB] * 8
    assert res["peak_allocated"] == 2 * MiB and res["peak_allocated_event"] == 3


def test_w6_tie_lowest_address():
    # eight 256K blocks; holes 256K@0 and 256K@1M; the tie goes to @0, so freeing e5
    # merges with the hole @1M into 512K, which A512K fits (highest-address ties -> 4 MiB)
    t = [A(256 * KiB)] * 8 + [F(0), F(4), A(256 * KiB), F(5), A(512 * KiB)]
    res, ser = both(t)
    assert ser == [2 * MiB] * 13
    assert res["peak_allocated"] == 2 * MiB and res["peak_allocated_event"] == 7


def test_w7_large_reuse_split():
    # 11 MiB -> 12 MiB segment; after the free it is one 12 MiB hole that 3 MiB splits
    res, ser = both([A(11 * MiB), F(0), A(3 * MiB)])
    assert ser == [12 * MiB] * 3
    assert res["peak_allocated"] == 11 * MiB and res["peak_allocated_event"] == 0
    assert res["max_free_blocks_large"] == 1


def test_w8_reclaim_then_oom():
    t = [A(MiB), F(0), A(19 * MiB)]
    # cap 20 MiB: 2 + 20 > 20 -> release the idle small segment -> 0 + 20 <= 20
    res, ser = both(t, oracle.paper_params(device_capacity_bytes=20 * MiB))
    assert ser == [2 * MiB, 2 * MiB, 20 * MiB]
    assert (res["segments_created"], res["segments_released"], res["status"]) == (2, 1, OK)
    assert res["peak_reserved"] == 20 * MiB and res["peak_reserved_event"] == 2
    # one byte less: even after reclaim 20 MiB > cap -> OOM at e2; the reclaim of the
    # failing event is not applied
    res, ser = both(t, oracle.paper_params(device_capacity_bytes=20 * MiB - 1))
    assert ser == [2 * MiB, 2 * MiB, -1]
    assert (res["status"], res["stop_event"]) == (OOM, 2)
    assert (res["peak_reserved"], res["peak_reserved_event"]) == (2 * MiB, 0)
    assert (res["segments_created"], res["segments_released"], res["final_reserved"]) == (1, 0, 2 * MiB)


def test_w8b_reclaim_skips_busy_segments():
    # the small segment still holds a live block, so nothing can be released -> OOM
    t = [A(MiB), A(19 * MiB)]
    res, ser = both(t, oracle.paper_params(device_capacity_bytes=21 * MiB))
    assert (res["status"], res["stop_event"], ser) == (OOM, 1, [2 * MiB, -1])


def test_w9_packing():
    res, ser = both([A(MiB)] * 5)
    assert ser == [2 * MiB * ((e + 2) // 2) for e in range(5)]


def test_w10_record_highs():
    t = [A(12 * MiB), F(0), A(10 * MiB), F(2), A(14 * MiB), F(4), A(12 * MiB), F(6), A(16 * MiB), F(8)]
    res, ser = both(t)
    assert res["peak_reserved"] == 42 * MiB and res["peak_reserved_event"] == 8
    assert ser == [12 * MiB] * 4 + [26 * MiB] * 4 + [42 * MiB] * 2


def test_w11_small_alternation():
    t = [A(MiB), F(0), A(512), F(2), A(700 * KiB), F(4), A(MiB), F(6), A(1), F(8)]
    res, ser = both(t)
    assert ser == [2 * MiB] * len(t)


def test_w13_split_threshold_preset():
    t = [A(3 * MiB), A(2 * MiB), A(2 * MiB), F(0), A(2 * MiB), F(1), A(3 * MiB), A(13 * MiB)]
    res, ser = both(t, P)
    assert ser == [20 * MiB] * 8
    assert res["peak_allocated"] == 20 * MiB and res["peak_allocated_event"] == 7
    # PYTORCH_LIKE: the 3 MiB hole is handed out whole for 2 MiB (1 MiB left is not
    # > 1 MiB), so e5's free cannot merge, A3MiB splits the 13 MiB hole and A13MiB
    # needs a 14 MiB segment: 20 + 14 = 34 MiB
    res, ser = both(t, PT)
    assert ser == [20 * MiB] * 7 + [34 * MiB]
    assert res["peak_allocated"] == 20 * MiB and res["peak_allocated_event"] == 7


def test_w14_split_at_exact_threshold():
    # small pool: 1 MiB + (1 MiB - 512) leaves exactly one granule, which IS split off
    # (remainder >= split_min), so a 512 B request fits it: one segment only
    res, ser = both([A(MiB), A(MiB - 512), A(512)])
    assert ser == [2 * MiB] * 3 and res["max_free_blocks_small"] == 1
    # large pool: 19 MiB in a 20 MiB segment leaves 1 MiB, a free block under the paper
    # parameters but not under PYTORCH_LIKE (needs > 1 MiB); 19 MiB - 512 leaves
    # 1 MiB + 512, a free block under both
    res, _ = both([A(19 * MiB)], P)
    assert res["max_free_blocks_large"] == 1
    res, _ = both([A(19 * MiB)], PT)
    assert res["max_free_blocks_large"] == 0
    res, _ = both([A(19 * MiB - 512)], PT)
    assert res["max_free_blocks_large"] == 1
    # the unsplit block is freed whole and merges back into one idle segment
    res, ser = both([A(19 * MiB), F(0), A(20 * MiB)], PT)
    assert ser == [20 * MiB] * 3 and res["segments_created"] == 1


def test_malformed_events():
    cases = [
        ([F(0)], BAD_FREE, 0),                         # h >= e
        ([A(512), F(1)], BAD_FREE, 1),                 # self reference
        ([A(512), F(0), F(0)], BAD_FREE, 2),           # double free
        ([A(0), F(0), F(0)], BAD_FREE, 2),             # double free of a no-op
        ([A(512), A(1024), F(1), F(2)], BAD_FREE, 3),  # frees a free event
        ([A(512), F(0) | (1 << 40)], BAD_EVENT, 1),    # nonzero bits 62:32
        ([A((1 << 48) + 1)], BAD_EVENT, 0),            # request above 2^48
        ([A(512), A(512), F(1), F(5)], BAD_FREE, 3),   # forward reference
    ]
    for t, st, e in cases:
        res, ser = both(t)
        assert (res["status"], res["stop_event"]) == (st, e), t
        assert ser[e:] == [-1] * (len(t) - e)
    res, ser = both([A(1 << 48)])                     # the largest legal request
    assert res["status"] == OK and res["peak_reserved"] == 1 << 48


def test_state_is_kept_at_stop():
    # stop at e3: everything reported is the state after e2
    res, ser = both([A(3 * MiB), A(MiB), F(1), F(7)])
    assert ser == [20 * MiB, 22 * MiB, 22 * MiB, -1]
    assert (res["final_allocated"], res["final_reserved"], res["peak_allocated"]) == (3 * MiB, 22 * MiB, 4 * MiB)


def test_pool_overflow():
    # every 2^48 request needs its own 2^48 segment; the 8193rd would pass 2^61
    n = 8193
    res, _ = oracle.replay_one([A(1 << 48)] * n, P, series=False)
    assert (int(res["status"]), int(res["stop_event"])) == (OVERFLOW, n - 1)
    assert int(res["peak_reserved"]) == 1 << 61 and int(res["final_allocated"]) == 1 << 61


def test_empty_and_batch_layout():
    ev = np.array([A(MiB), F(0), A(5 * MiB)], dtype=np.uint64)
    off = np.array([0, 0, 2, 2, 3, 3], dtype=np.int64)  # empty traces interleaved
    rc, out, ser = oracle.replay(ev, off, P, series=True)
    assert rc == 0
    for t in (0, 2, 4):
        assert int(out[t]["peak_reserved"]) == 0 and int(out[t]["peak_allocated_event"]) == -1
    assert int(out[1]["peak_reserved"]) == 2 * MiB and int(out[3]["peak_reserved"]) == 20 * MiB
    assert list(ser) == [2 * MiB, 2 * MiB, 20 * MiB]
    rc, out, _ = oracle.replay(np.zeros(0, np.uint64), np.array([0], np.int64), P)
    assert rc == 0 and len(out) == 0


def test_call_level_errors():
    ev = np.array([A(1)], dtype=np.uint64)
    assert oracle.replay(ev, np.array([1, 1], np.int64), P)[0] == -2
    assert oracle.replay(ev, np.array([0, 1, 0], np.int64), P)[0] == -2
    bad = [dict(P, round_bytes=384), dict(P, small_max_bytes=3 * MiB), dict(P, mid_segment_bytes=5 * MiB),
           dict(P, split_min_small_bytes=0), dict(P, device_capacity_bytes=0), dict(P, large_round_bytes=1000)]
    for b in bad:
        assert oracle.validate_params(b) == -1, b
        assert oracle.replay(ev, np.array([0, 1], np.int64), b)[0] == -1
    assert oracle.validate_params(P) == 0 and oracle.validate_params(PT) == 0


def test_oom_predicate_eq1():
    """Section 4.1, Eq. (1): OOM is predicted iff the estimated peak exceeds the device's maximum
    memory (a strict inequality).  The estimates come from the paper's own printed examples:
    a 1 MB tensor gets a 2 MB segment (Section 2.2.2), a 10 MB tensor a 20 MB one (Section 6.4),
    so their estimated peaks are 2,097,152 and 20,971,520 bytes."""
    ev = np.array([A(1_000_000), A(10_000_000)], dtype=np.uint64)
    rc, res, _ = oracle.replay(ev, np.array([0, 1, 2]), P)
    assert rc == 0 and list(res["peak_reserved"]) == [2 * MiB, 20 * MiB]
    for m_max, want in [(2 * MiB, [0, 1]), (2 * MiB - 1, [1, 1]), (20 * MiB, [0, 0]), (20 * MiB - 1, [0, 1]),
                        (0, [1, 1]), (1 << 62, [0, 0])]:
        rc, flags = oracle.oom_predicted(res, m_max)
        assert rc == 0 and list(flags) == want, (m_max, list(flags))


def test_oom_predicate_statuses():
    # W8 at cap 20 MiB - 1 stops with OOM: predicted, whatever m_max; a malformed trace and a
    # double free give no estimate; an empty trace has peak 0 (never predicted)
    t = [A(MiB), F(0), A(19 * MiB)]
    rc, oom, _ = oracle.replay(np.array(t, np.uint64), np.array([0, 3]),
                               oracle.paper_params(device_capacity_bytes=20 * MiB - 1))
    assert rc == 0 and oom["status"][0] == OOM
    rc, bad, _ = oracle.replay(np.array([A(1 << 49), A(8), F(1), F(1)], np.uint64), np.array([0, 1, 4, 4]), P)
    assert rc == 0 and list(bad["status"]) == [BAD_EVENT, BAD_FREE, OK]
    res = np.concatenate([oom, bad])
    rc, flags = oracle.oom_predicted(res, 1 << 62)
    assert rc == 0 and list(flags) == [1, -1, -1, 0]
    rc, flags = oracle.oom_predicted(res, 0)
    assert rc == 0 and list(flags) == [1, -1, -1, 0]
    assert oracle.oom_predicted(res, -1)[0] == -1
    rc, flags = oracle.oom_predicted(res[:0], 5)
    assert rc == 0 and len(flags) == 0
