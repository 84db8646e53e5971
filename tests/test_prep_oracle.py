"""Pins of the trace-preparation oracle (Sections 3.2 and 3.3), on the CPU.

* Hand-worked cases fix every reading: address reuse, persistence, a second allocation at an
  open address, unmatched frees, 0-byte events, each category rule, the order at equal times.
* An O(n^2) pairing written from the definition (scan forward from each allocation) and an
  orchestration re-derived with numpy (searchsorted for the markers, lexsort for the order)
  are compared with the oracle on seeded random inputs.
* The orchestrated words of a generated training trace are a valid Simulator input.
"""
import numpy as np
import pytest

import oracle
from oracle import BLOCK_DTYPE, PERSISTENT, RAW_DTYPE

pytestmark = pytest.mark.filterwarnings("ignore")
FREE = 1 << 63
P, CAT_PARAM, CAT_BATCH, CAT_GRAD, CAT_OPT = PERSISTENT, 1, 2, 3, 4


def raw(*evs):
    return np.array(list(evs), dtype=RAW_DTYPE)


def life(*evs):
    r = raw(*evs)
    rc, b, boff, unm = oracle.lifecycles(r, np.array([0, len(r)]))
    assert rc == 0
    return [(int(x["size"]), int(x["t_alloc"]), int(x["t_free"])) for x in b], int(unm[0])


# ---------------------------------------------------------------- Section 3.2 readings
def test_pairing_with_address_reuse():
    blocks, unm = life((0, 0x100, 64), (1, 0x100, -64), (2, 0x100, 32), (3, 0x100, -32))
    assert blocks == [(64, 0, 1), (32, 2, 3)] and unm == 0


def test_unfreed_block_is_persistent():
    blocks, _ = life((0, 0x100, 64), (1, 0x200, 8), (2, 0x200, -8))
    assert blocks == [(64, 0, P), (8, 1, 2)]


def test_second_allocation_at_open_address_leaves_first_persistent():
    blocks, unm = life((0, 0x100, 64), (1, 0x100, 16), (2, 0x100, -16))
    assert blocks == [(64, 0, P), (16, 1, 2)] and unm == 0


def test_unmatched_free_and_zero_bytes_ignored():
    blocks, unm = life((0, 0x100, -8), (1, 0x100, 0), (2, 0x100, 40), (3, 0x300, -40), (4, 0x100, -1))
    assert blocks == [(40, 2, 4)] and unm == 2  # the free's byte count is not checked


def test_blocks_in_allocation_order_across_traces():
    r = raw((0, 1, 5), (1, 2, 6), (2, 1, -5), (10, 1, 7), (11, 1, -7))
    rc, b, boff, unm = oracle.lifecycles(r, np.array([0, 3, 3, 5]))
    assert rc == 0 and list(boff) == [0, 2, 2, 3] and list(unm) == [0, 0, 0]
    assert [int(x) for x in b["size"]] == [5, 6, 7] and int(b["t_free"][1]) == P


def pairing_by_definition(evs):
    """For each allocation at index i, scan forward for the first event at its address: a free
    closes it, another allocation leaves it persistent.  Frees closing nothing are unmatched."""
    blocks, used = [], set()
    for i, (ts, addr, nb) in enumerate(evs):
        if nb <= 0:
            continue
        t_free = P
        for j in range(i + 1, len(evs)):
            tj, aj, bj = evs[j]
            if aj != addr or bj == 0:
                continue
            if bj < 0:
                t_free = tj
                used.add(j)
            break
        blocks.append((nb, ts, t_free))
    unmatched = sum(1 for j, e in enumerate(evs) if e[2] < 0 and j not in used)
    return blocks, unmatched


@pytest.mark.parametrize("seed", range(6))
def test_pairing_matches_definition(seed):
    rng = np.random.default_rng(seed)
    n = 400
    addrs = rng.integers(0, 12, n)
    kind = rng.choice([1, -1, 0], n, p=[0.5, 0.45, 0.05])
    evs = [(int(t) * 3, int(a) * 512, int(k) * int(rng.integers(1, 1 << 20))) for t, a, k in zip(range(n), addrs, kind)]
    assert life(*evs) == pairing_by_definition(evs)


def test_bad_offsets():
    r = raw((0, 1, 5))
    assert oracle.lifecycles(r, np.array([0, 2, 1]))[0] == -2


# ---------------------------------------------------------------- Section 3.3 readings
def orch(blocks, steps=(), zgs=()):
    b = np.array([(s, ta, tf, c, 0) for (s, ta, tf, c) in blocks], dtype=BLOCK_DTYPE)
    rc, ev, eoff = oracle.orchestrate(b, np.array([0, len(b)]), np.array(steps, np.int64),
                                      np.array([0, len(steps)]), np.array(zgs, np.int64), np.array([0, len(zgs)]))
    assert rc == 0
    return [int(x) for x in ev]


def test_activation_keeps_cpu_lifetime():
    assert orch([(10, 0, 5, 0), (20, 1, 3, 0)]) == [10, 20, FREE | 1, FREE | 0]


def test_parameters_and_optimizer_states_persist():
    assert orch([(10, 0, 5, CAT_PARAM), (20, 1, 3, CAT_OPT), (30, 2, 4, 0)]) == [10, 20, 30, FREE | 2]


def test_batch_data_bounded_by_the_iteration():
    # iteration boundaries at 10 and 20: a batch allocated at 2 and never freed on the CPU is
    # freed at 10; one freed on the CPU at 12 (before its boundary 20) keeps that free
    ev = orch([(8, 2, P, CAT_BATCH), (9, 11, 12, CAT_BATCH), (4, 25, P, CAT_BATCH)], steps=(10, 20))
    assert ev == [8, FREE | 0, 9, FREE | 2, 4]


def test_gradients_freed_at_next_zero_grad():
    # zero_grad at 5 and 30: a gradient made at 7 (CPU free at 8) is held until 30; one made
    # after the last zero_grad persists; one made exactly at 5 waits for 30
    ev = orch([(16, 7, 8, CAT_GRAD), (32, 31, 33, CAT_GRAD), (64, 5, 6, CAT_GRAD), (1, 9, 10, 0)], zgs=(5, 30))
    assert ev == [64, 16, 1, FREE | 2, FREE | 1, FREE | 0, 32]


def test_order_at_equal_times():
    # at time 5: the free of an earlier block, then allocations in block order, then the free of
    # a block allocated at 5 (zero length)
    ev = orch([(1, 0, 5, 0), (2, 5, 5, 0), (3, 5, 9, 0)])
    assert ev == [1, FREE | 0, 2, 3, FREE | 2, FREE | 3]
    # a free earlier than its allocation moves to the allocation time
    assert orch([(7, 4, 2, 0)]) == [7, FREE | 0]


def orchestrate_numpy(blocks, steps, zgs):
    """The same rules with numpy: markers by searchsorted, order by lexsort."""
    n = len(blocks)
    ta = blocks["t_alloc"].astype(np.int64)
    tf = blocks["t_free"].astype(np.int64).copy()
    cat = blocks["category"]
    steps, zgs = np.asarray(steps, np.int64), np.asarray(zgs, np.int64)
    i = np.searchsorted(steps, ta, side="right")
    nxt_step = np.where(i < len(steps), steps[np.minimum(i, max(len(steps) - 1, 0))] if len(steps) else P, P)
    j = np.searchsorted(zgs, ta, side="right")
    nxt_zg = np.where(j < len(zgs), zgs[np.minimum(j, max(len(zgs) - 1, 0))] if len(zgs) else P, P)
    tf = np.where((cat == CAT_PARAM) | (cat == CAT_OPT), P, tf)
    tf = np.where(cat == CAT_BATCH, np.minimum(tf, nxt_step), tf)
    tf = np.where(cat == CAT_GRAD, nxt_zg, tf)
    tf = np.where((tf != P) & (tf < ta), ta, tf)
    has_free = tf != P
    times = np.concatenate([ta, tf[has_free]])
    ranks = np.concatenate([np.ones(n, np.int64), np.where(tf[has_free] == ta[has_free], 2, 0)])
    blk = np.concatenate([np.arange(n), np.flatnonzero(has_free)])
    is_alloc = np.concatenate([np.ones(n, bool), np.zeros(int(has_free.sum()), bool)])
    order = np.lexsort((blk, ranks, times))
    pos = np.empty(n, np.int64)
    pos[blk[order][is_alloc[order]]] = np.flatnonzero(is_alloc[order])
    words = np.where(is_alloc[order], blocks["size"][blk[order]].astype(np.uint64),
                     np.uint64(FREE) | pos[blk[order]].astype(np.uint64))
    return [int(w) for w in words]


@pytest.mark.parametrize("seed", range(6))
def test_orchestration_matches_numpy(seed):
    rng = np.random.default_rng(100 + seed)
    n = 500
    ta = np.sort(rng.integers(0, 2000, n))
    life_ = rng.integers(0, 300, n)
    tf = np.where(rng.random(n) < 0.1, P, ta + life_)
    tf = np.where(rng.random(n) < 0.03, ta - 5, tf)  # a few frees before their allocation
    cat = rng.integers(0, 5, n)
    b = np.zeros(n, BLOCK_DTYPE)
    b["size"], b["t_alloc"], b["t_free"], b["category"] = rng.integers(1, 1 << 30, n), ta, tf, cat
    steps = np.sort(rng.choice(2000, 7, replace=False))
    zgs = np.sort(rng.choice(2000, 5, replace=False))
    got = orch([(int(x["size"]), int(x["t_alloc"]), int(x["t_free"]), int(x["category"])) for x in b], steps, zgs)
    assert got == orchestrate_numpy(b, steps, zgs)


def test_orchestration_bad_offsets():
    b = np.zeros(2, BLOCK_DTYPE)
    rc, _, _ = oracle.orchestrate(b, np.array([0, 2]), np.zeros(0, np.int64), np.array([1, 0]),
                                  np.zeros(0, np.int64), np.array([0, 0]))
    assert rc == -2


# ---------------------------------------------------------------- the three stages together
def _pipeline(pos, n_traces=4, n_events=12000):
    from tracegen import prep
    raw_, cat, roff, st, soff, zg, zoff = prep.batch_profiles(n_traces, n_events, pos=pos)
    rc, b, boff, unm = oracle.lifecycles(raw_.view(RAW_DTYPE), roff, cat)
    assert rc == 0 and (unm == 0).all()
    rc, ev, eoff = oracle.orchestrate(b, boff, st, soff, zg, zoff)
    assert rc == 0
    rc, res, _ = oracle.replay(ev, eoff, oracle.paper_params())
    assert rc == 0 and (res["status"] == 0).all()  # every free names an earlier, unfreed allocation
    return b, boff, ev, eoff, res


def test_orchestrated_training_trace_replays():
    from tracegen import prep
    b, boff, ev, eoff, res = _pipeline("POS1")
    _, _, _, st, soff, zg, zoff = prep.batch_profiles(4, 12000, pos="POS1")
    for t in range(2):  # the generated traces: oracle words == the numpy re-derivation
        words = [int(x) for x in ev[eoff[t]:eoff[t + 1]]]
        assert words == orchestrate_numpy(b[boff[t]:boff[t + 1]], st[soff[t]:soff[t + 1]], zg[zoff[t]:zoff[t + 1]])
    assert (res["peak_reserved"] >= res["peak_allocated"]).all()


def test_zero_grad_placement_changes_the_footprint():
    """Fig. 1: zero_grad just before the backward pass (POS0) keeps the previous gradients
    alive through the forward pass; at the iteration start (POS1) it does not."""
    *_, r0 = _pipeline("POS0")
    *_, r1 = _pipeline("POS1")
    assert (r0["peak_allocated"] > r1["peak_allocated"]).all()
    assert (r0["peak_reserved"] >= r1["peak_reserved"]).all() and (r0["peak_reserved"] != r1["peak_reserved"]).any()


# ---------------------------------------------------------------- Section 3.2 attribution
WIN_C, WIN_O = oracle.WIN_COMPONENT, oracle.WIN_OPERATOR


def windows(*ws):
    return np.array([(a, b, par, kind, cat, 0) for (a, b, par, kind, cat) in ws], dtype=oracle.WINDOW_DTYPE)


def attribute(blocks, wins, sizes=None):
    b = np.array([(1, ta, tf, 0, 0) for (ta, tf) in blocks], dtype=BLOCK_DTYPE)
    b["size"] = np.arange(1, len(b) + 1) if sizes is None else sizes
    rc, kept, koff, bw = oracle.attribute(b, np.array([0, len(b)]), wins, np.array([0, len(wins)]))
    assert rc == 0
    return [int(x) for x in bw], [(int(k["size"]), int(k["category"])) for k in kept]


def test_attribution_rules():
    W = windows((0, 100, -1, WIN_C, 0),          # 0 component
                (10, 50, 0, WIN_O, CAT_GRAD),    # 1 operator in 0
                (20, 30, 1, WIN_O, 0),           # 2 nested operator
                (60, 90, 0, WIN_C, 0),           # 3 component in 0
                (65, 70, 3, WIN_O, CAT_BATCH))   # 4 operator in 3
    bw, kept = attribute([(22, 28),    # (i) in 2
                          (22, 45),    # not (i)/(ii) in 2; (i) in 1
                          (12, 120),   # (ii) in 1: outlives component 0 -> its product
                          (55, 58),    # only component 0 contains it: dropped
                          (66, P),     # (ii) in 4: a persistent product
                          (66, 80),    # neither in 4, no operator outside: dropped
                          (5, 8),      # dropped
                          (50, 60),    # 1 contains 50 (end included) but neither rule holds
                          (30, 30),    # freed at 2's end: not strictly inside 2; (i) in 1
                          (20, 25),    # allocated at 2's start: not strictly inside 2; (i) in 1
                          (10, 49)],   # allocated at 1's start: (i) fails in 1, no operator above
                         W)
    assert bw == [2, 1, 1, -1, 4, -1, -1, -1, 1, 1, -1]
    assert kept == [(1, 0), (2, 0), (3, CAT_GRAD), (5, CAT_BATCH), (9, 0), (10, 0)]


def test_attribution_boundaries():
    # windows that start together nest in list order (the later one is inside); a block freed
    # exactly when its operator's component ends does not outlive it; rule (i) wants the
    # lifespan strictly inside the window (Section 3.2), so a block allocated at the common
    # start of the operators links to none of them, while one allocated a tick later does
    W = windows((200, 300, -1, WIN_C, 0),
                (200, 250, 0, WIN_O, CAT_PARAM),
                (200, 220, 1, WIN_O, CAT_BATCH))
    bw, kept = attribute([(200, 210), (240, 300), (240, 301), (201, 219), (201, 220), (219, 249)], W)
    assert bw == [-1, -1, 1, 2, 1, 1]
    assert kept == [(3, CAT_PARAM), (4, 0), (5, 0), (6, 0)]


def test_optimizer_states_by_parameter_size():
    """Section 3.3 item 5: blocks allocated during optimizer.step() whose sizes match model
    parameters are optimizer states.  Worked by hand: the parameters (products of the model.to
    operator) have sizes 1000 and 64.  In the step phase, the product of size 1000 becomes an
    optimizer state; the product of size 999 matches no parameter and keeps its operator's role;
    the temporary of size 64 (rule (i)) is no product and stays a temporary.  A product of size
    1000 outside the step phase keeps its operator's role."""
    W = windows((0, 100, -1, WIN_C, 0),                  # 0 model.to(device)
                (10, 20, 0, WIN_O, CAT_PARAM),           # 1 its operator
                (200, 300, -1, WIN_C, CAT_OPT),          # 2 optimizer.step(): the phase
                (210, 290, 2, WIN_O, 0),                 # 3 its operator, no role of its own
                (400, 500, -1, WIN_C, 0),                # 4 another component
                (410, 420, 4, WIN_O, CAT_BATCH))         # 5 an operator producing batch data
    blocks = [(12, P), (14, P),                  # parameters
              (220, P), (230, P), (240, 250),    # step phase: product, product, temporary
              (415, 600),                        # a product of operator 5, outside the phase
              (210, P)]                          # at the operator's start: still allocated during it
    sizes = [1000, 64, 1000, 999, 64, 1000, 64]
    bw, kept = attribute(blocks, W, sizes)
    assert bw == [1, 1, 3, 3, 3, 5, 3]
    assert kept == [(1000, CAT_PARAM), (64, CAT_PARAM), (1000, CAT_OPT), (999, 0), (64, 0), (1000, CAT_BATCH),
                    (64, CAT_OPT)]


def test_optimizer_rule_is_per_trace():
    """The parameter sizes of one trace do not make optimizer states in another."""
    W = windows((0, 100, -1, WIN_C, 0), (10, 20, 0, WIN_O, CAT_PARAM),
                (200, 300, -1, WIN_C, CAT_OPT), (210, 290, 2, WIN_O, 0))
    b = np.zeros(3, BLOCK_DTYPE)
    b["size"], b["t_alloc"], b["t_free"] = [777, 777, 777], [12, 220, 220], [P, P, P]
    rc, kept, koff, bw = oracle.attribute(b, np.array([0, 2, 3]), np.concatenate([W, W]), np.array([0, 4, 8]))
    assert rc == 0 and list(koff) == [0, 2, 3] and list(bw) == [1, 3, 3]
    assert list(kept["category"]) == [CAT_PARAM, CAT_OPT, 0]


def test_attribution_without_windows_drops_everything():
    bw, kept = attribute([(1, 2), (3, P)], windows())
    assert bw == [-1, -1] and kept == []


def attribution_by_depth(blocks, w):
    """Innermost containing window = the one with the most ancestors; then the rules outward."""
    def parent(i):
        p_ = int(w["parent"][i])
        return p_ if 0 <= p_ < i else -1

    def depth(i):
        d = 0
        while parent(i) >= 0:
            i, d = parent(i), d + 1
        return d

    out = []
    for ta, tf in blocks:
        cont = [i for i in range(len(w)) if w["start"][i] <= ta <= w["end"][i]]
        i = max(cont, key=lambda j: (depth(j), j)) if cont else -1
        got = (-1, 0, False)
        while i >= 0:
            if w["kind"][i] == WIN_O:
                c = parent(i)
                while c >= 0 and w["kind"][c] != WIN_C:
                    c = parent(c)
                if w["start"][i] < ta and tf < w["end"][i]:
                    got = (i, 0, False)
                    break
                if c >= 0 and tf > w["end"][c]:
                    got = (i, int(w["category"][i]), True)
                    break
            i = parent(i)
        out.append(got)
    return out


def optimizer_rule(blocks, sizes, w, linked):
    """Section 3.3 item 5 over the operator rule's result: a product allocated inside an
    optimizer.step() component with a parameter's size becomes an optimizer state."""
    params = {s for s, (i, c, prod) in zip(sizes, linked) if i >= 0 and prod and c == CAT_PARAM}
    steps = [(int(a), int(b)) for a, b, k, c in zip(w["start"], w["end"], w["kind"], w["category"])
             if k == WIN_C and c == CAT_OPT]
    out = []
    for (ta, _tf), s, (i, c, prod) in zip(blocks, sizes, linked):
        if i >= 0 and prod and s in params and any(a <= ta <= b for a, b in steps):
            c = CAT_OPT
        out.append((i, c))
    return out


def nested_windows(rng, n_top, t_end):
    """Properly nested random windows in start order (a random call tree)."""
    rows = []

    def gen(lo, hi, par, depth):
        t = lo
        while t < hi - 4 and len(rows) < 4000:
            a = int(rng.integers(t, min(hi - 2, t + (hi - t) // 2 + 1)))
            b = int(rng.integers(a + 1, min(hi, a + max(2, (hi - a) // 2)) + 1))
            rows.append([a, b, par, int(rng.integers(0, 2)), int(rng.integers(0, 5))])
            me = len(rows) - 1
            if depth < 5 and b - a > 6 and rng.random() < 0.7:
                gen(a + 1, b, me, depth + 1)
            t = b + int(rng.integers(0, 3))

    gen(0, t_end, -1, 0)
    return windows(*[tuple(r) for r in rows])


def _depth_search_case(seed):
    rng = np.random.default_rng(300 + seed)
    W = nested_windows(rng, 10, 20000)
    ta = np.sort(rng.integers(0, 20000, 600))
    tf = np.where(rng.random(600) < 0.1, P, ta + rng.integers(0, 4000, 600))
    blocks = list(zip(ta.tolist(), tf.tolist()))
    sizes = rng.integers(1, 40, 600)  # few distinct sizes, so that some match a parameter's
    bw, kept = attribute(blocks, W, sizes)
    want = optimizer_rule(blocks, sizes.tolist(), W, attribution_by_depth(blocks, W))
    assert bw == [i for i, _ in want]
    assert kept == [(int(s), c) for s, (i, c) in zip(sizes, want) if i >= 0]
    return sum(c == CAT_OPT for _, c in want)


@pytest.mark.parametrize("seed", range(5))
def test_attribution_matches_depth_search(seed):
    _depth_search_case(seed)


def test_depth_search_cases_exercise_the_optimizer_rule():
    assert sum(_depth_search_case(seed) > 0 for seed in range(5)) >= 2


def test_attribution_recovers_generated_roles():
    """On generated profiles, every block allocated inside an operator is kept with the role the
    generator planted, and only the script-level temporaries are dropped."""
    from tracegen import prep
    raw_, cat, roff, st, soff, zg, zoff, win, woff = prep.batch_profiles(3, 15000, windows=True)
    rc, b, boff, _ = oracle.lifecycles(raw_.view(RAW_DTYPE), roff)  # no roles given
    rc2, bc, _, _ = oracle.lifecycles(raw_.view(RAW_DTYPE), roff, cat)  # the planted roles
    rc3, kept, koff, bw = oracle.attribute(b, boff, win.view(oracle.WINDOW_DTYPE), woff)
    assert rc == rc2 == rc3 == 0
    keep = bw >= 0
    assert np.array_equal(kept["category"], bc["category"][keep])
    dropped = np.flatnonzero(~keep)
    assert 0 < len(dropped) < 0.05 * len(b)
    assert (bc["category"][dropped] == 0).all() and (b["size"][dropped] <= 4096).all()
