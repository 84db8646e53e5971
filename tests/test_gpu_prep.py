"""Parity of the HIP trace-preparation steps with the oracle (bit-exact): lifecycle pairing
(Section 3.2), orchestration (Section 3.3), and the three stages chained on the GPU
(raw allocator events -> blocks -> event words -> replay results).

Sizes span many 4096-element sort tiles with ragged tails; batches of up to 300 traces take
two radix passes for the trace key."""
import numpy as np
import pytest

import oracle
from gpu_util import compare, gpu_replay, log

pytestmark = pytest.mark.gpu
P = oracle.paper_params()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2510_21048_amd as xm
    xm.load()
    yield


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_lifecycles(raw, off, cat=None):
    import torch
    import paper_2510_21048_amd as xm
    T = len(off) - 1
    blocks, boff, unm, status = xm.lifecycles(_dev(raw.view(np.uint8)), _dev(off.astype(np.int64)),
                                              None if cat is None else _dev(cat.astype(np.int32)))
    torch.cuda.synchronize()
    boff = boff.cpu().numpy()
    b = blocks.cpu().numpy().reshape(-1).view(xm.BLOCK_DTYPE)[: int(boff[-1])]
    return b, boff, unm.cpu().numpy()[:T], int(status.cpu().item())


def gpu_orchestrate(blocks, boff, st, soff, zg, zoff):
    import torch
    import paper_2510_21048_amd as xm
    bl = blocks if len(blocks) else np.zeros(1, xm.BLOCK_DTYPE)
    ev, eoff, status = xm.orchestrate(_dev(bl.view(np.uint8)), _dev(boff.astype(np.int64)),
                                      _dev(st.astype(np.int64) if len(st) else np.zeros(1, np.int64)),
                                      _dev(soff.astype(np.int64)),
                                      _dev(zg.astype(np.int64) if len(zg) else np.zeros(1, np.int64)),
                                      _dev(zoff.astype(np.int64)))
    torch.cuda.synchronize()
    eoff = eoff.cpu().numpy()
    return ev.cpu().numpy().view(np.uint64)[: int(eoff[-1])], eoff, int(status.cpu().item())


def check_lifecycles(raw, off, cat=None, what=""):
    log(f"[gpu-prep] lifecycles {what}: {len(off) - 1} traces, {len(raw)} raw events")
    rc, wb, wboff, wunm = oracle.lifecycles(raw, off, cat)
    assert rc == 0
    gb, gboff, gunm, status = gpu_lifecycles(raw, off, cat)
    assert status == 0
    assert np.array_equal(gboff, wboff), what
    assert np.array_equal(gunm, wunm), what
    for f in ("size", "t_alloc", "t_free", "category"):
        bad = np.flatnonzero(gb[f] != wb[f])
        assert bad.size == 0, f"{what}: block field {f} differs at {bad[:5]}"
    return wb, wboff


def check_orchestrate(blocks, boff, st, soff, zg, zoff, what=""):
    log(f"[gpu-prep] orchestrate {what}: {len(boff) - 1} traces, {len(blocks)} blocks")
    rc, wev, weoff = oracle.orchestrate(blocks, boff, st, soff, zg, zoff)
    assert rc == 0
    gev, geoff, status = gpu_orchestrate(blocks, boff, st, soff, zg, zoff)
    assert status == 0
    assert np.array_equal(geoff, weoff), what
    bad = np.flatnonzero(gev != wev)
    assert bad.size == 0, f"{what}: event words differ at {bad[:5]}"
    return wev, weoff


def random_raw(seed, n_traces, max_len, n_addr=40):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, max_len, n_traces)
    lens[rng.random(n_traces) < 0.15] = 0  # empty traces
    n = int(lens.sum())
    raw = np.zeros(n, oracle.RAW_DTYPE)
    raw["ts"] = np.cumsum(rng.integers(0, 5, n))  # equal timestamps happen
    raw["addr"] = (rng.integers(0, n_addr, n) * 4096 + 0x7F0000000000).astype(np.uint64)
    kind = rng.choice([1, -1, 0], n, p=[0.5, 0.46, 0.04])
    raw["bytes"] = kind * rng.integers(1, 1 << 30, n)
    off = np.zeros(n_traces + 1, np.int64)
    off[1:] = np.cumsum(lens)
    cat = rng.integers(0, 5, n).astype(np.int32)
    return raw, off, cat


@pytest.mark.parametrize("seed,n_traces,max_len", [(1, 37, 20000), (2, 300, 1500), (3, 1, 70000)])
def test_lifecycles_random(seed, n_traces, max_len):
    raw, off, cat = random_raw(seed, n_traces, max_len)
    check_lifecycles(raw, off, cat, what=f"random seed {seed}")
    check_lifecycles(raw, off, None, what=f"random seed {seed}, no categories")


@pytest.mark.parametrize("span_bits,n_traces", [(63, 1), (64, 1), (20, 1000), (27, 128), (60, 300), (56, 255), (57, 256)])
def test_lifecycles_key_layouts(span_bits, n_traces):
    """Address spans that put the pairing sort on one key of (trace, address) bits -- up to 64 bits
    together, in an odd or an even number of 8-bit passes -- or on the address and then the trace.
    The pool of addresses holds 0 and 2^span_bits - 1, so the span is exact and no low bit is shared."""
    rng = np.random.default_rng(span_bits * 1000 + n_traces)
    hi = (1 << span_bits) - 1
    pool = np.concatenate([np.array([0, hi], np.uint64), rng.integers(0, hi, 62, dtype=np.uint64, endpoint=True)])
    lens = rng.integers(0, 3000, n_traces)
    n = int(lens.sum())
    raw = np.zeros(n, oracle.RAW_DTYPE)
    raw["ts"] = np.cumsum(rng.integers(0, 5, n))
    raw["addr"] = pool[rng.integers(0, len(pool), n)]
    raw["addr"][:2] = pool[:2]
    raw["bytes"] = rng.choice([1, -1, 0], n, p=[0.5, 0.46, 0.04]) * rng.integers(1, 1 << 30, n)
    raw["bytes"][:2] = 4096
    off = np.zeros(n_traces + 1, np.int64)
    off[1:] = np.cumsum(lens)
    check_lifecycles(raw, off, None, what=f"address span {span_bits} bits, {n_traces} traces")


def test_lifecycles_edge_cases():
    empty = np.zeros(0, oracle.RAW_DTYPE)
    check_lifecycles(empty, np.zeros(4, np.int64), what="all traces empty")
    only_frees = np.array([(i, 64 * i, -8) for i in range(5000)], dtype=oracle.RAW_DTYPE)
    check_lifecycles(only_frees, np.array([0, 5000]), what="only unmatched frees")
    one_addr = np.array([(i, 4096, 1 + i if i % 3 else -5) for i in range(9000)], dtype=oracle.RAW_DTYPE)
    check_lifecycles(one_addr, np.array([0, 4000, 9000]), what="one address, alloc-alloc-free")


def test_lifecycles_bad_offsets():
    raw, off, cat = random_raw(9, 4, 100)
    off = off.copy()
    off[1] = off[2] + 1  # decreasing
    _, gboff, _, status = gpu_lifecycles(raw, off, cat)
    assert status == 5 and (gboff == 0).all()


def random_blocks(seed, n_traces, max_blocks):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, max_blocks, n_traces)
    B = int(lens.sum())
    b = np.zeros(B, oracle.BLOCK_DTYPE)
    ta = np.concatenate([np.sort(rng.integers(-5000, 200000, l)) for l in lens]) if B else np.zeros(0, np.int64)
    tf = ta + rng.integers(0, 3000, B)
    tf = np.where(rng.random(B) < 0.1, oracle.PERSISTENT, tf)
    tf = np.where(rng.random(B) < 0.02, ta - 3, tf)
    b["size"], b["t_alloc"], b["t_free"], b["category"] = rng.integers(0, 1 << 34, B), ta, tf, rng.integers(0, 5, B)
    boff = np.zeros(n_traces + 1, np.int64)
    boff[1:] = np.cumsum(lens)
    ns, nz = rng.integers(0, 40, n_traces), rng.integers(0, 30, n_traces)
    st = np.concatenate([np.sort(rng.choice(250000, k, replace=False)) - 5000 for k in ns]).astype(np.int64)
    zg = np.concatenate([np.sort(rng.choice(250000, k, replace=False)) - 5000 for k in nz]).astype(np.int64)
    soff = np.concatenate([[0], np.cumsum(ns)]).astype(np.int64)
    zoff = np.concatenate([[0], np.cumsum(nz)]).astype(np.int64)
    return b, boff, st, soff, zg, zoff


@pytest.mark.parametrize("seed,n_traces,max_blocks", [(11, 29, 20000), (12, 300, 800), (13, 1, 60000)])
def test_orchestrate_random(seed, n_traces, max_blocks):
    check_orchestrate(*random_blocks(seed, n_traces, max_blocks), what=f"random seed {seed}")


@pytest.mark.parametrize("scale_bits,n_traces", [(30, 29), (36, 29), (40, 29), (40, 300), (30, 1)])
def test_orchestrate_time_layouts(scale_bits, n_traces):
    """Every time scaled by 2^scale_bits: the sort key of (trace, time, rank) takes an odd number of
    passes, or nearly 64 bits, or no longer fits, and the time and the trace are sorted apart
    (ending in either buffer by the trace passes)."""
    b, boff, st, soff, zg, zoff = random_blocks(20 + scale_bits + n_traces, n_traces, 4000)
    s = np.int64(1) << np.int64(scale_bits)
    live = b["t_free"] != oracle.PERSISTENT
    b["t_alloc"] = b["t_alloc"] * s
    b["t_free"] = np.where(live, b["t_free"] * s, b["t_free"])
    check_orchestrate(b, boff, st * s, soff, zg * s, zoff, what=f"times x 2^{scale_bits}, {n_traces} traces")


def test_orchestrate_bad_offsets():
    b, boff, st, soff, zg, zoff = random_blocks(19, 5, 200)
    zoff = zoff.copy()
    zoff[0] = 1
    _, geoff, status = gpu_orchestrate(b, boff, st, soff, zg, zoff)
    assert status == 5 and (geoff == 0).all()


@pytest.mark.parametrize("pos", ["POS0", "POS1"])
def test_pipeline_on_gpu(pos):
    """Raw profiler stream -> lifecycles -> orchestration -> replay, every stage on the GPU and
    every stage equal to the oracle's."""
    from tracegen import prep
    raw, cat, roff, st, soff, zg, zoff = prep.batch_profiles(12, 30000, pos=pos)
    raw = raw.view(oracle.RAW_DTYPE)
    wb, wboff = check_lifecycles(raw, roff, cat, what=f"training profiles {pos}")
    gb, gboff, _, _ = gpu_lifecycles(raw, roff, cat)
    wev, weoff = check_orchestrate(wb, wboff, st, soff, zg, zoff, what=f"training profiles {pos}")
    gev, geoff, _ = gpu_orchestrate(gb, gboff, st, soff, zg, zoff)
    gres, _ = gpu_replay(gev, geoff, P, series=False)
    rc, ores, _ = oracle.replay(wev, weoff, P, threads=8)
    assert rc == 0 and (ores["status"] == 0).all()
    compare(gres, ores, what=f"replay of orchestrated profiles {pos}")


# ---------------------------------------------------------------- time-window attribution
def gpu_attribute(blocks, boff, win, woff):
    import torch
    import paper_2510_21048_amd as xm
    bl = blocks if len(blocks) else np.zeros(1, xm.BLOCK_DTYPE)
    wn = win if len(win) else np.zeros(1, xm.WINDOW_DTYPE)
    kept, koff, bw, status = xm.attribute(_dev(bl.view(np.uint8)), _dev(boff.astype(np.int64)),
                                          _dev(wn.view(np.uint8)) if len(win) else _dev(np.zeros(0, np.uint8)),
                                          _dev(woff.astype(np.int64)))
    torch.cuda.synchronize()
    koff = koff.cpu().numpy()
    k = kept.cpu().numpy().reshape(-1).view(xm.BLOCK_DTYPE)[: int(koff[-1])]
    return k, koff, bw.cpu().numpy()[: len(blocks)], int(status.cpu().item())


def check_attribute(blocks, boff, win, woff, what=""):
    log(f"[gpu-prep] attribute {what}: {len(boff) - 1} traces, {len(blocks)} blocks, {len(win)} windows")
    rc, wk, wkoff, wbw = oracle.attribute(blocks, boff, win, woff)
    assert rc == 0
    gk, gkoff, gbw, status = gpu_attribute(blocks, boff, win, woff)
    assert status == 0
    assert np.array_equal(gkoff, wkoff), what
    assert np.array_equal(gbw, wbw), what
    assert gk.tobytes() == wk.tobytes(), what
    return wk, wkoff


def test_attribute_random():
    from test_prep_oracle import nested_windows
    rng = np.random.default_rng(41)
    bl, bo, wl, wo = [], [0], [], [0]
    for t in range(9):
        W = nested_windows(rng, 10, 30000) if t != 4 else np.zeros(0, oracle.WINDOW_DTYPE)  # one without windows
        nb = int(rng.integers(0, 6000))
        b = np.zeros(nb, oracle.BLOCK_DTYPE)
        # few distinct sizes in some traces, so that products of the optimizer.step() phases
        # match parameter sizes (Section 3.3 item 5); all distinct-ish in the others
        b["size"] = rng.integers(1, 50 if t % 2 else 1 << 30, nb)
        b["t_alloc"] = np.sort(rng.integers(0, 30000, nb))
        b["t_free"] = np.where(rng.random(nb) < 0.1, oracle.PERSISTENT, b["t_alloc"] + rng.integers(0, 5000, nb))
        bl.append(b); bo.append(bo[-1] + nb); wl.append(W); wo.append(wo[-1] + len(W))
    wk, _ = check_attribute(np.concatenate(bl), np.array(bo), np.concatenate(wl), np.array(wo),
                            what="random nested windows")
    assert (wk["category"] == oracle.CAT_OPTIMIZER).sum() > 0


def test_attribute_optimizer_rule_cases():
    """The hand-worked optimizer-state and strict-window cases of the oracle pins, on the GPU,
    in two traces (the parameter sizes of one trace do not count in the other)."""
    from test_prep_oracle import windows, WIN_C, WIN_O
    P_, CP, CB, CO = oracle.PERSISTENT, oracle.CAT_PARAMETER, oracle.CAT_BATCH, oracle.CAT_OPTIMIZER
    W = windows((0, 100, -1, WIN_C, 0), (10, 20, 0, WIN_O, CP), (200, 300, -1, WIN_C, CO), (210, 290, 2, WIN_O, 0),
                (400, 500, -1, WIN_C, 0), (410, 420, 4, WIN_O, CB))
    rows = [(1000, 12, P_), (64, 14, P_), (1000, 220, P_), (999, 230, P_), (64, 240, 250), (1000, 415, 600),
            (64, 210, P_), (5, 411, 419), (5, 410, 419), (5, 411, 420)]
    b = np.zeros(len(rows) + 2, oracle.BLOCK_DTYPE)
    b["size"][:len(rows)] = [r[0] for r in rows]
    b["t_alloc"][:len(rows)] = [r[1] for r in rows]
    b["t_free"][:len(rows)] = [r[2] for r in rows]
    b["size"][len(rows):], b["t_alloc"][len(rows):], b["t_free"][len(rows):] = 1000, 220, P_  # trace 1: no parameters
    wk, _ = check_attribute(b, np.array([0, len(rows), len(rows) + 2]), np.concatenate([W, W]),
                            np.array([0, len(W), 2 * len(W)]), what="optimizer rule cases")
    assert list(wk["category"][:3]) == [CP, CP, CO] and wk["category"][-1] == 0


def test_attribute_bad_offsets():
    from tracegen import prep
    raw, cat, roff, st, soff, zg, zoff, win, woff = prep.batch_profiles(2, 3000, windows=True)
    rc, b, boff, _ = oracle.lifecycles(raw.view(oracle.RAW_DTYPE), roff)
    woff = woff.copy()
    woff[-1] += 1  # does not end at the window count
    _, gkoff, _, status = gpu_attribute(b, boff, win.view(oracle.WINDOW_DTYPE), woff)
    assert status == 5 and (gkoff == 0).all()


@pytest.mark.parametrize("pos", ["POS0", "POS1"])
def test_full_pipeline_with_attribution(pos):
    """Raw allocator stream + execution windows -> lifecycles -> attribution -> orchestration ->
    replay, all on the GPU, each stage equal to the oracle's; the roles come from attribution."""
    from tracegen import prep
    raw, _cat, roff, st, soff, zg, zoff, win, woff = prep.batch_profiles(10, 30000, pos=pos, windows=True)
    raw, win = raw.view(oracle.RAW_DTYPE), win.view(oracle.WINDOW_DTYPE)
    wb, wboff = check_lifecycles(raw, roff, None, what=f"profiles {pos}")
    wk, wkoff = check_attribute(wb, wboff, win, woff, what=f"profiles {pos}")
    wev, weoff = check_orchestrate(wk, wkoff, st, soff, zg, zoff, what=f"attributed profiles {pos}")
    gb, gboff, _, _ = gpu_lifecycles(raw, roff, None)
    gk, gkoff, _, _ = gpu_attribute(gb, gboff, win, woff)
    gev, geoff, _ = gpu_orchestrate(gk, gkoff, st, soff, zg, zoff)
    gres, _ = gpu_replay(gev, geoff, P, series=False)
    rc, ores, _ = oracle.replay(wev, weoff, P, threads=8)
    assert rc == 0 and (ores["status"] == 0).all()
    compare(gres, ores, what=f"replay of the attributed pipeline {pos}")
