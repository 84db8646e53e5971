"""The no-allocation entry point (xmem_replay_batch_noalloc) against xmem_replay_batch_ex on the
same inputs, through the C ABI: results and the whole per-event reserved series, bit-exact.
Two calls in a row share the library's fixed workspace area; the second has a smaller input, so
it runs on whatever the first one left there."""
import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import compare, compare_series, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2510_21048_amd as xm
    xm.load()
    yield


def _noalloc(ev, off, p):
    import torch
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding
    T, N = len(off) - 1, len(ev)
    e = torch.from_numpy(np.ascontiguousarray(ev, dtype=np.uint64).view(np.int64)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(off, dtype=np.int64)).cuda()
    out = torch.full((T, 96), 0x5A, dtype=torch.uint8, device="cuda")
    ser = torch.full((N,), 7, dtype=torch.int64, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    rc = xm.xmem_replay_batch_noalloc(e, o, T, N, p, out, ser, st)
    assert rc == 0, xm.xmem_strerror(rc)
    torch.cuda.synchronize()
    return binding.to_numpy(out), ser.cpu().numpy()


def _ex(ev, off, p):
    import torch
    from paper_2510_21048_amd import binding
    e = torch.from_numpy(np.ascontiguousarray(ev, dtype=np.uint64).view(np.int64)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(off, dtype=np.int64)).cuda()
    out, ser = binding.replay(e, o, p, series=True)
    torch.cuda.synchronize()
    return binding.to_numpy(out), ser.cpu().numpy()


def _both(ev, off, pdict, what):
    import paper_2510_21048_amd as xm
    p = xm.params(**pdict)
    log(f"[no-alloc] {what}: {len(off) - 1} traces, {len(ev)} events")
    gres, gser = _noalloc(ev, off, p)
    wres, wser = _ex(ev, off, p)
    compare(gres, wres, what=what)
    compare_series(gser, wser, off, what=what)
    return gres


def _slices(cfg, nt, ne):
    ev, off = tracegen.generate(cfg, nt, ne)
    return ev, off


def test_noalloc_matches_ex_two_calls():
    P = oracle.paper_params()
    # 1) 24 GPT-style traces of 9,000 events: the library's own chunk grain fits the area
    ev, off = _slices(3, 24, 9000)
    _both(ev, off, P, "24 x 9000, chunked")
    # 2) smaller, right after: 5 CNN-shaped traces of 3,001 events
    ev2, off2 = _slices(2, 5, 3001)
    _both(ev2, off2, P, "5 x 3001, after a larger call")


def test_noalloc_serial_fallback_and_capacity():
    """A long trace whose small pool outgrows the LDS table (the paged-set kernel runs): its
    chunked workspace does not fit the area, so the serial replay with fewer paged slots runs;
    then a smaller batch under a finite capacity (reclaim and OOM), again after a larger call."""
    P = oracle.paper_params()
    ev, off = tracegen.generate(5, 1, 600000)
    res = _both(ev, off, P, "600K-event fragmented trace, serial fallback")
    assert int(res["max_free_blocks_small"][0]) > 1000
    ev2, off2 = _slices(4, 12, 6000)
    _, free_res, _ = oracle.replay(ev2, off2, P, threads=8)
    cap = int(np.median(free_res["peak_reserved"]) * 0.7)
    res2 = _both(ev2, off2, oracle.paper_params(device_capacity_bytes=cap), f"12 x 6000, capacity {cap}")
    assert (res2["status"] == 1).any()
