"""Helpers of the GPU tests: run the HIP path through the C ABI on numpy inputs
and compare it with the oracle field by field."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import paper_2510_21048_amd as xm
from paper_2510_21048_amd import binding

FIELDS = binding.RESULT_FIELDS


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_params(pdict: dict | None, chunks: int = 0):
    """Library parameters of an oracle parameter dict; chunks sets the chunk count of the
    chunked replay (flags bits [5:0]; 0 = automatic), which has no oracle counterpart."""
    pdict = oracle.paper_params() if pdict is None else pdict
    return xm.params(0, flags=chunks, **pdict)


def gpu_replay(ev: np.ndarray, off: np.ndarray, pdict: dict | None = None, series: bool = True, chunks: int = 0):
    """Replay on cuda:0 via xmem_replay_batch_ex; returns (results structured array, series or None)."""
    import torch

    dev = torch.device("cuda:0")
    e = torch.from_numpy(np.ascontiguousarray(ev, dtype=np.uint64).view(np.int64)).to(dev)
    o = torch.from_numpy(np.ascontiguousarray(off, dtype=np.int64)).to(dev)
    out, ser = binding.replay(e, o, gpu_params(pdict, chunks), series=series)
    torch.cuda.synchronize()
    res = binding.to_numpy(out)
    s = ser.cpu().numpy() if ser is not None else None
    del e, o, out, ser
    return res, s


def compare(gres, ores, traces=None, what=""):
    """Assert equality of every result field; report the first mismatching trace."""
    assert len(gres) == len(ores), (len(gres), len(ores))
    for f in FIELDS:
        a = np.asarray(gres[f], dtype=np.int64)
        b = np.asarray(ores[f], dtype=np.int64)
        bad = np.flatnonzero(a != b)
        if bad.size:
            t = int(bad[0])
            row_g = {k: int(gres[k][t]) for k in FIELDS}
            row_o = {k: int(ores[k][t]) for k in FIELDS}
            extra = f" trace={traces[t]}" if traces is not None and len(traces[t]) < 40 else ""
            raise AssertionError(f"{what}: field {f} differs in {bad.size} traces; first t={t}\n gpu={row_g}\n "
                                 f"oracle={row_o}{extra}")


def compare_series(gser, oser, off, what=""):
    bad = np.flatnonzero(gser != oser)
    if bad.size:
        e = int(bad[0])
        t = int(np.searchsorted(off, e, side="right") - 1)
        raise AssertionError(f"{what}: series differs at {bad.size} events; first global event {e} "
                             f"(trace {t}, local {e - off[t]}): gpu={int(gser[e])} oracle={int(oser[e])}")


def check(ev, off, pdict=None, series=True, threads=16, what="", traces=None, chunks=0):
    """GPU vs oracle on a whole batch, results and (optionally) the full series."""
    log(f"[gpu-parity] {what}: {len(off) - 1} traces, {len(ev)} events, chunks={chunks}")
    gres, gser = gpu_replay(ev, off, pdict, series=series, chunks=chunks)
    rc, ores, oser = oracle.replay(ev, off, pdict, series=series, threads=threads)
    assert rc == 0
    compare(gres, ores, traces, what)
    if series:
        compare_series(gser, oser, off, what)
    return gres, ores
