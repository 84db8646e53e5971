#!/usr/bin/env python3
"""Benchmark: allocator-trace events replayed per second on one MI355X.

One step = one xmem_replay_batch_ex call over the whole batch (plan, event-
stream pass, allocator replay, finalisation) with inputs already resident in
HBM.  Default workload: 256 ResNet-50-like traces of 65,536 events each
(batch 16..512), paper allocator parameters, unbounded capacity.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "allocator trace events replayed/sec (1 GPU) + % HBM roofline; peak exact-match"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
EVENT_BYTES = 8                 # algorithmic bytes per event: the event word, read once
SERIES_BYTES = 8                # plus one int64 written per event when the series is requested
SOURCE = os.path.join(ROOT, "paper_2510_21048_amd", "csrc", "xmem_replay.hip")
PROFILES = os.path.join(ROOT, "profiles")
COPY_CAL_BYTES = 1 << 30        # --copy-calibration: one kernel reading and writing 1 GiB each


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded (one runtime per process)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            h = ctypes.c_void_p()
            if self.lib.hipEventCreate(ctypes.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            out.append(h.value)
        return out

    def ms(self, a, b):
        f = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(f), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return f.value

    def destroy(self, evs):
        for h in evs:
            self.lib.hipEventDestroy(ctypes.c_void_p(h))


def source_sha256():
    import hashlib
    with open(SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload_key):
    """HBM bytes per launch of the replay phase, from the rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary committed for this workload, scaled by the copy-kernel calibration it records.
    None when no summary matches the workload or the kernel source changed since it was taken."""
    import glob
    sha = source_sha256()
    for path in sorted(glob.glob(os.path.join(PROFILES, "hbm_traffic_*.txt"))):
        kv = {}
        with open(path) as f:
            for ln in f:
                if ":" in ln and not ln.startswith("#"):
                    k, v = ln.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("workload_key") != workload_key or kv.get("source_sha256") != sha:
            continue
        fetch = float(kv["fetch_kib_per_launch"]) * float(kv["fetch_factor"])
        write = float(kv["write_kib_per_launch"]) * float(kv["write_factor"])
        return (fetch + write) * 1024.0
    return None


def copy_calibration():
    """A plain copy of known size, run under rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE to scale
    those counters to bytes."""
    import torch
    n = COPY_CAL_BYTES // 4
    x = torch.ones(n, dtype=torch.int32, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": COPY_CAL_BYTES, "copy_calibration_bytes_written": COPY_CAL_BYTES,
                      "launches": 3, "check": int(y[n - 1].item())}), flush=True)


def bench_prep(n_traces, n_events, steps, warmup, cpu_seconds, want_cpu):
    """Trace preparation on a batch of synthetic profiler streams: lifecycle pairing and
    time-window attribution (Section 3.2), then orchestration (Section 3.3).  n_traces traces of
    n_events raw allocator events with their execution windows, tiled from 16 generated training
    profiles; the roles come from the attribution.  Returns the "prep" object of the JSON line."""
    import numpy as np
    import torch

    import oracle
    import paper_2510_21048_amd as xm
    from tracegen import prep

    base = min(16, n_traces)
    gen = prep.batch_profiles(base, n_events, windows=True)
    raw0, _cat0, roff0, st0, soff0, zg0, zoff0, win0, woff0 = gen
    reps = (n_traces + base - 1) // base

    def tile(arr, off):
        parts = ([arr[off[t]:off[t + 1]] for t in range(base)] * reps)[:n_traces]
        o = np.zeros(n_traces + 1, np.int64)
        o[1:] = np.cumsum([len(x) for x in parts])
        return np.concatenate(parts), o

    raw, roff = tile(raw0, roff0)
    st, soff = tile(st0, soff0)
    zg, zoff = tile(zg0, zoff0)
    win, woff = tile(win0, woff0)
    dev = torch.device("cuda:0")
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_raw, d_roff = d(raw.view(np.uint8)), d(roff)
    d_win, d_woff = d(win.view(np.uint8)), d(woff)
    d_st, d_soff, d_zg, d_zoff = d(st), d(soff), d(zg), d(zoff)
    N, T, W = len(raw), n_traces, len(win)
    blocks = torch.empty((N, xm.BLOCK_DTYPE.itemsize), dtype=torch.uint8, device=dev)
    kept = torch.empty((N, xm.BLOCK_DTYPE.itemsize), dtype=torch.uint8, device=dev)
    boff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    koff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    unm = torch.empty(T, dtype=torch.int64, device=dev)
    status = torch.zeros(3, dtype=torch.int32, device=dev)
    events = torch.empty(2 * N, dtype=torch.int64, device=dev)
    eoff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    ws_bytes = xm.xmem_prep_workspace_bytes(T, max(2 * N, W))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    hip = HipEvents()
    hip.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    sizes = {}

    def mark(evs, i):
        if evs:
            hip.lib.hipEventRecord(ctypes.c_void_p(evs[i]), ctypes.c_void_p(stream.cuda_stream))

    def run(evs=None):
        mark(evs, 0)
        rc1 = xm.xmem_lifecycles(d_raw, None, d_roff, T, N, blocks, boff, unm, status[0:], ws, ws_bytes,
                                 stream.cuda_stream)
        mark(evs, 1)
        # block and kept counts live on the device; the host passes the sizes found by the
        # untimed first run (identical inputs give identical counts)
        rc2 = xm.xmem_attribute(blocks, boff, T, sizes["blocks"], d_win, d_woff, W, kept, koff, None,
                                status[1:], ws, ws_bytes, stream.cuda_stream)
        mark(evs, 2)
        rc3 = xm.xmem_orchestrate(kept, koff, T, sizes["kept"], d_st, d_soff, d_zg, d_zoff, events, eoff,
                                  status[2:], ws, ws_bytes, stream.cuda_stream)
        mark(evs, 3)
        if rc1 or rc2 or rc3:
            raise RuntimeError(f"prep: {xm.xmem_strerror(rc1 or rc2 or rc3)}")

    xm.xmem_lifecycles(d_raw, None, d_roff, T, N, blocks, boff, unm, status[0:], ws, ws_bytes, stream.cuda_stream)
    torch.cuda.synchronize()
    sizes["blocks"] = int(boff[-1].item())
    xm.xmem_attribute(blocks, boff, T, sizes["blocks"], d_win, d_woff, W, kept, koff, None, status[1:], ws,
                      ws_bytes, stream.cuda_stream)
    torch.cuda.synchronize()
    sizes["kept"] = int(koff[-1].item())
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    evs_all = [hip.create(4) for _ in range(steps)]
    t0 = time.perf_counter()
    for k in range(steps):
        run(evs_all[k])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    names = ["lifecycles", "attribute", "orchestrate"]
    stage_ms = {nm: float(np.mean([hip.ms(e[i], e[i + 1]) for e in evs_all])) for i, nm in enumerate(names)}
    for e in evs_all:
        hip.destroy(e)
    n_words = int(eoff[-1].item())
    g_eoff = eoff.cpu().numpy()
    g_ev = events.cpu().numpy().view(np.uint64)[:n_words]
    g_koff = koff.cpu().numpy()
    g_kept = kept.cpu().numpy().reshape(-1).view(xm.BLOCK_DTYPE)[: int(g_koff[-1])]

    def oracle_chain():  # on the 16 generated profiles; trace t of the batch is a copy of profile t % 16
        rc, wb, wbo, _ = oracle.lifecycles(raw0.view(oracle.RAW_DTYPE), roff0)
        rc2, wk, wko, _ = oracle.attribute(wb, wbo, win0.view(oracle.WINDOW_DTYPE), woff0)
        rc3, wev, weo = oracle.orchestrate(wk, wko, st0, soff0, zg0, zoff0)
        return rc | rc2 | rc3, wk, wko, wev, weo

    t1 = time.perf_counter()
    rc, w_kept, w_koff, w_ev, w_eoff = oracle_chain()
    cpu_once = time.perf_counter() - t1
    exact = rc == 0 and int(status.cpu().numpy().max()) == 0
    for t in range(T if exact else 0):
        b_ = t % base
        exact = exact and g_kept[g_koff[t]:g_koff[t + 1]].tobytes() == w_kept[w_koff[b_]:w_koff[b_ + 1]].tobytes() \
            and np.array_equal(g_ev[g_eoff[t]:g_eoff[t + 1]], w_ev[w_eoff[b_]:w_eoff[b_ + 1]])
    nb, nk = sizes["blocks"], sizes["kept"]
    alg = {"lifecycles": N * 24 + nb * 32,          # raw events read, blocks written
           "attribute": nb * 32 + W * 32 + nk * 32,  # blocks and windows read, kept blocks written
           "orchestrate": nk * 32 + n_words * 8}      # kept blocks read, event words written
    cpu = None
    if want_cpu:
        reps_cpu, tot = 1, cpu_once
        while tot < cpu_seconds:
            t1 = time.perf_counter()
            oracle_chain()
            tot += time.perf_counter() - t1
            reps_cpu += 1
        cpu = {"value": reps_cpu * len(raw0) / tot, "unit": "raw events/s", "cores": 1, "kind": "oracle",
               "sample": f"the {base} generated profiles ({len(raw0)} raw events, {len(win0)} windows) through the "
                         f"C++ oracle's lifecycle pairing, attribution (a scan of the trace's windows per block) "
                         f"and orchestration, {reps_cpu}x, one thread, {tot:.2f} s wall"}
    dom = max(stage_ms, key=stage_ms.get)
    achieved = alg[dom] / (stage_ms[dom] / 1e3) / 1e9
    return {
        "metric": "raw allocator events prepared/sec (lifecycle pairing + attribution + orchestration, 1 GPU)",
        "value": N / (wall if wall > 0 else 1e-9),
        "unit": "raw events/s",
        "ms_per_step": wall * 1e3,
        "stages_ms": stage_ms,
        "stages_hbm_frac": {k: alg[k] / (v / 1e3) / 1e9 / HBM_PEAK_GBS for k, v in stage_ms.items()},
        "config": {"workload": f"training profiler streams: {T} traces x {n_events} raw events with {W} execution "
                               f"windows (16 generated profiles tiled); {nb} blocks, {nk} attributed, "
                               f"{n_words} event words",
                   "traces": T, "raw_events": N, "windows": W, "blocks": nb, "kept_blocks": nk, "event_words": n_words},
        "exact_match": bool(exact),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes_per_launch": alg[dom]},
        "cpu_baseline": cpu,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, help="workload configuration (1-5); 2 is the headline")
    ap.add_argument("--traces", type=int, default=None)
    ap.add_argument("--events", type=int, default=None)
    ap.add_argument("--series", action="store_true", help="also write the per-event reserved series")
    ap.add_argument("--chunks", type=int, default=0,
                    help="chunks per pool chain of the chunked replay (0 = chosen by the library, 1 = serial)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=1.5, help="minimum wall time of the oracle sample")
    ap.add_argument("--no-prep", action="store_true", help="skip the trace-preparation measurement")
    ap.add_argument("--prep-traces", type=int, default=128)
    ap.add_argument("--prep-events", type=int, default=65536)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (the scale for rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py: this build replays on one GPU only (asked for --gpus {args.gpus}); "
              "traces shard across GPUs with no exchange, but no multi-GPU path is built.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import tracegen
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding

    xm.load()
    assert torch.cuda.is_available(), "bench needs a GPU"
    dev = torch.device("cuda:0")
    nt_def, ne_def = tracegen.default_shape(args.config)
    nt = args.traces or nt_def
    ne = args.events or ne_def
    log(f"generating config {args.config} ({tracegen.NAMES[args.config]}): {nt} traces x {ne} events")
    ev_np, off_np = tracegen.generate(args.config, nt, ne)
    N = int(off_np[-1])
    ev = torch.from_numpy(ev_np.view(np.int64)).to(dev)
    off = torch.from_numpy(off_np).to(dev)
    p = xm.params(flags=args.chunks)
    ws_bytes = xm.xmem_workspace_bytes(nt, N, p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((nt, 96), dtype=torch.uint8, device=dev)
    ser = torch.empty(N, dtype=torch.int64, device=dev) if args.series else None
    stream = torch.cuda.current_stream(dev)
    hip = HipEvents()
    nph = xm.XMEM_PHASE_EVENTS

    def step(evs=None):
        rc = xm.xmem_replay_batch_ex_timed(ev, off, nt, N, p, out, ser, ws, ws_bytes, stream.cuda_stream, evs)
        if rc != 0:
            raise RuntimeError(f"xmem_replay_batch_ex_timed: {xm.xmem_strerror(rc)}")

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [hip.create(nph) for _ in range(args.steps)]
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    phase_ms = {name: [] for name in xm.PHASES}
    for evs in events:
        for i, name in enumerate(xm.PHASES):
            phase_ms[name].append(hip.ms(evs[i], evs[i + 1]))
    for evs in events:
        hip.destroy(evs)
    avg = {k: float(np.mean(v)) for k, v in phase_ms.items()}
    ms_per_step = wall * 1e3 / args.steps
    value = N / (ms_per_step / 1e3)
    dominant = max(avg, key=avg.get)
    alg_bytes = N * (EVENT_BYTES + (SERIES_BYTES if args.series else 0))
    achieved = alg_bytes / (avg[dominant] / 1e3) / 1e9
    log(f"{ms_per_step:.3f} ms/step, {value:.3e} events/s; phases (ms): " +
        ", ".join(f"{k}={v:.3f}" for k, v in avg.items()))

    # peak exact-match against the oracle on the whole benchmark batch
    res = binding.to_numpy(out)
    import oracle
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    log(f"oracle check with {threads} threads")
    t1 = time.perf_counter()
    rc, want, _ = oracle.replay(ev_np, off_np, oracle.paper_params(), threads=threads)
    first = time.perf_counter() - t1
    bad_traces = int(np.any(np.stack([res[f].astype(np.int64) != want[f].astype(np.int64)
                                      for f in binding.RESULT_FIELDS]), axis=0).sum())
    workload_key = f"config{args.config} {nt}x{ne} series={int(bool(args.series))} phase={dominant}"
    traffic = measured_traffic(workload_key)
    cpu = None
    if not args.no_cpu_baseline:
        reps, tot = 1, first
        while tot < args.cpu_seconds:
            t1 = time.perf_counter()
            oracle.replay(ev_np, off_np, oracle.paper_params(), threads=threads)
            tot += time.perf_counter() - t1
            reps += 1
        cpu = {"value": reps * N / tot, "unit": "events/s", "cores": threads, "kind": "oracle",
               "sample": f"the whole benchmark batch ({nt} traces x {ne} events) replayed {reps}x by the C++ oracle "
                         f"(std::set best-fit index), one trace per task, {threads} threads, {tot:.2f} s wall"}
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": f"{tracegen.NAMES[args.config]}: {nt} traces x {ne} events, paper allocator parameters, "
                        f"unbounded capacity" + (", reserved series written" if args.series else ""),
            "traces": nt, "events_per_trace": ne, "total_events": N, "series": bool(args.series),
            "chunks": args.chunks or "auto",
        },
        "exact_match": bad_traces == 0,
        "mismatched_traces": bad_traces,
        "phases_ms": avg,
        # each phase against HBM with the same algorithmic bytes (the event words, 8 B each, read
        # once; plus 8 B written per event for the series)
        "phases_hbm_frac": {k: (alg_bytes / (v / 1e3) / 1e9 / HBM_PEAK_GBS if v > 0 else None)
                            for k, v in avg.items() if k in ("stream", "replay")},
        "roofline": {
            "bound": "hbm",
            "kernel": {"replay": "replay phase: chunk planner + k_chunk_sched (k_replay_fast when serial)",
                       "stream": "k_stream + k_link_check", "plan": "k_plan", "finalize": "k_finalize",
                       "series": "k_series"}[dominant],
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": alg_bytes,
        },
        "cpu_baseline": cpu,
    }
    if not args.no_prep:
        log(f"trace preparation: {args.prep_traces} traces x {args.prep_events} raw events")
        line["prep"] = bench_prep(args.prep_traces, args.prep_events, args.steps, args.warmup, args.cpu_seconds,
                                  not args.no_cpu_baseline)
        log(f"prep: {line['prep']['ms_per_step']:.3f} ms/step, {line['prep']['value']:.3e} raw events/s, "
            f"exact {line['prep']['exact_match']}")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
