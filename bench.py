#!/usr/bin/env python3
"""Benchmark: allocator-trace events replayed per second on one MI355X.

One step = one xmem_replay_batch_ex call over the whole batch (plan, event-
stream pass, allocator replay, finalisation) with inputs already resident in
HBM.  Headline workload: 1,024 GPT-style traces of 262,144 events each (the
largest single-GPU configuration), paper allocator parameters, unbounded
capacity; the other four configurations are measured as rows of "configs".

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
SALU_PEAK_GIPS = 256 * 2.4        # scalar instructions, G/s: one per CU per cycle, 256 CUs at 2.4 GHz
EVENT_BYTES = 8                 # algorithmic bytes per event: the event word, read once
SERIES_BYTES = 8                # plus one int64 written per event when the series is requested
SOURCE = os.path.join(ROOT, "paper_2510_21048_amd", "csrc", "xmem_replay.hip")
PREP_SOURCE = os.path.join(ROOT, "paper_2510_21048_amd", "csrc", "xmem_prep.hip")
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


def source_sha256(path=SOURCE):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload_key, source=SOURCE):
    """HBM bytes per launch of the dominant kernel (or per call of a preparation stage), from the
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary committed for this workload, scaled by the
    copy-kernel calibration it records.  None when no summary matches the workload or the kernel
    source changed since it was taken."""
    import glob
    sha = source_sha256(source)
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


def measured_issue(workload_key, source=SOURCE):
    """Scalar (SALU) instructions the dominant kernel issues per event, from the rocprofv3
    SQ_INSTS_SALU summary committed for this workload; None when none matches the workload or the
    kernel source changed since it was taken."""
    import glob
    sha = source_sha256(source)
    for path in sorted(glob.glob(os.path.join(PROFILES, "pmc_*.txt"))):
        kv = {}
        with open(path) as f:
            for ln in f:
                if ":" in ln and not ln.startswith("#"):
                    k, v = ln.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("issue_key") == workload_key and kv.get("source_sha256") == sha and "salu_per_event" in kv:
            return float(kv["salu_per_event"])
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


def bench_prep(n_traces, n_events, steps, warmup, cpu_seconds, want_cpu, threads=1):
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
        from concurrent.futures import ThreadPoolExecutor

        def oracle_range(a, b):  # traces [a, b) of the whole batch through the oracle's three stages
            def sl(arr, o):
                return arr[o[a]:o[b]], o[a:b + 1] - o[a]
            r_, ro = sl(raw, roff)
            w_, wo = sl(win, woff)
            s_, so = sl(st, soff)
            z_, zo = sl(zg, zoff)
            rc_, wb, wbo, _ = oracle.lifecycles(r_.view(oracle.RAW_DTYPE), ro)
            rc2_, wk, wko, _ = oracle.attribute(wb, wbo, w_.view(oracle.WINDOW_DTYPE), wo)
            rc3_, _, _ = oracle.orchestrate(wk, wko, s_, so, z_, zo)
            return rc_ | rc2_ | rc3_

        # every thread takes a contiguous range of traces (the oracle's calls release the GIL)
        cuts = [T * i // threads for i in range(threads + 1)]
        reps_cpu, tot = 0, 0.0
        with ThreadPoolExecutor(threads) as pool:
            while tot < cpu_seconds or reps_cpu == 0:
                t1 = time.perf_counter()
                assert not any(pool.map(lambda i: oracle_range(cuts[i], cuts[i + 1]), range(threads)))
                tot += time.perf_counter() - t1
                reps_cpu += 1
        reps1, tot1 = 1, cpu_once
        while tot1 < cpu_seconds / 2:
            t1 = time.perf_counter()
            oracle_chain()
            tot1 += time.perf_counter() - t1
            reps1 += 1
        cpu = {"value": reps_cpu * N / tot, "unit": "raw events/s", "cores": threads, "kind": "oracle",
               "sample": f"the whole batch ({T} traces, {N} raw events, {W} windows) through the C++ oracle's "
                         f"lifecycle pairing, attribution (a scan of the trace's windows per block) and "
                         f"orchestration, {reps_cpu}x, {threads} threads each on a contiguous range of traces, "
                         f"{tot:.2f} s wall; one thread: the {base} generated profiles ({len(raw0)} raw events) "
                         f"{reps1}x, {tot1:.2f} s",
               "value_one_thread": reps1 * len(raw0) / tot1, "cpu_model": cpu_model(), "host_cpus": os.cpu_count()}
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
        # the dominant stage: one C-ABI call of some tens of launches (the sort's passes among them)
        "roofline": {"bound": "hbm", "kernel": f"xmem_{dom} (one call)", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(f"prep {T}x{n_events} stage={dom}", PREP_SOURCE),
                     "algorithmic_bytes_per_launch": alg[dom]},
        "cpu_baseline": cpu,
    }


# the library's choice of replay kernel (the chunk grain rule of include/xmem.h), to name the
# dominant kernel in the roofline object: serial replay, rounds for a few traces, or the scheduler
# (its windowed instance when there is a chain per 4 of its wavefronts: 24 per CU on gfx950)
def replay_kernel(n_traces, chunks, bounded=False, cus=256, n_events=0):
    """The replay kernel the library launches for this batch (its grain and instance rules)."""
    if bounded:
        return "k_replay_fast<2>"
    k = chunks
    if k == 0:
        if 1 <= n_traces <= 2 and n_events // n_traces >= 1 << 20:
            return "k_replay_combo rounds"  # 127 (one trace) or 63 (two) chunks per pool
        if n_traces == 1 and n_events <= 4096:
            return "k_replay_fast<1>"  # serial
        want = 64512 // n_traces
        k = 63 if want > 63 else want if want >= 16 else (2 if n_traces < 16384 else 1)
    k = min(k, 63)
    if k <= 1:
        return "k_replay_fast<1>"
    if 2 * n_traces * k <= 128:
        return "k_replay_combo rounds"
    windowed = 4 * 2 * n_traces >= 24 * cus
    if windowed and k < 16:
        return "k_chunk_sched_aged"
    return "k_chunk_sched<true>" if windowed else "k_chunk_sched<false>"


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_config(cfg, nt, ne, steps, warmup, series, chunks, cpu_seconds, want_cpu, threads):
    """Generate a workload, time `steps` replays of the whole batch (inputs resident in HBM),
    check every trace against the oracle, optionally time the oracle.  Returns a dict."""
    import numpy as np
    import torch

    import oracle
    import tracegen
    import paper_2510_21048_amd as xm
    from paper_2510_21048_amd import binding

    dev = torch.device("cuda:0")
    log(f"generating config {cfg} ({tracegen.NAMES[cfg]}): {nt} traces x {ne} events")
    ev_np, off_np = tracegen.generate(cfg, nt, ne)
    N = int(off_np[-1])
    ev = torch.from_numpy(ev_np.view(np.int64)).to(dev)
    off = torch.from_numpy(off_np).to(dev)
    p = xm.params(flags=chunks)
    ws_bytes = xm.xmem_workspace_bytes(nt, N, p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((nt, 96), dtype=torch.uint8, device=dev)
    ser = torch.empty(N, dtype=torch.int64, device=dev) if series else None
    stream = torch.cuda.current_stream(dev)
    hip = HipEvents()
    nph = xm.XMEM_PHASE_EVENTS

    def step(evs=None):
        rc = xm.xmem_replay_batch_ex_timed(ev, off, nt, N, p, out, ser, ws, ws_bytes, stream.cuda_stream, evs)
        if rc != 0:
            raise RuntimeError(f"xmem_replay_batch_ex_timed: {xm.xmem_strerror(rc)}")

    log(f"C{cfg}: warmup {warmup} steps")
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    events = [hip.create(nph) for _ in range(steps)]
    log(f"C{cfg}: timing {steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
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
    ms_per_step = wall * 1e3 / steps
    log(f"C{cfg}: {ms_per_step:.3f} ms/step, {N / (ms_per_step / 1e3):.3e} events/s; phases (ms): " +
        ", ".join(f"{k}={v:.3f}" for k, v in avg.items()))

    # exact match against the oracle on every trace of the batch; the same run, repeated, is the
    # oracle's multi-threaded baseline
    res = binding.to_numpy(out)
    log(f"C{cfg}: oracle check with {threads} threads")
    t1 = time.perf_counter()
    rc, want, _ = oracle.replay(ev_np, off_np, oracle.paper_params(), threads=threads)
    first = time.perf_counter() - t1
    bad_traces = int(np.any(np.stack([res[f].astype(np.int64) != want[f].astype(np.int64)
                                      for f in binding.RESULT_FIELDS]), axis=0).sum()) if rc == 0 else nt
    cpu = None
    if want_cpu:
        reps, tot = 1, first
        while tot < cpu_seconds:
            t1 = time.perf_counter()
            oracle.replay(ev_np, off_np, oracle.paper_params(), threads=threads)
            tot += time.perf_counter() - t1
            reps += 1
        # one thread on a bounded sample: the first traces of the batch, about 1/64 of it
        ns = max(1, nt // 64)
        s_off = off_np[:ns + 1]
        s_ev = ev_np[:int(s_off[-1])]
        reps1, tot1 = 0, 0.0
        while tot1 < cpu_seconds / 2 or reps1 == 0:
            t1 = time.perf_counter()
            oracle.replay(s_ev, s_off, oracle.paper_params(), threads=1)
            tot1 += time.perf_counter() - t1
            reps1 += 1
        cpu = {"value": reps * N / tot, "unit": "events/s", "cores": threads, "kind": "oracle",
               "sample": f"the whole batch ({nt} traces x {ne} events) replayed {reps}x by the C++ oracle "
                         f"(std::set best-fit index), one trace per task, {threads} threads, {tot:.2f} s wall; "
                         f"one thread: the first {ns} traces ({int(s_off[-1])} events) {reps1}x, {tot1:.2f} s",
               "value_one_thread": reps1 * int(s_off[-1]) / tot1,
               "cpu_model": cpu_model(), "host_cpus": os.cpu_count()}
    alg_bytes = N * EVENT_BYTES
    return {
        "cfg": cfg, "nt": nt, "ne": ne, "N": N, "ms_per_step": ms_per_step, "value": N / (ms_per_step / 1e3),
        "phases_ms": avg, "alg_bytes": alg_bytes,
        "phases_hbm_frac": {k: (alg_bytes / (avg[k] / 1e3) / 1e9 / HBM_PEAK_GBS if avg[k] > 0 else None)
                            for k in ("stream", "replay")},
        "exact_match": bad_traces == 0, "mismatched_traces": bad_traces,
        "kernel": replay_kernel(nt, chunks, cus=torch.cuda.get_device_properties(0).multi_processor_count, n_events=N),
        "cpu": cpu,
        "workload": f"{tracegen.NAMES[cfg]}: {nt} traces x {ne} events, paper allocator parameters, unbounded capacity"
                    + (", reserved series written" if series else ""),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3,
                    help="headline workload configuration (1-5); 3, the largest single-GPU one, by default")
    ap.add_argument("--configs", default="1,2,4,5",
                    help="other configurations measured as rows of the 'configs' object ('' for none)")
    ap.add_argument("--traces", type=int, default=None)
    ap.add_argument("--events", type=int, default=None)
    ap.add_argument("--series", action="store_true", help="also write the per-event reserved series")
    ap.add_argument("--chunks", type=int, default=0,
                    help="chunks per pool chain of the chunked replay (0 = chosen by the library, 1 = serial)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=2.0, help="minimum wall time of each oracle sample")
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

    import torch

    import tracegen
    import paper_2510_21048_amd as xm

    xm.load()
    assert torch.cuda.is_available(), "bench needs a GPU"
    threads = max(1, len(os.sched_getaffinity(0)))
    nt_def, ne_def = tracegen.default_shape(args.config)
    nt = args.traces or nt_def
    ne = args.events or ne_def
    h = run_config(args.config, nt, ne, args.steps, args.warmup, args.series, args.chunks, args.cpu_seconds,
                   not args.no_cpu_baseline, threads)
    rows = {}
    for c in [int(x) for x in args.configs.split(",") if x.strip()]:
        if c == args.config:
            continue
        cnt, cne = tracegen.default_shape(c)
        steps = 2 if c == 5 else min(args.steps, 5)
        r = run_config(c, cnt, cne, steps, 1, False, args.chunks, args.cpu_seconds, False, threads)
        rows[f"C{c}"] = {"workload": r["workload"], "ms_per_step": r["ms_per_step"], "events_per_s": r["value"],
                         "steps": steps, "phases_ms": r["phases_ms"], "phases_hbm_frac": r["phases_hbm_frac"],
                         "replay_kernel": r["kernel"], "exact_match": r["exact_match"],
                         "mismatched_traces": r["mismatched_traces"]}
        torch.cuda.empty_cache()
    dom = h["kernel"]
    kernel_ms = h["phases_ms"]["replay"]
    achieved = h["alg_bytes"] / (kernel_ms / 1e3) / 1e9
    workload_key = f"config{args.config} {nt}x{ne} series={int(bool(args.series))} kernel={dom}"
    salu = measured_issue(workload_key)
    issue = None
    if salu is not None:  # the kernel's binding resource: one scalar instruction per CU per cycle
        rate = salu * h["N"] / (kernel_ms / 1e3) / 1e9
        issue = {"resource": "SALU issue", "unit": "G instructions/s", "per_event": salu, "achieved": rate,
                 "peak": SALU_PEAK_GIPS, "frac": rate / SALU_PEAK_GIPS}
    line = {
        "metric": METRIC,
        "value": h["value"],
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": h["workload"], "traces": nt, "events_per_trace": ne, "total_events": h["N"],
            "series": bool(args.series), "chunks": args.chunks or "auto",
        },
        "exact_match": h["exact_match"],
        "mismatched_traces": h["mismatched_traces"],
        "phases_ms": h["phases_ms"],
        # each phase against HBM with the same algorithmic bytes: the event words, 8 B each, read once
        "phases_hbm_frac": h["phases_hbm_frac"],
        "roofline": {
            "bound": "hbm",
            "kernel": dom,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": measured_traffic(workload_key),
            "algorithmic_bytes_per_launch": h["alg_bytes"],
            "kernel_ms": kernel_ms,
            # context, not the roofline: the scalar instructions the kernel issues (committed SQ
            # counters) against the chip's scalar issue rate
            "issue": issue,
        },
        "cpu_baseline": h["cpu"],
        "configs": rows,
    }
    if not args.no_prep:
        log(f"trace preparation: {args.prep_traces} traces x {args.prep_events} raw events")
        line["prep"] = bench_prep(args.prep_traces, args.prep_events, args.steps, args.warmup, args.cpu_seconds,
                                  not args.no_cpu_baseline, threads)
        log(f"prep: {line['prep']['ms_per_step']:.3f} ms/step, {line['prep']['value']:.3e} raw events/s, "
            f"exact {line['prep']['exact_match']}")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
