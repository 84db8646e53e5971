"""Seeded synthetic allocate/free traces shaped like training workloads.

The input generators of both sides: the CPU oracle (tests, CPU baseline) and
the HIP library (tests, benchmark) replay the same traces.  The C source
(``tracegen.c``) only writes event words; it holds no allocator logic.

Configurations (events per trace x traces at full size):
  1  MLP, strictly LIFO, balanced             4,096 x 1
  2  ResNet-50-like CNN, batch 16..512       65,536 x 256
  3  GPT-style decoder, 144 shapes          262,144 x 1,024
  4  Monte Carlo perturbation of 3           65,536 x 4,096
  5  long GPT trace, ~62K free holes 16,777,216 x 1
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "tracegen.c"
_LIB = _HERE / "libtracegen.so"

NAMES = {1: "mlp_lifo", 2: "resnet50_batch_sweep", 3: "gpt_shapes", 4: "gpt_monte_carlo", 5: "gpt_long_fragmented"}


def build(force: bool = False) -> Path:
    if force or not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
        tmp = _LIB.with_suffix(".so.tmp")
        subprocess.run(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", str(_SRC), "-o", str(tmp), "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not _LIB.exists():
            build()
        lib = ctypes.CDLL(str(_LIB))
        lib.tg_trace.restype = ctypes.c_int
        lib.tg_trace.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64,
                                 ctypes.c_void_p, ctypes.c_int64]
        lib.tg_trace_stage.restype = ctypes.c_int
        lib.tg_trace_stage.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64,
                                       ctypes.c_void_p, ctypes.c_int64, ctypes.c_int]
        lib.tg_default_traces.restype = ctypes.c_int64
        lib.tg_default_traces.argtypes = [ctypes.c_int]
        lib.tg_default_events.restype = ctypes.c_int64
        lib.tg_default_events.argtypes = [ctypes.c_int]
        _lib = lib
    return _lib


def default_shape(config: int) -> tuple[int, int]:
    lib = _load()
    return int(lib.tg_default_traces(config)), int(lib.tg_default_events(config))


def generate(config: int, n_traces: int | None = None, events_per_trace: int | None = None,
             seed: int = 0, frag_pairs: int = -1, first_trace: int = 0, threads: int | None = None):
    """Traces first_trace .. first_trace+n_traces-1 of a configuration, CSR layout.

    Returns (events uint64[n_traces * events_per_trace], offsets int64[n_traces + 1]).
    """
    lib = _load()
    dn, de = default_shape(config)
    n = dn if n_traces is None else int(n_traces)
    m = de if events_per_trace is None else int(events_per_trace)
    ev = np.empty(n * m, dtype=np.uint64)
    off = np.arange(n + 1, dtype=np.int64) * m
    base = ev.ctypes.data

    def one(i):
        rc = lib.tg_trace(config, first_trace + i, seed, frag_pairs, base + i * m * 8, m)
        if rc != 0:
            raise ValueError(f"tracegen: config {config} trace {first_trace + i} length {m} not supported")

    nthr = threads or min(16, os.cpu_count() or 1)
    if n <= 1 or nthr <= 1:
        for i in range(n):
            one(i)
    else:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(one, range(n)))
    return ev, off


def trace_stage(config: int, trace_index: int, n_events: int, stage: int, seed: int = 0,
                frag_pairs: int = -1) -> np.ndarray:
    """One trace at a stage of configuration 4's post-processing: 0 the base trace, 1 after the
    size jitter, 2 after the free-run shuffle (the final trace).  Other configurations ignore
    the stage."""
    out = np.zeros(n_events, dtype=np.uint64)
    rc = _load().tg_trace_stage(config, trace_index, seed, frag_pairs, out.ctypes.data if n_events else None,
                                n_events, stage)
    if rc != 0:
        raise ValueError(f"tg_trace_stage({config}, {trace_index}, {n_events}, {stage}) = {rc}")
    return out
