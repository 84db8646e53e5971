"""CPU oracle of the xMem Memory Simulator (Section 3.4) -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports, links or calls it.

The arithmetic lives in ``xmem_oracle.cpp`` (plain C++ with an ordered
``std::set`` per pool as the best-fit index) and, for the trace-preparation
steps upstream of the Simulator (Sections 3.2 and 3.3: lifecycle pairing and
orchestration), in ``xmem_prep_oracle.cpp``; this module only builds them with
g++ and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "xmem_oracle.cpp"
_SRC_PREP = _HERE / "xmem_prep_oracle.cpp"
_LIB = _HERE / "libxmem_oracle.so"

# status codes (same values as the public ABI)
T_OK, T_OOM, T_BAD_FREE, T_BAD_EVENT, T_OVERFLOW = 0, 1, 2, 3, 4

INT64_MAX = (1 << 63) - 1
MiB = 1 << 20


class OracleParams(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_uint32),
        ("flags", ctypes.c_uint32),
        ("round_bytes", ctypes.c_int64),
        ("small_max_bytes", ctypes.c_int64),
        ("small_segment_bytes", ctypes.c_int64),
        ("mid_segment_bytes", ctypes.c_int64),
        ("min_large_alloc_bytes", ctypes.c_int64),
        ("large_round_bytes", ctypes.c_int64),
        ("split_min_small_bytes", ctypes.c_int64),
        ("split_min_large_bytes", ctypes.c_int64),
        ("device_capacity_bytes", ctypes.c_int64),
    ]


RESULT_FIELDS = [
    "peak_allocated", "peak_reserved", "peak_allocated_event", "peak_reserved_event",
    "final_allocated", "final_reserved", "segments_created", "segments_released",
    "max_free_blocks_small", "max_free_blocks_large", "stop_event", "status",
]

# numpy view of the 96-byte result record
RESULT_DTYPE = np.dtype([(f, np.int64) for f in RESULT_FIELDS[:-1]] + [("status", np.int32), ("pad", np.int32)])
assert RESULT_DTYPE.itemsize == 96


def paper_params(**overrides) -> dict:
    """Values the paper states or exemplifies (Sections 2.2.1, 2.2.2, 3.4, 6.4)."""
    p = dict(
        round_bytes=512,
        small_max_bytes=1 * MiB,
        small_segment_bytes=2 * MiB,
        mid_segment_bytes=20 * MiB,
        min_large_alloc_bytes=10 * MiB,
        large_round_bytes=2 * MiB,
        split_min_small_bytes=512,
        split_min_large_bytes=512,
        device_capacity_bytes=INT64_MAX,
    )
    p.update(overrides)
    return p


def pytorch_like_params(**overrides) -> dict:
    """Paper values except that a large block is split only if >1 MiB remains."""
    return paper_params(split_min_large_bytes=MiB + 1, **overrides)


def build(force: bool = False) -> Path:
    """Compile the oracle with g++ -O2 (plain build, not tuned)."""
    newest = max(_SRC.stat().st_mtime, _SRC_PREP.stat().st_mtime)
    if force or not _LIB.exists() or _LIB.stat().st_mtime < newest:
        tmp = _LIB.with_suffix(".so.tmp")
        subprocess.run(
            ["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread", str(_SRC), str(_SRC_PREP), "-o", str(tmp)],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not _LIB.exists():
            build()
        lib = ctypes.CDLL(str(_LIB))
        lib.xmem_oracle_replay_batch.restype = ctypes.c_int
        lib.xmem_oracle_replay_batch.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(OracleParams),
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
        ]
        lib.xmem_oracle_oom_predicted.restype = ctypes.c_int
        lib.xmem_oracle_oom_predicted.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.xmem_oracle_validate_params.restype = ctypes.c_int
        lib.xmem_oracle_validate_params.argtypes = [ctypes.POINTER(OracleParams)]
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        lib.xmem_oracle_lifecycles.restype = ctypes.c_int
        lib.xmem_oracle_lifecycles.argtypes = [vp, vp, vp, i64, vp, vp, vp]
        lib.xmem_oracle_attribute.restype = ctypes.c_int
        lib.xmem_oracle_attribute.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp]
        lib.xmem_oracle_orchestrate.restype = ctypes.c_int
        lib.xmem_oracle_orchestrate.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp, vp]
        _lib = lib
    return _lib


def make_params(p: dict | None = None) -> OracleParams:
    p = paper_params() if p is None else p
    return OracleParams(abi_version=1, flags=0, **p)


def validate_params(p: dict) -> int:
    return _load().xmem_oracle_validate_params(ctypes.byref(make_params(p)))


def replay(events: np.ndarray, offsets: np.ndarray, params: dict | None = None,
           series: bool = False, threads: int = 1):
    """Replay a CSR batch of traces on the CPU.

    Returns (rc, results[n_traces] structured array, series int64[total] or None).
    """
    ev = np.ascontiguousarray(events, dtype=np.uint64)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    n = len(off) - 1
    out = np.zeros(max(n, 0), dtype=RESULT_DTYPE)
    ser = np.zeros(int(off[-1]) if n >= 0 else 0, dtype=np.int64) if series else None
    prm = make_params(params)
    rc = _load().xmem_oracle_replay_batch(
        ev.ctypes.data if ev.size else None, off.ctypes.data, n, ctypes.byref(prm),
        out.ctypes.data if n > 0 else None, ser.ctypes.data if (ser is not None and ser.size) else None,
        int(threads),
    )
    return rc, out, ser


def oom_predicted(results: np.ndarray, m_max: int):
    """Eq. (1) of Section 4.1 over replay results: 1 when a trace's estimated peak (its peak
    reserved bytes) exceeds m_max or its replay stopped with OOM, 0 when it does not, -1 when the
    replay stopped for another reason.  Returns (rc, flags int32[T])."""
    res = np.ascontiguousarray(results, dtype=RESULT_DTYPE)
    flags = np.zeros(len(res), dtype=np.int32)
    rc = _load().xmem_oracle_oom_predicted(res.ctypes.data if len(res) else None, len(res), int(m_max),
                                           flags.ctypes.data if len(res) else None)
    return rc, flags


def replay_one(events, params: dict | None = None, series: bool = True):
    """Convenience: one trace given as a list/array of event words."""
    ev = np.asarray(events, dtype=np.uint64)
    rc, out, ser = replay(ev, np.array([0, len(ev)], dtype=np.int64), params, series=series)
    assert rc == 0, rc
    return out[0], ser


# ------------------------------------------------------------------ trace preparation (Sections 3.2, 3.3)
PERSISTENT = INT64_MAX
CAT_OTHER, CAT_PARAMETER, CAT_BATCH, CAT_GRADIENT, CAT_OPTIMIZER = 0, 1, 2, 3, 4

# raw allocator instant event and memory-block records (same layouts as the public ABI)
RAW_DTYPE = np.dtype([("ts", np.int64), ("addr", np.uint64), ("bytes", np.int64)])
BLOCK_DTYPE = np.dtype([("size", np.int64), ("t_alloc", np.int64), ("t_free", np.int64),
                        ("category", np.int32), ("pad", np.int32)])
WINDOW_DTYPE = np.dtype([("start", np.int64), ("end", np.int64), ("parent", np.int32), ("kind", np.int32),
                         ("category", np.int32), ("pad", np.int32)])
WIN_COMPONENT, WIN_OPERATOR = 0, 1
assert RAW_DTYPE.itemsize == 24 and BLOCK_DTYPE.itemsize == 32 and WINDOW_DTYPE.itemsize == 32


def _ptr(a):
    return a.ctypes.data if a.size else None


def lifecycles(raw: np.ndarray, raw_off: np.ndarray, category: np.ndarray | None = None):
    """Pair raw allocator events into memory blocks (Section 3.2); a block takes the category of
    its allocation event (all 0 without `category`).
    Returns (rc, blocks[BLOCK_DTYPE], block_off int64[T+1], unmatched_frees int64[T])."""
    raw = np.ascontiguousarray(raw, dtype=RAW_DTYPE)
    cat = None if category is None else np.ascontiguousarray(category, dtype=np.int32)
    off = np.ascontiguousarray(raw_off, dtype=np.int64)
    T = len(off) - 1
    blocks = np.zeros(max(int(off[-1]), 0), dtype=BLOCK_DTYPE)
    boff = np.zeros(T + 1, dtype=np.int64)
    unm = np.zeros(T, dtype=np.int64)
    rc = _load().xmem_oracle_lifecycles(_ptr(raw), None if cat is None else _ptr(cat), off.ctypes.data, T,
                                        _ptr(blocks), boff.ctypes.data, _ptr(unm))
    return rc, blocks[:int(boff[-1])] if rc == 0 else blocks[:0], boff, unm


def attribute(blocks: np.ndarray, block_off: np.ndarray, windows: np.ndarray, window_off: np.ndarray):
    """Time-based attribution of blocks to operator windows (Section 3.2).
    Returns (rc, kept blocks[BLOCK_DTYPE], kept_off int64[T+1], block_window int32[B])."""
    blocks = np.ascontiguousarray(blocks, dtype=BLOCK_DTYPE)
    boff = np.ascontiguousarray(block_off, dtype=np.int64)
    win = np.ascontiguousarray(windows, dtype=WINDOW_DTYPE)
    woff = np.ascontiguousarray(window_off, dtype=np.int64)
    T = len(boff) - 1
    kept = np.zeros(max(int(boff[-1]), 0), dtype=BLOCK_DTYPE)
    koff = np.zeros(T + 1, dtype=np.int64)
    bw = np.zeros(max(int(boff[-1]), 0), dtype=np.int32)
    rc = _load().xmem_oracle_attribute(_ptr(blocks), boff.ctypes.data, T, _ptr(win), woff.ctypes.data, _ptr(kept),
                                       koff.ctypes.data, _ptr(bw))
    return rc, kept[:int(koff[-1])] if rc == 0 else kept[:0], koff, bw


def orchestrate(blocks: np.ndarray, block_off: np.ndarray, steps: np.ndarray, step_off: np.ndarray,
                zero_grads: np.ndarray, zg_off: np.ndarray):
    """Retime blocks by category and emit the Simulator's event words (Section 3.3).
    Returns (rc, events uint64[], event_off int64[T+1])."""
    blocks = np.ascontiguousarray(blocks, dtype=BLOCK_DTYPE)
    boff = np.ascontiguousarray(block_off, dtype=np.int64)
    st = np.ascontiguousarray(steps, dtype=np.int64)
    so = np.ascontiguousarray(step_off, dtype=np.int64)
    zg = np.ascontiguousarray(zero_grads, dtype=np.int64)
    zo = np.ascontiguousarray(zg_off, dtype=np.int64)
    T = len(boff) - 1
    ev = np.zeros(2 * max(int(boff[-1]), 0), dtype=np.uint64)
    eoff = np.zeros(T + 1, dtype=np.int64)
    rc = _load().xmem_oracle_orchestrate(_ptr(blocks), boff.ctypes.data, T, _ptr(st), so.ctypes.data, _ptr(zg),
                                         zo.ctypes.data, _ptr(ev), eoff.ctypes.data)
    return rc, ev[:int(eoff[-1])] if rc == 0 else ev[:0], eoff
