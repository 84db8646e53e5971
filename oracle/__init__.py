"""CPU oracle of the xMem Memory Simulator (Section 3.4) -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports, links or calls it.

The arithmetic lives in ``xmem_oracle.cpp`` (plain C++ with an ordered
``std::set`` per pool as the best-fit index); this module only builds it with
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
    if force or not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
        tmp = _LIB.with_suffix(".so.tmp")
        subprocess.run(
            ["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread", str(_SRC), "-o", str(tmp)],
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
        lib.xmem_oracle_validate_params.restype = ctypes.c_int
        lib.xmem_oracle_validate_params.argtypes = [ctypes.POINTER(OracleParams)]
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


def replay_one(events, params: dict | None = None, series: bool = True):
    """Convenience: one trace given as a list/array of event words."""
    ev = np.asarray(events, dtype=np.uint64)
    rc, out, ser = replay(ev, np.array([0, len(ev)], dtype=np.int64), params, series=series)
    assert rc == 0, rc
    return out[0], ser
