"""ctypes binding of libxmem_replay.so (argument marshalling only).

Every step of the replay runs in the library's HIP kernels.  The functions
named ``xmem_*`` mirror the C ABI one to one and take raw device pointers
(ints) or torch CUDA tensors; ``replay`` is a convenience wrapper that
allocates outputs and workspace with torch and calls ``xmem_replay_batch_ex``
on the current torch stream.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import numpy as np

_LIB_PATH = Path(__file__).resolve().parent / "libxmem_replay.so"

XMEM_ABI_VERSION = 1
XMEM_PRESET_PAPER, XMEM_PRESET_PYTORCH_LIKE = 0, 1
XMEM_OK = 0
INT64_MAX = (1 << 63) - 1


class XmemParams(ctypes.Structure):
    """xmem_allocator_params (include/xmem.h)."""
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

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_ if f not in ("abi_version", "flags")}


RESULT_FIELDS = [
    "peak_allocated", "peak_reserved", "peak_allocated_event", "peak_reserved_event",
    "final_allocated", "final_reserved", "segments_created", "segments_released",
    "max_free_blocks_small", "max_free_blocks_large", "stop_event", "status",
]
RESULT_DTYPE = np.dtype([(f, np.int64) for f in RESULT_FIELDS[:-1]] + [("status", np.int32), ("reserved_", np.int32)])
assert RESULT_DTYPE.itemsize == 96


class XmemError(RuntimeError):
    pass


_lib = None


def lib_path() -> Path:
    return _LIB_PATH


def load():
    """Load the HIP library; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is None:
        if not _LIB_PATH.exists():
            raise XmemError(f"{_LIB_PATH} is missing: build it with paper_2510_21048_amd.build.build()")
        lib = ctypes.CDLL(str(_LIB_PATH))
        P = ctypes.POINTER(XmemParams)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        lib.xmem_default_params.argtypes = [P, ctypes.c_int]
        lib.xmem_default_params.restype = ctypes.c_int
        lib.xmem_validate_params.argtypes = [P]
        lib.xmem_validate_params.restype = ctypes.c_int
        lib.xmem_workspace_bytes.argtypes = [i64, i64, P]
        lib.xmem_workspace_bytes.restype = ctypes.c_size_t
        lib.xmem_replay_batch.argtypes = [vp, vp, i64, P, vp]
        lib.xmem_replay_batch.restype = ctypes.c_int
        lib.xmem_replay_batch_ex.argtypes = [vp, vp, i64, i64, P, vp, vp, vp, ctypes.c_size_t, vp]
        lib.xmem_replay_batch_ex.restype = ctypes.c_int
        lib.xmem_replay_batch_ex_timed.argtypes = [vp, vp, i64, i64, P, vp, vp, vp, ctypes.c_size_t, vp,
                                                   ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]
        lib.xmem_replay_batch_ex_timed.restype = ctypes.c_int
        lib.xmem_strerror.argtypes = [ctypes.c_int]
        lib.xmem_strerror.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def xmem_default_params(preset: int = XMEM_PRESET_PAPER) -> XmemParams:
    p = XmemParams()
    rc = load().xmem_default_params(ctypes.byref(p), int(preset))
    if rc != XMEM_OK:
        raise XmemError(xmem_strerror(rc))
    return p


def params(preset: int = XMEM_PRESET_PAPER, **overrides) -> XmemParams:
    """Defaults of a preset with some fields replaced (byte counts)."""
    p = xmem_default_params(preset)
    for k, v in overrides.items():
        setattr(p, k, int(v))
    return p


def xmem_validate_params(p: XmemParams) -> int:
    return load().xmem_validate_params(ctypes.byref(p))


def xmem_workspace_bytes(n_traces: int, total_events: int, p: XmemParams) -> int:
    return int(load().xmem_workspace_bytes(int(n_traces), int(total_events), ctypes.byref(p)))


def xmem_strerror(code: int) -> str:
    return load().xmem_strerror(int(code)).decode()


def xmem_replay_batch(d_events, d_offsets, n_traces: int, p: XmemParams, d_out) -> int:
    return load().xmem_replay_batch(_ptr(d_events), _ptr(d_offsets), int(n_traces), ctypes.byref(p), _ptr(d_out))


def xmem_replay_batch_ex(d_events, d_offsets, n_traces: int, total_events: int, p: XmemParams, d_out,
                         d_series, d_workspace, workspace_bytes: int, stream) -> int:
    return load().xmem_replay_batch_ex(
        _ptr(d_events), _ptr(d_offsets), int(n_traces), int(total_events), ctypes.byref(p), _ptr(d_out),
        _ptr(d_series), _ptr(d_workspace), int(workspace_bytes), _ptr(stream) if not isinstance(stream, int) else stream)


XMEM_PHASE_EVENTS = 6
PHASES = ["plan", "stream", "replay", "finalize", "series"]


def xmem_replay_batch_ex_timed(d_events, d_offsets, n_traces: int, total_events: int, p: XmemParams, d_out,
                               d_series, d_workspace, workspace_bytes: int, stream, phase_events) -> int:
    """phase_events: sequence of XMEM_PHASE_EVENTS hipEvent_t handles (ints) or None."""
    arr = None
    if phase_events is not None:
        arr = (ctypes.c_void_p * len(phase_events))(*phase_events)
    return load().xmem_replay_batch_ex_timed(
        _ptr(d_events), _ptr(d_offsets), int(n_traces), int(total_events), ctypes.byref(p), _ptr(d_out),
        _ptr(d_series), _ptr(d_workspace), int(workspace_bytes), _ptr(stream) if not isinstance(stream, int) else stream,
        arr, len(phase_events) if phase_events is not None else 0)


def replay(events, offsets, p: XmemParams | None = None, series: bool = False, workspace=None, stream=None):
    """Replay a CSR batch held in torch CUDA tensors (uint64 events as int64, int64 offsets).

    Returns (results: torch.uint8 CUDA tensor [T, 96], series: int64 CUDA tensor or None).
    Decode results with ``to_numpy``.  Raises XmemError on a call-level error.
    """
    import torch

    p = xmem_default_params() if p is None else p
    T = offsets.numel() - 1
    N = events.numel()
    dev = events.device
    out = torch.empty((max(T, 0), 96), dtype=torch.uint8, device=dev)
    ser = torch.empty(N, dtype=torch.int64, device=dev) if series else None
    need = xmem_workspace_bytes(T, N, p)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream(dev).cuda_stream if stream is None else stream
    rc = xmem_replay_batch_ex(events, offsets, T, N, p, out, ser, workspace, workspace.numel(), st)
    if rc != XMEM_OK:
        raise XmemError(f"xmem_replay_batch_ex: {xmem_strerror(rc)} ({rc})")
    return out, ser


def to_numpy(results) -> np.ndarray:
    """Results tensor (or bytes) -> numpy structured array with RESULT_DTYPE."""
    arr = results.cpu().numpy() if hasattr(results, "cpu") else np.asarray(results)
    return np.ascontiguousarray(arr).reshape(-1).view(RESULT_DTYPE)
