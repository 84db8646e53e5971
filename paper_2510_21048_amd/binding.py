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
        lib.xmem_replay_batch_noalloc.argtypes = [vp, vp, i64, i64, P, vp, vp, vp]
        lib.xmem_replay_batch_noalloc.restype = ctypes.c_int
        lib.xmem_oom_predicted.argtypes = [vp, i64, i64, vp, vp]
        lib.xmem_oom_predicted.restype = ctypes.c_int
        lib.xmem_strerror.argtypes = [ctypes.c_int]
        lib.xmem_strerror.restype = ctypes.c_char_p
        lib.xmem_prep_workspace_bytes.argtypes = [i64, i64]
        lib.xmem_prep_workspace_bytes.restype = ctypes.c_size_t
        lib.xmem_lifecycles.argtypes = [vp, vp, vp, i64, i64, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        lib.xmem_lifecycles.restype = ctypes.c_int
        lib.xmem_orchestrate.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        lib.xmem_attribute.restype = ctypes.c_int
        lib.xmem_attribute.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        lib.xmem_orchestrate.restype = ctypes.c_int
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


XMEM_NOALLOC_SCRATCH_BYTES = 256 << 20
XMEM_ESCRATCH = -6


def xmem_replay_batch_noalloc(d_events, d_offsets, n_traces: int, total_events: int, p: XmemParams, d_out,
                              d_series, stream) -> int:
    return load().xmem_replay_batch_noalloc(
        _ptr(d_events), _ptr(d_offsets), int(n_traces), int(total_events), ctypes.byref(p), _ptr(d_out),
        _ptr(d_series), _ptr(stream) if not isinstance(stream, int) else stream)


XMEM_PHASE_EVENTS = 8
PHASES = ["plan", "stream", "chunk_plan", "replay", "fallback", "finalize", "series"]


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


def xmem_oom_predicted(d_results, n_traces: int, m_max_bytes: int, d_flags, stream) -> int:
    return load().xmem_oom_predicted(_ptr(d_results), int(n_traces), int(m_max_bytes), _ptr(d_flags),
                                     _ptr(stream) if not isinstance(stream, int) else stream)


def oom_predicted(results, m_max_bytes: int, stream=None):
    """Eq. (1) of Section 4.1 on replay results held in a torch CUDA tensor ([T, 96] uint8, as
    ``replay`` returns them): an int32 CUDA tensor of per-trace flags (1 OOM predicted, 0 not,
    -1 no estimate).  Raises XmemError on a call-level error."""
    import torch

    T = results.shape[0]
    flags = torch.empty(T, dtype=torch.int32, device=results.device)
    st = torch.cuda.current_stream(results.device).cuda_stream if stream is None else stream
    rc = xmem_oom_predicted(results, T, m_max_bytes, flags, st)
    if rc != XMEM_OK:
        raise XmemError(f"xmem_oom_predicted: {xmem_strerror(rc)} ({rc})")
    return flags


def to_numpy(results) -> np.ndarray:
    """Results tensor (or bytes) -> numpy structured array with RESULT_DTYPE."""
    arr = results.cpu().numpy() if hasattr(results, "cpu") else np.asarray(results)
    return np.ascontiguousarray(arr).reshape(-1).view(RESULT_DTYPE)


# ---------------------------------------------------------------- trace preparation (include/xmem_prep.h)
XMEM_PERSISTENT = INT64_MAX
XMEM_CAT_OTHER, XMEM_CAT_PARAMETER, XMEM_CAT_BATCH, XMEM_CAT_GRADIENT, XMEM_CAT_OPTIMIZER = 0, 1, 2, 3, 4
RAW_EVENT_DTYPE = np.dtype([("ts", np.int64), ("addr", np.uint64), ("bytes", np.int64)])
BLOCK_DTYPE = np.dtype([("size", np.int64), ("t_alloc", np.int64), ("t_free", np.int64),
                        ("category", np.int32), ("pad", np.int32)])
WINDOW_DTYPE = np.dtype([("start", np.int64), ("end", np.int64), ("parent", np.int32), ("kind", np.int32),
                         ("category", np.int32), ("pad", np.int32)])
XMEM_WIN_COMPONENT, XMEM_WIN_OPERATOR = 0, 1


def xmem_prep_workspace_bytes(n_traces: int, n_records: int) -> int:
    return load().xmem_prep_workspace_bytes(int(n_traces), int(n_records))


def xmem_lifecycles(d_raw, d_category, d_raw_offsets, n_traces: int, total_raw: int, d_blocks, d_block_offsets,
                    d_unmatched, d_status, d_workspace, workspace_bytes: int, stream) -> int:
    return load().xmem_lifecycles(_ptr(d_raw), _ptr(d_category), _ptr(d_raw_offsets), int(n_traces), int(total_raw),
                                  _ptr(d_blocks), _ptr(d_block_offsets), _ptr(d_unmatched), _ptr(d_status),
                                  _ptr(d_workspace), int(workspace_bytes), _ptr(stream))


def xmem_attribute(d_blocks, d_block_offsets, n_traces: int, total_blocks: int, d_windows, d_window_offsets,
                   total_windows: int, d_kept, d_kept_offsets, d_block_window, d_status, d_workspace,
                   workspace_bytes: int, stream) -> int:
    return load().xmem_attribute(_ptr(d_blocks), _ptr(d_block_offsets), int(n_traces), int(total_blocks),
                                 _ptr(d_windows), _ptr(d_window_offsets), int(total_windows), _ptr(d_kept),
                                 _ptr(d_kept_offsets), _ptr(d_block_window), _ptr(d_status), _ptr(d_workspace),
                                 int(workspace_bytes), _ptr(stream))


def xmem_orchestrate(d_blocks, d_block_offsets, n_traces: int, total_blocks: int, d_steps, d_step_offsets,
                     d_zero_grads, d_zg_offsets, d_events, d_event_offsets, d_status, d_workspace,
                     workspace_bytes: int, stream) -> int:
    return load().xmem_orchestrate(_ptr(d_blocks), _ptr(d_block_offsets), int(n_traces), int(total_blocks),
                                   _ptr(d_steps), _ptr(d_step_offsets), _ptr(d_zero_grads), _ptr(d_zg_offsets),
                                   _ptr(d_events), _ptr(d_event_offsets), _ptr(d_status), _ptr(d_workspace),
                                   int(workspace_bytes), _ptr(stream))


def _stream(dev, stream):
    import torch
    return torch.cuda.current_stream(dev).cuda_stream if stream is None else stream


def lifecycles(raw, raw_offsets, category=None, workspace=None, stream=None):
    """Lifecycle pairing on torch CUDA tensors: raw is uint8 [N, 24] (RAW_EVENT_DTYPE records),
    offsets int64 [T+1], category int32 [N] or None.
    Returns (blocks uint8 [N, 32], block_offsets int64 [T+1], unmatched int64 [T], status int32 [1])."""
    import torch
    dev = raw_offsets.device
    T = raw_offsets.numel() - 1
    N = raw.numel() // RAW_EVENT_DTYPE.itemsize
    blocks = torch.empty((max(N, 1), BLOCK_DTYPE.itemsize), dtype=torch.uint8, device=dev)
    boff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    unm = torch.empty(max(T, 1), dtype=torch.int64, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    need = xmem_prep_workspace_bytes(T, N)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    rc = xmem_lifecycles(raw if N else None, category, raw_offsets, T, N, blocks, boff, unm, status, workspace,
                         workspace.numel(), _stream(dev, stream))
    if rc != XMEM_OK:
        raise XmemError(f"xmem_lifecycles: {xmem_strerror(rc)} ({rc})")
    return blocks, boff, unm, status


def attribute(blocks, block_offsets, windows, window_offsets, workspace=None, stream=None):
    """Time-window attribution on torch CUDA tensors: blocks uint8 [>=B, 32] (B = block_offsets[-1]),
    windows uint8 [W, 32] (WINDOW_DTYPE records), both with int64 CSR offsets.
    Returns (kept uint8 [B, 32], kept_offsets int64 [T+1], block_window int32 [B], status int32 [1])."""
    import torch
    dev = block_offsets.device
    T = block_offsets.numel() - 1
    B = int(block_offsets[-1].item()) if T >= 0 else 0
    W = windows.numel() // WINDOW_DTYPE.itemsize
    kept = torch.empty((max(B, 1), BLOCK_DTYPE.itemsize), dtype=torch.uint8, device=dev)
    koff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    bw = torch.empty(max(B, 1), dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    need = xmem_prep_workspace_bytes(T, max(B, W))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    rc = xmem_attribute(blocks if B else None, block_offsets, T, B, windows if W else None, window_offsets, W,
                        kept if B else None, koff, bw if B else None, status, workspace, workspace.numel(),
                        _stream(dev, stream))
    if rc != XMEM_OK:
        raise XmemError(f"xmem_attribute: {xmem_strerror(rc)} ({rc})")
    return kept, koff, bw, status


def orchestrate(blocks, block_offsets, steps, step_offsets, zero_grads, zg_offsets, workspace=None, stream=None):
    """Orchestration on torch CUDA tensors: blocks uint8 [>=B, 32] (BLOCK_DTYPE records, B =
    block_offsets[-1] read by the caller as total), the marker arrays int64 CSR.
    Returns (events int64 [2B] (uint64 words), event_offsets int64 [T+1], status int32 [1])."""
    import torch
    dev = block_offsets.device
    T = block_offsets.numel() - 1
    B = int(block_offsets[-1].item()) if T >= 0 else 0
    events = torch.empty(max(2 * B, 1), dtype=torch.int64, device=dev)
    eoff = torch.empty(T + 1, dtype=torch.int64, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    need = xmem_prep_workspace_bytes(T, 2 * B)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    rc = xmem_orchestrate(blocks if B else None, block_offsets, T, B, steps, step_offsets, zero_grads, zg_offsets,
                          events if B else None, eoff, status, workspace, workspace.numel(), _stream(dev, stream))
    if rc != XMEM_OK:
        raise XmemError(f"xmem_orchestrate: {xmem_strerror(rc)} ({rc})")
    return events, eoff, status
