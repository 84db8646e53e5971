"""MI355X-native batched replay of tensor allocate/free traces through the
caching-allocator model of xMem's Memory Simulator (Section 3.4), and the
trace preparation upstream of it: lifecycle pairing of raw allocator events and
time-window attribution (Section 3.2), and orchestration into the Simulator's
event words (Section 3.3).

The compute lives in ``libxmem_replay.so`` (HIP, gfx950); this package is its
ctypes binding.  PyTorch only provides device memory and streams.
"""
from .binding import (  # noqa: F401
    RESULT_DTYPE, RESULT_FIELDS, XmemParams, XMEM_ABI_VERSION, XMEM_PRESET_PAPER, XMEM_PRESET_PYTORCH_LIKE,
    XmemError, lib_path, load, params, replay, xmem_default_params, xmem_replay_batch, xmem_replay_batch_ex,
    xmem_replay_batch_ex_timed, XMEM_PHASE_EVENTS, PHASES, to_numpy, oom_predicted, xmem_oom_predicted,
    xmem_replay_batch_noalloc, XMEM_NOALLOC_SCRATCH_BYTES, XMEM_ESCRATCH,
    xmem_strerror, xmem_validate_params, xmem_workspace_bytes,
    BLOCK_DTYPE, RAW_EVENT_DTYPE, WINDOW_DTYPE, XMEM_PERSISTENT, attribute, lifecycles, orchestrate, xmem_attribute,
    xmem_lifecycles, xmem_orchestrate, xmem_prep_workspace_bytes,
)
