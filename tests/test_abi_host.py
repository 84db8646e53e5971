"""The C ABI on the host (no GPU needed): the library loads, exports every
function include/*.h declares, the struct layouts match the headers, and
every host-side argument check returns its code before any device work."""
import ctypes
import re
import subprocess
from pathlib import Path

import pytest

import paper_2510_21048_amd as xm
from paper_2510_21048_amd import binding

ROOT = Path(__file__).resolve().parents[1]
HEADERS = sorted((ROOT / "include").glob("*.h"))


def declared_functions():
    text = "\n".join(h.read_text() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s+(xmem_[a-z_]+)\s*\(", text, flags=re.M)
    inline = set(re.findall(r"static inline [^(]*\b(xmem_[a-z_]+)\s*\(", text))
    return sorted(set(names) - inline)


def test_header_declares_the_entry_points():
    assert declared_functions() == sorted([
        "xmem_default_params", "xmem_validate_params", "xmem_workspace_bytes", "xmem_replay_batch",
        "xmem_replay_batch_ex", "xmem_replay_batch_ex_timed", "xmem_strerror", "xmem_oom_predicted",
        "xmem_replay_batch_noalloc",
        "xmem_prep_workspace_bytes", "xmem_lifecycles", "xmem_attribute", "xmem_orchestrate"])


def test_library_exports_every_declared_symbol():
    lib = xm.load()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", str(xm.lib_path())], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (xmem_\w+)", out))
    assert set(declared_functions()) <= exported


def test_struct_layouts_match_header():
    src = r'''
#include <stddef.h>
#include <stdio.h>
#include "xmem.h"
#include "xmem_prep.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu\n", sizeof(xmem_allocator_params), sizeof(xmem_trace_result),
         offsetof(xmem_trace_result, stop_event), offsetof(xmem_trace_result, status),
         offsetof(xmem_allocator_params, device_capacity_bytes), sizeof(xmem_raw_event),
         offsetof(xmem_raw_event, bytes), sizeof(xmem_block), offsetof(xmem_block, category),
         sizeof(xmem_window), offsetof(xmem_window, category));
  return 0;
}
'''
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        c = Path(d) / "l.c"
        c.write_text(src)
        subprocess.run(["gcc", "-std=c99", f"-I{ROOT / 'include'}", str(c), "-o", str(Path(d) / "l")], check=True)
        got = subprocess.run([str(Path(d) / "l")], capture_output=True, text=True).stdout.split()
    assert [int(x) for x in got] == [
        ctypes.sizeof(xm.XmemParams), xm.RESULT_DTYPE.itemsize, xm.RESULT_DTYPE.fields["stop_event"][1],
        xm.RESULT_DTYPE.fields["status"][1], xm.XmemParams.device_capacity_bytes.offset,
        xm.RAW_EVENT_DTYPE.itemsize, xm.RAW_EVENT_DTYPE.fields["bytes"][1], xm.BLOCK_DTYPE.itemsize,
        xm.BLOCK_DTYPE.fields["category"][1], xm.WINDOW_DTYPE.itemsize, xm.WINDOW_DTYPE.fields["category"][1]]


def test_default_params_and_presets():
    p = xm.xmem_default_params()
    assert p.round_bytes == 512 and p.small_segment_bytes == 2 << 20 and p.mid_segment_bytes == 20 << 20
    assert p.split_min_large_bytes == 512 and p.device_capacity_bytes == (1 << 63) - 1
    q = xm.xmem_default_params(xm.XMEM_PRESET_PYTORCH_LIKE)
    assert q.split_min_large_bytes == (1 << 20) + 1
    assert xm.xmem_validate_params(p) == 0 and xm.xmem_validate_params(q) == 0
    with pytest.raises(xm.XmemError):
        xm.xmem_default_params(7)


@pytest.mark.parametrize("field,value", [
    ("round_bytes", 384), ("round_bytes", 0), ("small_max_bytes", 3 << 20), ("mid_segment_bytes", 5 << 20),
    ("split_min_small_bytes", 0), ("device_capacity_bytes", 0), ("large_round_bytes", 1000),
    ("abi_version", 2), ("flags", 64), ("flags", 65), ("flags", 1 << 31),
    ("small_segment_bytes", (1 << 41)),
])
def test_invalid_params_rejected(field, value):
    p = xm.xmem_default_params()
    setattr(p, field, value)
    assert xm.xmem_validate_params(p) == -1
    assert xm.xmem_workspace_bytes(1, 10, p) == 0
    # both replay forms reject before touching the device
    assert xm.xmem_replay_batch(8, 16, 1, p, 32) == -1
    assert xm.xmem_replay_batch_ex(8, 16, 1, 10, p, 32, None, 64, 1 << 20, None) == -1


def test_chunk_flags():
    """flags bits [5:0] request a chunk count (0 automatic, 1..63); the chunked replay
    needs per-chunk state, so the workspace grows with the count under unbounded capacity
    and does not change under a finite one (chunking is off there)."""
    sizes = []
    for k in range(0, 64):
        p = xm.params(0, flags=k)
        assert xm.xmem_validate_params(p) == 0
        sizes.append(xm.xmem_workspace_bytes(4, 100000, p))
    # chunk states grow with the count; the paged chunk slots exist only while
    # 2 x traces x chunks <= 128 (here up to 16 chunks)
    assert sizes[1] < min(sizes[2:])
    assert sizes[2] < sizes[8] < sizes[16] and sizes[17] < sizes[32] < sizes[63] and sizes[17] < sizes[16]
    assert sizes[0] == sizes[63]  # 4 traces: the automatic count is the cap of 63
    assert xm.xmem_workspace_bytes(4096, 100000, xm.params(0)) > 0
    capped = [xm.xmem_workspace_bytes(4, 100000, xm.params(0, flags=k, device_capacity_bytes=1 << 40))
              for k in (0, 1, 8, 32)]
    assert len(set(capped)) == 1 and capped[0] == sizes[1]


def test_validation_agrees_with_oracle():
    import oracle
    for preset in (0, 1):
        p = xm.xmem_default_params(preset)
        for field, value in [("round_bytes", 1024), ("round_bytes", 768), ("small_max_bytes", 2 << 20),
                             ("small_max_bytes", (2 << 20) + 512), ("min_large_alloc_bytes", 21 << 20),
                             ("split_min_large_bytes", 1), ("split_min_large_bytes", 1 << 40),
                             ("split_min_large_bytes", (1 << 40) + 1), ("device_capacity_bytes", 1)]:
            q = xm.xmem_default_params(preset)
            setattr(q, field, value)
            assert xm.xmem_validate_params(q) == oracle.validate_params(q.as_dict()), (field, value)


def test_host_argument_errors_before_device_work():
    p = xm.xmem_default_params()
    ws = xm.xmem_workspace_bytes(3, 100, p)
    assert ws > 0
    assert xm.xmem_workspace_bytes(3, 200, p) > ws
    assert xm.xmem_workspace_bytes(-1, 5, p) == 0
    ex = xm.xmem_replay_batch_ex
    assert ex(8, None, 3, 100, p, 32, None, 256, ws, None) == -1        # no offsets
    assert ex(8, 16, 3, 100, p, None, None, 256, ws, None) == -1        # no output
    assert ex(None, 16, 3, 100, p, 32, None, 256, ws, None) == -1       # no events
    assert ex(8, 16, -1, 100, p, 32, None, 256, ws, None) == -1         # negative count
    assert ex(8, 16, 3, 100, p, 32, None, None, ws, None) == -5         # no workspace
    assert ex(8, 16, 3, 100, p, 32, None, 256, ws - 1, None) == -5      # workspace too small
    assert ex(8, 16, 3, 100, p, 32, None, 256 + 8, ws, None) == -5      # misaligned
    assert ex(None, 16, 0, 0, p, None, None, None, 0, None) == 0        # empty batch: nothing to do
    assert ex(8, 16, 0, 5, p, None, None, None, 0, None) == -2          # events without traces
    assert xm.xmem_replay_batch_ex_timed(8, 16, 3, 100, p, 32, None, 256, ws, None, [1, 2, 3]) == -1  # too few events
    assert xm.xmem_replay_batch(8, None, 1, p, 32) == -1
    assert xm.xmem_replay_batch(8, 16, 0, p, None) == 0


def test_noalloc_host_argument_errors():
    """The no-allocation entry point checks its arguments and its size limit on the host, before
    it touches a device."""
    p = xm.xmem_default_params()
    f = xm.xmem_replay_batch_noalloc
    assert f(None, 16, 0, 0, p, None, None, None) == 0               # empty batch: nothing to do
    assert f(8, None, 3, 100, p, 32, None, None) == -1               # no offsets
    assert f(8, 16, 3, 100, p, None, None, None) == -1               # no output
    assert f(None, 16, 3, 100, p, 32, None, None) == -1              # no events
    assert f(8, 16, 0, 5, p, None, None, None) == -2                 # events without traces
    assert f(8, 16, 3, 40_000_000, p, 32, None, None) == xm.XMEM_ESCRATCH  # past the fixed area
    assert f(8, 16, 3000, 4_000_000, p, 32, None, None) == xm.XMEM_ESCRATCH
    q = xm.params(round_bytes=3)
    assert f(8, 16, 3, 100, q, 32, None, None) == -1                 # invalid params
    assert "no-allocation" in xm.xmem_strerror(xm.XMEM_ESCRATCH)


def test_oom_predicted_host_argument_errors():
    f = xm.xmem_oom_predicted
    assert f(None, 0, 5, None, None) == 0          # nothing to do
    assert f(8, -1, 5, 16, None) == -1             # negative count
    assert f(8, 3, -1, 16, None) == -1             # negative m_max
    assert f(None, 3, 5, 16, None) == -1           # no results
    assert f(8, 3, 5, None, None) == -1            # no flags


def test_prep_host_argument_errors():
    ws = xm.xmem_prep_workspace_bytes(3, 100)
    assert ws > 0 and xm.xmem_prep_workspace_bytes(3, 1000) > ws
    assert xm.xmem_prep_workspace_bytes(-1, 5) == 0 and xm.xmem_prep_workspace_bytes(1, -5) == 0
    assert xm.xmem_prep_workspace_bytes(1, (1 << 32)) == 0
    life = xm.xmem_lifecycles
    assert life(8, None, None, 3, 100, 16, 24, None, 32, 256, ws, None) == -1      # no offsets
    assert life(None, None, 8, 3, 100, 16, 24, None, 32, 256, ws, None) == -1      # no events
    assert life(8, None, 8, 3, 100, 16, 24, None, None, 256, ws, None) == -1       # no status
    assert life(8, None, 8, -1, 100, 16, 24, None, 32, 256, ws, None) == -1        # negative count
    assert life(8, None, 8, 3, 1 << 33, 16, 24, None, 32, 256, ws, None) == -1     # too many records
    assert life(8, None, 8, 3, 100, 16, 24, None, 32, None, ws, None) == -5        # no workspace
    assert life(8, None, 8, 3, 100, 16, 24, None, 32, 256, ws - 1, None) == -5     # too small
    assert life(8, None, 8, 3, 100, 16, 24, None, 32, 264, ws, None) == -5         # misaligned
    ow = xm.xmem_prep_workspace_bytes(3, 200)
    orch = xm.xmem_orchestrate
    assert orch(8, None, 3, 100, 16, 24, 32, 40, 48, 56, 64, 256, ow, None) == -1  # no block offsets
    assert orch(8, 8, 3, 100, 16, None, 32, 40, 48, 56, 64, 256, ow, None) == -1   # no step offsets
    assert orch(None, 8, 3, 100, 16, 24, 32, 40, 48, 56, 64, 256, ow, None) == -1  # no blocks
    assert orch(8, 8, 3, 100, 16, 24, 32, 40, None, 56, 64, 256, ow, None) == -1   # no events
    assert orch(8, 8, 3, 100, 16, 24, 32, 40, 48, 56, 64, 256, ow - 1, None) == -5
    att = xm.xmem_attribute
    aw = xm.xmem_prep_workspace_bytes(3, 300)
    assert att(8, None, 3, 100, 16, 24, 300, 32, 40, None, 48, 256, aw, None) == -1   # no block offsets
    assert att(8, 8, 3, 100, None, 24, 300, 32, 40, None, 48, 256, aw, None) == -1    # no windows
    assert att(8, 8, 3, 100, 16, 24, 300, None, 40, None, 48, 256, aw, None) == -1    # no output
    assert att(8, 8, 3, -1, 16, 24, 300, 32, 40, None, 48, 256, aw, None) == -1       # negative count
    assert att(8, 8, 3, 100, 16, 24, 300, 32, 40, None, 48, 256, aw - 1, None) == -5  # sized by windows


def test_strerror_total():
    for code in (0, -1, -2, -3, -4, -5, -6, 1, 2, 3, 4, 5, 6, 99, -99):
        assert isinstance(xm.xmem_strerror(code), str) and xm.xmem_strerror(code)


def test_product_path_has_no_oracle_or_fallback():
    """The binding and the HIP source never reach the oracle or a CPU path."""
    for f in list((ROOT / "paper_2510_21048_amd").rglob("*.py")) + list((ROOT / "paper_2510_21048_amd").rglob("*.hip")):
        text = f.read_text()
        assert "oracle" not in text.replace("# no oracle", ""), f
        assert "import numpy" not in text or f.name == "binding.py", f
    src = (ROOT / "paper_2510_21048_amd" / "binding.py").read_text()
    assert "raise XmemError" in src and "is missing" in src


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "_LIB_PATH", tmp_path / "absent.so")
    with pytest.raises(xm.XmemError):
        binding.load()


def test_workspace_follows_the_grain_rules():
    """The automatic grain's special cases, seen through the workspace they size: a single trace
    of at most 4096 events is serial (no chunk state); one of 2^20 events or more takes 127
    chunks per pool on per-chunk paged sets (twice the slots of 63); two averaging 2^20 events
    take those slots at 63 chunks instead of the scheduler's queue; three or four keep the
    scheduler and hold the slots as well; five do not."""
    p = xm.params(0)
    W = lambda t, n: xm.xmem_workspace_bytes(t, n, p)
    assert W(1, 4096) < W(1, 4097) / 4                      # serial: no chunk state, no paged slots
    slot = (W(1, 1 << 20) - W(1, (1 << 20) - 1)) / (254 - 126)
    assert 8e6 < slot < 9e6                                  # 127 against 63 chunks, 8.4 MB a slot
    assert W(2, 2 << 20) - W(2, (2 << 20) - 2) > 240 * 8e6  # 2 x 2 x 63 slots
    assert W(3, 3 << 20) - W(3, (3 << 20) - 3) > 370 * 8e6  # 2 x 3 x 63 slots beside the queue
    assert W(5, 5 << 20) < 1e9                               # no paged slots past four traces
