"""Host-side parts of bench.py, on the CPU: the one-GPU rule of its command line, and the readers
that take a kernel's measured HBM traffic and scalar issue from the committed rocprofv3
summaries (matched by workload and by the sha256 of the kernel source)."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def write_summary(path, lines):
    with open(path, "w") as f:
        f.write("# a summary as the profiling script writes it\n")
        f.write("\n".join(lines) + "\n")


def test_traffic_reader_scales_and_matches_source(tmp_path, monkeypatch):
    bench = load_bench()
    src = tmp_path / "kernel.hip"
    src.write_text("__global__ void k() {}\n")
    sha = bench.source_sha256(str(src))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    write_summary(tmp_path / "hbm_traffic_a.txt",
                  ["workload_key: w1", f"source_sha256: {sha}", "fetch_kib_per_launch: 100",
                   "write_kib_per_launch: 30", "fetch_factor: 2.00", "write_factor: 1.00"])
    write_summary(tmp_path / "hbm_traffic_b.txt",
                  ["workload_key: w2", "source_sha256: 0", "fetch_kib_per_launch: 1",
                   "write_kib_per_launch: 1", "fetch_factor: 1.00", "write_factor: 1.00"])
    assert bench.measured_traffic("w1", str(src)) == (100 * 2.0 + 30 * 1.0) * 1024.0
    assert bench.measured_traffic("w2", str(src)) is None  # taken from another source
    assert bench.measured_traffic("w3", str(src)) is None  # no summary for that workload
    src.write_text("__global__ void k() { /* changed */ }\n")
    assert bench.measured_traffic("w1", str(src)) is None  # the kernel changed since


def test_issue_reader_matches_workload_and_source(tmp_path, monkeypatch):
    bench = load_bench()
    src = tmp_path / "kernel.hip"
    src.write_text("x\n")
    sha = bench.source_sha256(str(src))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    write_summary(tmp_path / "pmc_a.txt", ["counter  per launch", "issue_key: w1", f"source_sha256: {sha}",
                                           "salu_per_event: 55.180", "valu_per_event: 40.794"])
    assert bench.measured_issue("w1", str(src)) == 55.18
    assert bench.measured_issue("w2", str(src)) is None
    src.write_text("y\n")
    assert bench.measured_issue("w1", str(src)) is None


def test_committed_summaries_parse():
    """Every committed traffic or issue summary carries the keys its reader needs."""
    bench = load_bench()
    import glob
    for path in glob.glob(os.path.join(bench.PROFILES, "hbm_traffic_*.txt")) + \
            glob.glob(os.path.join(bench.PROFILES, "pmc_*.txt")):
        kv = {}
        with open(path) as f:
            for ln in f:
                if ":" in ln and not ln.startswith("#"):
                    k, v = ln.split(":", 1)
                    kv[k.strip()] = v.strip()
        if os.path.basename(path).startswith("hbm_traffic_"):
            for k in ("workload_key", "source_sha256", "fetch_kib_per_launch", "write_kib_per_launch",
                      "fetch_factor", "write_factor"):
                assert k in kv, (path, k)
            assert float(kv["fetch_factor"]) > 0 and float(kv["write_factor"]) > 0
        elif "issue_key" in kv:
            assert "source_sha256" in kv and float(kv["salu_per_event"]) > 0, path
