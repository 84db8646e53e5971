"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the CPU oracle (oracle/*.cpp) and the
trace generator (tracegen/tracegen.c), run on the CPU by a small driver (tests/sanitize/driver.cpp)
over every workload configuration, four parameter sets, one and four threads, malformed and
empty traces, the OOM prediction and the trace-preparation oracle.  A sanitizer report fails."""
import os
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc and g++")
def test_oracle_and_generator_under_sanitizers(tmp_path):
    tg = tmp_path / "tracegen.o"
    subprocess.run(["gcc", "-std=c11", *SAN, "-c", str(ROOT / "tracegen" / "tracegen.c"), "-o", str(tg)], check=True)
    exe = tmp_path / "driver"
    subprocess.run(["g++", "-std=c++17", *SAN, "-pthread", str(ROOT / "tests" / "sanitize" / "driver.cpp"),
                    str(ROOT / "oracle" / "xmem_oracle.cpp"), str(ROOT / "oracle" / "xmem_prep_oracle.cpp"), str(tg),
                    "-o", str(exe), "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-4000:]
    assert "driver ok" in r.stdout
