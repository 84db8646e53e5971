"""Build libxmem_replay.so (replay and trace preparation) in-tree with hipcc for gfx950."""
from __future__ import annotations

import os
import subprocess
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
SRCS = [PKG / "csrc" / "xmem_replay.hip", PKG / "csrc" / "xmem_prep.hip"]
LIB = PKG / "libxmem_replay.so"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed fp32 instructions anywhere (none are needed: the path is integer-only)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def build() -> Path:
    """Compile every time it is called (the library is small: a few seconds)."""
    tmp = LIB.with_suffix(".so.tmp")
    cmd = [HIPCC, *FLAGS, f"-I{ROOT / 'include'}", *map(str, SRCS), "-o", str(tmp)]
    subprocess.run(cmd, check=True, stderr=subprocess.PIPE)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
