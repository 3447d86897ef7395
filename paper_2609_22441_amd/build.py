"""Build the HIP library libccjoin.so for gfx950 (in-tree, no GPU needed)."""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
LIB = PKG / "libccjoin.so"
SOURCES = [CSRC / "cc_api.hip", CSRC / "join_kernels.hip", CSRC / "sort_kernels.hip",
           CSRC / "map_kernels.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # Packed fp32 instructions stay off (no arithmetic here needs them).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-fvisibility=hidden",
]


def build(out: Path = LIB, extra_flags=()) -> Path:
    out = Path(out)
    tmp = out.with_name(out.name + ".tmp")
    cmd = [HIPCC, *FLAGS, *extra_flags, f"-I{ROOT / 'include'}", f"-I{CSRC}",
           *map(str, SOURCES), "-o", str(tmp)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building libccjoin.so")
    tmp.replace(out)
    return out


if __name__ == "__main__":
    print(build())
