"""Build the HIP library libccjoin.so for gfx950 (in-tree, no GPU needed)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
LIB = PKG / "libccjoin.so"
SOURCES = [CSRC / "cc_api.hip", CSRC / "join_kernels.hip", CSRC / "sort_kernels.hip",
           CSRC / "map_kernels.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # Packed fp32 instructions stay off (no arithmetic here needs them).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-fvisibility=hidden",
]


def build(out: Path = LIB, extra_flags=()) -> Path:
    """Compile every source to an object (in parallel), then link the shared library."""
    out = Path(out)
    objdir = PKG / "_build"
    objdir.mkdir(exist_ok=True)
    inc = [f"-I{ROOT / 'include'}", f"-I{CSRC}"]

    def compile_one(src: Path):
        obj = objdir / (src.stem + ".o")
        r = subprocess.run([HIPCC, *FLAGS, *extra_flags, *inc, "-c", str(src), "-o", str(obj)],
                           capture_output=True, text=True)
        return src, obj, r

    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        results = list(ex.map(compile_one, SOURCES))
    for src, _, r in results:
        if r.returncode != 0:
            sys.stderr.write(r.stdout + r.stderr)
            raise RuntimeError(f"hipcc failed compiling {src.name}")
    tmp = out.with_name(out.name + ".tmp")
    r = subprocess.run([HIPCC, *FLAGS, *extra_flags, "-shared", *[str(o) for _, o, _ in results],
                        "-o", str(tmp)], capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed linking libccjoin.so")
    tmp.replace(out)
    return out


if __name__ == "__main__":
    print(build())
