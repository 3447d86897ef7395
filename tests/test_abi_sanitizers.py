"""The library's host code under the address and undefined-behaviour sanitizers (no GPU).

The four sources are compiled with both sanitizers on the host side only (each `-fsanitize=`
is given to the host pass; device code is built as usual and never runs here), linked into a
separate library, and `abi_sanitize.c` drives its argument checks: see that file's header.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import pytest

from paper_2609_22441_amd import build as B

HERE = Path(__file__).resolve().parent
CLANG = Path("/opt/rocm/llvm/bin/clang")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.mark.timeout(600)
def test_host_code_is_clean_under_sanitizers(tmp_path):
    if not (Path(B.HIPCC).exists() and CLANG.exists()):
        pytest.skip("hipcc or ROCm clang not available")
    inc = [f"-I{B.ROOT / 'include'}", f"-I{B.CSRC}"]
    flags = [f for f in B.FLAGS if f != "-O3"] + ["-O1", "-g"]

    def compile_one(src):
        obj = tmp_path / (src.stem + ".o")
        r = subprocess.run([B.HIPCC, *flags, *HOST_SAN, *inc, "-c", str(src), "-o", str(obj)],
                           capture_output=True, text=True)
        return obj, r

    with ThreadPoolExecutor(max_workers=min(4, os.cpu_count() or 1)) as ex:
        results = list(ex.map(compile_one, B.SOURCES))
    for obj, r in results:
        assert r.returncode == 0, r.stderr[-3000:]
    lib = tmp_path / "libccjoin_san.so"
    r = subprocess.run([B.HIPCC, "--offload-arch=gfx950", "-shared", *[str(o) for o, _ in results],
                        "-o", str(lib)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    exe = tmp_path / "abi_san"
    r = subprocess.run([str(CLANG), "-O1", "-g", "-std=c99", "-Wall", "-Wextra", "-Werror",
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                        "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", *inc,
                        str(HERE / "abi_sanitize.c"), f"-L{tmp_path}", "-lccjoin_san",
                        f"-Wl,-rpath,{tmp_path}", "-o", str(exe)],
                       capture_output=True, text=True)
    if r.returncode != 0 and "asan" in r.stderr.lower() and "cannot find" in r.stderr.lower():
        pytest.skip("the sanitizer runtime is not installed")
    assert r.returncode == 0, r.stderr[-3000:]
    # The HIP runtime keeps allocations until exit, so leak detection is off.
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr[-3000:]
    shutil.rmtree(tmp_path, ignore_errors=True)
