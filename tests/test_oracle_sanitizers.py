"""The CPU oracle under gcc's address and undefined-behaviour sanitizers.

`oracle_sanitize.c` drives every oracle entry point on a few thousand small random cases with
exactly sized buffers and cross-checks the results (see its header). It is built here together
with the oracle source; a one-element overflow planted in a copy of the oracle must stop it.
"""
import shutil
import subprocess
from pathlib import Path

import pytest

HERE = Path(__file__).resolve().parent
ORACLE_SRC = HERE.parent / "oracle" / "cc_oracle.c"
HARNESS = HERE / "oracle_sanitize.c"
FLAGS = ["-O1", "-g", "-std=c99", "-Wall", "-Wextra", "-Werror", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _build(oracle_src: Path, exe: Path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    r = subprocess.run(["gcc", *FLAGS, str(HARNESS), str(oracle_src), "-o", str(exe)],
                       capture_output=True, text=True, timeout=120)
    if r.returncode != 0 and "asan" in (r.stderr or "").lower():
        pytest.skip("the sanitizer runtime is not installed: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr


def _run(exe: Path):
    return subprocess.run([str(exe), "3000"], capture_output=True, text=True, timeout=300,
                          env={"ASAN_OPTIONS": "detect_leaks=1", "UBSAN_OPTIONS": "print_stacktrace=1"})


def test_oracle_is_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_san"
    _build(ORACLE_SRC, exe)
    r = _run(exe)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr[-2000:]


def test_planted_overflow_is_caught(tmp_path):
    """A sort that writes each viewer's keys one slot too far must stop the harness."""
    src = ORACLE_SRC.read_text()
    old = "keys_out[k0 + i] = keys_in[k0 + idx[i]];"
    assert src.count(old) == 1
    bad = tmp_path / "cc_oracle_bad.c"
    bad.write_text(src.replace(old, "keys_out[k0 + i + 1] = keys_in[k0 + idx[i]];"))
    exe = tmp_path / "oracle_san_bad"
    _build(bad, exe)
    r = _run(exe)
    assert r.returncode != 0
    assert "AddressSanitizer: heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
