"""CPU-side checks of the C ABI: the library loads, exports what the header declares, and
rejects bad host arguments before touching a device (no compute calls here)."""
from __future__ import annotations

import ctypes
import re
from pathlib import Path

import pytest

import paper_2609_22441_amd as P
from paper_2609_22441_amd import binding as B

ROOT = Path(__file__).resolve().parents[1]


def _declared():
    text = (ROOT / "include" / "cc_join.h").read_text()
    return sorted(set(re.findall(r"^CC_API\s+[\w\s\*]*?\b(cc_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_binding_surface():
    assert _declared() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(str(B.LIB_PATH))
    for name in _declared():
        assert hasattr(lib, name), name


def test_status_strings():
    assert P.cc_status_string(0) == "CC_OK"
    assert P.cc_status_string(1) == "CC_ERR_INVALID_ARGUMENT"
    assert P.cc_status_string(5) == "CC_ERR_NOT_SUPPORTED"
    assert P.cc_status_string(6) == "CC_ERR_STORE_FULL"
    assert P.cc_status_string(8) == "CC_ERR_TIMEOUT"
    assert P.cc_status_string(99) == "CC_UNKNOWN_STATUS"
    assert P.cc_last_device_error() == 0


@pytest.mark.parametrize("n_docs,ids,rows,width,flags", [
    (-1, None, None, 16, 1),          # negative size
    (4, 8, 8, 24, 1),                 # row width not a multiple of 16
    (4, 8, 8, 0, 1),                  # zero row width
    (4, 8, 8, (1 << 20) + 16, 1),     # row wider than 1 MiB
    (4, None, 8, 16, 1),              # missing author ids
    (4, 8, None, 16, 1),              # missing rows
    (0, None, None, 16, 3),           # unknown source flag
    (1 << 62, 8, 8, 16, 1),           # byte size overflows int64
])
def test_store_create_rejects_bad_arguments(n_docs, ids, rows, width, flags):
    lib = B.lib()
    h = ctypes.c_void_p(1234)
    st = lib.cc_store_create(ctypes.byref(h), n_docs, ids, rows, width, flags, None)
    assert st == B.CC_ERR_INVALID_ARGUMENT
    assert h.value is None


def test_store_create_without_output_pointer():
    assert B.lib().cc_store_create(None, 0, None, None, 16, 1, None) == B.CC_ERR_INVALID_ARGUMENT


def test_join_rejects_null_store():
    lib = B.lib()
    assert lib.cc_join(None, None, 0, None, 0, None, 16, None, None, 32, None, None) == 1
    assert lib.cc_join_batched(None, 0, None, None, 0, None, None, 0, None, 16, None, 1, None,
                               None, 32, None, None) == 1
    assert lib.cc_join_batched_authors(None, 0, None, None, None, 0, None, None, 0, None, 16,
                                       None, 1, None, None, 32, None, None) == 1
    # candidates without their author ids: refused before the store is looked at
    assert lib.cc_join_batched_authors(None, 1, 8, 8, None, 5, 8, None, 0, None, 16, None, 1,
                                       None, 16, 32, 8, None) == 1


def test_store_queries_reject_null():
    lib = B.lib()
    n = ctypes.c_int64()
    assert lib.cc_store_info(None, ctypes.byref(n), None) == 1
    assert lib.cc_store_invalid_count(None, ctypes.byref(n), None) == 1
    assert lib.cc_store_reset_invalid_count(None, None) == 1
    assert lib.cc_store_destroy(None) == 0


def test_validate_keys_rejects_bad_arguments():
    lib = B.lib()
    bad = ctypes.c_int64(7)
    assert lib.cc_validate_keys(None, None, 1, 0, None, None) == 1           # no output
    assert lib.cc_validate_keys(None, None, 1, 0, ctypes.byref(bad), None) == 1  # no offsets
    assert lib.cc_validate_keys(8, None, 1, 5, ctypes.byref(bad), None) == 1     # no keys
    assert lib.cc_validate_keys(12, 16, 1, 5, ctypes.byref(bad), None) == 1      # misaligned
    assert lib.cc_validate_keys(None, None, 0, 0, ctypes.byref(bad), None) == 0  # nothing to do
    assert bad.value == -1


def test_sort_workspace_size():
    lib = B.lib()
    assert lib.cc_sort_workspace_bytes(0, 3) == 0
    assert lib.cc_sort_workspace_bytes(-5, 3) == 0
    assert lib.cc_sort_workspace_bytes(100, 0) == 0
    assert lib.cc_sort_workspace_bytes(4097, 2) >= 2 * 16 * 4097 + 3 * 8   # ping-pong + plan
    assert lib.cc_sort_workspace_bytes(1 << 32, 1) == 0             # more than the sort takes


def test_sort_noalloc_rejects_bad_arguments_and_sizes_past_its_scratch():
    lib = B.lib()
    base = dict(nv=1, off=0x1000, kin=0x2000, rin=0x10000, rb=32, tk=1000, mk=0, kout=0x30000,
                rout=0x100000)

    def call(**kw):
        a = dict(base, **kw)
        return lib.cc_sort_affinity_noalloc(a["nv"], a["off"], a["kin"], a["rin"], a["rb"],
                                            a["tk"], a["mk"], a["kout"], a["rout"], None)

    assert B.SORT_NOALLOC_MAX_RECORDS == 1 << 20 and B.SORT_NOALLOC_MAX_VIEWERS == 1 << 16
    big = dict(kin=None, rin=None, kout=None, rout=None)
    assert call(tk=B.SORT_NOALLOC_MAX_RECORDS + 1, **big) == B.CC_ERR_TOO_LARGE
    assert call(nv=B.SORT_NOALLOC_MAX_VIEWERS + 1, **big) == B.CC_ERR_TOO_LARGE
    assert call(tk=1 << 32, **big) == B.CC_ERR_TOO_LARGE
    assert P.cc_status_string(B.CC_ERR_TOO_LARGE) == "CC_ERR_TOO_LARGE"
    assert call(rb=24) == 1                      # row width not a multiple of 16
    assert call(rb=(1 << 20) + 16) == 1          # row wider than 1 MiB
    assert call(tk=-1) == 1
    assert call(nv=-1) == 1
    assert call(mk=-1) == 1
    assert call(off=None) == 1
    assert call(kin=None) == 1
    assert call(rout=0x100008) == 1              # misaligned rows
    assert call(kout=0x2004) == 1                # misaligned keys
    assert call(kout=0x2000) == 1                # output keys alias the input keys
    assert call(rout=0x10000 + 64) == 1          # output rows overlap the input rows
    assert call(tk=0, **big) == 0                # no work: nothing touches a device


def test_sort_rejects_bad_arguments():
    lib = B.lib()
    ws = lib.cc_sort_workspace_bytes(1000, 1)
    base = dict(nv=1, off=0x1000, kin=0x2000, rin=0x10000, rb=32, tk=1000, mk=0, kout=0x30000,
                rout=0x100000, w=0x200000, wb=ws)

    def call(**kw):
        a = dict(base, **kw)
        return lib.cc_sort_affinity(a["nv"], a["off"], a["kin"], a["rin"], a["rb"], a["tk"],
                                    a["mk"], a["kout"], a["rout"], a["w"], a["wb"], None)

    assert call(rb=24) == 1                      # row width not a multiple of 16
    assert call(rb=(1 << 20) + 16) == 1          # row wider than 1 MiB
    assert call(rb=1 << 20, tk=0, kin=None, rin=None, kout=None, rout=None, w=None, wb=0) == 0
    assert call(tk=-1) == 1
    assert call(tk=1 << 32) == 1                 # record count must fit 32 bits
    assert call(nv=-1) == 1
    assert call(off=None) == 1
    assert call(kin=None) == 1
    assert call(wb=ws - 1) == 1                  # workspace too small
    assert call(rout=0x100008) == 1              # misaligned rows
    assert call(kout=0x2004) == 1                # misaligned keys
    assert call(kout=0x2000) == 1                # output keys alias the input keys
    assert call(rout=0x10000 + 64) == 1          # output rows overlap the input rows
    assert call(w=0x30000) == 1                  # workspace overlaps the output keys
    assert call(mk=-1) == 1                      # negative hint
    assert call(tk=0, kin=None, rin=None, kout=None, rout=None, w=None, wb=0) == 0   # no work


def test_sort_method_rejects_bad_arguments():
    """cc_sort_affinity_method: an unknown method or a key_bits bound outside [0, 64] is refused
    before anything is enqueued; the other checks are cc_sort_affinity's."""
    lib = B.lib()
    ws = lib.cc_sort_workspace_bytes(1000, 1)
    base = dict(m=2, kb=26, nv=1, off=0x1000, kin=0x2000, rin=0x10000, rb=32, tk=1000, mk=0,
                kout=0x30000, rout=0x100000, w=0x200000, wb=ws)

    def call(**kw):
        a = dict(base, **kw)
        return lib.cc_sort_affinity_method(a["m"], a["kb"], a["nv"], a["off"], a["kin"], a["rin"],
                                           a["rb"], a["tk"], a["mk"], a["kout"], a["rout"],
                                           a["w"], a["wb"], None)

    header = (ROOT / "include" / "cc_join.h").read_text()
    for name, value in (("CC_SORT_AUTO", B.SORT_AUTO), ("CC_SORT_MERGE", B.SORT_MERGE),
                        ("CC_SORT_RADIX", B.SORT_RADIX),
                        ("CC_SORT_RADIX_MIN_RECORDS", B.SORT_RADIX_MIN_RECORDS)):
        m = re.search(rf"#define {name} \(?(\d+)(?: << (\d+)\))?", header)
        assert m, name                           # the binding's constants are the header's
        assert int(m.group(1)) << int(m.group(2) or 0) == value, name
    assert call(m=3) == 1 and call(m=-1) == 1    # no such method
    assert call(kb=-1) == 1 and call(kb=65) == 1
    assert call(rb=24) == 1                      # the checks of cc_sort_affinity apply
    assert call(wb=ws - 1) == 1
    for m in (0, 1, 2):                          # no work: nothing touches a device
        for kb in (0, 1, 64):
            assert call(m=m, kb=kb, tk=0, kin=None, rin=None, kout=None, rout=None, w=None,
                        wb=0) == 0


def test_indexed_store_rejects_bad_arguments():
    lib = B.lib()
    h = ctypes.c_void_p(99)
    assert lib.cc_store_create_indexed(None, 10, 16, None) == 1
    assert lib.cc_store_create_indexed(ctypes.byref(h), -1, 16, None) == 1
    assert h.value is None
    assert lib.cc_store_create_indexed(ctypes.byref(h), 1 << 31, 16, None) == 1   # > INT32_MAX
    assert lib.cc_store_create_indexed(ctypes.byref(h), 10, 24, None) == 1        # row width
    assert lib.cc_store_create_indexed(ctypes.byref(h), 10, 0, None) == 1
    assert lib.cc_store_create_indexed(ctypes.byref(h), 10, (1 << 20) + 16, None) == 1


def test_upsert_and_resolve_reject_bad_arguments():
    lib = B.lib()
    n = ctypes.c_int64()
    assert lib.cc_store_upsert(None, 1, 8, 8, 16, 16, 1 << 20, ctypes.byref(n), None, None) == 1
    assert lib.cc_resolve_ids(None, 8, 1, 8, None) == 1
    assert lib.cc_set_ingestion_wait_limit(0) == 0    # no device touched
    assert lib.cc_set_ingestion_wait_limit(-1) == 0   # back to the default
    assert lib.cc_upsert_workspace_bytes(0) == 0
    assert lib.cc_upsert_workspace_bytes(-3) == 0
    assert lib.cc_upsert_workspace_bytes(1000) >= 12 * 1000
    assert lib.cc_upsert_workspace_bytes((1 << 30) + 1) == 0        # more than a batch takes


def test_library_has_no_cpu_fallback(monkeypatch, tmp_path):
    """The binding refuses to run when the HIP library is missing (no silent fallback)."""
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", tmp_path / "missing.so")
    with pytest.raises(RuntimeError, match="not built"):
        B.lib()


def test_product_path_does_not_import_the_oracle():
    for f in (ROOT / "paper_2609_22441_amd").rglob("*"):
        if f.suffix in (".py", ".hip", ".h", ".cpp"):
            text = f.read_text()
            assert "oracle" not in text.lower().replace("oracle-free", ""), f
