"""CPU tests of the oracle: its pins, edge cases, and planted mistakes the pins must catch."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import numpy as np
import pytest
import torch

import oracle
import workload as W

sys.path.insert(0, str(Path(__file__).resolve().parent))
import oracle_pins as P  # noqa: E402

HERE = Path(__file__).resolve().parent


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


def test_pin_golden(lib):
    P.pin_golden(lib)


def test_pin_scan(lib):
    P.pin_scan(lib)


def test_pin_alg1(lib):
    P.pin_alg1(lib)


def test_pin_invariants(lib):
    P.pin_invariants(lib)


def test_pin_padding(lib):
    P.pin_padding(lib)


def test_pin_sort(lib):
    P.pin_sort(lib)


# ---- edge cases of the readings --------------------------------------------------------------
def _one(lib, author, doc, cand, keys, edge, **kw):
    return oracle.join_single(np.asarray(author, np.int64), np.asarray(doc, np.uint8),
                              np.asarray(cand, np.int64), np.asarray(keys, np.int64),
                              np.asarray(edge, np.uint8).reshape(len(keys), 16), lib=lib,
                              fill=P.FILL, **kw)


def test_empty_key_list_is_all_miss(lib):
    doc = np.arange(48, dtype=np.uint8).reshape(3, 16)
    dflt = np.full(16, 9, np.uint8)
    out, hit, inv = _one(lib, [1, 2, 3], doc, [0, 2, 1], [], np.zeros((0, 16)), default_row=dflt)
    assert inv == 0 and not hit.any()
    assert (out[:, 16:] == 9).all() and np.array_equal(out[:, :16], doc[[0, 2, 1]])


def test_no_candidates(lib):
    out, hit, inv = _one(lib, [1], np.zeros((1, 16)), [], [1], np.ones((1, 16)))
    assert out.shape == (0, 32) and hit.shape == (0, 1) and inv == 0


def test_int64_extremes_and_negatives(lib):
    lo, hi = W.I64_MIN, W.I64_MAX
    author = [lo, hi, -5, 0, hi - 1]
    doc = np.arange(80, dtype=np.uint8).reshape(5, 16)
    keys = [lo, -5, hi]
    edge = np.repeat(np.array([[1], [2], [3]], np.uint8), 16, axis=1)
    out, hit, _ = _one(lib, author, doc, [0, 1, 2, 3, 4], keys, edge)
    assert hit[:, 0].tolist() == [1, 1, 1, 0, 0]
    assert out[:, 16].tolist() == [1, 3, 2, 0, 0]


def test_duplicate_keys_take_leftmost(lib):
    keys = [4, 4, 4, 9]
    edge = np.repeat(np.array([[1], [2], [3], [4]], np.uint8), 16, axis=1)
    for m in P.METHODS:
        out, hit, _ = _one(lib, [4, 9], np.zeros((2, 16)), [0, 1], keys, edge, method=m)
        assert out[:, 16].tolist() == [1, 4] and hit[:, 0].tolist() == [1, 1]


def test_invalid_positions(lib):
    n = 4
    bad = [-1, n, n + 10, W.I64_MIN, W.I64_MAX]
    dflt = np.full(16, 0x5A, np.uint8)
    out, hit, inv = _one(lib, [7] * n, np.ones((n, 16)), bad, [7], np.ones((1, 16)),
                         default_row=dflt)
    assert inv == len(bad) and not hit.any()
    assert (out[:, :16] == 0).all() and (out[:, 16:] == 0x5A).all()


def test_stride_padding_untouched(lib):
    out, _, _ = _one(lib, [3, 3], np.ones((2, 16)), [0, 1], [3], np.full((1, 16), 2),
                     out_stride=64)
    assert (out[:, 32:] == P.FILL).all()


def test_special_bit_patterns_copied(lib):
    g = W.gen("cpu", 5, 0)
    doc = W.salt_special_values(torch.randn(64, 16), 0.3, g)
    edge = W.salt_special_values(torch.rand(8, 8).to(torch.bfloat16), 0.3, g)
    author = torch.arange(64) % 10
    keys = torch.arange(0, 16, 2)
    cand = torch.randperm(64, generator=g)
    out, hit, _ = oracle.join_single(author, doc, cand, keys, edge, lib=lib)
    d = oracle.as_bytes(doc)
    e = oracle.as_bytes(edge)
    assert np.array_equal(out[:, :64], d[cand.numpy()])
    h = hit[:, 0].astype(bool)
    a = author.numpy()[cand.numpy()]
    assert np.array_equal(out[h, 64:], e[a[h] // 2])


def test_generator_hit_rate_closed_form():
    """Generator sanity (not the join): uniform keys over the author space hit with rate K/M."""
    s, r = W.shape(1, store_n_docs=200_000)
    st = W.make_store(s, 11)
    q = W.make_request(st, r, 11, 0)
    rate = torch.isin(st.author_id[q.cand_idx], q.keys).double().mean().item()
    expect = r.k / s.n_authors                       # 1%
    sd = (expect * (1 - expect) / r.n_cand) ** 0.5
    assert abs(rate - expect) < 5 * sd


# ---- planted mistakes --------------------------------------------------------------------------
MUTANTS = [
    ("search keeps going past equal keys", "if (keys[mid] < x)", "if (keys[mid] <= x)"),
    ("equality test dropped", "if (p < n && keys[p] == x)", "if (p < n)"),
    ("scan takes the last match", "        if (keys[i] == x)\n            return i;",
     "        if (keys[i] == x && i + 1 < n && keys[i + 1] != x)\n            return i;"),
    ("hash keeps the last duplicate", "if (t->idx[s] < 0) {          /* first occurrence",
     "if (1) {          /* first occurrence"),
    ("viewer offset dropped from the edge row", "edge_rows + (k0 + i) * edge_bytes",
     "edge_rows + i * edge_bytes"),
    ("doc row indexed by candidate slot", "doc_rows + c * doc_bytes", "doc_rows + j * doc_bytes"),
    ("author looked up by slot", "int64_t key = (l == 0) ? author_id[c]",
     "int64_t key = (l == 0) ? author_id[j % n_docs]"),
    ("negative positions accepted", "int valid = (c >= 0 && c < n_docs);",
     "int valid = (c >= -1 && c < n_docs);"),
    ("invalid count not kept", "                invalid++;", "                ;"),
    ("second segment overwrites the first", "row + doc_bytes + l * edge_bytes",
     "row + doc_bytes"),
    ("hit bit off by one", "(int8_t)(i >= 0)", "(int8_t)(i > 0)"),
    ("miss leaves the output unwritten", "                else\n                    memset(seg, 0, (size_t)edge_bytes);",
     "                else\n                    ;"),
    ("default row ignored", "                else if (default_row)\n                    memcpy(seg, default_row, (size_t)edge_bytes);",
     "                else if (0)\n                    memcpy(seg, default_row, (size_t)edge_bytes);"),
    ("actor key from the wrong candidate", "extra_keys[(l - 1) * total_cand + j]",
     "extra_keys[(l - 1) * total_cand + (j > c0 ? j - 1 : j)]"),
    ("invalid doc segment not cleared", "                memset(row, 0, (size_t)doc_bytes);\n",
     "\n"),
    ("sort loses stability", "if (keys[idx[j]] < keys[idx[i]])", "if (keys[idx[j]] <= keys[idx[i]])"),
    ("sorted rows not moved", "rows_in + (k0 + idx[i]) * row_bytes", "rows_in + (k0 + i) * row_bytes"),
    ("resolve reports positions one too high", "pos_out[j] = table_find(&t, queries[j]);",
     "pos_out[j] = table_find(&t, queries[j]) + (j > 0);"),
    ("stored ids not overwritten", "            ids_by_pos[p] = ids[i];\n        }\n",
     "            ids_by_pos[p] = ids[i];\n        } else\n            continue;\n"),
    ("reserved id stored", "        if (ids[i] == INT64_MIN)\n            continue;",
     "        if (0)\n            continue;"),
    ("capacity check off by one", "if (*n_docs + n_new > capacity)", "if (*n_docs + n_new >= capacity)"),
    ("stored ids counted as new",
     "if (table_find(&t, ids[i]) < 0 && table_find(&seen, ids[i]) < 0)",
     "if (table_find(&seen, ids[i]) < 0)"),
    ("author id not moved", "author[p] = authors_in[i];", "author[p] = authors_in[0];"),
]


def _check_mutant(args):
    name, old, new, tmp = args
    src = oracle.SRC.read_text()
    assert src.count(old) == 1, f"mutant '{name}': anchor not found exactly once"
    d = tmp / name.replace(" ", "_")
    d.mkdir()
    (d / "m.c").write_text(src.replace(old, new))
    so = oracle.build(out=d / "m.so", src=d / "m.c", werror=False)
    env = dict(os.environ, PYTHONPATH=str(HERE.parent))
    try:
        r = subprocess.run([sys.executable, str(HERE / "oracle_pins.py"), str(so)], env=env,
                           capture_output=True, text=True, timeout=120)
        return name, r.returncode
    except subprocess.TimeoutExpired:
        return name, "timeout"


def test_planted_mistakes_are_caught(tmp_path):
    """Every one-spot mistake planted in a copy of the oracle fails at least one pin."""
    jobs = [(n, o, w, tmp_path) for n, o, w in MUTANTS]
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(_check_mutant, jobs))
    survivors = [n for n, rc in results if rc == 0]
    assert not survivors, f"pins missed planted mistakes: {survivors}"


def test_unmutated_oracle_passes_pin_runner():
    env = dict(os.environ, PYTHONPATH=str(HERE.parent))
    r = subprocess.run([sys.executable, str(HERE / "oracle_pins.py"), str(oracle.LIB)], env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
