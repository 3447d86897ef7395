"""CPU oracle for the edge-feature join (Connected Content Retriever, §3.1, Eq. 1).

TEST INFRASTRUCTURE: only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import this package. The product path (the HIP library and its binding) never does.

The arithmetic lives in ``cc_oracle.c`` (plain C, built with gcc); this file only builds and
loads it and marshals numpy / CPU-torch arrays. ``join`` returns the full model-input rows
``[doc row | edge segment per lookup]``, the hit mask and the invalid-candidate count, exactly
as the C header comment defines them.

Parity pins: the three search methods (lower bound, naive scan, hash) are cross-checked in the
CPU tests against a pure-Python scan of Eq. 1, against NumPy's ``searchsorted`` route through
Alg. 1, against invariants, and against the hand-worked fixtures in ``tests/golden``.
"""
from __future__ import annotations

import ctypes
import subprocess
from pathlib import Path
from typing import Optional

import numpy as np

LOWER_BOUND, SCAN, HASH = 0, 1, 2

_HERE = Path(__file__).resolve().parent
SRC = _HERE / "cc_oracle.c"
LIB = _HERE / "libccoracle.so"

_lib = None


def build(out: Optional[Path] = None, src: Optional[Path] = None, werror: bool = True) -> Path:
    """Compile the oracle into a shared library (gcc, no GPU involved)."""
    out = Path(out) if out else LIB
    src = Path(src) if src else SRC
    tmp = out.with_suffix(".so.tmp")
    flags = ["-Wall", "-Wextra"] + (["-Werror"] if werror else ["-w"])
    subprocess.check_call(["gcc", "-O2", "-std=c99", *flags, "-fPIC", "-shared", "-o", str(tmp),
                           str(src)])
    tmp.replace(out)
    return out


def load(path: Optional[Path] = None):
    """Load a compiled oracle (building the default one if nothing is built yet)."""
    p = Path(path) if path else LIB
    if path is None and not p.exists():
        build()
    lib = ctypes.CDLL(str(p))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.ccor_join.restype = i64
    lib.ccor_join.argtypes = [ctypes.c_int,
                              i64, vp, vp, i64,
                              i64, vp, vp,
                              vp, vp,
                              vp, i64,
                              vp,
                              i64, vp,
                              vp, i64, vp]
    lib.ccor_sort_affinity.restype = ctypes.c_int
    lib.ccor_sort_affinity.argtypes = [i64, vp, vp, vp, i64, vp, vp]
    lib.ccor_resolve.restype = ctypes.c_int
    lib.ccor_resolve.argtypes = [i64, vp, i64, vp, vp]
    lib.ccor_upsert.restype = i64
    lib.ccor_upsert.argtypes = [i64, vp, vp, vp, vp, i64, i64, vp, vp, vp, vp]
    return lib


def _default_lib():
    global _lib
    if _lib is None:
        _lib = load()
    return _lib


def as_bytes(a) -> np.ndarray:
    """A 2-D array of any element type as a contiguous uint8 array of its rows' bytes."""
    if hasattr(a, "detach"):               # torch tensor (CPU)
        import torch
        t = a.detach().cpu().contiguous()
        if t.dim() == 1:
            t = t.reshape(-1, 1)
        width = int(np.prod(t.shape[1:])) * t.element_size()
        return t.view(torch.uint8).numpy().reshape(t.shape[0], width)
    a = np.ascontiguousarray(a)
    if a.ndim == 1:
        a = a.reshape(-1, 1)
    width = int(np.prod(a.shape[1:])) * a.itemsize
    return a.view(np.uint8).reshape(a.shape[0], width)


def _i64(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=np.int64)


def _ptr(a):
    return None if a is None else a.ctypes.data


def join(author_id, doc_rows, cand_offsets, cand_idx, key_offsets, keys, edge_rows,
         default_row=None, n_lookups: int = 1, extra_keys=None, out_stride: Optional[int] = None,
         method: int = LOWER_BOUND, lib=None, fill: int = 0):
    """Run the oracle join; returns (out uint8 [total, stride], hit int8 [total, L], invalid).

    ``extra_keys`` is a list of ``n_lookups - 1`` arrays of per-candidate keys. ``out`` starts
    filled with the byte ``fill`` so that a row the join forgets to write shows up.
    """
    lib = lib or _default_lib()
    author_id = _i64(author_id)
    doc = as_bytes(doc_rows)
    edge = as_bytes(edge_rows)
    co, ci, ko, ks = _i64(cand_offsets), _i64(cand_idx), _i64(key_offsets), _i64(keys)
    n_docs, wd = author_id.shape[0], doc.shape[1]
    if doc.shape[0] != n_docs:
        raise ValueError("doc_rows and author_id disagree on n_docs")
    we = edge.shape[1]
    if edge.shape[0] != ks.shape[0]:
        raise ValueError("edge_rows and keys disagree on K")
    total = int(co[-1])
    if ci.shape[0] != total:
        raise ValueError("cand_idx length != cand_offsets[-1]")
    stride = wd + n_lookups * we if out_stride is None else out_stride
    dflt = None
    if default_row is not None:
        dflt = as_bytes(default_row).reshape(-1)
        if dflt.shape[0] != we:
            raise ValueError("default_row width != edge row width")
    ex = None
    if n_lookups > 1:
        if extra_keys is None or len(extra_keys) != n_lookups - 1:
            raise ValueError("n_lookups - 1 extra key arrays are required")
        ex = np.ascontiguousarray(np.concatenate([_i64(e) for e in extra_keys]))
        if ex.shape[0] != (n_lookups - 1) * total:
            raise ValueError("extra key arrays must have one key per candidate")
    out = np.full((total, stride), fill, dtype=np.uint8)
    hit = np.zeros((total, n_lookups), dtype=np.int8)
    inv = lib.ccor_join(method, n_docs, _ptr(author_id), _ptr(doc), wd,
                        co.shape[0] - 1, _ptr(co), _ptr(ci), _ptr(ko), _ptr(ks),
                        _ptr(edge), we, _ptr(dflt), n_lookups, _ptr(ex),
                        _ptr(out), stride, _ptr(hit))
    if inv < 0:
        raise ValueError("oracle rejected its arguments")
    return out, hit, int(inv)


def sort_affinity(key_offsets, keys, rows, lib=None):
    """Alg. 1 Step 1 per viewer (stable): returns (sorted keys int64, rows moved with them)."""
    lib = lib or _default_lib()
    ko, ks = _i64(key_offsets), _i64(keys)
    r = as_bytes(rows)
    if r.shape[0] != ks.shape[0]:
        raise ValueError("rows and keys disagree on K")
    ko_out = np.empty_like(ks)
    r_out = np.empty_like(r)
    if lib.ccor_sort_affinity(ko.shape[0] - 1, _ptr(ko), _ptr(ks), _ptr(r), r.shape[1],
                              _ptr(ko_out), _ptr(r_out)) != 0:
        raise ValueError("oracle rejected its arguments")
    return ko_out, r_out


def pad_scatter(rows, hit, cand_offsets, n_max: int):
    """Padded batch layout of §6.3 (batching and padding for variable-length requests).

    Step 1 computes the scatter indices (batch_idx, pos_idx) of every valid row, step 2 is the
    flattened gather (here: the CSR rows the join produced, in order), step 3 scatters them into
    T[b, n_max, ...]. Pad slots keep zero bytes, hit 0 and valid 0. A request longer than n_max
    keeps its first n_max rows.
    """
    co = _i64(cand_offsets)
    b = co.shape[0] - 1
    n = np.minimum(co[1:] - co[:-1], n_max)
    batch_idx = np.repeat(np.arange(b), n)
    pos_idx = np.concatenate([np.arange(k) for k in n]) if b else np.zeros(0, np.int64)
    src = np.concatenate([co[v] + np.arange(n[v]) for v in range(b)]) if b else pos_idx
    T = np.zeros((b, n_max) + rows.shape[1:], dtype=rows.dtype)
    H = np.zeros((b, n_max) + hit.shape[1:], dtype=hit.dtype)
    valid = np.zeros((b, n_max), dtype=np.int8)
    T[batch_idx, pos_idx] = rows[src]
    H[batch_idx, pos_idx] = hit[src]
    valid[batch_idx, pos_idx] = 1
    return T, H, valid


def join_padded(author_id, doc_rows, cand_offsets, cand_idx, key_offsets, keys, edge_rows,
                n_max: int, **kw):
    """The join in the padded batch layout: (T uint8 [B, n_max, stride], hit, valid, invalid)."""
    co = _i64(cand_offsets)
    # Candidates beyond n_max in a request are dropped before the join (they produce no row).
    n = np.minimum(co[1:] - co[:-1], n_max)
    keep = np.concatenate([co[v] + np.arange(n[v]) for v in range(len(n))]) if len(n) else \
        np.zeros(0, np.int64)
    co_kept = np.zeros(len(n) + 1, np.int64)
    co_kept[1:] = np.cumsum(n)
    ci = _i64(cand_idx)[keep]
    extra = kw.pop("extra_keys", None)
    if extra is not None:
        extra = [_i64(e)[keep] for e in extra]
    out, hit, inv = join(author_id, doc_rows, co_kept, ci, key_offsets, keys, edge_rows,
                         extra_keys=extra, **kw)
    T, H, valid = pad_scatter(out, hit, co_kept, n_max)
    return T, H, valid, inv


INT64_MIN = -(1 << 63)


def resolve(index_ids, queries, lib=None):
    """Eq. 6 (§6.3.1): position of each query id in the index, or -1 (index_ids[p] = id at p)."""
    lib = lib or _default_lib()
    ix, q = _i64(index_ids), _i64(queries)
    out = np.empty_like(q)
    if lib.ccor_resolve(ix.shape[0], _ptr(ix), q.shape[0], _ptr(q), _ptr(out)) != 0:
        raise ValueError("oracle rejected its arguments")
    return out


class IndexState:
    """A document index under ingestion (§6.2): the id, author id and row at each position, and
    the number of stored documents. ``upsert`` applies one batch by sequential replay."""

    def __init__(self, capacity: int, row_bytes: int, lib=None):
        self.lib = lib or _default_lib()
        self.capacity = capacity
        self.n_docs = 0
        self.ids = np.full(capacity, INT64_MIN, np.int64)
        self.author = np.zeros(capacity, np.int64)
        self.rows = np.zeros((capacity, row_bytes), np.uint8)

    def upsert(self, ids, authors, rows):
        """Apply one batch; returns (n_new, n_rejected), or None when it does not fit (then the
        state is unchanged)."""
        i, a = _i64(ids), _i64(authors)
        r = as_bytes(rows)
        if not (i.shape[0] == a.shape[0] == r.shape[0]) or r.shape[1] != self.rows.shape[1]:
            raise ValueError("batch arrays disagree")
        nd = ctypes.c_int64(self.n_docs)
        rej = ctypes.c_int64(0)
        n_new = self.lib.ccor_upsert(self.capacity, ctypes.byref(nd), _ptr(self.ids),
                                     _ptr(self.author), _ptr(self.rows), self.rows.shape[1],
                                     i.shape[0], _ptr(i), _ptr(a), _ptr(r), ctypes.byref(rej))
        if n_new == -1:
            raise ValueError("oracle rejected its arguments")
        if n_new == -2:
            return None
        self.n_docs = nd.value
        return int(n_new), int(rej.value)

    def resolve(self, queries):
        return resolve(self.ids[:self.n_docs], queries, self.lib)


def join_single(author_id, doc_rows, cand_idx, keys, edge_rows, **kw):
    """One viewer: the batched form with offsets [0, N] and [0, K]."""
    n = len(cand_idx)
    k = len(keys)
    return join(author_id, doc_rows, np.array([0, n]), cand_idx, np.array([0, k]), keys,
                edge_rows, **kw)
