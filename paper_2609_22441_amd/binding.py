"""ctypes binding of libccjoin.so: argument marshalling only.

Tensor arguments are torch tensors. Before a call, each one is checked for what the C ABI
cannot see behind a pointer: element type, dense layout, enough elements for the sizes passed
with it, and GPU memory. A failed check raises ValueError or TypeError and nothing is enqueued.
Plain integers in place of 1-D arrays are taken as raw device pointers and are not checked.
The stream defaults to torch's current stream on the current device.
"""
from __future__ import annotations

import ctypes
from pathlib import Path
from typing import Optional, Sequence

LIB_PATH = Path(__file__).resolve().with_name("libccjoin.so")

# Every symbol that include/cc_join.h declares.
EXPORTS = (
    "cc_store_create", "cc_store_destroy", "cc_store_info", "cc_store_invalid_count",
    "cc_store_reset_invalid_count", "cc_join", "cc_join_batched", "cc_join_batched_authors",
    "cc_join_batched_tuned",
    "cc_join_batched_padded", "cc_sort_workspace_bytes", "cc_sort_affinity",
    "cc_sort_affinity_method", "cc_sort_affinity_noalloc",
    "cc_store_create_indexed", "cc_set_ingestion_wait_limit", "cc_upsert_workspace_bytes",
    "cc_store_upsert", "cc_store_read",
    "cc_store_layout",
    "cc_resolve_ids",
    "cc_validate_keys", "cc_status_string", "cc_last_device_error",
)

CC_OK, CC_ERR_INVALID_ARGUMENT, CC_ERR_OUT_OF_MEMORY, CC_ERR_DEVICE = 0, 1, 2, 3
CC_ERR_UNSORTED_KEYS, CC_ERR_NOT_SUPPORTED, CC_ERR_STORE_FULL, CC_ERR_TOO_LARGE = 4, 5, 6, 7
CC_ERR_TIMEOUT = 8
SORT_NOALLOC_MAX_RECORDS, SORT_NOALLOC_MAX_VIEWERS = 1 << 20, 1 << 16
CC_SRC_HOST, CC_SRC_DEVICE = 1, 2


class CCError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.device_error = _lib.cc_last_device_error() if _lib is not None else 0
        super().__init__(f"{where}: {cc_status_string(status)}"
                         + (f" (hipError {self.device_error})" if status == CC_ERR_DEVICE else ""))


class Tuning(ctypes.Structure):
    """Launch tuning (cc_tuning); zero fields mean automatic. Results never depend on it."""
    _fields_ = [("fence_stride", ctypes.c_int32), ("lds_keys", ctypes.c_int32),
                ("workgroups", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None


def lib():
    """Load libccjoin.so (no fallback: raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(str(LIB_PATH))
        i64, i32, u32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p
        st = ctypes.c_int
        P64 = ctypes.POINTER(i64)
        sig = {
            "cc_store_create": [ctypes.POINTER(vp), i64, vp, vp, i32, u32, vp],
            "cc_store_destroy": [vp],
            "cc_store_info": [vp, P64, ctypes.POINTER(i32)],
            "cc_store_invalid_count": [vp, P64, vp],
            "cc_store_reset_invalid_count": [vp, vp],
            "cc_join": [vp, vp, i64, vp, i64, vp, i32, vp, vp, i64, vp, vp],
            "cc_join_batched": [vp, i32, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                ctypes.POINTER(vp), vp, i64, vp, vp],
            "cc_join_batched_authors": [vp, i32, vp, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                        ctypes.POINTER(vp), vp, i64, vp, vp],
            "cc_join_batched_tuned": [vp, i32, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                      ctypes.POINTER(vp), vp, i64, vp, ctypes.POINTER(Tuning),
                                      vp],
            "cc_join_batched_padded": [vp, i32, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                       ctypes.POINTER(vp), i64, vp, i64, vp, vp, vp],
            "cc_sort_affinity": [i32, vp, vp, vp, i32, i64, i64, vp, vp, vp, i64, vp],
            "cc_sort_affinity_method": [i32, i32, i32, vp, vp, vp, i32, i64, i64, vp, vp, vp, i64,
                                        vp],
            "cc_sort_affinity_noalloc": [i32, vp, vp, vp, i32, i64, i64, vp, vp, vp],
            "cc_store_create_indexed": [ctypes.POINTER(vp), i64, i32, vp],
            "cc_set_ingestion_wait_limit": [i32],
            "cc_store_upsert": [vp, i64, vp, vp, vp, vp, i64, P64, P64, vp],
            "cc_resolve_ids": [vp, vp, i64, vp, vp],
            "cc_store_read": [vp, i64, i64, vp, vp, vp],
            "cc_store_layout": [vp, ctypes.POINTER(i32), P64],
            "cc_validate_keys": [vp, vp, i32, i64, P64, vp],
            "cc_status_string": [st],
            "cc_last_device_error": [],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = st
        L.cc_status_string.restype = ctypes.c_char_p
        L.cc_sort_workspace_bytes.argtypes = [i64, i32]
        L.cc_sort_workspace_bytes.restype = i64
        L.cc_upsert_workspace_bytes.argtypes = [i64]
        L.cc_upsert_workspace_bytes.restype = i64
        _lib = L
    return _lib


def cc_status_string(status: int) -> str:
    return lib().cc_status_string(int(status)).decode()


def cc_last_device_error() -> int:
    return lib().cc_last_device_error()


def _check(status: int, where: str):
    if status != CC_OK:
        raise CCError(status, where)


_RAW_STREAM = None


def _current_stream() -> int:
    """Handle of torch's current stream on the current device. torch's raw-stream query costs
    a tenth of building a Stream object (about 0.3 us against 3 us per call); the public call
    is the fallback where the query is missing."""
    global _RAW_STREAM
    import torch
    if _RAW_STREAM is None:
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        _RAW_STREAM = (lambda: raw(torch.cuda.current_device())) if raw is not None else \
            (lambda: torch.cuda.current_stream().cuda_stream)
    return _RAW_STREAM()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return _current_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _prod(xs):
    p = 1
    for x in xs:
        p *= int(x)
    return p


# ---- checks the C ABI cannot make ----
# The library receives plain pointers. A host pointer, a buffer shorter than the sizes passed
# with it, or a strided view would reach a kernel as an out-of-bounds or unmapped access, so
# every tensor argument is checked here before the call: element type, dense layout, length
# and GPU residency. Offsets and keys held in device memory are not read here; the kernels
# clamp them.

def _fail(name: str, what: str, exc=ValueError):
    raise exc(f"{name}: {what}")


_DTYPES = None


def _i64():
    global _DTYPES
    if _DTYPES is None:
        import torch
        _DTYPES = (torch.int64, torch.int8)
    return _DTYPES[0]


def _i8():
    _i64()
    return _DTYPES[1]


def _row_bytes(x) -> int:
    """Bytes per row (dim 0 indexes rows; the trailing dims make up a row)."""
    if x.dim() == 2:
        return x.shape[1] * x.element_size()
    return _prod(x.shape[1:]) * x.element_size()


def _dense_from(x, d: int) -> bool:
    """Dims d.. of x are laid out row-major without gaps."""
    expect = 1
    for size, st in zip(reversed(x.shape[d:]), reversed(x.stride()[d:])):
        if size != 1 and st != expect:
            return False
        expect *= size
    return True


def _arr(x, name: str, dtype=None, numel: int = 0, optional: bool = False,
         gpu: bool = True) -> Optional[int]:
    """Pointer of a dense array of at least `numel` elements of `dtype`, in GPU memory unless
    `gpu` is False. None is allowed when `optional` or nothing is needed; an int is a raw device
    pointer and is passed through unchecked."""
    if x is None:
        if optional or numel == 0:
            return None
        _fail(name, "is required")
    if isinstance(x, int):
        return x
    if ((dtype is not None and x.dtype != dtype) or not x.is_contiguous()
            or x.numel() < numel or (gpu and not x.is_cuda)):
        if dtype is not None and x.dtype != dtype:
            _fail(name, f"must be {dtype} (is {x.dtype})", TypeError)
        if not x.is_contiguous():
            _fail(name, "must be contiguous")
        if x.numel() < numel:
            _fail(name, f"needs at least {numel} elements (has {x.numel()})")
        _fail(name, f"must be in GPU memory (is on {x.device})")
    return x.data_ptr()


def _bytes_arr(x, name: str, nbytes: int) -> Optional[int]:
    """Device pointer of a dense buffer of at least `nbytes` bytes (any element type), or None."""
    if x is None or isinstance(x, int):
        return x
    if x.numel() * x.element_size() < nbytes:
        _fail(name, f"needs at least {nbytes} bytes (has {x.numel() * x.element_size()})")
    return _arr(x, name)


def _rows(x, name: str, n: int, row_bytes: Optional[int] = None) -> Optional[int]:
    """Device pointer of a dense [>= n, ...] array of rows (of `row_bytes` bytes, if given)."""
    if x is None:
        if n == 0:
            return None
        _fail(name, "is required")
    if x.dim() < 1 or x.shape[0] < n:
        _fail(name, f"needs at least {n} rows (shape {tuple(x.shape)})")
    if row_bytes is not None and _row_bytes(x) != row_bytes:
        _fail(name, f"rows must be {row_bytes} bytes (are {_row_bytes(x)})")
    return _arr(x, name)


def _out_rows(out, name: str, n: int, width: int, per_group: int = 0):
    """(pointer, row stride in bytes) of an output of n rows whose rows may sit inside a wider
    tensor. Each row (the trailing dims) must be dense and hold `width` bytes. With per_group,
    a 3-D output [groups, per_group, row] is addressed as groups * per_group rows, so its outer
    stride must equal per_group row strides."""
    if out.dim() == 2 and out.stride(1) == 1:
        # the common case: [rows, bytes-per-row] with any row stride
        rows, rb, stride = out.shape[0], out.shape[1] * out.element_size(), out.stride(0)
    else:
        lead = 1
        if out.dim() == 3 and per_group:
            lead = 2
            if out.shape[1] != per_group:
                _fail(name, f"dim 1 must be n_max = {per_group} (shape {tuple(out.shape)})")
            if out.shape[0] > 1 and out.stride(0) != per_group * out.stride(1):
                _fail(name, "must address its slots with one row stride")
        if out.dim() <= lead or not _dense_from(out, lead):
            _fail(name, "rows must be dense (the trailing dims contiguous)")
        rows = _prod(out.shape[:lead])
        rb = _prod(out.shape[lead:]) * out.element_size()
        stride = out.stride(lead - 1)
    if rows < n:
        _fail(name, f"needs at least {n} rows (shape {tuple(out.shape)})")
    if rb < width:
        _fail(name, f"rows must hold at least {width} bytes (hold {rb})")
    if not out.is_cuda:
        _fail(name, f"must be in GPU memory (is on {out.device})")
    return out.data_ptr(), stride * out.element_size()


def _doc_row_bytes(store: int) -> int:
    return cc_store_info(store)[1]


def cc_store_create(author_ids, doc_rows, stream=None) -> int:
    """Copy (author_ids [n] int64, doc_rows [n, ...]) into a new device store; returns its handle.
    Both are host tensors or both are GPU tensors."""
    n = author_ids.numel()
    on_gpu = bool(author_ids.is_cuda)
    if bool(doc_rows.is_cuda) != on_gpu:
        _fail("doc_rows", "must be in the same memory (host or GPU) as author_ids")
    if doc_rows.dim() < 1 or doc_rows.shape[0] != n:
        _fail("doc_rows", f"needs {n} rows, one per author id (shape {tuple(doc_rows.shape)})")
    pa = _arr(author_ids, "author_ids", _i64(), gpu=on_gpu)
    pr = _arr(doc_rows, "doc_rows", gpu=on_gpu)
    flags = CC_SRC_DEVICE if on_gpu else CC_SRC_HOST
    h = ctypes.c_void_p()
    _check(lib().cc_store_create(ctypes.byref(h), n, pa, pr, _row_bytes(doc_rows), flags,
                                 _stream(stream)), "cc_store_create")
    return h.value


def cc_store_create_indexed(capacity: int, doc_row_bytes: int, stream=None) -> int:
    """An empty store with a document-id map for `capacity` documents; returns its handle."""
    h = ctypes.c_void_p()
    _check(lib().cc_store_create_indexed(ctypes.byref(h), capacity, doc_row_bytes,
                                         _stream(stream)), "cc_store_create_indexed")
    return h.value


def cc_set_ingestion_wait_limit(polls: int) -> None:
    """Bound (in polls) on every device-side wait of an ingestion batch; a batch in which one
    gives up is rolled back and cc_store_upsert raises CCError(CC_ERR_TIMEOUT). 0 makes every
    such wait give up at once; a negative value restores the default. Process-wide."""
    _check(lib().cc_set_ingestion_wait_limit(int(polls)), "cc_set_ingestion_wait_limit")


def cc_upsert_workspace_bytes(n_records: int) -> int:
    return lib().cc_upsert_workspace_bytes(n_records)


def cc_store_upsert(store: int, doc_ids, author_ids, doc_rows, workspace, stream=None):
    """Apply one ingestion batch (§6.2); returns (n_new, n_rejected). Synchronises the stream.
    Raises CCError with status CC_ERR_STORE_FULL (store unchanged) when the batch does not fit,
    CC_ERR_TIMEOUT (store unchanged) when a bounded device-side wait gave up."""
    n = doc_ids.numel()
    pi = _arr(doc_ids, "doc_ids", _i64())
    pa = _arr(author_ids, "author_ids", _i64(), n)
    pr = _rows(doc_rows, "doc_rows", n, _doc_row_bytes(store))
    pw = _arr(workspace, "workspace", optional=True)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    nn, nr = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().cc_store_upsert(store, n, pi, pa, pr, pw, ws_bytes, ctypes.byref(nn),
                                 ctypes.byref(nr), _stream(stream)), "cc_store_upsert")
    return nn.value, nr.value


def cc_store_read(store: int, first: int, count: int, author_out=None, rows_out=None,
                  stream=None) -> None:
    """Copy positions [first, first + count) of the store into device buffers."""
    n = max(int(count), 0)
    pa = _arr(author_out, "author_out", _i64(), n, optional=True)
    pr = None if rows_out is None else _bytes_arr(rows_out, "rows_out",
                                                  n * _doc_row_bytes(store))
    _check(lib().cc_store_read(store, first, count, pa, pr, _stream(stream)), "cc_store_read")


def cc_resolve_ids(store: int, doc_ids, positions, stream=None) -> None:
    """Eq. 6 (§6.3.1): positions[i] = store position of doc_ids[i], or -1."""
    n = doc_ids.numel()
    pi = _arr(doc_ids, "doc_ids", _i64())
    pp = _arr(positions, "positions", _i64(), n)
    _check(lib().cc_resolve_ids(store, pi, n, pp, _stream(stream)), "cc_resolve_ids")


def cc_store_destroy(store: int) -> None:
    _check(lib().cc_store_destroy(store), "cc_store_destroy")


def cc_store_info(store: int):
    n, w = ctypes.c_int64(), ctypes.c_int32()
    _check(lib().cc_store_info(store, ctypes.byref(n), ctypes.byref(w)), "cc_store_info")
    return n.value, w.value


def cc_store_layout(store: int):
    """(author id bytes the joins read: 4 or 8, capacity)."""
    b, c = ctypes.c_int32(), ctypes.c_int64()
    _check(lib().cc_store_layout(store, ctypes.byref(b), ctypes.byref(c)), "cc_store_layout")
    return b.value, c.value


def cc_store_invalid_count(store: int, stream=None) -> int:
    c = ctypes.c_int64()
    _check(lib().cc_store_invalid_count(store, ctypes.byref(c), _stream(stream)),
           "cc_store_invalid_count")
    return c.value


def cc_store_reset_invalid_count(store: int, stream=None) -> None:
    _check(lib().cc_store_reset_invalid_count(store, _stream(stream)),
           "cc_store_reset_invalid_count")


def _edge_args(edge_keys, edge_feats, tk: int, default_row):
    """Checked pointers (keys, rows, default row) and the edge row width in bytes."""
    pk = _arr(edge_keys, "edge_keys", _i64(), tk)
    ew = _row_bytes(edge_feats)
    pf = _rows(edge_feats, "edge_feats", tk)
    pd = _bytes_arr(default_row, "default_row", ew)
    return pk, pf, pd, ew


def cc_join(store: int, cand_idx, edge_keys, edge_feats, out, hit_mask, default_row=None,
            stream=None) -> None:
    """One viewer (see include/cc_join.h). out is [n_cand, >= doc+edge bytes] (any dtype)."""
    n = cand_idx.numel()
    pc = _arr(cand_idx, "cand_idx", _i64())
    pk, pf, pd, ew = _edge_args(edge_keys, edge_feats, edge_keys.numel(), default_row)
    po, stride = _out_rows(out, "out", n, _doc_row_bytes(store) + ew)
    ph = _arr(hit_mask, "hit_mask", _i8(), n)
    _check(lib().cc_join(store, pc, n, pk, edge_keys.numel(), pf, ew, pd, po, stride, ph,
                         _stream(stream)), "cc_join")


class PreparedJoin:
    """cc_join with its arguments checked once, for serving loops that reuse the same buffers.

    The constructor runs every check of cc_join on buffers sized for the largest request and keeps
    the tensors alive. A call then writes the next request's candidates and keys into those
    buffers' leading elements and passes only the counts: ``prepared(n_cand, n_keys)`` joins
    cand_idx[:n_cand] against edge_keys[:n_keys] / edge_feats[:n_keys] into out[:n_cand] and
    hit_mask[:n_cand]. Counts default to the full buffers and must not exceed them. Same C call
    and semantics as cc_join; only the per-call Python work is smaller. The object keeps its
    tensors referenced and their device pointers fixed: resizing a buffer in place
    (``Tensor.resize_``, ``set_``) would leave it with a stale pointer, so build a new one instead.
    """

    def __init__(self, store: int, cand_idx, edge_keys, edge_feats, out, hit_mask,
                 default_row=None):
        self._cap_n = cand_idx.numel()
        self._cap_k = edge_keys.numel()
        pc = _arr(cand_idx, "cand_idx", _i64())
        pk, pf, pd, ew = _edge_args(edge_keys, edge_feats, self._cap_k, default_row)
        po, stride = _out_rows(out, "out", self._cap_n, _doc_row_bytes(store) + ew)
        ph = _arr(hit_mask, "hit_mask", _i8(), self._cap_n)
        self._keep = (cand_idx, edge_keys, edge_feats, out, hit_mask, default_row)
        self._head = (store, pc)
        self._mid = (pk,)
        self._tail = (pf, ew, pd, po, stride, ph)
        self._fn = lib().cc_join

    def __call__(self, n_cand: Optional[int] = None, n_keys: Optional[int] = None,
                 stream=None) -> None:
        n = self._cap_n if n_cand is None else n_cand
        k = self._cap_k if n_keys is None else n_keys
        if not (0 <= n <= self._cap_n and 0 <= k <= self._cap_k):
            _fail("counts", f"must lie in [0, {self._cap_n}] and [0, {self._cap_k}] "
                            f"(got {n}, {k})")
        st = self._fn(*self._head, n, *self._mid, k, *self._tail, _stream(stream))
        if st != CC_OK:
            raise CCError(st, "cc_join")


class PreparedJoinBatched:
    """cc_join_batched with its arguments checked once (see PreparedJoin).

    Buffers are sized for the largest batch. A call passes the batch's viewer count and totals:
    ``prepared(n_viewers, total_cand, total_keys)`` joins the CSR batch described by
    cand_offsets[:n_viewers + 1] and key_offsets[:n_viewers + 1] (device contents written by the
    caller, as for cc_join_batched) over the leading elements of the other buffers. Counts
    default to the full buffers and must not exceed them.
    """

    def __init__(self, store: int, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats,
                 out, hit_mask, default_row=None, extra_keys: Optional[Sequence] = None,
                 author_ids=None):
        B, L, tc, tk, pco, pc, pko, pk, pf, pd, ex, ew = _batched_args(
            store, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, default_row,
            extra_keys, None, None)
        po, stride = _out_rows(out, "out", tc, _doc_row_bytes(store) + L * ew)
        ph = _arr(hit_mask, "hit_mask", _i8(), tc * L)
        self._cap = (B, tc, tk)
        self._keep = (cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, out, hit_mask,
                      default_row, extra_keys, ex, author_ids)
        self._a = (store, pco, pc, pko, pk, pf, ew, pd, L, ex, po, stride, ph)
        # With author_ids ([total_cand] int64 buffer), cc_join_batched_authors.
        self._pa = None if author_ids is None else _arr(author_ids, "author_ids", _i64(), tc)
        self._fn = lib().cc_join_batched

    def __call__(self, n_viewers: Optional[int] = None, total_cand: Optional[int] = None,
                 total_keys: Optional[int] = None, stream=None) -> None:
        B, tc, tk = self._cap
        b = B if n_viewers is None else n_viewers
        n = tc if total_cand is None else total_cand
        k = tk if total_keys is None else total_keys
        if not (0 <= b <= B and 0 <= n <= tc and 0 <= k <= tk):
            _fail("counts", f"must lie in [0, {B}], [0, {tc}] and [0, {tk}] (got {b}, {n}, {k})")
        store, pco, pc, pko, pk, pf, ew, pd, L, ex, po, stride, ph = self._a
        if self._pa is not None:
            st = lib().cc_join_batched_authors(store, b, pco, pc, self._pa, n, pko, pk, k, pf, ew,
                                               pd, L, ex, po, stride, ph, _stream(stream))
            if st != CC_OK:
                raise CCError(st, "cc_join_batched_authors")
            return
        st = self._fn(store, b, pco, pc, n, pko, pk, k, pf, ew, pd, L, ex, po, stride, ph,
                      _stream(stream))
        if st != CC_OK:
            raise CCError(st, "cc_join_batched")


def _batched_args(store, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats,
                  default_row, extra_keys, total_cand, total_keys):
    """Checked inputs of the batched joins: (B, L, pointers..., extra array, edge width)."""
    n_lookups = 1 + (len(extra_keys) if extra_keys else 0)
    B = cand_offsets.numel() - 1
    tc = cand_idx.numel() if total_cand is None else int(total_cand)
    tk = edge_keys.numel() if total_keys is None else int(total_keys)
    pco = _arr(cand_offsets, "cand_offsets", _i64(), 1)
    pko = _arr(key_offsets, "key_offsets", _i64(), B + 1)
    pc = _arr(cand_idx, "cand_idx", _i64(), tc)
    pk, pf, pd, ew = _edge_args(edge_keys, edge_feats, tk, default_row)
    ex = None
    if extra_keys:
        ex = (ctypes.c_void_p * len(extra_keys))(
            *[_arr(e, f"extra_keys[{i}]", _i64(), tc) for i, e in enumerate(extra_keys)])
    return B, n_lookups, tc, tk, pco, pc, pko, pk, pf, pd, ex, ew


def cc_join_batched(store: int, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, out,
                    hit_mask, default_row=None, extra_keys: Optional[Sequence] = None,
                    total_cand: Optional[int] = None, total_keys: Optional[int] = None,
                    tuning: Optional[Tuning] = None, stream=None, author_ids=None) -> None:
    """B viewers in CSR form, 1 + len(extra_keys) lookups (see include/cc_join.h). With
    `author_ids` ([total_cand] int64), lookup 0 searches the caller's author id of each
    candidate instead of the store's (cc_join_batched_authors)."""
    B, L, tc, tk, pco, pc, pko, pk, pf, pd, ex, ew = _batched_args(
        store, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, default_row,
        extra_keys, total_cand, total_keys)
    po, stride = _out_rows(out, "out", tc, _doc_row_bytes(store) + L * ew)
    ph = _arr(hit_mask, "hit_mask", _i8(), tc * L)
    if author_ids is not None:
        if tuning is not None:
            raise ValueError("author_ids and tuning cannot be combined")
        pa = _arr(author_ids, "author_ids", _i64(), tc)
        _check(lib().cc_join_batched_authors(store, B, pco, pc, pa, tc, pko, pk, tk, pf, ew, pd,
                                             L, ex, po, stride, ph, _stream(stream)),
               "cc_join_batched_authors")
        return
    args = (store, B, pco, pc, tc, pko, pk, tk, pf, ew, pd, L, ex, po, stride, ph)
    if tuning is None:
        _check(lib().cc_join_batched(*args, _stream(stream)), "cc_join_batched")
    else:
        _check(lib().cc_join_batched_tuned(*args, ctypes.byref(tuning), _stream(stream)),
               "cc_join_batched_tuned")


def cc_join_batched_padded(store: int, cand_offsets, cand_idx, key_offsets, edge_keys,
                           edge_feats, n_max: int, out, hit_mask, valid_mask, default_row=None,
                           extra_keys: Optional[Sequence] = None,
                           total_cand: Optional[int] = None, total_keys: Optional[int] = None,
                           stream=None) -> None:
    """B viewers written into the padded [B, n_max] layout (see include/cc_join.h). out is
    [B, n_max, >= row bytes] or [B * n_max, >= row bytes]."""
    B, L, tc, tk, pco, pc, pko, pk, pf, pd, ex, ew = _batched_args(
        store, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, default_row,
        extra_keys, total_cand, total_keys)
    slots = max(B, 0) * max(int(n_max), 0)
    po, stride = _out_rows(out, "out", slots, _doc_row_bytes(store) + L * ew,
                           per_group=max(int(n_max), 0))
    ph = _arr(hit_mask, "hit_mask", _i8(), slots * L)
    pv = _arr(valid_mask, "valid_mask", _i8(), slots)
    _check(lib().cc_join_batched_padded(store, B, pco, pc, tc, pko, pk, tk, pf, ew, pd, L, ex,
                                        n_max, po, stride, ph, pv, _stream(stream)),
           "cc_join_batched_padded")


def cc_sort_workspace_bytes(total_keys: int, n_viewers: int) -> int:
    return lib().cc_sort_workspace_bytes(total_keys, n_viewers)


SORT_AUTO, SORT_MERGE, SORT_RADIX = 0, 1, 2
SORT_RADIX_MIN_RECORDS = 1 << 20       # CC_SORT_AUTO takes the radix method from this many records


def cc_sort_affinity(key_offsets, keys_in, rows_in, keys_out, rows_out, workspace,
                     max_keys: int = 0, total_keys: Optional[int] = None, stream=None,
                     method: int = SORT_AUTO, key_bits: int = 0) -> None:
    """Stable per-viewer sort of affinity records (Alg. 1 Step 1; see include/cc_join.h).
    With the defaults this is cc_sort_affinity; a `method` (CC_SORT_MERGE, CC_SORT_RADIX) or a
    `key_bits` bound on the keys' span calls cc_sort_affinity_method."""
    B = key_offsets.numel() - 1
    tk = keys_in.numel() if total_keys is None else int(total_keys)
    rb = _row_bytes(rows_in)
    pko = _arr(key_offsets, "key_offsets", _i64(), 1)
    pki = _arr(keys_in, "keys_in", _i64(), tk)
    pri = _rows(rows_in, "rows_in", tk)
    pk = _arr(keys_out, "keys_out", _i64(), tk)
    pr = _rows(rows_out, "rows_out", tk, rb)
    pw = _arr(workspace, "workspace")
    ws_bytes = workspace.numel() * workspace.element_size()
    if method == SORT_AUTO and key_bits == 0:
        _check(lib().cc_sort_affinity(B, pko, pki, pri, rb, tk, max_keys, pk, pr, pw, ws_bytes,
                                      _stream(stream)), "cc_sort_affinity")
    else:
        _check(lib().cc_sort_affinity_method(int(method), int(key_bits), B, pko, pki, pri, rb, tk,
                                             max_keys, pk, pr, pw, ws_bytes, _stream(stream)),
               "cc_sort_affinity_method")


def cc_sort_affinity_noalloc(key_offsets, keys_in, rows_in, keys_out, rows_out,
                             max_keys: int = 0, total_keys: Optional[int] = None,
                             stream=None) -> None:
    """cc_sort_affinity with the library's fixed per-device scratch instead of a workspace (for
    callers that cannot allocate; calls on one device must not overlap)."""
    B = key_offsets.numel() - 1
    tk = keys_in.numel() if total_keys is None else int(total_keys)
    rb = _row_bytes(rows_in)
    pko = _arr(key_offsets, "key_offsets", _i64(), 1)
    pki = _arr(keys_in, "keys_in", _i64(), tk)
    pri = _rows(rows_in, "rows_in", tk)
    pk = _arr(keys_out, "keys_out", _i64(), tk)
    pr = _rows(rows_out, "rows_out", tk, rb)
    _check(lib().cc_sort_affinity_noalloc(B, pko, pki, pri, rb, tk, max_keys, pk, pr,
                                          _stream(stream)), "cc_sort_affinity_noalloc")


def cc_validate_keys(key_offsets, edge_keys, total_keys: Optional[int] = None, stream=None):
    """Returns -1 when every viewer's keys are strictly increasing, else the first bad viewer."""
    bad = ctypes.c_int64()
    tk = edge_keys.numel() if total_keys is None else int(total_keys)
    pko = _arr(key_offsets, "key_offsets", _i64(), 1)
    pk = _arr(edge_keys, "edge_keys", _i64(), tk)
    st = lib().cc_validate_keys(pko, pk, key_offsets.numel() - 1, tk, ctypes.byref(bad),
                                _stream(stream))
    if st == CC_ERR_UNSORTED_KEYS:
        return bad.value
    _check(st, "cc_validate_keys")
    return -1
