"""ctypes binding of libccjoin.so: argument marshalling only.

Tensor arguments are anything with ``data_ptr()``, ``numel()``, ``element_size()`` and
``shape`` (torch tensors in practice); plain integers are taken as raw device pointers. The
stream defaults to torch's current stream on the current device.
"""
from __future__ import annotations

import ctypes
from pathlib import Path
from typing import Optional, Sequence

LIB_PATH = Path(__file__).resolve().with_name("libccjoin.so")

# Every symbol that include/cc_join.h declares.
EXPORTS = (
    "cc_store_create", "cc_store_destroy", "cc_store_info", "cc_store_invalid_count",
    "cc_store_reset_invalid_count", "cc_join", "cc_join_batched", "cc_join_batched_tuned",
    "cc_join_batched_padded", "cc_sort_workspace_bytes", "cc_sort_affinity",
    "cc_store_create_indexed", "cc_upsert_workspace_bytes", "cc_store_upsert", "cc_store_read",
    "cc_store_layout",
    "cc_resolve_ids",
    "cc_validate_keys", "cc_status_string", "cc_last_device_error",
)

CC_OK, CC_ERR_INVALID_ARGUMENT, CC_ERR_OUT_OF_MEMORY, CC_ERR_DEVICE = 0, 1, 2, 3
CC_ERR_UNSORTED_KEYS, CC_ERR_NOT_SUPPORTED, CC_ERR_STORE_FULL = 4, 5, 6
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
            "cc_join_batched_tuned": [vp, i32, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                      ctypes.POINTER(vp), vp, i64, vp, ctypes.POINTER(Tuning),
                                      vp],
            "cc_join_batched_padded": [vp, i32, vp, vp, i64, vp, vp, i64, vp, i32, vp, i32,
                                       ctypes.POINTER(vp), i64, vp, i64, vp, vp, vp],
            "cc_sort_affinity": [i32, vp, vp, vp, i32, i64, i64, vp, vp, vp, i64, vp],
            "cc_store_create_indexed": [ctypes.POINTER(vp), i64, i32, vp],
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


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _prod(xs):
    p = 1
    for x in xs:
        p *= int(x)
    return p


def _out_stride(out) -> int:
    return out.stride(0) * out.element_size()


def cc_store_create(author_ids, doc_rows, stream=None) -> int:
    """Copy (author_ids [n] int64, doc_rows [n, ...]) into a new device store; returns its handle."""
    n = author_ids.numel()
    flags = CC_SRC_DEVICE if getattr(author_ids, "is_cuda", False) else CC_SRC_HOST
    h = ctypes.c_void_p()
    _check(lib().cc_store_create(ctypes.byref(h), n, _ptr(author_ids), _ptr(doc_rows),
                                 int(_prod(doc_rows.shape[1:])) * doc_rows.element_size(),
                                 flags, _stream(stream)), "cc_store_create")
    return h.value


def cc_store_create_indexed(capacity: int, doc_row_bytes: int, stream=None) -> int:
    """An empty store with a document-id map for `capacity` documents; returns its handle."""
    h = ctypes.c_void_p()
    _check(lib().cc_store_create_indexed(ctypes.byref(h), capacity, doc_row_bytes,
                                         _stream(stream)), "cc_store_create_indexed")
    return h.value


def cc_upsert_workspace_bytes(n_records: int) -> int:
    return lib().cc_upsert_workspace_bytes(n_records)


def cc_store_upsert(store: int, doc_ids, author_ids, doc_rows, workspace, stream=None):
    """Apply one ingestion batch (§6.2); returns (n_new, n_rejected). Synchronises the stream.
    Raises CCError with status CC_ERR_STORE_FULL (store unchanged) when the batch does not fit."""
    n = doc_ids.numel()
    nn, nr = ctypes.c_int64(), ctypes.c_int64()
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().cc_store_upsert(store, n, _ptr(doc_ids), _ptr(author_ids), _ptr(doc_rows),
                                 _ptr(workspace), ws_bytes, ctypes.byref(nn), ctypes.byref(nr),
                                 _stream(stream)), "cc_store_upsert")
    return nn.value, nr.value


def cc_store_read(store: int, first: int, count: int, author_out=None, rows_out=None,
                  stream=None) -> None:
    """Copy positions [first, first + count) of the store into device buffers."""
    _check(lib().cc_store_read(store, first, count, _ptr(author_out), _ptr(rows_out),
                               _stream(stream)), "cc_store_read")


def cc_resolve_ids(store: int, doc_ids, positions, stream=None) -> None:
    """Eq. 6 (§6.3.1): positions[i] = store position of doc_ids[i], or -1."""
    _check(lib().cc_resolve_ids(store, _ptr(doc_ids), doc_ids.numel(), _ptr(positions),
                                _stream(stream)), "cc_resolve_ids")


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


def cc_join(store: int, cand_idx, edge_keys, edge_feats, out, hit_mask, default_row=None,
            stream=None) -> None:
    """One viewer (see include/cc_join.h). out is [n_cand, >= doc+edge bytes] (any dtype)."""
    ew = int(_prod(edge_feats.shape[1:])) * edge_feats.element_size()
    _check(lib().cc_join(store, _ptr(cand_idx), cand_idx.numel(), _ptr(edge_keys),
                         edge_keys.numel(), _ptr(edge_feats), ew, _ptr(default_row), _ptr(out),
                         _out_stride(out), _ptr(hit_mask), _stream(stream)), "cc_join")


def cc_join_batched(store: int, cand_offsets, cand_idx, key_offsets, edge_keys, edge_feats, out,
                    hit_mask, default_row=None, extra_keys: Optional[Sequence] = None,
                    total_cand: Optional[int] = None, total_keys: Optional[int] = None,
                    tuning: Optional[Tuning] = None, stream=None) -> None:
    """B viewers in CSR form, 1 + len(extra_keys) lookups (see include/cc_join.h)."""
    n_lookups = 1 + (len(extra_keys) if extra_keys else 0)
    ex = None
    if extra_keys:
        ex = (ctypes.c_void_p * len(extra_keys))(*[_ptr(e) for e in extra_keys])
    ew = int(_prod(edge_feats.shape[1:])) * edge_feats.element_size()
    tc = cand_idx.numel() if total_cand is None else total_cand
    tk = edge_keys.numel() if total_keys is None else total_keys
    args = (store, cand_offsets.numel() - 1, _ptr(cand_offsets), _ptr(cand_idx), tc,
            _ptr(key_offsets), _ptr(edge_keys), tk, _ptr(edge_feats), ew, _ptr(default_row),
            n_lookups, ex, _ptr(out), _out_stride(out), _ptr(hit_mask))
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
    """B viewers written into the padded [B, n_max] layout (see include/cc_join.h)."""
    n_lookups = 1 + (len(extra_keys) if extra_keys else 0)
    ex = None
    if extra_keys:
        ex = (ctypes.c_void_p * len(extra_keys))(*[_ptr(e) for e in extra_keys])
    ew = int(_prod(edge_feats.shape[1:])) * edge_feats.element_size()
    tc = cand_idx.numel() if total_cand is None else total_cand
    tk = edge_keys.numel() if total_keys is None else total_keys
    stride = out.stride(-2) * out.element_size() if out.dim() == 3 else _out_stride(out)
    _check(lib().cc_join_batched_padded(
        store, cand_offsets.numel() - 1, _ptr(cand_offsets), _ptr(cand_idx), tc,
        _ptr(key_offsets), _ptr(edge_keys), tk, _ptr(edge_feats), ew, _ptr(default_row),
        n_lookups, ex, n_max, _ptr(out), stride, _ptr(hit_mask), _ptr(valid_mask),
        _stream(stream)), "cc_join_batched_padded")


def cc_sort_workspace_bytes(total_keys: int, n_viewers: int) -> int:
    return lib().cc_sort_workspace_bytes(total_keys, n_viewers)


def cc_sort_affinity(key_offsets, keys_in, rows_in, keys_out, rows_out, workspace,
                     max_keys: int = 0, total_keys: Optional[int] = None, stream=None) -> None:
    """Stable per-viewer sort of affinity records (Alg. 1 Step 1; see include/cc_join.h)."""
    tk = keys_in.numel() if total_keys is None else total_keys
    rb = int(_prod(rows_in.shape[1:])) * rows_in.element_size()
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().cc_sort_affinity(key_offsets.numel() - 1, _ptr(key_offsets), _ptr(keys_in),
                                  _ptr(rows_in), rb, tk, max_keys, _ptr(keys_out),
                                  _ptr(rows_out), _ptr(workspace), ws_bytes, _stream(stream)),
           "cc_sort_affinity")


def cc_validate_keys(key_offsets, edge_keys, total_keys: Optional[int] = None, stream=None):
    """Returns -1 when every viewer's keys are strictly increasing, else the first bad viewer."""
    bad = ctypes.c_int64()
    tk = edge_keys.numel() if total_keys is None else total_keys
    st = lib().cc_validate_keys(_ptr(key_offsets), _ptr(edge_keys), key_offsets.numel() - 1, tk,
                                ctypes.byref(bad), _stream(stream))
    if st == CC_ERR_UNSORTED_KEYS:
        return bad.value
    _check(st, "cc_validate_keys")
    return -1
