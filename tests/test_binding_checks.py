"""The Python binding's argument checks (CPU only).

The C ABI receives plain pointers and cannot see a buffer's length, element type, layout or
memory kind, so the binding checks them before every call. These tests run the checks on the
CPU: `OnGpu` wraps a host tensor and reports GPU residency, and a stub library records the calls
that get through, so no call reaches the real library.
"""
import pytest
import torch

import paper_2609_22441_amd.binding as B


class OnGpu:
    """A host tensor that reports GPU residency, so the binding's checks run on the CPU."""
    is_cuda = True

    def __init__(self, t):
        self.t = t

    def __getattr__(self, k):
        return getattr(self.t, k)


class StubLib:
    """Records each library call; every call succeeds."""

    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def call(*args):
            self.calls.append((name, args))
            return 0
        return call


DOC_BYTES = 32


@pytest.fixture
def stub(monkeypatch):
    s = StubLib()
    monkeypatch.setattr(B, "lib", lambda: s)
    monkeypatch.setattr(B, "_doc_row_bytes", lambda store: DOC_BYTES)
    return s


def g(*shape, dtype=torch.int64):
    return OnGpu(torch.zeros(*shape, dtype=dtype))


def join_args(n=10, k=6, ew=16):
    return dict(cand_idx=g(n), edge_keys=g(k), edge_feats=g(k, ew, dtype=torch.uint8),
                out=g(n, DOC_BYTES + ew, dtype=torch.uint8), hit_mask=g(n, 1, dtype=torch.int8))


def test_valid_join_reaches_the_library(stub):
    a = join_args()
    B.cc_join(1, stream=0, **a)
    (name, args), = stub.calls
    assert name == "cc_join"
    assert args[2] == 10 and args[4] == 6 and args[6] == 16    # n_cand, n_keys, edge row bytes
    assert args[9] == DOC_BYTES + 16                           # row stride in bytes


def test_rows_inside_a_wider_tensor(stub):
    a = join_args()
    wide = torch.zeros(10, 80, dtype=torch.uint8)
    a["out"] = OnGpu(wide[:, :DOC_BYTES + 16])                 # rows 80 bytes apart
    B.cc_join(1, stream=0, **a)
    assert stub.calls[0][1][9] == 80


@pytest.mark.parametrize("arg,bad,exc,match", [
    ("cand_idx", torch.zeros(10, dtype=torch.int64), ValueError, "GPU memory"),
    ("cand_idx", g(10, dtype=torch.int32), TypeError, "int64"),
    ("cand_idx", OnGpu(torch.zeros(20, dtype=torch.int64)[::2]), ValueError, "contiguous"),
    ("edge_keys", g(6, dtype=torch.float64), TypeError, "int64"),
    ("edge_feats", g(5, 16, dtype=torch.uint8), ValueError, "rows"),
    ("hit_mask", g(9, 1, dtype=torch.int8), ValueError, "elements"),
    ("hit_mask", g(10, 1, dtype=torch.bool), TypeError, "int8"),
    ("out", g(9, DOC_BYTES + 16, dtype=torch.uint8), ValueError, "rows"),
    ("out", g(10, DOC_BYTES, dtype=torch.uint8), ValueError, "bytes"),
    ("out", OnGpu(torch.zeros(DOC_BYTES + 16, 10, dtype=torch.uint8).t()), ValueError, "dense"),
    ("out", torch.zeros(10, DOC_BYTES + 16, dtype=torch.uint8), ValueError, "GPU memory"),
])
def test_join_rejects(stub, arg, bad, exc, match):
    a = join_args()
    a[arg] = bad
    with pytest.raises(exc, match=match):
        B.cc_join(1, stream=0, **a)
    assert stub.calls == []


def test_default_row_must_cover_an_edge_row(stub):
    a = join_args()
    with pytest.raises(ValueError, match="bytes"):
        B.cc_join(1, default_row=g(8, dtype=torch.uint8), stream=0, **a)
    B.cc_join(1, default_row=g(16, dtype=torch.uint8), stream=0, **a)
    assert len(stub.calls) == 1


def batched_args(b=3, n=12, k=9, ew=16, lookups=1):
    return dict(cand_offsets=g(b + 1), cand_idx=g(n), key_offsets=g(b + 1), edge_keys=g(k),
                edge_feats=g(k, ew, dtype=torch.uint8),
                out=g(n, DOC_BYTES + lookups * ew, dtype=torch.uint8),
                hit_mask=g(n, lookups, dtype=torch.int8),
                extra_keys=[g(n)] if lookups == 2 else None)


def test_valid_batched_join_reaches_the_library(stub):
    B.cc_join_batched(1, stream=0, **batched_args(lookups=2))
    (name, args), = stub.calls
    assert name == "cc_join_batched"
    assert args[1] == 3 and args[4] == 12 and args[7] == 9 and args[11] == 2
    assert args[14] == DOC_BYTES + 32


@pytest.mark.parametrize("arg,bad,match", [
    ("key_offsets", g(3), "elements"),                         # needs B + 1 = 4
    ("cand_offsets", g(0), "elements"),
    ("hit_mask", g(12, 1, dtype=torch.int8), "elements"),      # two lookups need 24
    ("out", g(12, DOC_BYTES + 16, dtype=torch.uint8), "bytes"),
    ("extra_keys", [g(11)], "elements"),
])
def test_batched_join_rejects(stub, arg, bad, match):
    a = batched_args(lookups=2)
    a[arg] = bad
    with pytest.raises(ValueError, match=match):
        B.cc_join_batched(1, stream=0, **a)
    assert stub.calls == []


def test_explicit_totals_must_fit_the_arrays(stub):
    with pytest.raises(ValueError, match="cand_idx"):
        B.cc_join_batched(1, total_cand=13, stream=0, **batched_args())
    with pytest.raises(ValueError, match="edge_keys"):
        B.cc_join_batched(1, total_keys=10, stream=0, **batched_args())
    B.cc_join_batched(1, total_cand=5, total_keys=4, stream=0, **batched_args())
    assert stub.calls[0][1][4] == 5 and stub.calls[0][1][7] == 4


def padded_args(b=3, n_max=4, ew=16):
    a = batched_args(b=b, ew=ew)
    a.update(out=g(b, n_max, DOC_BYTES + ew, dtype=torch.uint8),
             hit_mask=g(b, n_max, 1, dtype=torch.int8), valid_mask=g(b, n_max, dtype=torch.int8),
             n_max=n_max)
    return a


def test_padded_layouts(stub):
    B.cc_join_batched_padded(1, stream=0, **padded_args())
    assert stub.calls[-1][1][15] == DOC_BYTES + 16
    a = padded_args()
    a["out"] = g(12, DOC_BYTES + 16, dtype=torch.uint8)       # flat [B * n_max, row]
    B.cc_join_batched_padded(1, stream=0, **a)
    assert len(stub.calls) == 2


@pytest.mark.parametrize("arg,bad,match", [
    ("out", g(3, 5, DOC_BYTES + 16, dtype=torch.uint8), "n_max"),
    ("out", OnGpu(torch.zeros(3, 8, DOC_BYTES + 16, dtype=torch.uint8)[:, :4]), "one row stride"),
    ("valid_mask", g(3, 3, dtype=torch.int8), "elements"),
    ("hit_mask", g(3, 3, 1, dtype=torch.int8), "elements"),
])
def test_padded_rejects(stub, arg, bad, match):
    a = padded_args()
    a[arg] = bad
    with pytest.raises(ValueError, match=match):
        B.cc_join_batched_padded(1, stream=0, **a)
    assert stub.calls == []


def sort_args(b=2, n=10, rb=64):
    return dict(key_offsets=g(b + 1), keys_in=g(n), rows_in=g(n, rb, dtype=torch.uint8),
                keys_out=g(n), rows_out=g(n, rb, dtype=torch.uint8),
                workspace=g(4096, dtype=torch.uint8))


@pytest.mark.parametrize("arg,bad,match", [
    (None, None, None),
    ("rows_out", g(10, 32, dtype=torch.uint8), "bytes"),
    ("rows_out", g(9, 64, dtype=torch.uint8), "rows"),
    ("keys_out", g(9), "elements"),
    ("rows_in", g(9, 64, dtype=torch.uint8), "rows"),
    ("workspace", torch.zeros(4096, dtype=torch.uint8), "GPU memory"),
])
def test_sort_checks(stub, arg, bad, match):
    a = sort_args()
    if arg is None:
        B.cc_sort_affinity(stream=0, **a)
        assert stub.calls[0][1][4] == 64 and stub.calls[0][1][5] == 10
        return
    a[arg] = bad
    with pytest.raises(ValueError, match=match):
        B.cc_sort_affinity(stream=0, **a)
    assert stub.calls == []


def test_store_and_map_checks(stub):
    ids, rows = g(5), g(5, DOC_BYTES, dtype=torch.uint8)
    with pytest.raises(ValueError, match="same memory"):
        B.cc_store_create(ids, torch.zeros(5, DOC_BYTES, dtype=torch.uint8), stream=0)
    with pytest.raises(ValueError, match="5 rows"):
        B.cc_store_create(ids, g(4, DOC_BYTES, dtype=torch.uint8), stream=0)
    with pytest.raises(TypeError, match="int64"):
        B.cc_store_create(torch.zeros(5, dtype=torch.int32),
                          torch.zeros(5, DOC_BYTES, dtype=torch.uint8), stream=0)
    with pytest.raises(ValueError, match="elements"):
        B.cc_resolve_ids(1, ids, g(4), stream=0)
    with pytest.raises(ValueError, match="bytes"):
        B.cc_store_upsert(1, ids, ids, g(5, 16, dtype=torch.uint8), g(64, dtype=torch.uint8),
                          stream=0)
    with pytest.raises(ValueError, match="bytes"):
        B.cc_store_read(1, 0, 5, None, g(4, DOC_BYTES, dtype=torch.uint8), stream=0)
    with pytest.raises(ValueError, match="elements"):
        B.cc_validate_keys(g(3), g(4), total_keys=5, stream=0)
    assert stub.calls == []
    # host tensors for a store are copied from host memory
    B.cc_store_create(torch.zeros(5, dtype=torch.int64),
                      torch.zeros(5, DOC_BYTES, dtype=torch.uint8), stream=0)
    B.cc_resolve_ids(1, ids, g(5), stream=0)
    B.cc_store_upsert(1, ids, ids, rows, g(64, dtype=torch.uint8), stream=0)
    B.cc_store_read(1, 0, 5, g(5), rows, stream=0)
    assert [c[0] for c in stub.calls] == ["cc_store_create", "cc_resolve_ids",
                                          "cc_store_upsert", "cc_store_read"]
    assert stub.calls[0][1][5] == B.CC_SRC_HOST


def test_prepared_join_passes_the_same_arguments_and_counts(stub):
    a = join_args()
    B.cc_join(1, stream=0, **a)
    p = B.PreparedJoin(1, **a)
    p(stream=0)
    p(3, 2, stream=0)
    (_, full), (_, prep), (_, part) = stub.calls
    assert prep == full                                       # same call as cc_join
    assert part[2] == 3 and part[4] == 2                      # n_cand, n_keys
    assert part[:2] + part[3:4] + part[5:] == full[:2] + full[3:4] + full[5:]


@pytest.mark.parametrize("arg,bad,exc,match", [
    ("cand_idx", torch.zeros(10, dtype=torch.int64), ValueError, "GPU memory"),
    ("edge_keys", g(6, dtype=torch.float64), TypeError, "int64"),
    ("hit_mask", g(9, 1, dtype=torch.int8), ValueError, "elements"),
    ("out", g(10, DOC_BYTES, dtype=torch.uint8), ValueError, "bytes"),
])
def test_prepared_join_checks_its_buffers_once(stub, arg, bad, exc, match):
    a = join_args()
    a[arg] = bad
    with pytest.raises(exc, match=match):
        B.PreparedJoin(1, **a)
    assert stub.calls == []


@pytest.mark.parametrize("n,k", [(11, 6), (10, 7), (-1, 0), (0, -1)])
def test_prepared_join_counts_must_fit_the_buffers(stub, n, k):
    p = B.PreparedJoin(1, **join_args())
    with pytest.raises(ValueError, match="counts"):
        p(n, k, stream=0)
    assert stub.calls == []


def test_prepared_batched_join_passes_the_same_arguments_and_counts(stub):
    a = batched_args(lookups=2)
    B.cc_join_batched(1, stream=0, **a)
    p = B.PreparedJoinBatched(1, **a)
    p(stream=0)
    p(2, 7, 5, stream=0)
    (_, full), (_, prep), (_, part) = stub.calls
    same = lambda x: list(x) if hasattr(x, "_length_") else x   # ctypes arrays by contents
    assert [same(x) for x in prep] == [same(x) for x in full]
    assert part[1] == 2 and part[4] == 7 and part[7] == 5     # viewers, candidates, keys
    with pytest.raises(ValueError, match="counts"):
        p(4, 7, 5, stream=0)                                    # more viewers than the offsets
    with pytest.raises(ValueError, match="counts"):
        p(2, 13, 5, stream=0)
    assert len(stub.calls) == 3


def test_prepared_batched_join_checks_its_buffers_once(stub):
    a = batched_args(lookups=2)
    a["extra_keys"] = [g(11)]
    with pytest.raises(ValueError, match="elements"):
        B.PreparedJoinBatched(1, **a)
    assert stub.calls == []
