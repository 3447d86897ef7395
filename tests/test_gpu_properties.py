"""Property-based GPU parity on inputs that hypothesis draws from an id pool with the int64
extremes: the HIP join equals the oracle byte for byte (repeated keys, invalid positions, one
or two lookups, an optional default row) under launch tunings that force every search path
(automatic, whole list in LDS, fixed strides, LDS tables so small that windows exceed the
16-key scan); ingestion and resolution equal the oracle's replay; the device sort equals the
oracle's stable sort."""
from __future__ import annotations

import numpy as np
import pytest
import torch
from hypothesis import given, strategies as st

import oracle
import paper_2609_22441_amd as P
from gpu_common import FILL, assert_same, gpu_join, note, oracle_join, row_bytes
from test_gpu_map import DeviceIndex
from test_oracle_properties import ID_POOL, SETTINGS, cases

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

TUNINGS = [None, (1, 4096, 0), (4, 0, 0), (16, 8, 0), (0, 2, 0), (2, 3, 8), (0, 0, 1)]


@pytest.fixture(scope="module", autouse=True)
def _name_the_case():
    note("property-based join parity (hypothesis cases, every tuning)")


@SETTINGS
@given(cases(), st.sampled_from(TUNINGS), st.integers(0, 1))
def test_join_equals_the_oracle(tc, tuning, extra_stride):
    b = tc.batch.to(DEV)
    wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
    stride = wd + tc.n_lookups * we + 16 * extra_stride
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        d = None if tc.default_row is None else tc.default_row.to(DEV)
        tun = None if tuning is None else P.Tuning(*tuning, 0)
        got = gpu_join(store, None, b, wd, we, tc.n_lookups, default_row=d, stride=stride,
                       tuning=tun)
        want = oracle_join(tc.author_id, tc.doc_rows, tc.batch, tc.n_lookups,
                           default_row=tc.default_row, stride=stride)
        assert_same(got, want, f"tuning {tuning}")
        assert P.cc_store_invalid_count(store) == want[2]
    finally:
        P.cc_store_destroy(store)


@SETTINGS
@given(st.integers(0, 12),
       st.lists(st.lists(st.tuples(st.sampled_from(ID_POOL), st.sampled_from(ID_POOL),
                                   st.binary(min_size=16, max_size=16)), max_size=8),
                max_size=5),
       st.lists(st.sampled_from(ID_POOL), max_size=12))
def test_ingestion_and_resolution_equal_the_oracle(capacity, batches, queries):
    """Batch after batch (repeats, the reserved id, refused batches, author ids wider than 32
    bits), the device store equals the oracle's sequential replay; then Eq. 6 resolution."""
    ix = DeviceIndex(capacity, 16)
    try:
        for k, batch in enumerate(batches):
            rows = torch.frombuffer(bytearray(b"".join(r for _, _, r in batch)) or bytearray(16),
                                    dtype=torch.uint8)[:16 * len(batch)].reshape(len(batch), 16)
            ix.upsert([i for i, _, _ in batch], [a for _, a, _ in batch], rows)
            ix.check_state(f"batch {k}")
        ix.resolve(queries, "queries")
    finally:
        ix.close()


@SETTINGS
@given(st.lists(st.lists(st.sampled_from(ID_POOL + list(range(-5, 40))), max_size=40),
                min_size=1, max_size=5),
       st.sampled_from([16, 32, 64]), st.booleans(),
       st.sampled_from([P.SORT_AUTO, P.SORT_MERGE, P.SORT_RADIX]))
def test_sort_equals_the_oracle(viewers, row_bytes, hint, method):
    """Alg. 1 Step 1 on the device against the oracle's stable sort, with each sort method; the
    pool's int64 extremes force the wide element form, small ids alone allow the packed one."""
    keys = torch.tensor([k for v in viewers for k in v], dtype=torch.int64)
    ko = torch.tensor(np.cumsum([0] + [len(v) for v in viewers]), dtype=torch.int64)
    n = keys.numel()
    rows = torch.arange(n * row_bytes, dtype=torch.int64).to(torch.uint8).reshape(n, row_bytes)
    rows[:, :8] = torch.arange(n, dtype=torch.int64).view(torch.uint8).reshape(n, 8) if n else 0
    want_k, want_r = oracle.sort_affinity(ko.numpy(), keys.numpy(), rows.numpy())
    k_out = torch.full((max(n, 1),), -7, dtype=torch.int64, device=DEV)
    r_out = torch.full((max(n, 1), row_bytes), FILL, dtype=torch.uint8, device=DEV)
    ws = torch.empty(max(16, P.cc_sort_workspace_bytes(n, len(viewers))), dtype=torch.uint8,
                     device=DEV)
    mk = max(len(v) for v in viewers) if hint else 0
    P.cc_sort_affinity(ko.to(DEV), keys.to(DEV), rows.to(DEV), k_out, r_out, ws, max_keys=mk,
                       total_keys=n, method=method)
    torch.cuda.synchronize()
    assert np.array_equal(k_out.cpu().numpy()[:n], want_k)
    assert np.array_equal(r_out.cpu().numpy()[:n], want_r)
