"""Property-based GPU parity: the HIP join equals the oracle byte for byte on inputs that
hypothesis draws (the id pool with the int64 extremes, repeated keys, invalid positions, one or
two lookups, an optional default row), under launch tunings that force every search path:
automatic, whole list in LDS, fixed strides, and LDS tables so small that windows exceed the
16-key scan."""
from __future__ import annotations

import pytest
import torch
from hypothesis import given, strategies as st

import paper_2609_22441_amd as P
from gpu_common import assert_same, gpu_join, note, oracle_join, row_bytes
from test_oracle_properties import SETTINGS, cases

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
