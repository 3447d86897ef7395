"""GPU parity of the padded batch layout (§6.3, batching and padding) against the oracle."""
from __future__ import annotations

import json
from pathlib import Path

import numpy as np
import pytest
import torch

import oracle
import paper_2609_22441_amd as P
import workload as W
from gpu_common import FILL, note, row_bytes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
GOLDEN = Path(__file__).resolve().parent / "golden"


def _gpu_padded(store, b, wd, we, L, n_max, default_row=None, stride=None):
    B = b.n_viewers
    stride = stride or wd + L * we
    out = torch.full((B, n_max, stride), FILL, dtype=torch.uint8, device=DEV)
    hit = torch.full((B, n_max, L), -7, dtype=torch.int8, device=DEV)
    valid = torch.full((B, n_max), -7, dtype=torch.int8, device=DEV)
    P.cc_join_batched_padded(store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys,
                             b.edge_rows, n_max, out, hit, valid, default_row=default_row,
                             extra_keys=[b.actor] if L == 2 else None)
    torch.cuda.synchronize()
    return out.cpu().numpy(), hit.cpu().numpy(), valid.cpu().numpy()


def _check(got, want, width, what):
    go, gh, gv = got
    T, H, V = want[0], want[1], want[2]
    assert np.array_equal(gv, V), f"{what}: valid mask"
    assert np.array_equal(gh, H), f"{what}: hit mask"
    assert np.array_equal(go[:, :, :width], T[:, :, :width]), f"{what}: rows"
    assert (go[:, :, width:] == FILL).all(), f"{what}: stride padding written"


def test_paper_padding_example():
    note("padding example of the paper")
    g = json.loads((GOLDEN / "padding_worked.json").read_text())
    feat = torch.arange(100 * 16, dtype=torch.int64).to(torch.uint8).reshape(100, 16)
    feat[:, 0] = torch.arange(100).to(torch.uint8)
    author = torch.full((100,), 7, dtype=torch.int64)
    pos = g["positions"]
    reqs = [W.Request(torch.zeros(0, dtype=torch.int64), torch.zeros(0, 16, dtype=torch.uint8),
                      torch.tensor(p, dtype=torch.int64), None) for p in pos]
    b = W.pack(reqs).to(DEV)
    store = P.cc_store_create(author.to(DEV), feat.to(DEV))
    try:
        out, hit, valid = _gpu_padded(store, b, 16, 16, 1, g["n_max"])
        assert valid.tolist() == g["expected_valid"]
        for v, want in enumerate(g["expected_rows"]):
            for i, p in enumerate(want):
                if p is None:
                    assert not out[v, i].any() and not hit[v, i].any()
                else:
                    assert np.array_equal(out[v, i, :16], feat[p].numpy())
    finally:
        P.cc_store_destroy(store)


@pytest.mark.parametrize("mode", ["exact", "slack", "truncate"])
def test_tiny_padded_cases(mode):
    note(f"padded tiny cases ({mode})")
    for seed in range(30):
        tc = W.tiny_case(5000 + seed, max_k=120, max_n=700, max_viewers=5)
        b = tc.batch
        n = np.diff(b.cand_offsets.numpy())
        n_max = max(1, int(n.max()) + {"exact": 0, "slack": 37, "truncate": -50}[mode])
        wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
        stride = wd + tc.n_lookups * we + 16 * (seed % 2)
        store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
        try:
            d = None if tc.default_row is None else tc.default_row.to(DEV)
            got = _gpu_padded(store, b.to(DEV), wd, we, tc.n_lookups, n_max, default_row=d,
                              stride=stride)
            want = oracle.join_padded(tc.author_id, tc.doc_rows, b.cand_offsets, b.cand_idx,
                                      b.key_offsets, b.keys, b.edge_rows, n_max,
                                      default_row=tc.default_row, n_lookups=tc.n_lookups,
                                      extra_keys=[b.actor] if tc.n_lookups == 2 else None)
            _check(got, want, wd + tc.n_lookups * we, f"seed {seed} {mode}")
            assert P.cc_store_invalid_count(store) == want[3]
        finally:
            P.cc_store_destroy(store)


def test_padded_without_candidates_fills_pads():
    note("padded layout with no candidates")
    tc = W.tiny_case(11)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        co = torch.zeros(4, dtype=torch.int64, device=DEV)
        empty = torch.zeros(0, dtype=torch.int64, device=DEV)
        keys = torch.zeros(0, dtype=torch.int64, device=DEV)
        edge = torch.zeros(0, 16, dtype=torch.uint8, device=DEV)
        wd = row_bytes(tc.doc_rows)
        b = W.Batch(co, empty, co.clone(), keys, edge, None)
        out, hit, valid = _gpu_padded(store, b, wd, 16, 1, 5)
        assert not valid.any() and not hit.any() and not out[:, :, :wd + 16].any()
    finally:
        P.cc_store_destroy(store)


@pytest.mark.timeout(300)
def test_workload3_padded():
    note("workload 3 in the padded layout")
    s, r = W.SHAPES[3]
    st = W.make_store(s, 2, device=DEV)
    reqs = W.make_requests(st, r, 3)
    b = W.pack(reqs)
    n_max = r.n_cand + 64
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        got = _gpu_padded(store, b, wd, we, 1, n_max)
        bc = b.to("cpu")
        want = oracle.join_padded(st.author_id.cpu(), st.doc_rows.cpu(), bc.cand_offsets,
                                  bc.cand_idx, bc.key_offsets, bc.keys, bc.edge_rows, n_max)
        _check(got, want, wd + we, "workload 3 padded")
    finally:
        P.cc_store_destroy(store)
