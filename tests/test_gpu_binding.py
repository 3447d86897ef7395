"""The binding enqueues on torch's current stream: the stream handle it passes is the one
torch reports, on the default stream and inside a stream context, and work launched there is
ordered with torch's own work on that stream."""
from __future__ import annotations

import pytest
import torch

import paper_2609_22441_amd as P
from paper_2609_22441_amd import binding as B
import workload as W
from gpu_common import assert_same, note, oracle_join, row_bytes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def test_launch_stream_is_torchs_current_stream():
    note("binding: current stream")
    torch.cuda.set_device(DEV)
    assert B._stream(None) == torch.cuda.current_stream().cuda_stream
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        assert B._stream(None) == side.cuda_stream
    assert B._stream(None) == torch.cuda.current_stream().cuda_stream


def test_join_on_a_side_stream_is_ordered_with_torch_work():
    """Inputs written by torch on a side stream, the join launched on that stream without a
    synchronisation in between, and the output read back after the stream ends."""
    note("binding: side-stream ordering")
    tc = W.tiny_case(77, n_lookups=1, max_n=600, max_viewers=3)
    wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        b = tc.batch
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            cand = torch.empty_like(b.cand_idx, device=DEV)
            cand.copy_(b.cand_idx, non_blocking=False)
            out = torch.full((b.cand_idx.numel(), wd + we), 0xEE, dtype=torch.uint8, device=DEV)
            hit = torch.full((b.cand_idx.numel(), 1), -7, dtype=torch.int8, device=DEV)
            P.cc_join_batched(store, b.cand_offsets.to(DEV), cand, b.key_offsets.to(DEV),
                              b.keys.to(DEV), b.edge_rows.to(DEV), out, hit)
        side.synchronize()
        want = oracle_join(tc.author_id, tc.doc_rows, b, 1)
        assert_same((out.cpu().numpy(), hit.cpu().numpy()), want, "side stream")
    finally:
        P.cc_store_destroy(store)


def test_prepared_join_equals_cc_join():
    """PreparedJoin over the leading elements of its buffers gives the bytes cc_join gives for
    the same slices, for full, partial and empty counts; the full case also against the oracle."""
    note("binding: prepared join")
    tc = W.tiny_case(91, n_lookups=1, max_n=900, max_k=300, max_viewers=1)
    b = tc.batch
    wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        cand, keys, feats = b.cand_idx.to(DEV), b.keys.to(DEV), b.edge_rows.to(DEV)
        n_all, k_all = cand.numel(), keys.numel()
        out = torch.full((n_all, wd + we), 0x5A, dtype=torch.uint8, device=DEV)
        hit = torch.full((n_all, 1), -7, dtype=torch.int8, device=DEV)
        prepared = P.PreparedJoin(store, cand, keys, feats, out, hit)
        for n, k in ((n_all, k_all), (n_all // 2, k_all // 3), (0, k_all), (n_all, 0)):
            out.fill_(0x5A)
            hit.fill_(-7)
            prepared(n, k)
            ref_out = torch.full((n, wd + we), 0x5A, dtype=torch.uint8, device=DEV)
            ref_hit = torch.full((n, 1), -7, dtype=torch.int8, device=DEV)
            P.cc_join(store, cand[:n], keys[:k], feats[:k], ref_out, ref_hit)
            torch.cuda.synchronize()
            assert torch.equal(out[:n], ref_out) and torch.equal(hit[:n], ref_hit), (n, k)
            assert bool((hit[n:] == -7).all()) and bool((out[n:] == 0x5A).all()), (n, k)
            if (n, k) == (n_all, k_all):
                want = oracle_join(tc.author_id, tc.doc_rows, b, 1)
                assert_same((out.cpu().numpy(), hit.cpu().numpy()), want, "prepared join")
    finally:
        P.cc_store_destroy(store)


def test_prepared_batched_join_with_author_ids():
    """PreparedJoinBatched with caller-supplied author ids gives the bytes of
    cc_join_batched(..., author_ids=...) for every CSR prefix (that call is checked against
    the oracle in test_gpu_join.py)."""
    note("binding: prepared batched join, caller author ids")
    tc = W.tiny_case(94, max_n=400, max_k=200, max_viewers=5)
    b = tc.batch
    wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        d = b.to(DEV)
        n_all = d.cand_idx.numel()
        g = torch.Generator().manual_seed(3)
        pool = torch.cat([b.keys, tc.author_id]) if b.keys.numel() + tc.author_id.numel() else \
            torch.zeros(1, dtype=torch.int64)
        authors = pool[torch.randint(0, pool.numel(), (n_all,), generator=g)].to(DEV)
        out = torch.full((n_all, wd + we), 0x5A, dtype=torch.uint8, device=DEV)
        hit = torch.full((n_all, 1), -7, dtype=torch.int8, device=DEV)
        prepared = P.PreparedJoinBatched(store, d.cand_offsets, d.cand_idx, d.key_offsets, d.keys,
                                         d.edge_rows, out, hit, author_ids=authors)
        co, ko = b.cand_offsets.tolist(), b.key_offsets.tolist()
        for nv in range(len(co) - 1, -1, -1):
            n, k = co[nv], ko[nv]
            out.fill_(0x5A)
            hit.fill_(-7)
            prepared(nv, n, k)
            ref_out = torch.full((n, wd + we), 0x5A, dtype=torch.uint8, device=DEV)
            ref_hit = torch.full((n, 1), -7, dtype=torch.int8, device=DEV)
            P.cc_join_batched(store, d.cand_offsets[:nv + 1], d.cand_idx[:n],
                              d.key_offsets[:nv + 1], d.keys[:k], d.edge_rows[:k], ref_out,
                              ref_hit, author_ids=authors[:n])
            torch.cuda.synchronize()
            assert torch.equal(out[:n], ref_out) and torch.equal(hit[:n], ref_hit), nv
            assert bool((hit[n:] == -7).all()), nv
    finally:
        P.cc_store_destroy(store)


def test_prepared_batched_join_equals_cc_join_batched():
    """PreparedJoinBatched on its first b viewers gives the bytes cc_join_batched gives for the
    same CSR prefix, two lookups, b from all viewers down to none."""
    note("binding: prepared batched join")
    tc = W.tiny_case(93, n_lookups=2, max_n=400, max_k=200, max_viewers=5)
    b = tc.batch
    wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        d = b.to(DEV)
        n_all = d.cand_idx.numel()
        out = torch.full((n_all, wd + 2 * we), 0x5A, dtype=torch.uint8, device=DEV)
        hit = torch.full((n_all, 2), -7, dtype=torch.int8, device=DEV)
        prepared = P.PreparedJoinBatched(store, d.cand_offsets, d.cand_idx, d.key_offsets, d.keys,
                                         d.edge_rows, out, hit, extra_keys=[d.actor])
        co, ko = b.cand_offsets.tolist(), b.key_offsets.tolist()
        for nv in range(len(co) - 1, -1, -1):
            n, k = co[nv], ko[nv]
            out.fill_(0x5A)
            hit.fill_(-7)
            prepared(nv, n, k)
            ref_out = torch.full((n, wd + 2 * we), 0x5A, dtype=torch.uint8, device=DEV)
            ref_hit = torch.full((n, 2), -7, dtype=torch.int8, device=DEV)
            P.cc_join_batched(store, d.cand_offsets[:nv + 1], d.cand_idx[:n],
                              d.key_offsets[:nv + 1], d.keys[:k], d.edge_rows[:k], ref_out,
                              ref_hit, extra_keys=[d.actor[:n]])
            torch.cuda.synchronize()
            assert torch.equal(out[:n], ref_out) and torch.equal(hit[:n], ref_hit), nv
            assert bool((hit[n:] == -7).all()), nv
            if nv == len(co) - 1:
                want = oracle_join(tc.author_id, tc.doc_rows, b, 2)
                assert_same((out.cpu().numpy(), hit.cpu().numpy()), want, "prepared batched")
    finally:
        P.cc_store_destroy(store)
