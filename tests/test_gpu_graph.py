"""The per-request calls are safe inside a HIP graph (no synchronisation, allocation or memset):
a counter reset, resolve (Eq. 6) and join (Eq. 1) captured once and replayed with new inputs,
every replay checked against the same calls made eagerly."""
from __future__ import annotations

import pytest
import torch

import paper_2609_22441_amd as P
import workload as W
from gpu_common import note

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def test_resolve_then_join_replays_in_a_graph():
    note("graph: resolve then join, captured and replayed")
    spec = W.IndexSpec(100_000, 20_000, 64, torch.bfloat16, 2, 3000, 0.05, 0, 0.0, 0.0)
    store = P.cc_store_create_indexed(spec.n_index, 128)
    try:
        ids, authors, rows = W.index_records(spec, torch.arange(spec.n_index), 4, 1, DEV)
        ws = torch.empty(P.cc_upsert_workspace_bytes(spec.n_index), dtype=torch.uint8, device=DEV)
        P.cc_store_upsert(store, ids, authors, rows, ws)
        g = W.gen(DEV, 4, 2)
        B, N, K = spec.batch, spec.ids_per_request, 1500
        co = torch.arange(0, B * N + 1, N, device=DEV)
        ko = torch.arange(0, B * K + 1, K, device=DEV)
        keys = torch.sort(torch.randperm(spec.n_authors, generator=g, device=DEV)[:B * K]
                          .view(B, K), dim=1).values.reshape(-1)
        edge = torch.randn(B * K, 32, generator=g, device=DEV).to(torch.bfloat16)
        # static buffers the graph reads and writes
        q = torch.empty(B * N, dtype=torch.int64, device=DEV)
        pos = torch.empty_like(q)
        out = torch.empty(B * N, 192, dtype=torch.uint8, device=DEV)
        hit = torch.empty(B * N, 1, dtype=torch.int8, device=DEV)

        def queries(seed):
            gq = W.gen(DEV, seed, 5)
            items = torch.randint(0, spec.n_index + spec.n_index // 20, (B * N,), generator=gq,
                                  device=DEV)          # about 5% past the index: absent
            return W.doc_ids(items, 4)

        def request():
            P.cc_store_reset_invalid_count(store)
            P.cc_resolve_ids(store, q, pos)
            P.cc_join_batched(store, co, pos, ko, keys, edge, out, hit)

        q.copy_(queries(100))
        request()                                   # warm-up outside the capture
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            with torch.cuda.graph(graph, stream=s):
                request()
        torch.cuda.synchronize()
        for rep in range(4):
            q.copy_(queries(200 + rep))
            out.fill_(0xCD)
            hit.fill_(-7)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            got_out, got_hit, got_pos = out.clone(), hit.clone(), pos.clone()
            # the join counts every position of -1 (an absent id) since the captured reset
            assert P.cc_store_invalid_count(store) == int((got_pos < 0).sum()), \
                f"replay {rep}: invalid count"
            out.fill_(0x5A)
            request()                               # the same calls, eagerly
            torch.cuda.synchronize()
            assert torch.equal(got_pos, pos), f"replay {rep}: positions"
            assert torch.equal(got_out, out), f"replay {rep}: rows"
            assert torch.equal(got_hit, hit), f"replay {rep}: hit mask"
            assert 0.9 * B * N < int((got_pos >= 0).sum()) < B * N, f"replay {rep}: hits"
    finally:
        P.cc_store_destroy(store)
