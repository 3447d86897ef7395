"""GPU parity of the HIP join against the oracle: edge cases, every search strategy, the
argument checks that need a real store, and the store's counters. Bit-exact (tolerance 0)."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import torch

import paper_2609_22441_amd as P
from paper_2609_22441_amd import binding as B
import workload as W
from gpu_common import FILL, assert_same, gpu_join, note, oracle_join, row_bytes

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")

# (fence_stride, lds_keys, workgroups): automatic, whole list in LDS, fixed strides, tiny LDS
# tables that force strides beyond the 16-key window, and a single workgroup doing everything.
TUNINGS = [None, (1, 4096, 0), (4, 0, 0), (16, 8, 0), (0, 2, 0), (2, 3, 8), (0, 0, 1)]


def _tuning(t):
    return None if t is None else P.Tuning(*t, 0)


def _tiny(tc, tuning=None, stride_extra=0, what=""):
    b = tc.batch.to(DEV)
    wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
    stride = wd + tc.n_lookups * we + stride_extra
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        d = None if tc.default_row is None else tc.default_row.to(DEV)
        got = gpu_join(store, None, b, wd, we, tc.n_lookups, default_row=d, stride=stride,
                       tuning=_tuning(tuning))
        want = oracle_join(tc.author_id, tc.doc_rows, tc.batch, tc.n_lookups,
                           default_row=tc.default_row, stride=stride)
        assert_same(got, want, what)
        assert P.cc_store_invalid_count(store) == want[2], f"{what}: invalid count"
    finally:
        P.cc_store_destroy(store)


@pytest.mark.parametrize("tuning", TUNINGS)
def test_tiny_random_cases(tuning):
    note(f"tiny random cases, tuning {tuning}")
    for seed in range(40):
        tc = W.tiny_case(seed, max_k=120, max_n=700, max_viewers=5)
        _tiny(tc, tuning, stride_extra=16 * (seed % 2), what=f"seed {seed} tuning {tuning}")


def _caller_authors(tc, seed):
    """Per-candidate author ids for the caller-supplied form: the store's id at the candidate's
    position for a third of them, a key of the batch (a likely hit) for a third, an arbitrary
    int64 for the rest."""
    c = tc.batch.cand_idx
    n, nd = c.numel(), tc.author_id.numel()
    g = torch.Generator().manual_seed(seed)
    own = tc.author_id[c.clamp(0, nd - 1)] if nd else torch.zeros_like(c)
    keys = tc.batch.keys
    pick = keys[torch.randint(0, keys.numel(), (n,), generator=g)] if keys.numel() else own
    wild = torch.randint(-(1 << 62), 1 << 62, (n,), generator=g, dtype=torch.int64)
    which = torch.randint(0, 3, (n,), generator=g)
    return torch.where(which == 0, own, torch.where(which == 1, pick, wild)).contiguous()


def _oracle_caller_authors(tc, authors, stride):
    """Eq. 1 with caller-supplied author ids, as the plain oracle join over a store holding one
    document per candidate (its doc row, the caller's author id), each valid candidate pointing
    at its own document and each invalid one at -1."""
    c = tc.batch.cand_idx
    n, nd = c.numel(), tc.author_id.numel()
    valid = (c >= 0) & (c < nd)
    rows = torch.zeros((n,) + tuple(tc.doc_rows.shape[1:]), dtype=tc.doc_rows.dtype)
    rows[valid] = tc.doc_rows[c[valid]]
    own_pos = torch.where(valid, torch.arange(n), torch.full_like(c, -1))
    b = tc.batch
    b2 = W.Batch(b.cand_offsets, own_pos, b.key_offsets, b.keys, b.edge_rows, b.actor)
    return oracle_join(authors, rows, b2, tc.n_lookups, default_row=tc.default_row,
                       stride=stride)


def test_caller_supplied_author_ids():
    """cc_join_batched_authors (lookup 0 searches the caller's author id of each candidate, Alg.
    1's input form) against the oracle over a store remapped to those ids, on random tiny
    cases with one and two lookups, invalid positions and defaults."""
    note("caller-supplied author ids")
    for seed in range(30):
        tc = W.tiny_case(4000 + seed, max_k=150, max_n=900, max_viewers=5)
        if tc.batch.cand_idx.numel() == 0:
            continue
        authors = _caller_authors(tc, seed)
        b = tc.batch.to(DEV)
        wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
        stride = wd + tc.n_lookups * we + 16 * (seed % 2)
        store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
        try:
            n = b.cand_idx.numel()
            out = torch.full((n, stride), FILL, dtype=torch.uint8, device=DEV)
            hit = torch.full((n, tc.n_lookups), -7, dtype=torch.int8, device=DEV)
            d = None if tc.default_row is None else tc.default_row.to(DEV)
            P.cc_join_batched(store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys,
                              b.edge_rows, out, hit, default_row=d,
                              extra_keys=[b.actor] if tc.n_lookups == 2 else None,
                              author_ids=authors.to(DEV))
            torch.cuda.synchronize()
            want = _oracle_caller_authors(tc, authors, stride)
            assert_same((out.cpu().numpy(), hit.cpu().numpy()), want, f"seed {seed}")
            assert P.cc_store_invalid_count(store) == want[2], f"seed {seed}: invalid count"
        finally:
            P.cc_store_destroy(store)


def test_duplicate_keys_leftmost():
    note("duplicate keys")
    for seed in range(20):
        tc = W.tiny_case(1000 + seed, max_k=200, max_n=500, dup_keys=True)
        for t in (None, (4, 0, 0), (0, 2, 0)):
            _tiny(tc, t, what=f"dup seed {seed} tuning {t}")


def test_empty_and_degenerate_viewers():
    note("empty viewers, K=0, N=0")
    # viewers with no candidates, no keys, and both, in every position
    for seed in range(12):
        tc = W.tiny_case(2000 + seed, max_k=30, max_n=40, max_viewers=6,
                         k_values=[0, 5, 0, 17, 1, 0])
        _tiny(tc, what=f"degenerate seed {seed}")


def test_no_candidates_is_a_no_op():
    st = W.tiny_case(3)
    store = P.cc_store_create(st.author_id.to(DEV), st.doc_rows.to(DEV))
    try:
        empty = torch.empty(0, dtype=torch.int64, device=DEV)
        keys = torch.tensor([1, 2], dtype=torch.int64, device=DEV)
        edge = torch.zeros(2, 16, dtype=torch.uint8, device=DEV)
        out = torch.empty(0, row_bytes(st.doc_rows) + 16, dtype=torch.uint8, device=DEV)
        hit = torch.empty(0, 1, dtype=torch.int8, device=DEV)
        P.cc_join(store, empty, keys, edge, out, hit)
        torch.cuda.synchronize()
    finally:
        P.cc_store_destroy(store)


def test_store_from_host_memory():
    """A store copied from host memory (CC_SRC_HOST) joins exactly like one copied from device
    memory, and both match the oracle."""
    note("store from host memory")
    for seed in range(6):
        tc = W.tiny_case(4000 + seed, n_lookups=1)
        b = tc.batch.to(DEV)
        wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
        want = oracle_join(tc.author_id, tc.doc_rows, tc.batch, 1, default_row=tc.default_row)
        d = None if tc.default_row is None else tc.default_row.to(DEV)
        for src in ("host", "device"):
            a, r = (tc.author_id, tc.doc_rows) if src == "host" else \
                (tc.author_id.to(DEV), tc.doc_rows.to(DEV))
            store = P.cc_store_create(a, r)
            try:
                assert P.cc_store_info(store) == (tc.author_id.numel(), wd)
                got = gpu_join(store, None, b, wd, we, 1, default_row=d)
                assert_same(got, want, f"seed {seed}, store from {src} memory")
            finally:
                P.cc_store_destroy(store)


def test_empty_store_makes_every_position_invalid():
    """A store of 0 documents: every candidate position is out of range, so each row is a zero
    doc segment plus the default edge row, every hit bit is 0 and every candidate is counted."""
    note("empty store")
    store = P.cc_store_create(torch.zeros(0, dtype=torch.int64),
                              torch.zeros(0, 32, dtype=torch.uint8))
    try:
        assert P.cc_store_info(store) == (0, 32)
        cand = torch.tensor([0, 1, -1, 7, 0], dtype=torch.int64)
        keys = torch.tensor([0, 1, 7], dtype=torch.int64)
        edge = torch.arange(3 * 16, dtype=torch.int64).to(torch.uint8).reshape(3, 16)
        default = torch.full((16,), 0xAB, dtype=torch.uint8)
        batch = W.pack([W.Request(keys, edge, cand, None)])
        got = gpu_join(store, None, batch.to(DEV), 32, 16, 1, default_row=default.to(DEV))
        want = oracle_join(torch.zeros(0, dtype=torch.int64), torch.zeros(0, 32, dtype=torch.uint8),
                           batch, 1, default_row=default)
        assert_same(got, want, "empty store")
        assert (got[0][:, :32] == 0).all() and (got[0][:, 32:] == 0xAB).all()
        assert not got[1].any()
        assert P.cc_store_invalid_count(store) == cand.numel()
    finally:
        P.cc_store_destroy(store)


def _scaled_store(seed, cfg=2, **kw):
    kw = {"store_n_docs": 300_000, "store_n_authors": 200_000, **kw}
    s, r = W.shape(cfg, **kw)
    st = W.make_store(s, seed, device=DEV)
    return st, r


@pytest.mark.parametrize("k", [1, 2, 15, 16, 17, 511, 512, 513, 4095, 4096, 4097, 8192, 8193, 18432, 18433,
                               19456, 19457, 40000, 100_000])
def test_key_count_thresholds(k):
    """K around every table-size and stride boundary, automatic tuning, two lookups."""
    note(f"K threshold {k}")
    st, r = _scaled_store(7, cfg=4, store_n_authors=10_000_000, req_k=k, req_n_cand=6_000,
                          req_n_viewers=2)
    reqs = W.make_requests(st, r, 7)
    b = W.pack(reqs)
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        for t in (None, (1, 18432, 0), (8, 0, 0)):
            got = gpu_join(store, None, b, wd, we, 2, tuning=_tuning(t))
            want = oracle_join(st.author_id.cpu(), st.doc_rows.cpu(), b.to("cpu"), 2)
            assert_same(got, want, f"K={k} tuning {t}")
    finally:
        P.cc_store_destroy(store)


def test_single_viewer_entry_point():
    note("cc_join single viewer, scaled production shape")
    st, r = _scaled_store(9, req_k=3000, req_n_cand=20_000)
    q = W.make_request(st, r, 9, 0)
    b = W.pack([q])
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        dflt = torch.arange(we, dtype=torch.uint8, device=DEV)
        got = gpu_join(store, None, b, wd, we, 1, default_row=dflt, single=True)
        want = oracle_join(st.author_id.cpu(), st.doc_rows.cpu(), b.to("cpu"), 1,
                           default_row=dflt)
        assert_same(got, want, "cc_join")
    finally:
        P.cc_store_destroy(store)


def test_special_bit_patterns_are_copied_exactly():
    note("NaN payloads, signed zeros, subnormals")
    st, r = _scaled_store(10, req_k=2000, req_n_cand=10_000, req_n_viewers=3)
    g = W.gen(DEV, 10, 77)
    W.salt_special_values(st.doc_rows, 0.2, g)
    reqs = W.make_requests(st, r, 10)
    for q in reqs:
        W.salt_special_values(q.edge_rows, 0.2, g)
    b = W.pack(reqs)
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        got = gpu_join(store, None, b, wd, we, 1)
        want = oracle_join(st.author_id.cpu(), st.doc_rows.cpu(), b.to("cpu"), 1)
        assert_same(got, want, "special values")
    finally:
        P.cc_store_destroy(store)


def test_fp32_rows_of_the_tiny_shape():
    note("fp32 rows (16 + 8 columns)")
    s, r = W.shape(1, store_n_docs=100_000)
    st = W.make_store(s, 12, device=DEV)
    b = W.pack([W.make_request(st, r, 12, 0)])
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        got = gpu_join(store, None, b, wd, we, 1, single=True)
        want = oracle_join(st.author_id.cpu(), st.doc_rows.cpu(), b.to("cpu"), 1)
        assert_same(got, want, "fp32")
    finally:
        P.cc_store_destroy(store)


def test_odd_row_widths_use_the_generic_copy():
    note("generic widths 48 + 80 bytes")
    tc = W.tiny_case(4242, max_k=100, max_n=900, doc_bytes=48, edge_bytes=80, n_lookups=2)
    _tiny(tc, what="generic widths")


def test_invalid_counter_and_reset():
    note("invalid counter")
    tc = W.tiny_case(77, max_n=500, n_lookups=1)
    b = tc.batch.to(DEV)
    n_docs = tc.author_id.numel()
    b.cand_idx[::3] = -1
    b.cand_idx[1::7] = n_docs
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    try:
        wd, we = row_bytes(tc.doc_rows), row_bytes(tc.batch.edge_rows)
        ci = b.cand_idx.cpu()
        bad = int(((ci < 0) | (ci >= n_docs)).sum())
        gpu_join(store, None, b, wd, we, 1)
        gpu_join(store, None, b, wd, we, 1)
        assert P.cc_store_invalid_count(store) == 2 * bad
        P.cc_store_reset_invalid_count(store)
        assert P.cc_store_invalid_count(store) == 0
        assert P.cc_store_info(store) == (n_docs, wd)
    finally:
        P.cc_store_destroy(store)


def test_validate_keys():
    note("cc_validate_keys")
    ko = torch.tensor([0, 3, 3, 7, 9], dtype=torch.int64, device=DEV)
    good = torch.tensor([1, 5, 9, -4, 0, 2, 8, 3, 4], dtype=torch.int64, device=DEV)
    assert P.cc_validate_keys(ko, good) == -1
    dup = good.clone()
    dup[5] = 0                      # viewer 2 now has a repeat
    assert P.cc_validate_keys(ko, dup) == 2
    uns = good.clone()
    uns[8] = 1                      # viewer 3 now descends
    assert P.cc_validate_keys(ko, uns) == 3


def test_argument_errors_with_a_real_store():
    note("host argument checks")
    tc = W.tiny_case(5, n_lookups=1, doc_bytes=32, edge_bytes=16)
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    lib = B.lib()
    try:
        n = 8
        cand = torch.zeros(n, dtype=torch.int64, device=DEV)
        keys = torch.arange(4, dtype=torch.int64, device=DEV)
        edge = torch.zeros(4, 16, dtype=torch.uint8, device=DEV)
        out = torch.zeros(n, 64, dtype=torch.uint8, device=DEV)
        hit = torch.zeros(n, 2, dtype=torch.int8, device=DEV)
        s = torch.cuda.current_stream().cuda_stream
        p = lambda t: t.data_ptr()

        def join(**kw):
            a = dict(cand=p(cand), n=n, keys=p(keys), k=4, edge=p(edge), ew=16, d=None,
                     out=p(out), stride=48, hit=p(hit))
            a.update(kw)
            return lib.cc_join(store, a["cand"], a["n"], a["keys"], a["k"], a["edge"], a["ew"],
                               a["d"], a["out"], a["stride"], a["hit"], s)

        assert join() == 0
        assert join(out=p(out) + 8) == 1                    # misaligned output
        assert join(edge=p(edge) + 4) == 1                  # misaligned edge rows
        assert join(cand=p(cand) + 4) == 1                  # misaligned candidates
        assert join(d=p(edge) + 8) == 1                     # misaligned default row
        assert join(stride=40) == 1                         # stride below the row width
        assert join(stride=56) == 1                         # stride not a multiple of 16
        assert join(ew=24) == 1                             # edge width not a multiple of 16
        assert join(ew=(1 << 20) + 16, stride=(1 << 20) + 64) == 1   # edge row above 1 MiB
        assert join(n=-1) == 1
        assert join(k=-1) == 1
        assert join(cand=None) == 1
        assert join(keys=None) == 1                         # K > 0 needs keys
        assert join(keys=None, edge=None, k=0) == 0         # K = 0 needs neither
        co = torch.tensor([0, n], dtype=torch.int64, device=DEV)
        ko = torch.tensor([0, 4], dtype=torch.int64, device=DEV)

        def batched(L=1, extra=None, **kw):
            return lib.cc_join_batched(store, 1, p(co), p(cand), n, p(ko), p(keys), 4, p(edge),
                                       16, None, L, extra, p(out), kw.get("stride", 64),
                                       p(hit), s)

        assert batched() == 0
        assert batched(L=3) == 1
        assert batched(L=2) == 1                            # no extra key arrays
        arr = (ctypes.c_void_p * 1)(None)
        assert batched(L=2, extra=arr) == 1                 # null extra key array
        arr = (ctypes.c_void_p * 1)(p(cand))
        assert batched(L=2, extra=arr) == 0
        assert batched(L=2, extra=arr, stride=48) == 1      # two lookups need 64 bytes
        assert lib.cc_join_batched(store, 1, None, p(cand), n, p(ko), p(keys), 4, p(edge), 16,
                                   None, 1, None, p(out), 64, p(hit), s) == 1
        tun = P.Tuning(3, 0, 0, 0)                          # stride not a power of two
        assert lib.cc_join_batched_tuned(store, 1, p(co), p(cand), n, p(ko), p(keys), 4,
                                         p(edge), 16, None, 1, None, p(out), 64, p(hit),
                                         ctypes.byref(tun), s) == 1
        tun = P.Tuning(0, 20000, 0, 0)                      # LDS table too large
        assert lib.cc_join_batched_tuned(store, 1, p(co), p(cand), n, p(ko), p(keys), 4,
                                         p(edge), 16, None, 1, None, p(out), 64, p(hit),
                                         ctypes.byref(tun), s) == 1
        torch.cuda.synchronize()
    finally:
        P.cc_store_destroy(store)


def test_concurrent_streams_share_a_store():
    note("two streams, one store")
    st, r = _scaled_store(13, req_k=2500, req_n_cand=15_000, req_n_viewers=2)
    reqs = W.make_requests(st, r, 13)
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        torch.cuda.synchronize()
        wd = row_bytes(st.doc_rows)
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        outs = []
        for q, sm in zip(reqs, streams):
            b = W.pack([q])
            we = row_bytes(b.edge_rows)
            out = torch.full((b.cand_idx.numel(), wd + we), FILL, dtype=torch.uint8, device=DEV)
            hit = torch.zeros(b.cand_idx.numel(), 1, dtype=torch.int8, device=DEV)
            with torch.cuda.stream(sm):
                P.cc_join(store, b.cand_idx, b.keys, b.edge_rows, out, hit, stream=sm)
            outs.append((b, out, hit))
        torch.cuda.synchronize()
        for i, (b, out, hit) in enumerate(outs):
            want = oracle_join(st.author_id.cpu(), st.doc_rows.cpu(), b.to("cpu"), 1)
            assert_same((out.cpu().numpy(), hit.cpu().numpy()), want, f"stream {i}")
    finally:
        P.cc_store_destroy(store)


def _remap_ids(tc, f):
    """The same case with every author id, key and actor id passed through the increasing map f
    (ranks of the distinct ids -> new ids), so keys stay sorted and every match is kept."""
    b = tc.batch
    parts = [tc.author_id, b.keys] + ([b.actor] if b.actor is not None else [])
    ids = torch.unique(torch.cat(parts))
    rank = lambda t: torch.searchsorted(ids, t)
    new = lambda t: None if t is None else f(rank(t))
    nb = W.Batch(b.cand_offsets, b.cand_idx, b.key_offsets, new(b.keys), b.edge_rows, new(b.actor))
    return W.TinyCase(new(tc.author_id), tc.doc_rows, nb, tc.default_row, tc.n_lookups)


def test_author_column_layouts():
    """Stores whose author ids fit in 32 bits keep a 32-bit column that the joins read; wider
    ids keep the 64-bit column. Both give the oracle's result, including ids at the int32
    limits and negative ids."""
    note("author column layouts")
    lo, hi = -(1 << 31), (1 << 31) - 1
    maps = {
        4: [lambda r: r - 7, lambda r: lo + r, lambda r: hi - 40 + r],
        8: [lambda r: (r - 3) << 33, lambda r: hi - 3 + r],       # the second crosses 2^31
    }
    for seed in range(16):
        tc = W.tiny_case(5000 + seed, max_k=60, max_n=300, max_viewers=4, max_docs=40)
        for width, fs in maps.items():
            for k, f in enumerate(fs):
                t = _remap_ids(tc, f)
                store = P.cc_store_create(t.author_id.to(DEV), t.doc_rows.to(DEV))
                try:
                    got_w = P.cc_store_layout(store)[0]
                    fits = bool(((t.author_id >= lo) & (t.author_id <= hi)).all())
                    assert got_w == (4 if fits else 8), f"seed {seed}: layout {got_w}"
                    if width == 4:
                        assert got_w == 4
                finally:
                    P.cc_store_destroy(store)
                for tu in (None, (4, 0, 0)):
                    _tiny(t, tu, what=f"seed {seed} map {width}/{k} tuning {tu}")


def test_outputs_overlapping_inputs_are_rejected():
    """The join refuses outputs that overlap an input or each other (checked on the host)."""
    note("overlapping outputs")
    tc = W.tiny_case(77, max_k=30, max_n=100, max_viewers=2, n_lookups=1, doc_bytes=32,
                     edge_bytes=16)
    b = tc.batch.to(DEV)
    n, k = b.cand_idx.numel(), b.keys.numel()
    assert n > 0 and k > 0
    store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
    lib = B.lib()
    out = torch.zeros(n, 48, dtype=torch.uint8, device=DEV)
    hit = torch.zeros(n, 1, dtype=torch.int8, device=DEV)
    stream = torch.cuda.current_stream().cuda_stream

    def call(out_p, hit_p):
        return lib.cc_join_batched(store, b.n_viewers, b.cand_offsets.data_ptr(),
                                   b.cand_idx.data_ptr(), n, b.key_offsets.data_ptr(),
                                   b.keys.data_ptr(), k, b.edge_rows.data_ptr(), 16, None, 1, None,
                                   out_p, 48, hit_p, stream)
    try:
        assert call(b.cand_idx.data_ptr(), hit.data_ptr()) == 1        # out over the positions
        assert call(b.edge_rows.data_ptr(), hit.data_ptr()) == 1       # out over the edge rows
        assert call(out.data_ptr(), out.data_ptr() + 32) == 1          # hit mask inside out
        assert call(out.data_ptr(), b.keys.data_ptr()) == 1            # hit mask over the keys
        assert call(out.data_ptr(), hit.data_ptr()) == 0               # disjoint: accepted
        torch.cuda.synchronize()
    finally:
        P.cc_store_destroy(store)


@pytest.mark.parametrize("tuning", [None, (1, 4096, 0), (4, 0, 0), (16, 8, 0), (0, 2, 0)])
def test_unsorted_keys_stay_in_bounds(tuning):
    """Keys out of order give an unspecified result, but every access stays in bounds and the
    output is consistent: doc segments are exact, a miss carries the default row and hit 0,
    and a hit carries one of the same viewer's edge rows."""
    note(f"unsorted keys, tuning {tuning}")
    for seed in range(12):
        tc = W.tiny_case(9100 + seed, max_k=120, max_n=400, max_viewers=4, n_lookups=1,
                         dup_keys=False)
        b = tc.batch
        ko = b.key_offsets.tolist()
        g = W.gen("cpu", seed, 11)
        keys = b.keys.clone()
        for v in range(len(ko) - 1):
            if ko[v + 1] > ko[v]:
                keys[ko[v]:ko[v + 1]] = keys[ko[v]:ko[v + 1]][
                    torch.randperm(ko[v + 1] - ko[v], generator=g)]
        ub = W.Batch(b.cand_offsets, b.cand_idx, b.key_offsets, keys, b.edge_rows, None)
        wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
        store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
        try:
            d = None if tc.default_row is None else tc.default_row.to(DEV)
            out, hit = gpu_join(store, None, ub.to(DEV), wd, we, 1, default_row=d,
                                tuning=_tuning(tuning))
        finally:
            P.cc_store_destroy(store)
        want, _, _ = oracle_join(tc.author_id, tc.doc_rows, b, 1, default_row=tc.default_row)
        assert np.array_equal(out[:, :wd], want[:, :wd]), f"seed {seed}: doc segments"
        assert set(np.unique(hit).tolist()) <= {0, 1}
        default = (np.zeros(we, np.uint8) if tc.default_row is None
                   else tc.default_row.numpy())
        edge = b.edge_rows.numpy().reshape(b.edge_rows.shape[0], -1).view(np.uint8)
        co = b.cand_offsets.tolist()
        for v in range(len(co) - 1):
            rows_v = {bytes(r) for r in edge[ko[v]:ko[v + 1]]}
            for j in range(co[v], co[v + 1]):
                seg = out[j, wd:wd + we]
                if hit[j, 0]:
                    assert bytes(seg) in rows_v, f"seed {seed}: hit row from another viewer"
                else:
                    assert np.array_equal(seg, default), f"seed {seed}: miss row"


def test_thousands_of_small_viewers():
    """3,000 viewers with 0 to 40 candidates and 0 to 60 keys each (many workgroups cross
    several viewers): bit-exact with the oracle."""
    note("3,000 small viewers")
    g = W.gen("cpu", 31, 4)
    n_docs = 5000
    author = torch.randint(0, 2000, (n_docs,), generator=g)
    doc = torch.randint(0, 256, (n_docs, 32), generator=g, dtype=torch.int64).to(torch.uint8)
    reqs = []
    for v in range(3000):
        k = int(torch.randint(0, 61, (1,), generator=g))
        keys = torch.sort(torch.randperm(2000, generator=g)[:k]).values
        edge = torch.randint(0, 256, (k, 16), generator=g, dtype=torch.int64).to(torch.uint8)
        n = int(torch.randint(0, 41, (1,), generator=g))
        cand = torch.randint(-1, n_docs + 1, (n,), generator=g)
        reqs.append(W.Request(keys, edge, cand, None))
    tc = W.TinyCase(author, doc, W.pack(reqs), None, 1)
    for t in (None, (4, 0, 0), (0, 0, 8)):
        _tiny(tc, t, what=f"3000 viewers tuning {t}")


def _skewed_batch(n_viewers, seed, n_lookups):
    """Viewers with skewed work: about 10% without candidates, every 97th with 3,000, the rest
    0 to 300; lists of 0 to 200 keys, every 50th with 9,000 to 12,000 (beyond the LDS table)."""
    g = W.gen("cpu", seed, n_viewers)
    n_docs, n_ids = 20_000, 40_000
    author = torch.randint(0, n_ids, (n_docs,), generator=g)
    doc = torch.randint(0, 256, (n_docs, 64), generator=g, dtype=torch.int64).to(torch.uint8)
    reqs = []
    for v in range(n_viewers):
        big = v % 50 == 7
        k = int(torch.randint(9_000, 12_001, (1,), generator=g)) if big else \
            int(torch.randint(0, 201, (1,), generator=g))
        keys = torch.sort(torch.randperm(n_ids, generator=g)[:k]).values
        edge = torch.randint(0, 256, (k, 32), generator=g, dtype=torch.int64).to(torch.uint8)
        if v % 10 == 3:
            n = 0
        elif v % 97 == 5:
            n = 3_000
        else:
            n = int(torch.randint(0, 301, (1,), generator=g))
        cand = torch.randint(-1, n_docs + 1, (n,), generator=g)
        actor = None
        if n_lookups == 2:
            pick = keys[torch.randint(0, max(k, 1), (n,), generator=g)] if k else \
                torch.full((n,), -1, dtype=torch.int64)
            actor = torch.where(torch.rand(n, generator=g) < 0.5, pick, torch.full_like(pick, -1))
        reqs.append(W.Request(keys, edge, cand, actor))
    return W.TinyCase(author, doc, W.pack(reqs), None, n_lookups)


@pytest.mark.parametrize("n_viewers", [2, 255, 256, 257, 700, 1024, 1025])
def test_weighted_ranges_around_the_viewer_limit(n_viewers):
    """CSR batches of up to 1,024 viewers split their candidates by estimated cost (more than
    one 256-viewer chunk of the prefix for 257 and up); 1,025 falls back to equal ranges. Every
    split must cover each candidate once: bit-exact with the oracle, automatic and fixed grids."""
    note(f"weighted ranges, {n_viewers} viewers")
    for n_lookups in (1, 2):
        tc = _skewed_batch(n_viewers, 41, n_lookups)
        for t in (None, (0, 0, 8), (0, 0, 1000)):
            _tiny(tc, t, what=f"{n_viewers} viewers, {n_lookups} lookups, tuning {t}")


@pytest.mark.parametrize("tuning", [None, (0, 0, 8), (4, 0, 0)])
def test_offsets_that_break_the_rules_stay_in_bounds(tuning):
    """Offsets that break the CSR rules (a decreasing pair, a negative entry, entries past the
    totals) give an unspecified result, but the kernels clamp them: the call completes, and
    every row it writes has its candidate's exact doc segment and a hit byte of 0 or 1."""
    note(f"offsets that break the CSR rules, tuning {tuning}")
    for seed in range(8):
        tc = W.tiny_case(9300 + seed, max_k=120, max_n=300, max_viewers=6, n_lookups=1,
                         dup_keys=False)
        b = tc.batch
        B = b.cand_offsets.numel() - 1
        co, ko = b.cand_offsets.clone(), b.key_offsets.clone()
        tc_n, tk_n = b.cand_idx.numel(), b.keys.numel()
        kind = seed % 4
        if kind == 0 and B >= 2:
            co[1], co[2] = co[2].item() + 5, max(co[1].item() - 3, 0)
        elif kind == 1:
            co[B] = tc_n + 1000
            ko[B] = tk_n + 1000
        elif kind == 2 and B >= 2:
            co[1] = -50
            ko[1] = -7
        else:
            ko[:] = ko.flip(0)
        bad = W.Batch(co, b.cand_idx, ko, b.keys, b.edge_rows, None)
        wd, we = row_bytes(tc.doc_rows), row_bytes(b.edge_rows)
        store = P.cc_store_create(tc.author_id.to(DEV), tc.doc_rows.to(DEV))
        try:
            out, hit = gpu_join(store, None, bad.to(DEV), wd, we, 1, tuning=_tuning(tuning))
        finally:
            P.cc_store_destroy(store)
        doc = tc.doc_rows.numpy()
        cand = b.cand_idx.tolist()
        for j in np.flatnonzero(hit[:, 0] != -7):
            assert hit[j, 0] in (0, 1), f"seed {seed}: hit byte {hit[j, 0]}"
            c = cand[j]
            want = doc[c] if 0 <= c < doc.shape[0] else np.zeros(wd, np.uint8)
            assert np.array_equal(out[j, :wd], want), f"seed {seed}: doc segment of row {j}"


def test_store_too_large_for_the_device_is_out_of_memory():
    """A store that cannot fit returns CC_ERR_OUT_OF_MEMORY, frees what it had allocated, and
    leaves the library usable (2^31 - 1 rows of 1 MiB: its id column fits, its rows do not)."""
    note("store larger than device memory")
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    with pytest.raises(B.CCError) as err:
        P.cc_store_create_indexed((1 << 31) - 1, 1 << 20)
    assert err.value.status == B.CC_ERR_OUT_OF_MEMORY
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert abs(free1 - free0) < (64 << 20), (free0, free1)      # nothing left allocated
    tc = W.tiny_case(77, max_viewers=3, n_lookups=1)
    _tiny(tc, None, what="a join after the failed allocation")
