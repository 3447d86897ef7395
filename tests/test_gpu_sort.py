"""GPU parity of the affinity-record sort (Alg. 1 Step 1) against the oracle's stable sort."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2609_22441_amd as P
import workload as W
from gpu_common import note, row_bytes

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _shuffle_within(key_offsets, keys, rows, seed):
    g = W.gen("cpu", seed, 9)
    ko = key_offsets.cpu().numpy()
    k, r = keys.clone().cpu(), rows.clone().cpu()
    for v in range(len(ko) - 1):
        p = torch.randperm(int(ko[v + 1] - ko[v]), generator=g) + int(ko[v])
        k[ko[v]:ko[v + 1]] = keys.cpu()[p]
        r[ko[v]:ko[v + 1]] = rows.cpu()[p]
    return k, r


METHODS = (P.SORT_MERGE, P.SORT_RADIX)


def _gpu_sort(ko, keys, rows, max_keys=0, method=P.SORT_AUTO, key_bits=0):
    n = keys.numel()
    ws = torch.empty(max(16, P.cc_sort_workspace_bytes(n, ko.numel() - 1)), dtype=torch.uint8,
                     device=DEV)
    ko_d, k_d, r_d = ko.to(DEV), keys.to(DEV), rows.to(DEV)
    k_out = torch.full_like(k_d, -7)
    r_out = torch.full_like(r_d, 0xCD) if r_d.dtype == torch.uint8 else torch.empty_like(r_d)
    P.cc_sort_affinity(ko_d, k_d, r_d, k_out, r_out, ws, max_keys=max_keys, method=method,
                       key_bits=key_bits)
    torch.cuda.synchronize()
    return k_out.cpu().numpy(), oracle.as_bytes(r_out.cpu())


def _check(ko, keys, rows, what, max_keys=0):
    """Both sort methods (merge rounds; radix passes and a row gather) against the oracle."""
    wk, wr = oracle.sort_affinity(ko, keys, rows)
    for method in METHODS:
        gk, gr = _gpu_sort(ko, keys, rows, max_keys, method)
        assert np.array_equal(gk, wk), f"{what}, method {method}: keys"
        assert np.array_equal(gr, wr), f"{what}, method {method}: rows"


def test_tiny_sorts_with_duplicates_and_empty_viewers():
    note("sort: tiny cases")
    for seed in range(40):
        tc = W.tiny_case(8000 + seed, max_k=300, max_viewers=6, dup_keys=bool(seed % 2),
                         k_values=None if seed % 3 else [0, 250, 3, 0, 100, 1])
        b = tc.batch
        k, r = _shuffle_within(b.key_offsets, b.keys, b.edge_rows, seed)
        mk = int(b.key_offsets.diff().max()) if seed % 4 == 0 else 0    # with and without hint
        _check(b.key_offsets, k, r, f"seed {seed}", max_keys=mk)


@pytest.mark.parametrize("n", [1, 4095, 4096, 4097, 8192, 8193, 12289, 100_000])
def test_one_viewer_tile_boundaries(n):
    note(f"sort: one viewer, {n} records")
    g = W.gen("cpu", n, 3)
    keys = torch.randint(-1000, 1000, (n,), generator=g)        # many repeats
    rows = torch.randint(0, 256, (n, 32), generator=g, dtype=torch.int64).to(torch.uint8)
    _check(torch.tensor([0, n]), keys, rows, f"n={n}")


def test_many_ragged_viewers():
    """Viewers from empty to several tiles in one call: each viewer runs its own number of
    merge rounds and its result sits in the ping-pong array that matches that count."""
    note("sort: 300 ragged viewers")
    g = W.gen("cpu", 77, 3)
    sizes = torch.tensor([0, 1, 4095, 4096, 4097, 9000, 20000, 0, 70000, 3] * 30)
    sizes = sizes[torch.randperm(sizes.numel(), generator=g)]
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    keys = torch.randint(-(1 << 40), 1 << 40, (n,), generator=g)
    keys[::7] = 5                                                # repeats across tiles
    rows = torch.randint(0, 256, (n, 16), generator=g, dtype=torch.int64).to(torch.uint8)
    _check(ko, keys, rows, "ragged")
    _check(ko, keys, rows, "ragged with hint", max_keys=int(sizes.max()))


@pytest.mark.timeout(300)
@pytest.mark.parametrize("cfg", [3, 5])
def test_workload_record_sets(cfg):
    note(f"sort: workload {cfg} record sets")
    s, r = W.SHAPES[cfg]
    s = W.StoreSpec(1_000_000, s.n_authors, s.zipf_s, s.doc_cols, s.doc_dtype)
    st = W.make_store(s, 2, device=DEV)
    b = W.pack(W.make_requests(st, r, cfg))
    k, rw = _shuffle_within(b.key_offsets, b.keys, b.edge_rows, cfg)
    _check(b.key_offsets.cpu(), k, rw, f"workload {cfg}")
    _check(b.key_offsets.cpu(), k, rw, f"workload {cfg} with hint",
           max_keys=int(b.key_offsets.diff().max()))


def test_sort_then_join_equals_oracle():
    note("sort then join")
    s, r = W.shape(2, store_n_docs=300_000, store_n_authors=200_000, req_k=3000,
                   req_n_cand=20_000, req_n_viewers=3)
    st = W.make_store(s, 4, device=DEV)
    b = W.pack(W.make_requests(st, r, 4))
    k, rw = _shuffle_within(b.key_offsets, b.keys, b.edge_rows, 4)
    ws = torch.empty(P.cc_sort_workspace_bytes(k.numel(), 3), dtype=torch.uint8, device=DEV)
    ko_d = b.key_offsets
    k_s, r_s = torch.empty_like(b.keys), torch.empty_like(b.edge_rows)
    P.cc_sort_affinity(ko_d, k.to(DEV), rw.to(DEV), k_s, r_s, ws)
    store = P.cc_store_create(st.author_id, st.doc_rows)
    try:
        wd, we = row_bytes(st.doc_rows), row_bytes(b.edge_rows)
        out = torch.empty(b.cand_idx.numel(), wd + we, dtype=torch.uint8, device=DEV)
        hit = torch.empty(b.cand_idx.numel(), 1, dtype=torch.int8, device=DEV)
        P.cc_join_batched(store, b.cand_offsets, b.cand_idx, ko_d, k_s, r_s, out, hit)
        torch.cuda.synchronize()
        bc = b.to("cpu")
        ks, rs = oracle.sort_affinity(bc.key_offsets, k, rw)
        want = oracle.join(st.author_id.cpu(), st.doc_rows.cpu(), bc.cand_offsets, bc.cand_idx,
                           bc.key_offsets, ks, rs)
        assert np.array_equal(out.cpu().numpy(), want[0]) and np.array_equal(hit.cpu().numpy(), want[1])
    finally:
        P.cc_store_destroy(store)


def test_key_span_at_the_packed_limit():
    """Records whose keys span just under, and exactly at, the limit of the 8-byte element form
    (2^(64 - b) - 1 for b position bits): the first is sorted packed, the second wide; both
    must match the oracle."""
    note("sort: key span at the packed limit")
    n = 1000                                     # b = 10 position bits
    g = W.gen("cpu", 5, 3)
    rows = torch.randint(0, 256, (n, 16), generator=g, dtype=torch.int64).to(torch.uint8)
    for span in ((1 << 54) - 2, (1 << 54) - 1, (1 << 63) - 1):
        base = -(1 << 62)
        keys = base + torch.randint(0, 50, (n,), generator=g) * (span // 49)
        keys[0], keys[1] = base, base + span    # the span is exact
        keys[2:6] = base + span // 2            # repeats
        _check(torch.tensor([0, n]), keys, rows, f"span {span}")
        _check(torch.tensor([0, n]), keys, rows, f"span {span} with hint", max_keys=n)


def test_thousands_of_small_viewers():
    """5,000 viewers of 0 to 40 records: the tile plan scans the viewers in several chunks and
    every tile finds its viewer by search."""
    note("sort: 5,000 small viewers")
    g = W.gen("cpu", 21, 3)
    sizes = torch.randint(0, 41, (5000,), generator=g)
    sizes[::97] = 0
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    keys = torch.randint(-50, 50, (n,), generator=g)
    rows = torch.randint(0, 256, (n, 16), generator=g, dtype=torch.int64).to(torch.uint8)
    _check(ko, keys, rows, "5000 viewers")


@pytest.mark.parametrize("max_keys", [0, 20_000])
def test_many_viewers_with_merge_rounds(max_keys):
    """1,300 viewers (more than one round of the workgroup-wide viewer search) where every 50th
    has 5,000 to 20,000 records, so the merge rounds also look up viewers past the first 512;
    the rest hold 0 to 60 records. Packed elements; without and with the max_keys hint."""
    note(f"sort: 1,300 viewers with merge rounds, max_keys {max_keys}")
    g = W.gen("cpu", 23, 5)
    sizes = torch.randint(0, 61, (1300,), generator=g)
    sizes[::50] = torch.randint(5_000, 20_001, (26,), generator=g)
    sizes[3::97] = 0
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    keys = torch.randint(0, 3_000, (n,), generator=g)            # many equal keys: stability
    rows = torch.randint(0, 256, (n, 32), generator=g, dtype=torch.int64).to(torch.uint8)
    _check(ko, keys, rows, f"1300 viewers, max_keys {max_keys}", max_keys=max_keys)


@pytest.mark.parametrize("max_keys", [1, 4095, 6000, 20_000])
def test_viewers_above_the_max_keys_bound_are_copied_through(max_keys):
    """A max_keys hint below some viewer's record count: that viewer is copied to the output in
    input order (keys and rows), every other viewer is sorted as usual."""
    sizes = [5000, 20_000, 300, 0, 6001, 1]
    ko = torch.tensor([0] + np.cumsum(sizes).tolist(), dtype=torch.int64)
    g = torch.Generator().manual_seed(max_keys)
    n = int(ko[-1])
    keys = torch.randint(-500, 500, (n,), generator=g)
    rows = torch.randint(0, 256, (n, 48), generator=g, dtype=torch.int64).to(torch.uint8)
    note(f"sort: viewers {sizes}, max_keys {max_keys}")
    wk, wr = oracle.sort_affinity(ko, keys, rows)
    kn, rn = keys.numpy(), oracle.as_bytes(rows)
    for method in METHODS:
        gk, gr = _gpu_sort(ko, keys, rows, max_keys, method)
        for v, size in enumerate(sizes):
            sl = slice(int(ko[v]), int(ko[v + 1]))
            want_k, want_r = (kn[sl], rn[sl]) if size > max_keys else (wk[sl], wr[sl])
            assert np.array_equal(gk[sl], want_k), f"method {method}, viewer {v} ({size}): keys"
            assert np.array_equal(gr[sl], want_r), f"method {method}, viewer {v} ({size}): rows"


@pytest.mark.parametrize("key_bits", [9, 18, 26, 27, 64])
def test_radix_passes_bounded_by_key_bits(key_bits):
    """A key_bits bound that holds launches only the passes it needs (1 to 3 here, 8 at 64):
    the output is still the oracle's. Viewers of several tiles, keys spanning just under
    2^min(key_bits, 26), with repeats."""
    note(f"sort: radix with key_bits {key_bits}")
    g = W.gen("cpu", 40 + key_bits, 3)
    sizes = torch.tensor([30_000, 9_000, 100, 17_000, 4097])
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    span = 1 << min(key_bits, 26)
    keys = 1_000_000_000 + torch.randint(0, span, (n,), generator=g)
    keys[::5] = 1_000_000_000 + span - 1                         # the span is exact, repeats
    rows = torch.randint(0, 256, (n, 32), generator=g, dtype=torch.int64).to(torch.uint8)
    gk, gr = _gpu_sort(ko, keys, rows, 0, P.SORT_RADIX, key_bits)
    wk, wr = oracle.sort_affinity(ko, keys, rows)
    assert np.array_equal(gk, wk), "keys"
    assert np.array_equal(gr, wr), "rows"


def test_radix_with_a_key_bits_bound_that_does_not_hold():
    """Keys spanning 40 bits under a 9-bit bound: every viewer still gets a permutation of its
    own records, each key with its own row (the order is unspecified), and nothing outside the
    outputs changes."""
    note("sort: radix with a key_bits bound that does not hold")
    g = W.gen("cpu", 41, 3)
    sizes = torch.tensor([20_000, 3_000, 12_000])
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    keys = torch.randint(0, 1 << 40, (n,), generator=g)
    rows = torch.zeros(n, 16, dtype=torch.uint8)
    rows.view(torch.int64)[:, 0] = keys                          # each row names its key
    rows.view(torch.int64)[:, 1] = torch.arange(n)
    gk, gr = _gpu_sort(ko, keys, rows, 0, P.SORT_RADIX, 9)
    gr64 = gr.view(np.int64).reshape(n, 2)
    assert np.array_equal(gr64[:, 0], gk), "every key travels with its own row"
    for v in range(len(sizes)):
        lo, hi = int(ko[v]), int(ko[v + 1])
        src = gr64[lo:hi, 1]
        assert np.array_equal(np.sort(src), np.arange(lo, hi)), f"viewer {v}: a permutation"


def test_multi_tile_viewers_with_wide_keys():
    """Viewers of several tiles whose keys span all 64 bits: the radix method takes the wide
    16-byte elements (4,096-record tiles) and all 8 digit passes, the last 5 of them on the
    looping workgroups; repeats across tiles check stability. Both methods against the oracle."""
    note("sort: multi-tile viewers, 64-bit key span")
    g = W.gen("cpu", 43, 3)
    sizes = torch.tensor([12_000, 4_097, 9_000, 1])
    ko = torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(sizes, 0)])
    n = int(ko[-1])
    keys = torch.randint(-(1 << 62), 1 << 62, (n,), generator=g) * 2
    keys[0], keys[1] = -(1 << 63), (1 << 63) - 1                 # the full span
    keys[::11] = 12345                                           # repeats across tiles
    rows = torch.randint(0, 256, (n, 16), generator=g, dtype=torch.int64).to(torch.uint8)
    _check(ko, keys, rows, "64-bit span")

