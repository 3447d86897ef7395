"""The allocation-free sort entry point (cc_sort_affinity_noalloc) against the workspace sort
(cc_sort_affinity) through the C ABI: bit-exact, on two calls in a row, the second smaller than
the first (the fixed scratch keeps the first call's contents)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2609_22441_amd as P
from paper_2609_22441_amd import binding as B
from gpu_common import note

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _records(n_viewers, total, row_bytes, seed, extremes):
    """Ragged CSR records: random viewer sizes summing to `total`, keys with repeats (and the
    int64 extremes when `extremes`, which forces the sort's 16-byte element form)."""
    g = torch.Generator().manual_seed(seed)
    cuts = torch.sort(torch.randint(0, total + 1, (n_viewers - 1,), generator=g)).values
    off = torch.cat([torch.zeros(1, dtype=torch.int64), cuts, torch.tensor([total])])
    keys = torch.randint(-(1 << 20), 1 << 20, (total,), generator=g)
    if extremes:
        pick = torch.randint(0, total, (total // 50,), generator=g)
        keys[pick] = torch.tensor([-(1 << 63), (1 << 63) - 1, -1, 0],
                                  dtype=torch.int64)[torch.randint(0, 4, (pick.numel(),),
                                                                   generator=g)]
    rows = torch.randint(0, 256, (total, row_bytes), generator=g, dtype=torch.int64).to(torch.uint8)
    return off, keys, rows


def _sort_both(off, keys, rows, max_keys):
    o, k, r = off.to(DEV), keys.to(DEV), rows.to(DEV)
    k_ref = torch.full_like(k, 7)
    r_ref = torch.full_like(r, 0xCD)
    ws = torch.empty(P.cc_sort_workspace_bytes(k.numel(), o.numel() - 1), dtype=torch.uint8,
                     device=DEV)
    P.cc_sort_affinity(o, k, r, k_ref, r_ref, ws, max_keys=max_keys)
    k_got = torch.full_like(k, 9)
    r_got = torch.full_like(r, 0xAB)
    P.cc_sort_affinity_noalloc(o, k, r, k_got, r_got, max_keys=max_keys)
    torch.cuda.synchronize()
    return (k_ref.cpu().numpy(), r_ref.cpu().numpy()), (k_got.cpu().numpy(), r_got.cpu().numpy())


@pytest.mark.timeout(300)
def test_noalloc_sort_equals_the_workspace_sort_on_two_calls():
    cases = [
        # at both limits: 2^20 records over 2^16 viewers, packed 8-byte elements
        (B.SORT_NOALLOC_MAX_VIEWERS, B.SORT_NOALLOC_MAX_RECORDS, 32, 11, False),
        # 2^20 records over 16 viewers of several tiles: the radix method's digit passes and
        # look-back words in the fixed scratch
        (16, B.SORT_NOALLOC_MAX_RECORDS, 32, 13, False),
        # smaller, with int64 extremes (16-byte elements) and viewers of several tiles
        (7, 60_000, 64, 12, True),
    ]
    for nv, total, rb, seed, extremes in cases:
        off, keys, rows = _records(nv, total, rb, seed, extremes)
        max_keys = int((off[1:] - off[:-1]).max())
        note(f"noalloc sort: {nv} viewers, {total} records, {rb}-byte rows, "
             f"largest viewer {max_keys}")
        want, got = _sort_both(off, keys, rows, max_keys)
        assert np.array_equal(got[0], want[0]), "sorted keys differ from cc_sort_affinity"
        assert np.array_equal(got[1], want[1]), "moved rows differ from cc_sort_affinity"
        ko, ro = oracle.sort_affinity(off, keys, rows)
        assert np.array_equal(got[0], ko) and np.array_equal(got[1], ro), "differs from oracle"


def test_noalloc_sort_refuses_sizes_past_its_scratch():
    off = torch.tensor([0, B.SORT_NOALLOC_MAX_RECORDS + 1], dtype=torch.int64, device=DEV)
    keys = torch.zeros(B.SORT_NOALLOC_MAX_RECORDS + 1, dtype=torch.int64, device=DEV)
    rows = torch.zeros(keys.numel(), 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(P.CCError) as e:
        P.cc_sort_affinity_noalloc(off, keys, rows, torch.empty_like(keys),
                                   torch.empty_like(rows))
    assert e.value.status == B.CC_ERR_TOO_LARGE
