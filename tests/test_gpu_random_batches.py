"""Random valid batches against the oracle, bit-exact: 1 to 1,100 viewers (either side of the
weighted-split limit) with skewed candidate counts, some empty viewers, some lists longer than
the LDS table, one or two lookups, specialised and generic row widths, and several tunings."""
from __future__ import annotations

import pytest
import torch

import paper_2609_22441_amd as P
import workload as W
from gpu_common import assert_same, gpu_join, note, oracle_join

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
WIDTHS = [(64, 32), (128, 64), (128, 128), (48, 16), (16, 48)]
TUNINGS = [None, (4, 0, 0), (0, 0, 8), (0, 2048, 0), (0, 0, 600), (16, 64, 0)]


def _case(seed: int):
    g = torch.Generator().manual_seed(7100 + seed)
    ri = lambda lo, hi: int(torch.randint(lo, hi + 1, (1,), generator=g))
    B = ri(1, 1100) if seed % 3 else ri(1, 8)
    wd, we = WIDTHS[seed % len(WIDTHS)]
    L = 1 + seed % 2
    n_docs, n_ids = ri(1, 100_000), ri(10, 50_000)
    author = torch.randint(0, n_ids, (n_docs,), generator=g)
    doc = torch.randint(0, 256, (n_docs, wd), generator=g, dtype=torch.int64).to(torch.uint8)
    nc = torch.randint(0, max(2, 300_000 // B), (B,), generator=g)
    nc[torch.rand(B, generator=g) < 0.1] = 0
    kc = torch.randint(0, 300, (B,), generator=g)
    big = torch.rand(B, generator=g) < 0.05
    kc[big] = torch.randint(8_000, 30_000, (int(big.sum()),), generator=g)
    kc = torch.minimum(kc, torch.tensor(n_ids))
    co = torch.zeros(B + 1, dtype=torch.int64)
    co[1:] = torch.cumsum(nc, 0)
    ko = torch.zeros(B + 1, dtype=torch.int64)
    ko[1:] = torch.cumsum(kc, 0)
    keys = torch.cat([torch.sort(torch.randperm(n_ids, generator=g)[:k]).values
                      for k in kc.tolist()])
    edge = torch.randint(0, 256, (int(ko[-1]), we), generator=g, dtype=torch.int64).to(torch.uint8)
    tc = int(co[-1])
    cand = torch.randint(-2, n_docs + 2, (tc,), generator=g)
    actor = torch.randint(-1, n_ids, (tc,), generator=g) if L == 2 else None
    return author, doc, W.Batch(co, cand, ko, keys, edge, actor), wd, we, L


@pytest.mark.timeout(300)
@pytest.mark.parametrize("seed", range(12))
def test_random_batch(seed):
    author, doc, b, wd, we, L = _case(seed)
    t = TUNINGS[seed % len(TUNINGS)]
    note(f"random batch {seed}: B={b.n_viewers} cand={b.cand_idx.numel()} keys={b.keys.numel()} "
         f"widths={wd}/{we} L={L} tuning={t}")
    store = P.cc_store_create(author.to(DEV), doc.to(DEV))
    try:
        got = gpu_join(store, None, b.to(DEV), wd, we, L,
                       tuning=None if t is None else P.Tuning(*t, 0))
        want = oracle_join(author, doc, b, L)
        assert_same(got, want, f"random batch {seed}")
        assert P.cc_store_invalid_count(store) == want[2]
    finally:
        P.cc_store_destroy(store)
