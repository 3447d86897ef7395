"""Seeded synthetic inputs for the edge-feature join (Connected Content Retriever, §3.1).

This module only draws random inputs and packs them; it computes no part of the join
(no key search, no match test, no row selection). Both sides of every parity check, the
CPU oracle and the device library, take their inputs from here.

The paper's workloads are internal to its authors (LinkedIn Feed sessions and edge-affinity
data), so these generators stand in for them with the shapes the paper states in §3.1 (N in
the tens of thousands of candidates, K in the few thousands of affinity records) and the five
shapes named in the recipe table below.

Recipe (every draw comes from a ``torch.Generator`` seeded with
``seed * 1_000_003 + stream``; stream 0 is the store, stream 1 + v is viewer v):

* store: ``author_id`` int64 either uniform over ``[0, n_authors)`` or Zipf(s) over
  ``n_authors`` ids. Zipf ranks r = 1..M have weight r^-s and are sampled by inverse CDF on a
  float64 cumulative sum; rank -> id goes through a seeded random permutation so popularity is
  not correlated with key order. Doc features are N(0,1) draws in fp32, rounded to the stored
  dtype (bf16 rounds to nearest even).
* viewer keys: K unique ids, sorted ascending (signed int64). "uniform" draws them uniformly
  without replacement from ``[0, n_authors)``; "top1_half" takes half from the ids of the top 1%
  Zipf ranks and half uniformly from all ids, disjoint from the first half. K is fixed or
  log-uniform, ``floor(exp(U(ln lo, ln hi)))``.
* edge features: U(0,1) in fp32, rounded to the edge dtype.
* candidates: a fraction ``in_net_frac`` is sampled from the docs whose author is one of the
  viewer's keys (with or without replacement), the rest uniformly over all docs; the two parts
  are concatenated and shuffled. Duplicate candidates are allowed.
* actor keys (second lookup): half of the candidates carry an actor drawn uniformly from the
  viewer's keys, the other half carry -1 ("no actor").
* document ids (id map and ingestion, §6.3.1 and §6.2): item i has the id
  ``((i * A) mod 2^62) xor salt(seed)`` with A odd, a bijection on [0, 2^62), so ids are
  distinct and never the reserved INT64_MIN. The index holds items [0, n_index). A resolve
  batch has ``batch`` requests of ``ids_per_request`` ids; a share ``miss_rate`` are items past
  the index (absent), the rest uniform over stored items. An ingestion batch draws a share
  ``new_rate`` of new items (fresh indices), the rest uniform over stored items, then a share
  ``repeat_rate`` of its records repeat another record's id; the order is shuffled. Author
  ids are uniform over ``[0, n_authors)``, rows N(0,1) rounded to the row dtype.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import List, Optional, Sequence

import torch

__all__ = [
    "StoreSpec", "RequestSpec", "SHAPES", "Store", "Request", "Batch",
    "gen", "make_store", "make_requests", "pack", "salt_special_values", "shape",
    "IndexSpec", "INDEX_SHAPE", "doc_ids", "index_records", "resolve_queries", "upsert_batch",
]


@dataclass(frozen=True)
class StoreSpec:
    n_docs: int
    n_authors: int          # author ids lie in [0, n_authors)
    zipf_s: float           # 0.0 means uniform author ids
    doc_cols: int
    doc_dtype: torch.dtype


@dataclass(frozen=True)
class RequestSpec:
    n_viewers: int
    k: int                                  # keys per viewer when k_range is None
    k_range: Optional[tuple]                # (lo, hi): log-uniform keys per viewer
    key_mode: str                           # "uniform" or "top1_half"
    edge_cols: int
    edge_dtype: torch.dtype
    n_cand: int                             # candidates per viewer
    in_net_frac: float                      # share of candidates drawn from in-network docs
    in_net_replace: bool                    # in-network part drawn with replacement
    uniform_replace: bool                   # uniform part drawn with replacement
    actor: bool = False                     # second lookup key per candidate


F32, BF16 = torch.float32, torch.bfloat16

# The five workload shapes: (store, requests).
SHAPES = {
    # Single viewer, tiny: 1M docs, uniform authors over [0,1e5), 16 fp32 doc cols;
    # K=1000 uniform keys, 8 fp32 edge cols; N=10k uniform candidates without replacement.
    1: (StoreSpec(1_000_000, 100_000, 0.0, 16, F32),
        RequestSpec(1, 1_000, None, "uniform", 8, F32, 10_000, 0.0, False, False)),
    # Single viewer, production-shaped: 10M docs, Zipf(1.1) over 1e7 ids, 64 bf16 cols;
    # K=5000 (half top-1%), 32 bf16 edge cols; N=50k, 70% in-network.
    2: (StoreSpec(10_000_000, 10_000_000, 1.1, 64, BF16),
        RequestSpec(1, 5_000, None, "top1_half", 32, BF16, 50_000, 0.7, False, True)),
    # Batched ragged: same store; B=64 viewers, K log-uniform in [100, 30000]; N=30k each,
    # 70% in-network drawn with replacement (small-K viewers have small pools).
    3: (StoreSpec(10_000_000, 10_000_000, 1.1, 64, BF16),
        RequestSpec(64, 0, (100, 30_000), "top1_half", 32, BF16, 30_000, 0.7, True, True)),
    # Second-degree double join: K=20000, N=100k, author + actor lookups.
    4: (StoreSpec(10_000_000, 10_000_000, 1.1, 64, BF16),
        RequestSpec(1, 20_000, None, "top1_half", 32, BF16, 100_000, 0.7, False, True, actor=True)),
    # Large scale: 200M docs, Zipf(1.1) over 5e7 ids; B=32 viewers x K=100k, 64 bf16 edge
    # cols; 31,250 in-network candidates per viewer (1M per batch).
    5: (StoreSpec(200_000_000, 50_000_000, 1.1, 64, BF16),
        RequestSpec(32, 100_000, None, "top1_half", 64, BF16, 31_250, 1.0, False, True)),
}


def shape(i: int, **scale) -> tuple:
    """Return (StoreSpec, RequestSpec) of workload i, with optional field overrides.

    Overrides are given as ``store_<field>=`` / ``req_<field>=`` keyword arguments, e.g.
    ``shape(2, store_n_docs=100_000, req_n_cand=2_000)`` for a scaled-down copy.
    """
    s, r = SHAPES[i]
    s = replace(s, **{k[6:]: v for k, v in scale.items() if k.startswith("store_")})
    r = replace(r, **{k[4:]: v for k, v in scale.items() if k.startswith("req_")})
    return s, r


def gen(device, seed: int, stream: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1_000_003 + int(stream))
    return g


@dataclass
class Store:
    spec: StoreSpec
    author_id: torch.Tensor           # int64 [n_docs]
    doc_rows: torch.Tensor            # doc_dtype [n_docs, doc_cols]
    top_ids: Optional[torch.Tensor]   # ids of the top-1% Zipf ranks (None when uniform)
    _by_author: Optional[tuple] = None

    @property
    def device(self):
        return self.author_id.device

    def docs_by_author(self):
        """CSR from author id to the docs that author owns: (order, offsets[n_authors+1])."""
        if self._by_author is None:
            order = torch.argsort(self.author_id, stable=True)
            counts = torch.bincount(self.author_id, minlength=self.spec.n_authors)
            offsets = torch.zeros(self.spec.n_authors + 1, dtype=torch.int64, device=self.device)
            torch.cumsum(counts, 0, out=offsets[1:])
            self._by_author = (order, offsets)
        return self._by_author


@dataclass
class Request:
    keys: torch.Tensor                # int64 [K], strictly increasing
    edge_rows: torch.Tensor           # edge_dtype [K, edge_cols]
    cand_idx: torch.Tensor            # int64 [N]
    actor: Optional[torch.Tensor]     # int64 [N] or None


@dataclass
class Batch:
    cand_offsets: torch.Tensor        # int64 [B+1]
    cand_idx: torch.Tensor            # int64 [sum N]
    key_offsets: torch.Tensor         # int64 [B+1]
    keys: torch.Tensor                # int64 [sum K]
    edge_rows: torch.Tensor           # [sum K, edge_cols]
    actor: Optional[torch.Tensor]     # int64 [sum N] or None

    @property
    def n_viewers(self) -> int:
        return self.cand_offsets.numel() - 1

    def to(self, device):
        mv = lambda t: None if t is None else t.to(device)
        return Batch(mv(self.cand_offsets), mv(self.cand_idx), mv(self.key_offsets),
                     mv(self.keys), mv(self.edge_rows), mv(self.actor))


def _zipf_ids(n: int, m: int, s: float, perm: torch.Tensor, g, device, chunk=1 << 24):
    # The CDF is accumulated on the host: a device scan adds its tiles in a timing-dependent
    # order, so the CDF's last bits, and with them a few ids, could change from run to run.
    ranks = torch.arange(1, m + 1, dtype=torch.float64)
    cdf = torch.cumsum(ranks.pow_(-s), 0).to(device)
    del ranks
    total = cdf[-1].item()
    out = torch.empty(n, dtype=torch.int64, device=device)
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        u = torch.rand(hi - lo, dtype=torch.float64, device=device, generator=g) * total
        r = torch.searchsorted(cdf, u, right=True).clamp_(max=m - 1)
        out[lo:hi] = perm[r]
    return out


def make_store(spec: StoreSpec, seed: int, device="cpu", chunk_rows: int = 1 << 23) -> Store:
    device = torch.device(device)
    g = gen(device, seed, 0)
    if spec.zipf_s == 0.0:
        author = torch.randint(0, spec.n_authors, (spec.n_docs,), generator=g, device=device)
        top = None
    else:
        perm = torch.randperm(spec.n_authors, generator=g, device=device)
        author = _zipf_ids(spec.n_docs, spec.n_authors, spec.zipf_s, perm, g, device)
        top = perm[: max(1, spec.n_authors // 100)].clone()
        del perm
    rows = torch.empty(spec.n_docs, spec.doc_cols, dtype=spec.doc_dtype, device=device)
    for lo in range(0, spec.n_docs, chunk_rows):
        hi = min(spec.n_docs, lo + chunk_rows)
        rows[lo:hi] = torch.randn(hi - lo, spec.doc_cols, generator=g, device=device,
                                  dtype=torch.float32).to(spec.doc_dtype)
    return Store(spec, author, rows, top)


def _uniform_unique(m: int, count: int, exclude: Optional[torch.Tensor], g, device):
    """`count` distinct ids uniform over [0, m), none of them in `exclude`."""
    if count == 0:
        return torch.empty(0, dtype=torch.int64, device=device)
    if m <= 4 * (count + (0 if exclude is None else exclude.numel())):
        pool = torch.randperm(m, generator=g, device=device)
        if exclude is not None and exclude.numel():
            pool = pool[~torch.isin(pool, exclude)]
        assert pool.numel() >= count, "id space too small for the requested key count"
        return pool[:count]
    draw = 2 * count + 64
    while True:
        x = torch.unique(torch.randint(0, m, (draw,), generator=g, device=device))
        if exclude is not None and exclude.numel():
            x = x[~torch.isin(x, exclude)]
        if x.numel() >= count:
            return x[torch.randperm(x.numel(), generator=g, device=device)[:count]]
        draw *= 2


def _keys(store: Store, r: RequestSpec, k: int, g, device):
    m = store.spec.n_authors
    if r.key_mode == "uniform" or store.top_ids is None:
        keys = _uniform_unique(m, k, None, g, device)
    elif r.key_mode == "top1_half":
        h1 = k // 2
        top = store.top_ids
        if top.numel() < h1:
            raise ValueError(f"{h1} keys requested from only {top.numel()} top-1% ids")
        first = top[torch.randperm(top.numel(), generator=g, device=device)[:h1]]
        second = _uniform_unique(m, k - h1, first, g, device)
        keys = torch.cat([first, second])
    else:
        raise ValueError(r.key_mode)
    return torch.sort(keys).values


def _in_network_pool(store: Store, keys: torch.Tensor):
    """All docs whose author id is one of `keys` (CSR indexing by author id, no search)."""
    order, offsets = store.docs_by_author()
    ok = (keys >= 0) & (keys < store.spec.n_authors)
    k = keys[ok]
    lo, hi = offsets[k], offsets[k + 1]
    lens = hi - lo
    total = int(lens.sum().item())
    if total == 0:
        return order[:0]
    starts = torch.repeat_interleave(lo - (torch.cumsum(lens, 0) - lens), lens)
    return order[starts + torch.arange(total, device=keys.device)]


def _edge_rows(k, cols, dtype, g, device):
    return torch.rand(k, cols, generator=g, device=device, dtype=torch.float32).to(dtype)


def make_request(store: Store, r: RequestSpec, seed: int, viewer: int) -> Request:
    device = store.device
    g = gen(device, seed, 1 + viewer)
    if r.k_range is None:
        k = r.k
    else:
        lo, hi = r.k_range
        u = torch.rand(1, generator=g, device=device, dtype=torch.float64).item()
        k = int(math.floor(math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))))
    keys = _keys(store, r, k, g, device)
    edge = _edge_rows(k, r.edge_cols, r.edge_dtype, g, device)
    n_in = int(round(r.in_net_frac * r.n_cand))
    parts = []
    if n_in:
        pool = _in_network_pool(store, keys)
        if pool.numel() == 0:
            n_in = 0
        elif r.in_net_replace or pool.numel() < n_in:
            parts.append(pool[torch.randint(0, pool.numel(), (n_in,), generator=g, device=device)])
        else:
            parts.append(pool[torch.randperm(pool.numel(), generator=g, device=device)[:n_in]])
    n_un = r.n_cand - n_in
    if n_un:
        n = store.spec.n_docs
        if r.uniform_replace:
            parts.append(torch.randint(0, n, (n_un,), generator=g, device=device))
        else:
            parts.append(torch.randperm(n, generator=g, device=device)[:n_un])
    cand = torch.cat(parts) if parts else torch.empty(0, dtype=torch.int64, device=device)
    cand = cand[torch.randperm(cand.numel(), generator=g, device=device)]
    actor = None
    if r.actor:
        n = cand.numel()
        has = torch.zeros(n, dtype=torch.bool, device=device)
        has[torch.randperm(n, generator=g, device=device)[: n // 2]] = True
        if k:
            pick = keys[torch.randint(0, k, (n,), generator=g, device=device)]
        else:
            pick = torch.full((n,), -1, dtype=torch.int64, device=device)
        actor = torch.where(has, pick, torch.full_like(pick, -1))
    return Request(keys.contiguous(), edge.contiguous(), cand.contiguous(), actor)


def make_requests(store: Store, r: RequestSpec, seed: int, first_viewer: int = 0,
                  n_viewers: Optional[int] = None) -> List[Request]:
    n = r.n_viewers if n_viewers is None else n_viewers
    return [make_request(store, r, seed, first_viewer + v) for v in range(n)]


def pack(reqs: Sequence[Request]) -> Batch:
    """Concatenate requests into CSR form (offsets are running sums of the sizes)."""
    dev = reqs[0].cand_idx.device
    co = torch.zeros(len(reqs) + 1, dtype=torch.int64)
    ko = torch.zeros(len(reqs) + 1, dtype=torch.int64)
    co[1:] = torch.cumsum(torch.tensor([q.cand_idx.numel() for q in reqs], dtype=torch.int64), 0)
    ko[1:] = torch.cumsum(torch.tensor([q.keys.numel() for q in reqs], dtype=torch.int64), 0)
    actor = None
    if reqs[0].actor is not None:
        actor = torch.cat([q.actor for q in reqs])
    return Batch(co.to(dev), torch.cat([q.cand_idx for q in reqs]), ko.to(dev),
                 torch.cat([q.keys for q in reqs]), torch.cat([q.edge_rows for q in reqs]),
                 actor)


# Bit patterns that a pure copy must carry unchanged (quiet/signalling NaN with payloads,
# both zeros, both infinities, smallest and largest subnormals, the extreme normals).
_SPECIAL_F32 = [0x7FC00001, 0x7F800001, 0xFFC12345, 0x7FBFFFFF, 0x80000000, 0x00000000,
                0x7F800000, 0xFF800000, 0x00000001, 0x807FFFFF, 0x7F7FFFFF, 0x00800000]
_SPECIAL_BF16 = [0x7FC1, 0x7F81, 0xFFC5, 0x7FBF, 0x8000, 0x0000, 0x7F80, 0xFF80, 0x0001,
                 0x807F, 0x7F7F, 0x0080]


def salt_special_values(t: torch.Tensor, frac: float, g) -> torch.Tensor:
    """Overwrite a random `frac` of the entries of fp32/bf16 tensor `t` with special bit patterns."""
    if t.dtype == torch.float32:
        view, pats, idt = t.view(torch.int32), _SPECIAL_F32, torch.int32
        pats = [p - (1 << 32) if p >= 1 << 31 else p for p in pats]
    elif t.dtype == torch.bfloat16:
        view, pats, idt = t.view(torch.int16), _SPECIAL_BF16, torch.int16
        pats = [p - (1 << 16) if p >= 1 << 15 else p for p in pats]
    else:
        raise TypeError(t.dtype)
    flat = view.reshape(-1)
    n = flat.numel()
    m = int(n * frac)
    if m:
        pos = torch.randint(0, n, (m,), generator=g, device=t.device)
        which = torch.randint(0, len(pats), (m,), generator=g, device=t.device)
        flat[pos] = torch.tensor(pats, dtype=idt, device=t.device)[which]
    return t


# ---------------------------------------------------------------------------------------------
# Tiny randomized cases with edge values, for exhaustive small checks.

I64_MIN, I64_MAX = -(1 << 63), (1 << 63) - 1
_EDGE_IDS = [I64_MIN, I64_MIN + 1, -(1 << 40), -1, 0, 1, (1 << 40), I64_MAX - 1, I64_MAX]
_BAD_POS = [-1, -2, I64_MIN, I64_MAX, -(1 << 40)]


@dataclass
class TinyCase:
    author_id: torch.Tensor      # int64 [n_docs]
    doc_rows: torch.Tensor       # uint8 [n_docs, doc_bytes]
    batch: Batch                 # edge_rows are uint8 [sum K, edge_bytes]
    default_row: Optional[torch.Tensor]   # uint8 [edge_bytes] or None
    n_lookups: int


def tiny_case(seed: int, device="cpu", max_docs=48, max_k=40, max_n=64, max_viewers=4,
              n_lookups: Optional[int] = None, dup_keys: Optional[bool] = None,
              doc_bytes: Optional[int] = None, edge_bytes: Optional[int] = None,
              k_values: Optional[Sequence[int]] = None) -> TinyCase:
    """A small random join input whose ids collide often and include the int64 extremes.

    Keys are sorted ascending; with dup_keys they may repeat. Some candidate positions are
    invalid (negative, == n_docs, or far out of range).
    """
    g = gen("cpu", seed, 7)
    ri = lambda lo, hi: int(torch.randint(lo, hi + 1, (1,), generator=g).item())
    n_docs = ri(1, max_docs)
    b = ri(1, max_viewers)
    if n_lookups is None:
        n_lookups = ri(1, 2)
    if dup_keys is None:
        dup_keys = ri(0, 3) == 0
    wd = doc_bytes if doc_bytes is not None else 16 * ri(1, 4)
    we = edge_bytes if edge_bytes is not None else 16 * ri(1, 3)
    pool = torch.tensor(list(range(-12, 13)) + _EDGE_IDS, dtype=torch.int64)
    pick = lambda n: pool[torch.randint(0, pool.numel(), (n,), generator=g)]
    author = pick(n_docs)
    doc = torch.randint(0, 256, (n_docs, wd), generator=g, dtype=torch.int64).to(torch.uint8)
    reqs = []
    for v in range(b):
        k = ri(0, max_k) if k_values is None else int(k_values[v % len(k_values)])
        if dup_keys:
            keys = torch.sort(pick(k)).values
        else:
            k = min(k, pool.numel())
            keys = torch.sort(pool[torch.randperm(pool.numel(), generator=g)[:k]]).values
        n = ri(0, max_n)
        cand = torch.randint(0, n_docs, (n,), generator=g)
        bad = torch.rand(n, generator=g) < 0.1
        if bad.any():
            choices = torch.tensor(_BAD_POS + [n_docs, n_docs + 3], dtype=torch.int64)
            cand[bad] = choices[torch.randint(0, choices.numel(), (int(bad.sum()),), generator=g)]
        edge = torch.randint(0, 256, (keys.numel(), we), generator=g,
                             dtype=torch.int64).to(torch.uint8)
        actor = None
        if n_lookups == 2:
            actor = pick(n)
            if keys.numel():
                use = torch.rand(n, generator=g) < 0.5
                actor[use] = keys[torch.randint(0, keys.numel(), (int(use.sum()),), generator=g)]
        reqs.append(Request(keys, edge, cand, actor))
    batch = pack(reqs)
    default = None
    if ri(0, 1):
        default = torch.randint(0, 256, (we,), generator=g, dtype=torch.int64).to(torch.uint8)
    tc = TinyCase(author, doc, batch, default, n_lookups)
    if torch.device(device).type != "cpu":
        tc = TinyCase(author.to(device), doc.to(device), batch.to(device),
                      None if default is None else default.to(device), n_lookups)
    return tc


# ---- document ids: the id map (§6.3.1, Eq. 6) and ingestion batches (§6.2) ----

@dataclass(frozen=True)
class IndexSpec:
    n_index: int            # documents in the index (items [0, n_index))
    n_authors: int
    row_cols: int
    row_dtype: torch.dtype
    batch: int              # requests per resolve batch (the paper's b)
    ids_per_request: int    # candidate ids per request ("tens of thousands")
    miss_rate: float        # share of query ids not in the index
    upsert_batch: int       # records per ingestion batch
    new_rate: float         # share of an ingestion batch's records with new ids
    repeat_rate: float      # share of records repeating another record's id in the batch


# The one-shard index of the largest store shape (200M documents with 64 bf16 columns); resolve
# batches of b = 8 requests x 50,000 ids (§6.3.1 quotes batch 8 with tens of thousands of ids
# per request against a few-hundred-million-entry index); ingestion batches of 300,000 records
# (§6.2: bootstrap batches of hundreds of thousands of documents).
INDEX_SHAPE = IndexSpec(200_000_000, 50_000_000, 64, BF16, 8, 50_000, 0.02, 300_000, 0.2, 0.05)

_ID_MASK = (1 << 62) - 1
_ID_MULT = 0x2545F4914F6CDD1D & _ID_MASK       # odd


def doc_ids(items: torch.Tensor, seed: int) -> torch.Tensor:
    """Distinct document ids for item indices (int64 tensor, any device)."""
    salt = (seed * 0x9E3779B97F4A7C15 + 0x632BE59BD9B4E019) & _ID_MASK
    return ((items * _ID_MULT) & _ID_MASK) ^ salt


def index_records(spec: IndexSpec, items: torch.Tensor, seed: int, stream: int, device="cpu"):
    """(doc ids, author ids, rows) for the given item indices."""
    g = gen(device, seed, stream)
    n = items.numel()
    ids = doc_ids(items.to(device), seed)
    authors = torch.randint(0, spec.n_authors, (n,), generator=g, device=device)
    rows = torch.randn(n, spec.row_cols, generator=g, device=device).to(spec.row_dtype)
    return ids, authors, rows


def resolve_queries(spec: IndexSpec, n_stored: int, seed: int, device="cpu") -> torch.Tensor:
    """[batch * ids_per_request] query ids: stored items, and a share of absent ones."""
    g = gen(device, seed, 11)
    m = spec.batch * spec.ids_per_request
    items = torch.randint(0, max(n_stored, 1), (m,), generator=g, device=device)
    miss = torch.rand(m, generator=g, device=device) < spec.miss_rate
    absent = n_stored + torch.randint(0, 1 << 40, (m,), generator=g, device=device)
    return doc_ids(torch.where(miss | (n_stored == 0), absent, items), seed)


def upsert_batch(spec: IndexSpec, n_stored: int, next_item: int, seed: int, stream: int,
                 device="cpu", n: Optional[int] = None):
    """One ingestion batch: (ids, authors, rows, n_fresh_items). Fresh items are
    [next_item, next_item + n_fresh_items); the caller advances next_item by that much."""
    g = gen(device, seed, stream)
    n = spec.upsert_batch if n is None else n
    n_new = int(round(n * spec.new_rate)) if n_stored > 0 else n
    items = torch.cat([torch.arange(next_item, next_item + n_new, device=device),
                       torch.randint(0, max(n_stored, 1), (n - n_new,), generator=g,
                                     device=device)])
    rep = torch.nonzero(torch.rand(n, generator=g, device=device) < spec.repeat_rate).flatten()
    if n > 0 and rep.numel():
        items[rep] = items[torch.randint(0, n, (rep.numel(),), generator=g, device=device)]
    items = items[torch.randperm(n, generator=g, device=device)]
    ids, authors, rows = index_records(spec, items, seed, stream + 1, device)
    return ids, authors, rows, n_new
