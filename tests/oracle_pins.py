"""Pins that tie the CPU oracle to something other than itself.

Each pin takes a loaded oracle library (``oracle.load(path)``) so the planted-mistake test can
run the same pins against deliberately broken copies of the oracle. The references used here
are independent of the oracle's code:

* ``pin_golden``      -- the hand-worked Eq. 1 example in ``tests/golden/eq1_worked.json``;
* ``pin_scan``        -- a pure-Python scan of Eq. 1 on tiny random inputs (the naive O(N K)
                         scan of §3.1), including duplicates, int64 extremes, invalid positions;
* ``pin_alg1``        -- a first-record map built from NumPy's stable ``argsort`` and
                         ``np.unique`` (each id gets the row of its first record once records
                         are stably sorted, the record Eq. 1 picks after Alg. 1 Step 1), given
                         the keys in shuffled order;
* ``pin_invariants``  -- properties of the result on generated workloads: hit iff the key is
                         in the viewer's key set, miss rows equal the default row, valid doc
                         segments equal the store row, equivariance under a permutation of the
                         candidates, batched == per-viewer concatenation, the second lookup does
                         not disturb the first, and the hit count equals the membership count;
* ``pin_padding`` / ``pin_sort`` -- the padded layout of §6.3.1 and Alg. 1 Step 1;
* ``pin_index_golden`` -- the hand-worked ingestion example in ``tests/golden/upsert_worked.json``;
* ``pin_resolve``     -- Eq. 6 against a brute-force scan and a sorted-search route;
* ``pin_upsert``      -- the sequential replay against the four-step batch protocol of §6.2
                         written with NumPy set operations.
"""
from __future__ import annotations

import json
import sys
from pathlib import Path

import numpy as np
import torch

import oracle
import workload as W

GOLDEN = Path(__file__).resolve().parent / "golden"
METHODS = (oracle.LOWER_BOUND, oracle.SCAN, oracle.HASH)
FILL = 0xCD


def _np(t):
    return t.detach().cpu().numpy()


def _run(lib, tc: W.TinyCase, method, **kw):
    b = tc.batch
    extra = [b.actor] if tc.n_lookups == 2 else None
    return oracle.join(tc.author_id, tc.doc_rows, b.cand_offsets, b.cand_idx, b.key_offsets,
                       b.keys, b.edge_rows, default_row=tc.default_row,
                       n_lookups=tc.n_lookups, extra_keys=extra, method=method, lib=lib,
                       fill=FILL, **kw)


# --------------------------------------------------------------------------------------------
def pin_golden(lib):
    g = json.loads((GOLDEN / "eq1_worked.json").read_text())
    i32 = lambda x: np.asarray(x, dtype=np.int32)
    author = np.asarray(g["author_id"], dtype=np.int64)
    doc, edge = i32(g["doc_rows"]), i32(g["edge_rows"])
    want2 = i32(g["expected_out_two_lookups"])
    hit2 = np.asarray(g["expected_hit_two_lookups"], dtype=np.int8)
    for m in METHODS:
        out, hit, inv = oracle.join(author, doc, g["cand_offsets"], g["cand_idx"],
                                    g["key_offsets"], g["keys"], edge, n_lookups=2,
                                    extra_keys=[g["actor_keys"]], method=m, lib=lib, fill=FILL)
        assert np.array_equal(out.view(np.int32), want2), f"golden two-lookup rows, method {m}"
        assert np.array_equal(hit, hit2), f"golden two-lookup hits, method {m}"
        assert inv == g["expected_invalid"], f"golden invalid count, method {m}"
        out1, hit1, inv1 = oracle.join(author, doc, g["cand_offsets"], g["cand_idx"],
                                       g["key_offsets"], g["keys"], edge, method=m, lib=lib,
                                       fill=FILL)
        assert np.array_equal(out1.view(np.int32), want2[:, :8]), f"golden one-lookup, {m}"
        assert np.array_equal(hit1[:, 0], hit2[:, 0]), f"golden one-lookup hits, {m}"
        assert inv1 == g["expected_invalid"]
        # A non-zero default row replaces every miss segment and nothing else.
        dflt = np.array([-7, 8, -9, 10], dtype=np.int32)
        out3, _, _ = oracle.join(author, doc, g["cand_offsets"], g["cand_idx"],
                                 g["key_offsets"], g["keys"], edge, n_lookups=2,
                                 extra_keys=[g["actor_keys"]], default_row=dflt.view(np.uint8),
                                 method=m, lib=lib, fill=FILL)
        want3 = want2.copy()
        for j in range(want3.shape[0]):
            for l in range(2):
                if hit2[j, l] == 0:
                    want3[j, 4 + 4 * l: 8 + 4 * l] = dflt
        assert np.array_equal(out3.view(np.int32), want3), f"golden default row, method {m}"


# --------------------------------------------------------------------------------------------
def scan_reference(tc: W.TinyCase):
    """Eq. 1 by a plain scan, in pure Python (tiny inputs only)."""
    b = tc.batch
    author = _np(tc.author_id).tolist()
    doc = _np(tc.doc_rows)
    edge = _np(b.edge_rows)
    co, ko = _np(b.cand_offsets).tolist(), _np(b.key_offsets).tolist()
    cand, keys = _np(b.cand_idx).tolist(), _np(b.keys).tolist()
    actor = _np(b.actor).tolist() if tc.n_lookups == 2 else None
    n_docs, wd, we = len(author), doc.shape[1], edge.shape[1]
    L = tc.n_lookups
    dflt = bytes(we) if tc.default_row is None else bytes(_np(tc.default_row).tolist())
    rows, hits, invalid = [], [], 0
    for v in range(len(co) - 1):
        vkeys = keys[ko[v]:ko[v + 1]]
        for j in range(co[v], co[v + 1]):
            c = cand[j]
            if not (0 <= c < n_docs):
                invalid += 1
                rows.append(bytes(wd) + dflt * L)
                hits.append([0] * L)
                continue
            row = bytes(doc[c].tolist())
            h = []
            for l in range(L):
                key = author[c] if l == 0 else actor[j]
                found = None
                for i, a in enumerate(vkeys):
                    if a == key:
                        found = i
                        break
                if found is None:
                    row += dflt
                    h.append(0)
                else:
                    row += bytes(edge[ko[v] + found].tolist())
                    h.append(1)
            rows.append(row)
            hits.append(h)
    return rows, hits, invalid


def pin_scan(lib, seeds=range(60)):
    for seed in seeds:
        tc = W.tiny_case(seed)
        rows, hits, invalid = scan_reference(tc)
        for m in METHODS:
            out, hit, inv = _run(lib, tc, m)
            assert inv == invalid, f"seed {seed} method {m}: invalid count"
            assert [bytes(r.tolist()) for r in out] == rows, f"seed {seed} method {m}: rows"
            assert hit.tolist() == hits, f"seed {seed} method {m}: hit mask"


# --------------------------------------------------------------------------------------------
def first_record_rows(query_ids, record_ids, record_rows):
    """Eq. 1 for one viewer whose affinity records arrive in any order, from library routines.

    A query id receives the row of the first record carrying that id, where "first" is the
    order a stable sort by id leaves (records with equal ids keep their input order); a query
    id that no record carries receives the zero row. The map id -> first record comes from a
    stable argsort and np.unique's first-occurrence indices; membership from np.isin.
    Returns (rows [n, row_bytes], found [n] bool).
    """
    by_id = np.argsort(record_ids, kind="stable")
    distinct, first_in_sorted = np.unique(record_ids[by_id], return_index=True)
    first_record = dict(zip(distinct.tolist(), by_id[first_in_sorted].tolist()))
    found = np.isin(query_ids, distinct)
    rows = np.zeros((query_ids.shape[0], record_rows.shape[1]), dtype=record_rows.dtype)
    which = [first_record[q] for q in query_ids[found].tolist()]
    rows[found] = record_rows[np.asarray(which, dtype=np.int64)]
    return rows, found


def pin_alg1(lib, seeds=range(40)):
    rng = np.random.default_rng(12345)
    for seed in seeds:
        tc = W.tiny_case(seed, max_viewers=1, n_lookups=1, k_values=[int(rng.integers(1, 40))])
        b = tc.batch
        keys, edge = _np(b.keys), oracle.as_bytes(b.edge_rows)
        cand = _np(b.cand_idx)
        n_docs = tc.author_id.numel()
        ok = (cand >= 0) & (cand < n_docs)
        d = _np(tc.author_id)[np.where(ok, cand, 0)]
        # Alg. 1 receives the records in a shuffled order and sorts them itself (Step 1).
        # Equal keys keep their relative order in the shuffle, so its stable sort puts them
        # back in the order the oracle sees and the leftmost rule picks the same row.
        slot = rng.permutation(keys.shape[0])          # record i goes to position slot[i]
        for k in np.unique(keys):
            members = np.flatnonzero(keys == k)
            slot[members] = np.sort(slot[members])
        shuffled_keys = np.empty_like(keys)
        shuffled_edge = np.empty_like(edge)
        shuffled_keys[slot], shuffled_edge[slot] = keys, edge
        O, valid = first_record_rows(d, shuffled_keys, shuffled_edge)
        out, hit, _ = oracle.join(tc.author_id, tc.doc_rows, b.cand_offsets, b.cand_idx,
                                  b.key_offsets, b.keys, b.edge_rows, lib=lib, fill=FILL)
        wd = tc.doc_rows.shape[1]
        assert np.array_equal(hit[ok, 0].astype(bool), valid[ok]), f"seed {seed}: Alg.1 valid"
        assert np.array_equal(out[ok, wd:], O[ok]), f"seed {seed}: Alg.1 rows"


# --------------------------------------------------------------------------------------------
def _scaled_case(seed, cfg=2, lookups=False, viewers=3):
    s, r = W.shape(cfg, store_n_docs=60_000, store_n_authors=50_000, req_k=700,
                   req_n_cand=4_000, req_n_viewers=viewers, req_actor=lookups,
                   req_k_range=None)
    st = W.make_store(s, seed)
    reqs = W.make_requests(st, r, seed)
    return st, reqs


def pin_invariants(lib, seeds=(3, 4)):
    for seed in seeds:
        st, reqs = _scaled_case(seed, lookups=True)
        b = W.pack(reqs)
        author = _np(st.author_id)
        doc = oracle.as_bytes(st.doc_rows)
        wd = doc.shape[1]
        we = oracle.as_bytes(b.edge_rows).shape[1]
        g = W.gen("cpu", seed, 99)
        dflt = torch.randint(0, 256, (we,), generator=g, dtype=torch.int64).to(torch.uint8)
        # Plant a few invalid positions.
        cand = b.cand_idx.clone()
        cand[::97] = -1
        cand[5::211] = st.spec.n_docs
        out, hit, inv = oracle.join(st.author_id, st.doc_rows, b.cand_offsets, cand,
                                    b.key_offsets, b.keys, b.edge_rows, default_row=dflt,
                                    n_lookups=2, extra_keys=[b.actor], lib=lib, fill=FILL)
        cn = _np(cand)
        ok = (cn >= 0) & (cn < st.spec.n_docs)
        assert inv == int((~ok).sum()), "invalid count"
        edge = oracle.as_bytes(b.edge_rows)
        co, ko = _np(b.cand_offsets), _np(b.key_offsets)
        keys, actor = _np(b.keys), _np(b.actor)
        dn = _np(dflt)
        for v in range(len(reqs)):
            sl = slice(co[v], co[v + 1])
            vkeys = keys[ko[v]:ko[v + 1]]
            first = {}
            for i, k in enumerate(vkeys.tolist()):
                first.setdefault(k, i)
            for l, qk in enumerate((author[np.where(ok[sl], cn[sl], 0)], actor[sl])):
                member = np.isin(qk, vkeys) & ok[sl]
                h = hit[sl, l].astype(bool)
                # (i) hit iff the key is in the viewer's key set (and the position is valid)
                assert np.array_equal(h, member), f"seed {seed} viewer {v} lookup {l}: membership"
                seg = out[sl, wd + l * we: wd + (l + 1) * we]
                # (ii) a miss carries the default row
                assert (seg[~h] == dn).all(), "miss segment != default row"
                # hit rows are the edge row of that key
                rows = np.array([ko[v] + first[k] for k in qk[h].tolist()], dtype=np.int64)
                assert np.array_equal(seg[h], edge[rows]), "hit segment != edge row of key"
                # (vii) number of hits == size of the multiset intersection
                assert int(h.sum()) == int(member.sum())
            # (iii) valid doc segments are the store rows, invalid ones are zero
            assert np.array_equal(out[sl][ok[sl], :wd], doc[cn[sl][ok[sl]]]), "doc segment"
            assert (out[sl][~ok[sl], :wd] == 0).all(), "invalid doc segment"
        # (iv) equivariance: permuting candidates within each viewer permutes the rows
        perm = np.concatenate([co[v] + np.random.default_rng(seed + v).permutation(co[v + 1] - co[v])
                               for v in range(len(reqs))])
        outp, hitp, invp = oracle.join(st.author_id, st.doc_rows, b.cand_offsets, cn[perm],
                                       b.key_offsets, b.keys, b.edge_rows, default_row=dflt,
                                       n_lookups=2, extra_keys=[actor[perm]], lib=lib, fill=FILL)
        assert np.array_equal(outp, out[perm]) and np.array_equal(hitp, hit[perm])
        assert invp == inv
        # (v) batched == concatenation of single-viewer joins
        parts = []
        for v, q in enumerate(reqs):
            o1, h1, _ = oracle.join_single(st.author_id, st.doc_rows, cn[co[v]:co[v + 1]], q.keys,
                                           q.edge_rows, default_row=dflt, n_lookups=2,
                                           extra_keys=[q.actor], lib=lib, fill=FILL)
            parts.append((o1, h1))
        assert np.array_equal(np.concatenate([p[0] for p in parts]), out), "batched != singles"
        assert np.array_equal(np.concatenate([p[1] for p in parts]), hit)
        # (vi) the first lookup of a two-lookup join equals the one-lookup join
        o1, h1, _ = oracle.join(st.author_id, st.doc_rows, b.cand_offsets, cand, b.key_offsets,
                                b.keys, b.edge_rows, default_row=dflt, lib=lib, fill=FILL)
        assert np.array_equal(o1, out[:, :wd + we]) and np.array_equal(h1[:, 0], hit[:, 0])


# --------------------------------------------------------------------------------------------
def pin_padding(lib):
    """§6.3's padding example, then the padded layout against the CSR join on random inputs."""
    g = json.loads((GOLDEN / "padding_worked.json").read_text())
    feat = np.arange(100 * 16, dtype=np.int64).astype(np.uint8).reshape(100, 16)
    feat[:, 0] = np.arange(100)                       # row p starts with the byte p
    pos = g["positions"]
    co = np.array([0, len(pos[0]), len(pos[0]) + len(pos[1])])
    ci = np.array(pos[0] + pos[1])
    T, H, V, inv = oracle.join_padded(np.full(100, 7, np.int64), feat, co, ci, np.zeros(3, np.int64),
                                      np.zeros(0, np.int64), np.zeros((0, 16), np.uint8),
                                      g["n_max"], lib=lib)
    assert V.tolist() == g["expected_valid"], "padding example: valid mask"
    for b, want in enumerate(g["expected_rows"]):
        for i, p in enumerate(want):
            if p is None:
                assert not T[b, i].any() and not H[b, i].any(), "padding example: pad slot"
            else:
                assert np.array_equal(T[b, i, :16], feat[p]), "padding example: gathered row"
    got_idx = [[int(b), int(i)] for b, i in zip(*np.nonzero(V))]
    assert got_idx == g["scatter_indices"], "padding example: scatter indices"
    for seed in range(12):
        tc = W.tiny_case(3000 + seed, max_viewers=5)
        b = tc.batch
        n = np.diff(b.cand_offsets.numpy())
        n_max = int(n.max()) + (seed % 3) - 1 if n.max() > 0 else 1   # includes truncation
        n_max = max(n_max, 1)
        extra = [b.actor] if tc.n_lookups == 2 else None
        T, H, V, inv = oracle.join_padded(tc.author_id, tc.doc_rows, b.cand_offsets, b.cand_idx,
                                          b.key_offsets, b.keys, b.edge_rows, n_max,
                                          default_row=tc.default_row, n_lookups=tc.n_lookups,
                                          extra_keys=extra, lib=lib)
        out, hit, _ = _run(lib, tc, oracle.LOWER_BOUND)
        co = b.cand_offsets.numpy()
        for v in range(len(n)):
            k = min(n[v], n_max)
            assert np.array_equal(T[v, :k], out[co[v]:co[v] + k]), f"padded rows, seed {seed}"
            assert np.array_equal(H[v, :k], hit[co[v]:co[v] + k]), f"padded hits, seed {seed}"
            assert V[v, :k].all() and not V[v, k:].any(), f"padded valid, seed {seed}"
            assert not T[v, k:].any() and not H[v, k:].any(), f"padded pads, seed {seed}"


# --------------------------------------------------------------------------------------------
def pin_sort(lib):
    """Alg. 1 Step 1: the oracle's per-viewer sort against Python's stable sorted(), then the
    whole of Alg. 1 (sort, then join) against the NumPy route, on shuffled records."""
    for seed in range(40):
        tc = W.tiny_case(7000 + seed, max_k=60, max_viewers=4, dup_keys=bool(seed % 2))
        b = tc.batch
        ko = b.key_offsets.numpy()
        g = W.gen("cpu", seed, 5)
        keys = b.keys.clone()
        rows = b.edge_rows.clone()
        for v in range(len(ko) - 1):          # shuffle each viewer's records
            p = torch.randperm(int(ko[v + 1] - ko[v]), generator=g) + int(ko[v])
            keys[ko[v]:ko[v + 1]] = b.keys[p]
            rows[ko[v]:ko[v + 1]] = b.edge_rows[p]
        ks, rs = oracle.sort_affinity(ko, keys, rows, lib=lib)
        kn, rn = keys.numpy(), oracle.as_bytes(rows)
        for v in range(len(ko) - 1):
            sl = slice(ko[v], ko[v + 1])
            order = sorted(range(int(ko[v + 1] - ko[v])), key=lambda i: int(kn[sl][i]))
            assert ks[sl].tolist() == [int(kn[sl][i]) for i in order], f"sort keys, seed {seed}"
            assert np.array_equal(rs[sl], rn[sl][order]), f"sort rows, seed {seed}"
        # whole Alg. 1 on one viewer: shuffled records -> sort -> join == the NumPy first-record
        # map on the shuffled records
        v0 = slice(ko[0], ko[1])
        if ko[1] > ko[0]:
            cand = b.cand_idx[b.cand_offsets[0]:b.cand_offsets[1]].numpy()
            ok = (cand >= 0) & (cand < tc.author_id.numel())
            d = tc.author_id.numpy()[np.where(ok, cand, 0)]
            O, valid = first_record_rows(d, kn[v0], rn[v0])
            out, hit, _ = oracle.join_single(tc.author_id, tc.doc_rows, cand, ks[v0], rs[v0],
                                             lib=lib, fill=FILL)
            wd = tc.doc_rows.shape[1]
            assert np.array_equal(hit[ok, 0].astype(bool), valid[ok]), f"Alg.1 valid, seed {seed}"
            assert np.array_equal(out[ok, wd:], O[ok]), f"Alg.1 rows, seed {seed}"


def _golden_int(x):
    return oracle.INT64_MIN if x == "INT64_MIN" else int(x)


def _golden_state(st, d):
    rb = st.rows.shape[1]
    n = st.n_docs
    assert st.ids[:n].tolist() == [_golden_int(x) for x in d["ids"]]
    assert st.author[:n].tolist() == d["authors"]
    assert np.array_equal(st.rows[:n], np.repeat(np.array(d["row_fill"], np.uint8)[:, None], rb, 1))


def pin_index_golden(lib):
    """The hand-worked ingestion and id-resolution example in tests/golden/upsert_worked.json."""
    g = json.loads((GOLDEN / "upsert_worked.json").read_text())
    st = oracle.IndexState(g["capacity"], g["row_bytes"], lib=lib)
    for k, bt in enumerate(g["batches"]):
        ids = [_golden_int(x) for x in bt["ids"]]
        rows = np.repeat(np.array(bt["row_fill"], np.uint8)[:, None], g["row_bytes"], 1)
        r = st.upsert(ids, bt["authors"], rows)
        if bt.get("fits", True):
            assert r == (bt["n_new"], bt["n_rejected"]), f"upsert golden batch {k}: {r}"
        else:
            assert r is None, f"upsert golden batch {k} should not fit"
        _golden_state(st, bt["after"])
    q = [_golden_int(x) for x in g["resolve"]["queries"]]
    assert st.resolve(q).tolist() == g["resolve"]["positions"], "resolve golden"


def _random_ids(rng, n, lo=-(1 << 63) + 1, hi=(1 << 63) - 1):
    out = set()
    while len(out) < n:
        out.add(int(rng.integers(lo, hi, dtype=np.int64, endpoint=True)))
    return list(out)


def pin_resolve(lib):
    """Eq. 6: the oracle's map against a brute-force scan of the index (tiny inputs, int64
    extremes, the reserved id) and against a sorted-search route (argsort + searchsorted) on a
    larger index; every stored id resolves to its own position."""
    rng = np.random.default_rng(11)
    for seed in range(30):
        n = int(rng.integers(0, 40))
        ix = _random_ids(rng, n)
        if n and seed % 3 == 0:
            ix[0] = (1 << 63) - 1
            ix[-1] = oracle.INT64_MIN + 1
        extra = [0, -1, (1 << 63) - 1, oracle.INT64_MIN] + _random_ids(rng, 5)
        q = ix + extra
        rng.shuffle(q)
        want = []
        for x in q:
            p = -1
            for i, y in enumerate(ix):
                if y == x:
                    p = i
                    break
            want.append(p)
        got = oracle.resolve(np.array(ix, np.int64), np.array(q, np.int64), lib=lib)
        assert got.tolist() == want, f"resolve brute force, seed {seed}"
    n = 200_000
    ix = np.array(_random_ids(rng, n), np.int64)
    q = np.concatenate([ix[rng.integers(0, n, 50_000)], rng.integers(-(1 << 62), 1 << 62, 50_000)])
    order = np.argsort(ix, kind="stable")
    s = ix[order]
    k = np.searchsorted(s, q, side="left")
    kc = np.minimum(k, n - 1)
    want = np.where((k < n) & (s[kc] == q), order[kc], -1)
    got = oracle.resolve(ix, q, lib=lib)
    assert np.array_equal(got, want), "resolve vs sorted search"
    assert np.array_equal(oracle.resolve(ix, ix, lib=lib), np.arange(n)), "resolve identity"


def bootstrap_numpy(state, ids, authors, rows):
    """The four-step batch protocol of §6.2 in NumPy: (1) identify new vs stored ids (a tensor
    membership test), (2) prefix-sum positions for the new ids in order of first appearance,
    (3) scatter each id's last row to its position, (4) record the new ids in the map."""
    ids_all, author, table, n_docs, cap = state
    ok = ids != oracle.INT64_MIN
    i_ok = np.nonzero(ok)[0]
    ids_ok = ids[i_ok]
    stored = np.isin(ids_ok, ids_all[:n_docs])                              # step 1
    uniq, first = np.unique(ids_ok, return_index=True)
    is_new_first = np.zeros(len(ids_ok), bool)
    is_new_first[first] = ~stored[first]
    n_new = int(is_new_first.sum())
    if n_docs + n_new > cap:
        return None
    new_pos = n_docs + np.cumsum(is_new_first) - 1                          # step 2
    pos_of = dict(zip(ids_all[:n_docs].tolist(), range(n_docs)))
    for j in np.nonzero(is_new_first)[0]:
        pos_of[int(ids_ok[j])] = int(new_pos[j])
    rev_u, rev_first = np.unique(ids_ok[::-1], return_index=True)
    last = len(ids_ok) - 1 - rev_first                                      # last occurrences
    tgt = np.array([pos_of[int(x)] for x in ids_ok[last]], np.int64)
    table[tgt] = rows[i_ok[last]]                                           # step 3
    author[tgt] = authors[i_ok[last]]
    ids_all[new_pos[is_new_first]] = ids_ok[is_new_first]                   # step 4
    return n_docs + n_new, n_new, int((~ok).sum())


def pin_upsert(lib):
    """Ingestion: the oracle's sequential replay against the four-step batch protocol written
    with NumPy set operations, over batches mixing new ids, stored ids, repeats inside a batch,
    the reserved id, and batches that do not fit; then invariants of the final index."""
    rng = np.random.default_rng(5)
    cap, rb = 1500, 16
    st = oracle.IndexState(cap, rb, lib=lib)
    ref = [np.full(cap, oracle.INT64_MIN, np.int64), np.zeros(cap, np.int64),
           np.zeros((cap, rb), np.uint8), 0, cap]
    universe = np.array(_random_ids(rng, 4000), np.int64)
    last_row = {}
    for b in range(25):
        m = int(rng.integers(0, 400))
        ids = universe[rng.integers(0, 250 + 150 * b, m)]        # widening pool: new + stored
        if m and b % 4 == 1:
            ids[rng.integers(0, m, 3)] = oracle.INT64_MIN
        authors = rng.integers(-(1 << 40), 1 << 40, m)
        rows = rng.integers(0, 256, (m, rb)).astype(np.uint8)
        r = st.upsert(ids, authors, rows)
        w = bootstrap_numpy(ref, ids, authors, rows)
        if w is None:
            assert r is None, f"batch {b}: replay accepted a batch that does not fit"
        else:
            ref[3] = w[0]
            assert r == (w[1], w[2]), f"batch {b}: counts {r} vs {w[1:]}"
            for i in range(m):
                if ids[i] != oracle.INT64_MIN:
                    last_row[int(ids[i])] = (int(authors[i]), rows[i].copy())
        assert st.n_docs == ref[3], f"batch {b}: n_docs"
        n = st.n_docs
        assert np.array_equal(st.ids[:n], ref[0][:n]), f"batch {b}: ids by position"
        assert np.array_equal(st.author[:n], ref[1][:n]), f"batch {b}: authors"
        assert np.array_equal(st.rows[:n], ref[2][:n]), f"batch {b}: rows"
    n = st.n_docs
    assert len(set(st.ids[:n].tolist())) == n == len(last_row), "positions are a bijection"
    for x, (a, row) in last_row.items():
        p = int(st.resolve([x])[0])
        assert st.author[p] == a and np.array_equal(st.rows[p], row), "last write wins"


ALL_PINS = (pin_golden, pin_scan, pin_alg1, pin_invariants, pin_padding, pin_sort,
            pin_index_golden, pin_resolve, pin_upsert)


def run_all(lib_path=None):
    lib = oracle.load(lib_path)
    for p in ALL_PINS:
        p(lib)


if __name__ == "__main__":      # used by the planted-mistake test, one broken oracle per run
    try:
        run_all(sys.argv[1])
    except AssertionError as e:
        print("PIN FAILED:", e)
        sys.exit(3)
    sys.exit(0)
