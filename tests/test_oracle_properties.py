"""Property-based pins of the oracle (CPU only), on inputs that hypothesis draws and shrinks:
* join (Eq. 1): all three ways to find the leftmost equal key (lower bound, linear scan, hash
  map) give Eq. 1 written out as a plain Python scan, and the join is equivariant under a
  permutation of each viewer's candidates;
* ingestion (§6.2) and resolution (Eq. 6): the sequential replay equals plain Python over a
  dict, batch after batch, including refused batches and the reserved id;
* the sort (Alg. 1 Step 1): equals Python's stable sort within each viewer.
Ids come from a small pool that includes the int64 extremes, so keys collide and repeat often."""
from __future__ import annotations

import numpy as np
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import workload as W
from oracle_pins import scan_reference

ID_POOL = [-(1 << 63), -(1 << 63) + 1, -3, -1, 0, 1, 2, 3, 7, 1000, (1 << 62), (1 << 63) - 1]
ids = st.sampled_from(ID_POOL)


@st.composite
def cases(draw):
    n_docs = draw(st.integers(1, 12))
    wd = 16 * draw(st.integers(1, 2))
    we = 16 * draw(st.integers(1, 2))
    n_lookups = draw(st.integers(1, 2))
    author = draw(st.lists(ids, min_size=n_docs, max_size=n_docs))
    doc = draw(st.lists(st.integers(0, 255), min_size=n_docs * wd, max_size=n_docs * wd))
    reqs = []
    for _ in range(draw(st.integers(1, 3))):
        keys = sorted(draw(st.lists(ids, max_size=8)))          # may repeat: leftmost wins
        edge = draw(st.lists(st.integers(0, 255), min_size=len(keys) * we,
                             max_size=len(keys) * we))
        cand = draw(st.lists(st.integers(-2, n_docs + 1), max_size=10))   # some invalid
        actor = draw(st.lists(ids, min_size=len(cand), max_size=len(cand)))
        reqs.append(W.Request(torch.tensor(keys, dtype=torch.int64),
                              torch.tensor(edge, dtype=torch.uint8).reshape(len(keys), we),
                              torch.tensor(cand, dtype=torch.int64),
                              torch.tensor(actor, dtype=torch.int64) if n_lookups == 2 else None))
    default = None
    if draw(st.booleans()):
        default = torch.tensor(draw(st.lists(st.integers(0, 255), min_size=we, max_size=we)),
                               dtype=torch.uint8)
    return W.TinyCase(torch.tensor(author, dtype=torch.int64),
                      torch.tensor(doc, dtype=torch.uint8).reshape(n_docs, wd),
                      W.pack(reqs), default, n_lookups)


def run(tc, method, perm=None):
    b = tc.batch
    cand = b.cand_idx if perm is None else b.cand_idx[perm]
    actor = b.actor if (b.actor is None or perm is None) else b.actor[perm]
    return oracle.join(tc.author_id, tc.doc_rows, b.cand_offsets, cand, b.key_offsets, b.keys,
                       b.edge_rows, default_row=tc.default_row, n_lookups=tc.n_lookups,
                       extra_keys=[actor] if tc.n_lookups == 2 else None, method=method)


SETTINGS = settings(max_examples=300, deadline=None, derandomize=True, database=None,
                    suppress_health_check=[HealthCheck.too_slow])


@SETTINGS
@given(cases())
def test_every_method_is_eq1(tc):
    rows, hits, invalid = scan_reference(tc)
    width = tc.doc_rows.shape[1] + tc.n_lookups * tc.batch.edge_rows.shape[1]
    want_out = np.frombuffer(b"".join(rows), dtype=np.uint8).reshape(len(rows), width)
    want_hit = np.array(hits, dtype=np.int8).reshape(len(rows), tc.n_lookups)
    for method in (oracle.LOWER_BOUND, oracle.SCAN, oracle.HASH):
        out, hit, inv = run(tc, method)
        assert inv == invalid
        assert np.array_equal(hit, want_hit)
        assert np.array_equal(out, want_out)


@SETTINGS
@given(cases(), st.randoms(use_true_random=False))
def test_candidate_permutation_permutes_rows(tc, rnd):
    """Within each viewer, permuting the candidates permutes the output rows the same way."""
    b = tc.batch
    co = b.cand_offsets.tolist()
    perm = []
    for v in range(len(co) - 1):
        seg = list(range(co[v], co[v + 1]))
        rnd.shuffle(seg)
        perm += seg
    perm = torch.tensor(perm, dtype=torch.int64)
    out, hit, inv = run(tc, oracle.LOWER_BOUND)
    pout, phit, pinv = run(tc, oracle.LOWER_BOUND, perm)
    assert pinv == inv
    assert np.array_equal(pout, out[perm.numpy()])
    assert np.array_equal(phit, hit[perm.numpy()])


# ---- ingestion (§6.2) and id resolution (Eq. 6) ----

class DictModel:
    """Ingestion written as plain Python over a dict: records applied one at a time; a batch
    whose new ids do not fit in the capacity leaves everything unchanged."""

    def __init__(self, capacity, row_bytes):
        self.capacity, self.pos, self.ids, self.author, self.rows = capacity, {}, [], [], []
        self.row_bytes = row_bytes

    def upsert(self, batch):
        pos, ids = dict(self.pos), list(self.ids)
        author, rows = list(self.author), list(self.rows)
        rejected = 0
        for i, a, r in batch:
            if i == -(1 << 63):
                rejected += 1
                continue
            if i not in pos:
                if len(ids) == self.capacity:
                    return None
                pos[i] = len(ids)
                ids.append(i)
                author.append(0)
                rows.append(bytes(self.row_bytes))
            author[pos[i]] = a
            rows[pos[i]] = r
        n_new = len(ids) - len(self.ids)
        self.pos, self.ids, self.author, self.rows = pos, ids, author, rows
        return n_new, rejected


@SETTINGS
@given(st.integers(0, 10), st.lists(st.lists(st.tuples(ids, ids, st.binary(min_size=16,
                                                                           max_size=16)),
                                             max_size=8), max_size=5),
       st.lists(ids, max_size=12))
def test_upsert_replay_matches_a_dict(capacity, batches, queries):
    state = oracle.IndexState(capacity, 16)
    model = DictModel(capacity, 16)
    for batch in batches:
        ids_ = np.array([b[0] for b in batch], dtype=np.int64)
        authors = np.array([b[1] for b in batch], dtype=np.int64)
        rows = np.frombuffer(b"".join(b[2] for b in batch), dtype=np.uint8).reshape(len(batch), 16)
        got = state.upsert(ids_, authors, rows)
        assert got == model.upsert(batch)
        n = state.n_docs
        assert n == len(model.ids)
        assert state.ids[:n].tolist() == model.ids
        assert state.author[:n].tolist() == model.author
        assert [bytes(r) for r in state.rows[:n]] == model.rows
    got = state.resolve(np.array(queries, dtype=np.int64))
    want = [model.pos.get(q, -1) if q != -(1 << 63) else -1 for q in queries]
    assert np.asarray(got).tolist() == want


# ---- Alg. 1 Step 1: the per-viewer stable sort ----

@SETTINGS
@given(st.lists(st.lists(ids, max_size=12), min_size=1, max_size=4))
def test_sort_is_pythons_stable_sort_per_viewer(viewers):
    keys = [k for v in viewers for k in v]
    offs = np.cumsum([0] + [len(v) for v in viewers]).astype(np.int64)
    # row j carries its input index, so the test sees which record went where
    rows = np.zeros((len(keys), 16), dtype=np.uint8)
    rows[:, :8] = np.arange(len(keys), dtype=np.int64).view(np.uint8).reshape(-1, 8)
    k_out, r_out = oracle.sort_affinity(offs, np.array(keys, dtype=np.int64), rows)
    want = []
    for v in range(len(viewers)):
        want += sorted(range(offs[v], offs[v + 1]), key=lambda j: keys[j])   # stable
    src = r_out[:, :8].copy().view(np.int64).ravel().tolist()
    assert src == want
    assert k_out.tolist() == [keys[j] for j in want]
