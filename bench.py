"""Benchmark of the edge-feature join on one MI355X (prints one JSON line).

Headline workload: the production-shaped single-viewer request (10M-document store with
Zipf(1.1) author ids, 64 bf16 document columns; K = 5,000 sorted affinity keys with 32 bf16
columns; N = 50,000 candidates, 70% in-network). A step joins 64 distinct such requests in one
cc_join_batched launch (3.2M candidates). Steps cycle through 4 distinct batches.

Each timed step starts with cold caches: a 1 GiB read before the step leaves none of the join's
data in L2 or the 256 MB Infinity Cache. The step itself is timed with HIP events on the launch
stream; the flush lies outside the events.

Reported:
  value           joined candidates/s: candidates per step / mean cold step time
  warm            the same steps back to back, without the flush
  roofline        algorithmic bytes per launch (8-byte author id per candidate) / mean cold launch
                  time, against 8 TB/s; the figure with the store's 4-byte author column is
                  given beside it
  latency         per-request latency of single cc_join calls (hip events on the stream, and
                  host wall time to completion); PreparedJoin; the two-lookup request
  configs         every workload shape at full size (1-5, and workload 4's request 64 per
                  launch), cold and warm, each with its algorithmic bandwidth; the record sorts
  cpu_baseline    the CPU oracle on one thread and on all the threads this job may use, on
                  bounded samples of every workload
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

METRIC = "joined candidates/sec + achieved HBM GB/s (% peak); p99 per-request join ms"
PEAK_GBPS = 8000.0
REQS_PER_STEP = 64
N_BATCHES = 4
KERNEL_SRC = ROOT / "paper_2609_22441_amd" / "csrc" / "join_kernels.hip"
TRAFFIC = ROOT / "profiles" / "traffic_production_x64.json"
HEADLINE_KERNEL = "join_kernel<8, 4, 1, true, true>"


def parse(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--latency-calls", type=int, default=1024)
    ap.add_argument("--cpu-seconds", type=float, default=1.5,
                    help="length of each CPU-baseline leg (one workload, one thread count)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload entries (headline step and latency only)")
    ap.add_argument("--seed", type=int, default=2)
    ap.add_argument("--all-configs", action="store_true",
                    help="also the padded layout, the id map, ingestion, the merge-path probe "
                         "and a reference device copy")
    ap.add_argument("--only-headline", action="store_true",
                    help="only the headline steps (warm-up, cold steps, warm steps): for counter "
                         "passes on the headline launch")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (known bytes) for counter scaling")
    ap.add_argument("--only-sorts", default="",
                    help="time only the record sorts of these workload shapes (2, 3 and/or 5): "
                         "for counter passes on the sort")
    ap.add_argument("--only-index", action="store_true",
                    help="run only the id-map part (index build, resolve, ingestion batches): for "
                         "counter passes on those kernels")
    ap.add_argument("--only-workloads", default="",
                    help="time only the joins of these workload shapes (e.g. 3,5 or 4x64), "
                         "without the headline, the sort or the id map: for per-workload "
                         "counter passes")
    return ap.parse_args(argv)


def algorithmic_bytes(torch, st, batch, wd, we, n_lookups=1, author_bytes=8):
    """Bytes the method must move for one launch: per candidate its position, author id
    (author_bytes wide), doc row, output row, hit bytes and (second lookup) its extra key; per
    viewer its keys and each distinct edge row that some lookup hits."""
    n = batch.cand_idx.numel()
    per_cand = 8 + author_bytes + wd + (wd + n_lookups * we) + n_lookups + 8 * (n_lookups - 1)
    keys_bytes = batch.keys.numel() * 8
    co, ko = batch.cand_offsets.tolist(), batch.key_offsets.tolist()
    rows = 0
    for v in range(len(co) - 1):
        q = st.author_id[batch.cand_idx[co[v]:co[v + 1]]]
        if n_lookups == 2:
            q = torch.cat([q, batch.actor[co[v]:co[v + 1]]])
        rows += int(torch.isin(torch.unique(q), batch.keys[ko[v]:ko[v + 1]]).sum())
    return n * per_cand + keys_bytes + rows * we


class Flush:
    """Reads 1 GiB on the current stream: afterwards neither L2 nor the 256 MB Infinity Cache
    holds any of the join's data. A read leaves clean lines; a write would leave dirty lines
    whose write-back the next launch would pay for."""

    def __init__(self, torch, dev):
        self.buf = torch.ones(1 << 27, dtype=torch.int64, device=dev)

    def __call__(self):
        self.buf.amax()


def time_launches(torch, fn, iters, flush=None, warm=5):
    """Per-launch times (ms) of `fn` on the current stream, each bracketed by HIP events; with
    `flush`, a cache flush runs before each launch (outside the events). Returns
    {median, mean, min, max, n}."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(iters)]
    for a, b in evs:
        if flush is not None:
            flush()
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    return {"median": ms[len(ms) // 2], "mean": sum(ms) / len(ms), "min": ms[0], "max": ms[-1],
            "n": len(ms)}


def rates(n_cand, alg, alg_stored, t_cold, t_warm):
    """A per-workload entry's rates from cold and warm launch times (ms medians)."""
    bw = lambda b, ms: b / (ms / 1e3) / 1e9
    return {"ms_median": t_cold["median"], "ms_mean": t_cold["mean"],
            "ms_median_warm": t_warm["median"],
            "candidates_per_s": n_cand / (t_cold["median"] / 1e3),
            "algorithmic_bytes": alg, "hbm_gbps": bw(alg, t_cold["median"]),
            "frac": bw(alg, t_cold["median"]) / PEAK_GBPS,
            "frac_warm": bw(alg, t_warm["median"]) / PEAK_GBPS,
            "algorithmic_bytes_stored_author": alg_stored,
            "frac_stored_author": bw(alg_stored, t_cold["median"]) / PEAK_GBPS}


def calibration_copy(torch, dev):
    """Four plain 256 MiB device-to-device copies: known bytes for scaling traffic counters."""
    src = torch.empty(1 << 28, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def kernel_hash():
    return hashlib.sha256(KERNEL_SRC.read_bytes()).hexdigest()[:16]


def load_traffic():
    """HBM bytes per launch from committed rocprofv3 counter runs, if they match this kernel."""
    if not TRAFFIC.exists():
        return None
    t = json.loads(TRAFFIC.read_text())
    return t.get("bytes_per_launch") if t.get("kernel_sha") == kernel_hash() else None


# ---------------------------------------------------------------------------------------------
# Per-workload joins


class JoinCase:
    """One join launch of a workload shape: its inputs on the device, output buffers and the
    algorithmic bytes (8-byte author id, and the store's own author width)."""

    def __init__(self, torch, P, st, store, reqs, wd, we, n_lookups, single, dev,
                 authors=False):
        import workload as W
        self.P, self.store, self.n_lookups, self.single = P, store, n_lookups, single
        self.reqs = reqs
        self.b = W.pack(reqs)
        # With `authors`, every launch passes each candidate's author id (Alg. 1's input form,
        # cc_join_batched_authors), gathered once here, outside the timed launches.
        self.authors = st.author_id[self.b.cand_idx].contiguous() if authors else None
        self.n = self.b.cand_idx.numel()
        self.out = torch.empty(self.n, wd + n_lookups * we, dtype=torch.uint8, device=dev)
        self.hit = torch.empty(self.n, n_lookups, dtype=torch.int8, device=dev)
        self.alg = algorithmic_bytes(torch, st, self.b, wd, we, n_lookups, 8)
        self.alg_stored = algorithmic_bytes(torch, st, self.b, wd, we, n_lookups,
                                            P.cc_store_layout(store)[0])

    def __call__(self, key_offsets=None):
        b, P = self.b, self.P
        if self.single:
            P.cc_join(self.store, b.cand_idx, b.keys, b.edge_rows, self.out, self.hit)
        else:
            P.cc_join_batched(self.store, b.cand_offsets, b.cand_idx,
                              b.key_offsets if key_offsets is None else key_offsets, b.keys,
                              b.edge_rows, self.out, self.hit,
                              extra_keys=[b.actor] if self.n_lookups == 2 else None,
                              author_ids=self.authors)

    def entry(self, torch, flush, iters, floor=False):
        t_cold = time_launches(torch, self, max(10, iters // 2), flush=flush)
        t_warm = time_launches(torch, self, iters)
        e = {"entry": "cc_join" if self.single else
             ("cc_join_batched_authors" if self.authors is not None else "cc_join_batched"),
             "viewers": self.b.n_viewers, "candidates": self.n, "keys": self.b.keys.numel(),
             "lookups": self.n_lookups}
        e.update(rates(self.n, self.alg, self.alg_stored, t_cold, t_warm))
        if floor and not self.single:
            # The same launch with every key list empty: no search and no edge rows, only the
            # positions, author ids, doc rows and output rows. Its time bounds what any search
            # could reach on this launch; `frac_at_floor` is the launch's algorithmic bytes
            # over that time.
            z = torch.zeros_like(self.b.key_offsets)
            f_cold = time_launches(torch, lambda: self(z), max(10, iters // 2), flush=flush)
            f_warm = time_launches(torch, lambda: self(z), iters)
            e["no_keys_floor"] = {
                "ms_median": f_cold["median"], "ms_median_warm": f_warm["median"],
                "frac_at_floor": self.alg / (f_cold["median"] / 1e3) / 1e9 / PEAK_GBPS}
        return e


def sort_entry(torch, P, b, we, dev, tag, n_authors):
    """Alg. 1 Step 1 on a batch's records, shuffled within each viewer: the sort that precedes
    the join when affinity records arrive unsorted. The keys are author ids below n_authors, a
    bound the caller knows, passed as the span bound key_bits."""
    ko = b.key_offsets
    nk = b.keys.numel()
    perm = torch.argsort(torch.rand(nk, device=dev) + 2.0 * torch.repeat_interleave(
        torch.arange(ko.numel() - 1, device=dev), ko[1:] - ko[:-1]))
    k_in, r_in = b.keys[perm].contiguous(), b.edge_rows[perm].contiguous()
    k_out, r_out = torch.empty_like(k_in), torch.empty_like(r_in)
    ws = torch.empty(P.cc_sort_workspace_bytes(nk, ko.numel() - 1), dtype=torch.uint8, device=dev)
    mk = int((ko[1:] - ko[:-1]).max())
    kb = max(1, (n_authors - 1).bit_length())
    t = time_launches(torch, lambda: P.cc_sort_affinity(ko, k_in, r_in, k_out, r_out, ws,
                                                        max_keys=mk, key_bits=kb), 30)
    alg = nk * (16 + 2 * we)
    return {"entry": "cc_sort_affinity_method", "workload": tag, "viewers": ko.numel() - 1,
            "method": "radix" if nk >= P.SORT_RADIX_MIN_RECORDS else "merge", "key_bits": kb,
            "records": nk, "row_bytes": we, "ms_median": t["median"], "ms_mean": t["mean"],
            "records_per_s": nk / (t["median"] / 1e3), "algorithmic_bytes": alg,
            "hbm_gbps": alg / (t["median"] / 1e3) / 1e9,
            "frac": alg / (t["median"] / 1e3) / 1e9 / PEAK_GBPS}


def merge_path_probe(torch, P, st, b, dev):
    """The sort step of the merge-path alternative to the fence search (sort each viewer's
    candidates by author id, merge with the key list, write rows back in candidate order): the
    records are (author id of candidate j, j) per viewer, moved with a 16-byte row. Only the
    sort is timed: it is a lower bound on that alternative's cost."""
    keys = st.author_id[b.cand_idx].contiguous()
    n = keys.numel()
    rows = torch.zeros(n, 2, dtype=torch.int64, device=dev)
    rows[:, 0] = torch.arange(n, device=dev)
    co = b.cand_offsets
    k_out, r_out = torch.empty_like(keys), torch.empty_like(rows)
    ws = torch.empty(P.cc_sort_workspace_bytes(n, co.numel() - 1), dtype=torch.uint8, device=dev)
    mk = int((co[1:] - co[:-1]).max())
    kb = max(1, (st.spec.n_authors - 1).bit_length())
    t = time_launches(torch, lambda: P.cc_sort_affinity(co, keys, rows, k_out, r_out, ws,
                                                        max_keys=mk, key_bits=kb), 30)
    return {"entry": "cc_sort_affinity_method", "what": "candidates sorted by author id, per viewer",
            "records": n, "row_bytes": 16, "ms_median": t["median"], "ms_mean": t["mean"]}


def reference_copy(torch, dev, flush):
    """A reference point on this GPU: a plain 1 GiB device copy with PyTorch's own kernel
    (streaming reads and writes, the best access pattern there is)."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    tc = time_launches(torch, lambda: dst.copy_(src), 20, flush=flush)
    tw = time_launches(torch, lambda: dst.copy_(src), 20)
    nbytes = 2 * (1 << 30)
    del src, dst
    torch.cuda.empty_cache()
    res = {"reference-copy": {"entry": "torch copy_ (PyTorch's own kernel)", "bytes": nbytes,
                              "ms_median": tc["median"], "ms_median_warm": tw["median"],
                              "gbps": nbytes / (tc["median"] / 1e3) / 1e9,
                              "gbps_warm": nbytes / (tw["median"] / 1e3) / 1e9}}
    # Random 8-byte writes, as an ingestion batch's map update makes them: 25M values into a
    # 6.4 GB table at random distinct places, with PyTorch's own scatter kernel.
    n, m = 25_000_000, 800_000_000
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    table = torch.zeros(m, dtype=torch.int64, device=dev)
    idx = torch.randperm(m, generator=g, device=dev)[:n].contiguous()
    val = torch.arange(n, dtype=torch.int64, device=dev)
    tw = time_launches(torch, lambda: table.index_copy_(0, idx, val), 10, flush=flush)
    res["reference-random-writes"] = {
        "entry": "torch index_copy_ (PyTorch's own kernel)", "writes": n, "bytes_each": 8,
        "table_bytes": m * 8, "ms_median": tw["median"],
        "writes_per_s": n / (tw["median"] / 1e3)}
    del table, idx, val
    torch.cuda.empty_cache()
    return res


def workload_entries(torch, P, W, dev, seed, flush, only=None, sorts=True, sorts_only=False,
                     extra=False, cpu=None, floors=True):
    """Full-size entries of every workload shape (or those in `only`). With `cpu`, also collect
    the CPU oracle tasks of each shape into cpu[shape] (host copies of the inputs). With
    `floors`, workloads 3, 4 x64 and 5 also time their launch with empty key lists."""
    want = lambda k: only is None or k in only
    res = {}

    def oracle_tasks(author, rows, reqs, n_lookups):
        import oracle
        lib = oracle.load()

        def task(q):
            def run():
                ex = [q.actor] if n_lookups == 2 else None
                oracle.join_single(author, rows, q.cand_idx, q.keys, q.edge_rows,
                                   n_lookups=n_lookups, extra_keys=ex, lib=lib)
                return q.cand_idx.numel()
            return run
        return [task(W.Request(q.keys.cpu(), q.edge_rows.cpu(), q.cand_idx.cpu(),
                               None if q.actor is None else q.actor.cpu())) for q in reqs]

    # Workload 1: its own 1M-document store.
    if want("1"):
        s, r = W.SHAPES[1]
        st = W.make_store(s, seed, device=dev)
        store = P.cc_store_create(st.author_id, st.doc_rows)
        reqs = W.make_requests(st, r, seed)
        c = JoinCase(torch, P, st, store, reqs, 64, 32, 1, True, dev)
        if not sorts_only:
            res["1"] = c.entry(torch, flush, 200)
        if cpu is not None:
            cpu["1"] = oracle_tasks(st.author_id.cpu(), st.doc_rows.cpu(), reqs, 1)
        P.cc_store_destroy(store)
        del st, c
        torch.cuda.empty_cache()
    # Workloads 2-4 share the 10M-document store.
    if any(want(k) for k in ("2", "2x8", "3", "4", "4x64")):
        s, r2 = W.SHAPES[2]
        st = W.make_store(s, seed, device=dev)
        store = P.cc_store_create(st.author_id, st.doc_rows)
        host = (st.author_id.cpu(), st.doc_rows.cpu()) if cpu is not None else None
        _, r3 = W.SHAPES[3]
        _, r4 = W.SHAPES[4]
        cases = []
        if want("2"):
            cases.append(("2", W.make_requests(st, r2, seed), 1, True, 200))
        if want("2x8"):
            cases.append(("2x8", W.make_requests(st, r2, seed, n_viewers=8), 1, False, 100))
        if want("3"):
            cases.append(("3", W.make_requests(st, r3, seed), 1, False, 40))
        if want("4"):
            cases.append(("4", W.make_requests(st, r4, seed), 2, False, 200))
        if want("4x64"):
            cases.append(("4x64", W.make_requests(st, r4, seed, n_viewers=64), 2, False, 20))
        for tag, reqs, L, single, iters in cases:
            c = JoinCase(torch, P, st, store, reqs, 128, 64, L, single, dev)
            if tag in ("3", "4x64") and want(tag + "-authors") and not sorts_only:
                # the same launch with the candidates' author ids passed by the caller
                ca = JoinCase(torch, P, st, store, reqs, 128, 64, L, single, dev, authors=True)
                res[tag + "-authors"] = ca.entry(torch, flush, iters)
                del ca
            if not sorts_only:
                res[tag] = c.entry(torch, flush, iters, floor=floors and tag in ("3", "4x64"))
            if cpu is not None and tag in ("2", "3", "4"):
                src = reqs if tag != "2" else W.make_requests(st, r2, seed, n_viewers=16)
                cpu[tag] = oracle_tasks(host[0], host[1], src if tag != "4" else reqs, L)
            if tag == "3" and extra and not sorts_only:
                res["3-padded"] = padded_entry(torch, P, c, r3.n_cand, 128, 64, dev)
            if sorts and tag in ("2x8", "3") and want(tag):
                bs = c.b if tag == "3" else W.pack(W.make_requests(st, r2, seed, n_viewers=64))
                res[("2" if tag == "2x8" else "3") + "-sort"] = sort_entry(
                    torch, P, bs, 64, dev, tag, st.spec.n_authors)
            del c
            torch.cuda.empty_cache()
        if cpu is not None and "4" in cpu and want("4x64"):
            cpu["4x64"] = cpu["4"]
        P.cc_store_destroy(store)
        del st, host, cases
        torch.cuda.empty_cache()
    # Workload 5: the 200M-document store (27 GB), generated on the device.
    if want("5"):
        s, r = W.SHAPES[5]
        st = W.make_store(s, seed, device=dev)
        reqs = W.make_requests(st, r, seed)
        st._by_author = None
        store = P.cc_store_create(st.author_id, st.doc_rows)
        c = JoinCase(torch, P, st, store, reqs, 128, 128, 1, False, dev)
        ca = JoinCase(torch, P, st, store, reqs, 128, 128, 1, False, dev, authors=True) \
            if want("5-authors") else None
        if cpu is not None:
            # The oracle's store: only the documents the candidates name (the result is the same
            # as against the whole store; the 27 GB store never reaches the host).
            uniq, inv = torch.unique(c.b.cand_idx, return_inverse=True)
            author, rows = st.author_id[uniq].cpu(), st.doc_rows[uniq].cpu()
            co = c.b.cand_offsets.tolist()
            compact = [W.Request(q.keys, q.edge_rows, inv[co[v]:co[v + 1]], None)
                       for v, q in enumerate(reqs)]
            cpu["5"] = oracle_tasks(author, rows, compact, 1)
        if extra and not sorts_only:
            res["5-merge-path-sort"] = merge_path_probe(torch, P, st, c.b, dev)
        del st
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        if not sorts_only:
            res["5"] = c.entry(torch, flush, 40, floor=floors)
            if ca is not None:
                res["5-authors"] = ca.entry(torch, flush, 40)
        if sorts:
            res["5-sort"] = sort_entry(torch, P, c.b, 128, dev, "5", s.n_authors)
        P.cc_store_destroy(store)
        del c, ca
        torch.cuda.empty_cache()
    return res


def padded_entry(torch, P, c, n_max, wd, we, dev):
    """The same requests written into the padded [B, n_max] layout of the paper's batching (pad
    rows and the valid mask are extra output bytes)."""
    b = c.b
    slots = b.n_viewers * n_max
    outp = torch.empty(b.n_viewers, n_max, wd + we, dtype=torch.uint8, device=dev)
    hitp = torch.empty(b.n_viewers, n_max, 1, dtype=torch.int8, device=dev)
    valid = torch.empty(b.n_viewers, n_max, dtype=torch.int8, device=dev)
    t = time_launches(torch, lambda: P.cc_join_batched_padded(
        c.store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys, b.edge_rows, n_max, outp,
        hitp, valid), 30)
    alg = c.alg + (slots - c.n) * (wd + we + 1) + slots
    return {"entry": "cc_join_batched_padded", "viewers": b.n_viewers, "candidates": c.n,
            "n_max": n_max, "ms_median": t["median"], "ms_mean": t["mean"],
            "candidates_per_s": c.n / (t["median"] / 1e3), "algorithmic_bytes": alg,
            "hbm_gbps": alg / (t["median"] / 1e3) / 1e9,
            "frac": alg / (t["median"] / 1e3) / 1e9 / PEAK_GBPS}


# ---------------------------------------------------------------------------------------------
# Id map and ingestion (--all-configs)


def index_workloads(torch, P, W, dev, seed):
    """The document-id map (§6.3.1, Eq. 6) and ingestion (§6.2) on the one-shard index: build it
    by ingestion, resolve b x tens-of-thousands ids, and apply ingestion batches."""
    spec = W.INDEX_SHAPE
    n = spec.n_index
    rb = spec.row_cols * 2
    n_batches = 20
    res = {}
    store = P.cc_store_create_indexed(n + n_batches * spec.upsert_batch, rb)
    step = 25_000_000
    ws = torch.empty(P.cc_upsert_workspace_bytes(step), dtype=torch.uint8, device=dev)
    t_build = 0.0
    for first in range(0, n, step):
        ids, authors, rows = W.index_records(spec, torch.arange(first, first + step, device=dev),
                                             seed, 100, dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.cc_store_upsert(store, ids, authors, rows, ws)
        t_build += time.perf_counter() - t0
        del ids, authors, rows
    del ws
    res["index-build"] = {"entry": "cc_store_upsert", "documents": n, "batch": step,
                          "seconds": t_build, "records_per_s": n / t_build}
    # Eq. 6: b requests x ids_per_request ids, 2% absent
    q = W.resolve_queries(spec, n, seed, dev)
    pos = torch.empty_like(q)
    t = time_launches(torch, lambda: P.cc_resolve_ids(store, q, pos), 200)
    m = q.numel()
    alg = m * (8 + 8 + 64)            # id in, position out, one 64-byte probe group
    res["resolve"] = {"entry": "cc_resolve_ids", "index": n, "ids": m, "requests": spec.batch,
                      "ms_median": t["median"], "ms_mean": t["mean"],
                      "ids_per_s": m / (t["median"] / 1e3), "algorithmic_bytes": alg,
                      "hbm_gbps": alg / (t["median"] / 1e3) / 1e9,
                      "frac": alg / (t["median"] / 1e3) / 1e9 / PEAK_GBPS}
    res.update(request_latency(torch, P, W, dev, seed, store, spec))
    # §6.2 ingestion: bootstrap-size batches, then steady-state batches (a third of the size)
    next_item = n
    for tag, size, count in (("upsert", spec.upsert_batch, 10),
                             ("upsert-steady", spec.upsert_batch // 3, 10)):
        wsb = torch.empty(P.cc_upsert_workspace_bytes(size), dtype=torch.uint8, device=dev)
        times, fresh = [], 0
        for k in range(count):
            n_stored = P.cc_store_info(store)[0]
            ids, authors, rows, n_new = W.upsert_batch(spec, n_stored, next_item, seed,
                                                       200 + 2 * k + (0 if tag == "upsert" else 50),
                                                       dev, n=size)
            next_item += n_new
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            got = P.cc_store_upsert(store, ids, authors, rows, wsb)
            times.append(time.perf_counter() - t0)
            fresh += got[0]
            del ids, authors, rows
        times.sort()
        med = times[len(times) // 2]
        alg = size * (8 + 8 + rb + 16 + 12) + size * (rb + 8)   # read in + map, write rows
        res[tag] = {"entry": "cc_store_upsert", "records": size, "batches": count,
                    "new_ids": fresh, "ms_median": med * 1e3, "records_per_s": size / med,
                    "algorithmic_bytes": alg, "hbm_gbps": alg / med / 1e9,
                    "note": "host wall clock per call, including its one stream synchronisation"}
    P.cc_store_destroy(store)
    torch.cuda.empty_cache()
    return res


def request_latency(torch, P, W, dev, seed, store, spec, calls=400):
    n, k = spec.ids_per_request, 5000
    g = W.gen(dev, seed, 40)
    items = torch.randint(0, spec.n_index + spec.n_index // 50, (n,), generator=g, device=dev)
    q = W.doc_ids(items, seed)
    pos = torch.empty_like(q)
    keys = torch.sort(torch.randperm(spec.n_authors, generator=g, device=dev)[:k]).values
    edge = torch.randn(k, 32, generator=g, device=dev).to(torch.bfloat16)
    out = torch.empty(n, spec.row_cols * 2 + 64, dtype=torch.uint8, device=dev)
    hit = torch.empty(n, 1, dtype=torch.int8, device=dev)

    def request():
        P.cc_resolve_ids(store, q, pos)
        P.cc_join(store, pos, keys, edge, out, hit)

    def percentiles(fn):
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(calls)]
        for a, b in evs:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        ms = sorted(a.elapsed_time(b) for a, b in evs)
        return ms[len(ms) // 2], ms[int(len(ms) * 0.99)]

    eager = percentiles(request)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            request()
    torch.cuda.synchronize()
    replay = percentiles(graph.replay)
    return {"request-eager": {"entry": "cc_resolve_ids + cc_join", "ids": n, "keys": k,
                              "ms_median": eager[0], "p99_ms": eager[1]},
            "request-graph": {"entry": "cc_resolve_ids + cc_join, replayed HIP graph", "ids": n,
                              "keys": k, "ms_median": replay[0], "p99_ms": replay[1]}}


# ---------------------------------------------------------------------------------------------
# CPU baseline


def cpu_threads():
    """(threads this job may use, CPUs in its affinity mask, where the cap came from). The
    job's share of the host is its affinity mask, further capped by OMP_NUM_THREADS when that is
    set (a GPU job's share of a shared host)."""
    avail = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS", "")
    if cap.isdigit() and 0 < int(cap) < avail:
        return int(cap), avail, "OMP_NUM_THREADS"
    return avail, avail, "affinity mask"


def cpu_leg(tasks, threads, seconds):
    """Run the oracle tasks (each returns its candidate count) on `threads` threads, round
    robin, until `seconds` have passed and every thread has run at least one task. Returns
    (candidates/s, requests, seconds)."""
    done = n_req = 0
    t0 = time.perf_counter()
    if threads == 1:
        while True:
            done += tasks[n_req % len(tasks)]()
            n_req += 1
            if time.perf_counter() - t0 >= seconds:
                break
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            i = 0
            while True:
                batch = [tasks[(i + k) % len(tasks)] for k in range(threads)]
                i += threads
                for c in ex.map(lambda f: f(), batch):
                    done += c
                    n_req += 1
                if time.perf_counter() - t0 >= seconds:
                    break
    dt = time.perf_counter() - t0
    return done / dt, n_req, dt


def cpu_baseline(tasks_by_shape, seconds):
    threads, avail, source = cpu_threads()
    per = {}
    total_s = 0.0
    for tag, tasks in tasks_by_shape.items():
        if tag == "4x64":
            continue
        r1, n1, d1 = cpu_leg(tasks, 1, seconds)
        rn, nn, dn = cpu_leg(tasks, threads, seconds)
        total_s += d1 + dn
        per[tag] = {"threads_1": {"candidates_per_s": r1, "requests": n1, "seconds": d1},
                    f"threads_{threads}": {"candidates_per_s": rn, "requests": nn, "seconds": dn}}
    head = per.get("2")
    value = head[f"threads_{threads}"]["candidates_per_s"] if head else None
    return {"value": value, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": (f"lower-bound oracle (C), one request per task, {seconds:.1f} s per leg; "
                       f"value = workload 2's production-shaped requests (50,000 candidates, "
                       f"16 distinct) on {threads} threads; per_workload has 1 and {threads} "
                       f"threads for workloads 1-5 (workload 5 on the candidates' captured store "
                       f"rows); host CPU: {cpu_model()}"),
            "threads": threads, "threads_source": source, "host_cpus_in_affinity": avail,
            "host_cpu_count": os.cpu_count(), "cpu_model": cpu_model(),
            "value_1_thread": head["threads_1"]["candidates_per_s"] if head else None,
            "per_workload": per, "seconds_total": total_s}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------------------------


def headline(torch, P, W, dev, args, flush):
    """The headline step: timed cold (flush before each step), then warm (back to back)."""
    s, r = W.SHAPES[2]
    st = W.make_store(s, args.seed, device=dev)
    store = P.cc_store_create(st.author_id, st.doc_rows)
    batches = []
    for i in range(N_BATCHES):
        reqs = W.make_requests(st, r, args.seed, first_viewer=i * REQS_PER_STEP,
                               n_viewers=REQS_PER_STEP)
        batches.append((reqs, W.pack(reqs)))
    wd = st.doc_rows.shape[1] * st.doc_rows.element_size()
    we = r.edge_cols * 2
    total = batches[0][1].cand_idx.numel()
    out = torch.empty(total, wd + we, dtype=torch.uint8, device=dev)
    hit = torch.empty(total, 1, dtype=torch.int8, device=dev)
    alg8 = [algorithmic_bytes(torch, st, b, wd, we, 1, 8) for _, b in batches]
    alg_st = [algorithmic_bytes(torch, st, b, wd, we, 1, P.cc_store_layout(store)[0])
              for _, b in batches]
    torch.cuda.synchronize()

    def step(i):
        b = batches[i % N_BATCHES][1]
        P.cc_join_batched(store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys, b.edge_rows,
                          out, hit)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # Timed region: K cold steps, bracketed by device synchronisations.
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i, (a, b) in enumerate(evs):
        flush()
        a.record()
        step(i)
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    cold = [a.elapsed_time(b) for a, b in evs]
    ms_step = sum(cold) / len(cold)
    cold_sorted = sorted(cold)
    alg8_mean = sum(alg8[i % N_BATCHES] for i in range(args.steps)) / args.steps
    alg_st_mean = sum(alg_st[i % N_BATCHES] for i in range(args.steps)) / args.steps
    # Warm: the same K steps back to back.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms_warm = e0.elapsed_time(e1) / args.steps
    # Reference: the same launches with every key list empty (no search, no edge rows: the
    # candidate positions, author ids, doc rows and output rows only).
    nk = torch.zeros(REQS_PER_STEP + 1, dtype=torch.int64, device=dev)
    no_keys = time_launches(torch, lambda: P.cc_join_batched(
        store, batches[0][1].cand_offsets, batches[0][1].cand_idx, nk, batches[0][1].keys[:0],
        batches[0][1].edge_rows[:0], out, hit), 20, flush=flush)
    # The same steps with each candidate's author id passed by the caller (Alg. 1's input
    # form, cc_join_batched_authors): no read of the store's author column. The ids are
    # gathered once, outside the timed launches.
    authors = [st.author_id[b.cand_idx].contiguous() for _, b in batches]
    it = [0]

    def step_authors():
        k = it[0] % N_BATCHES
        it[0] += 1
        b = batches[k][1]
        P.cc_join_batched(store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys, b.edge_rows,
                          out, hit, author_ids=authors[k])

    with_authors = time_launches(torch, step_authors, 40, flush=flush)
    with_authors_warm = time_launches(torch, step_authors, 40)
    del authors
    res = {"no_keys_ms": no_keys["median"], "store": store, "st": st, "batches": batches,
           "authors_ms": with_authors["median"], "authors_ms_warm": with_authors_warm["median"],
           "wd": wd, "we": we, "total": total,
           "ms_step": ms_step, "ms_median": cold_sorted[len(cold) // 2],
           "ms_p99": cold_sorted[min(len(cold) - 1, int(0.99 * len(cold)))],
           "ms_warm": ms_warm, "wall": wall, "alg8": alg8_mean, "alg_stored": alg_st_mean}
    return res


def latency(torch, P, W, dev, args, h):
    """Per-request latency: one request at a time on an idle stream, cycling through 64
    distinct requests. Each call is timed twice: HIP events around it on the stream, and host
    wall time from the call until the stream has finished it."""
    store, st, batches, wd, we = h["store"], h["st"], h["batches"], h["wd"], h["we"]

    def timed_calls(calls, n):
        ev, wall = [], []
        for i in range(n):
            call = calls[i % len(calls)]
            torch.cuda.synchronize()
            a, bb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            a.record()
            call()
            bb.record()
            bb.synchronize()
            wall.append((time.perf_counter() - t0) * 1e3)
            ev.append(a.elapsed_time(bb))
        ev.sort()
        wall.sort()
        pick = lambda xs, p: xs[min(len(xs) - 1, int(p * len(xs)))]
        return {"p50_ms": pick(ev, 0.50), "p99_ms": pick(ev, 0.99),
                "wall_p50_ms": pick(wall, 0.50), "wall_p99_ms": pick(wall, 0.99), "calls": n}

    def single(q, o, hh):
        return lambda: P.cc_join(store, q.cand_idx, q.keys, q.edge_rows, o, hh)
    singles = [single(q, torch.empty(q.cand_idx.numel(), wd + we, dtype=torch.uint8, device=dev),
                      torch.empty(q.cand_idx.numel(), 1, dtype=torch.int8, device=dev))
               for q in batches[0][0]]
    timed_calls(singles, 32)                            # warm-up
    lat = timed_calls(singles, args.latency_calls)
    lat["candidates_per_request"] = batches[0][0][0].cand_idx.numel()
    # PreparedJoin: buffers checked once, then only counts per call (a serving loop that
    # reuses its buffers).
    prepared = [P.PreparedJoin(store, q.cand_idx, q.keys, q.edge_rows,
                               torch.empty(q.cand_idx.numel(), wd + we, dtype=torch.uint8,
                                           device=dev),
                               torch.empty(q.cand_idx.numel(), 1, dtype=torch.int8, device=dev))
                for q in batches[0][0]]
    timed_calls(prepared, 32)
    lat["prepared"] = timed_calls(prepared, args.latency_calls)
    del prepared
    # The second-degree double join (100,000 candidates, 20,000 keys, two lookups), one request
    # per launch on the same store.
    _, r4 = W.SHAPES[4]
    dj, dj_args = [], []
    for q in W.make_requests(st, r4, args.seed, n_viewers=16):
        b1 = W.pack([q])
        o = torch.empty(q.cand_idx.numel(), wd + 2 * we, dtype=torch.uint8, device=dev)
        hh = torch.empty(q.cand_idx.numel(), 2, dtype=torch.int8, device=dev)
        dj_args.append((b1, o, hh))
        dj.append((lambda b1=b1, o=o, hh=hh: P.cc_join_batched(
            store, b1.cand_offsets, b1.cand_idx, b1.key_offsets, b1.keys, b1.edge_rows, o,
            hh, extra_keys=[b1.actor])))
    timed_calls(dj, 16)
    lat["double_join"] = timed_calls(dj, min(args.latency_calls, 512))
    lat["double_join"]["candidates_per_request"] = r4.n_cand
    djp = [P.PreparedJoinBatched(store, b1.cand_offsets, b1.cand_idx, b1.key_offsets, b1.keys,
                                 b1.edge_rows, o, hh, extra_keys=[b1.actor])
           for b1, o, hh in dj_args]
    timed_calls(djp, 16)
    lat["double_join"]["prepared"] = timed_calls(djp, min(args.latency_calls, 512))
    return lat


def main(argv=None):
    args = parse(argv)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the join runs on a single MI355X and the library "
              "has no multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_22441_amd as P
    from paper_2609_22441_amd import binding
    import workload as W

    if not binding.LIB_PATH.exists():
        import __graft_entry__
        __graft_entry__.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    flush = Flush(torch, dev)
    if args.only_index:
        res = index_workloads(torch, P, W, dev, args.seed)
        if args.calibration_copy:
            calibration_copy(torch, dev)
        print(json.dumps({"metric": METRIC, "only_index": True, "configs": res}), flush=True)
        return
    if args.only_workloads or args.only_sorts:
        ids = [x.strip() for x in (args.only_workloads or args.only_sorts).split(",")]
        res = workload_entries(torch, P, W, dev, args.seed, flush, only=set(ids),
                               sorts=bool(args.only_sorts), sorts_only=bool(args.only_sorts),
                               floors=False)
        if args.calibration_copy:
            calibration_copy(torch, dev)
        key = "only_workloads" if args.only_workloads else "only_sorts"
        print(json.dumps({"metric": METRIC, key: ids, "configs": res}), flush=True)
        return

    h = headline(torch, P, W, dev, args, flush)
    lat = None
    if args.latency_calls and not args.only_headline:
        lat = latency(torch, P, W, dev, args, h)
    if args.calibration_copy:
        calibration_copy(torch, dev)
    P.cc_store_destroy(h["store"])
    total, ms_step = h["total"], h["ms_step"]
    achieved = h["alg8"] / (ms_step / 1e3) / 1e9
    achieved_stored = h["alg_stored"] / (ms_step / 1e3) / 1e9
    warm_gbps = h["alg8"] / (h["ms_warm"] / 1e3) / 1e9
    del h["st"], h["batches"]
    torch.cuda.empty_cache()

    configs, cpu = None, None
    if not args.no_configs and not args.only_headline:
        tasks = {} if not args.no_cpu_baseline else None
        configs = workload_entries(torch, P, W, dev, args.seed, flush, extra=args.all_configs,
                                   cpu=tasks)
        if args.all_configs:
            configs.update(index_workloads(torch, P, W, dev, args.seed))
            configs.update(reference_copy(torch, dev, flush))
        if tasks:
            cpu = cpu_baseline(tasks, args.cpu_seconds)
    line = {
        "metric": METRIC,
        "value": total / (ms_step / 1e3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": "production single-viewer shape x64 per step: 10M-doc store "
                        "(Zipf(1.1) authors, 64 bf16 doc cols), K=5000 keys with 32 bf16 edge "
                        "cols, N=50000 candidates (70% in-network); one cc_join_batched launch "
                        "of 64 requests; cold caches (1 GiB read before each step)",
            "requests_per_step": REQS_PER_STEP,
            "candidates_per_step": total,
            "payload": "bf16 rows copied bit-exact",
            "distinct_batches": N_BATCHES,
        },
        "hbm_gbps": achieved,
        "hbm_frac_of_peak": achieved / PEAK_GBPS,
        "ms_per_step_median": h["ms_median"],
        "ms_per_step_p99": h["ms_p99"],
        "warm": {"ms_per_step": h["ms_warm"], "candidates_per_s": total / (h["ms_warm"] / 1e3),
                 "hbm_gbps": warm_gbps, "frac": warm_gbps / PEAK_GBPS},
        "caller_author_ids": {
            "entry": "cc_join_batched_authors", "ms_median": h["authors_ms"],
            "ms_median_warm": h["authors_ms_warm"],
            "frac": h["alg8"] / (h["authors_ms"] / 1e3) / 1e9 / PEAK_GBPS,
            "frac_warm": h["alg8"] / (h["authors_ms_warm"] / 1e3) / 1e9 / PEAK_GBPS,
            "what": "the same steps with each candidate's author id passed by the caller (the "
                    "input form of Alg. 1), cold and warm medians"},
        "no_keys_reference": {"ms_median": h["no_keys_ms"],
                              "what": "the same launch with every key list empty (cold)"},
        "latency": lat,
        "p99_ms": None if lat is None else lat["p99_ms"],
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_GBPS, "unit": "GB/s",
            "frac": achieved / PEAK_GBPS, "traffic": load_traffic(),
            "kernel": HEADLINE_KERNEL, "algorithmic_bytes_per_launch": h["alg8"],
            "author_id_bytes": 8,
            "algorithmic_bytes_per_launch_stored_author": h["alg_stored"],
            "frac_stored_author": achieved_stored / PEAK_GBPS,
        },
        "cpu_baseline": cpu,
        "wall_s_timed_region": h["wall"],
        "configs": configs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
