"""Benchmark of the edge-feature join on one MI355X (prints one JSON line).

Workload: the production-shaped single-viewer request (10M-document store with Zipf(1.1)
author ids, 64 bf16 document columns; K = 5,000 sorted affinity keys with 32 bf16 columns;
N = 50,000 candidates, 70% in-network). A step joins 64 distinct such requests in one
cc_join_batched launch (3.2M candidates). Steps cycle through 4 distinct batches so that
only the store's hot columns can stay in the caches between steps.

Reported:
  value           joined candidates/s over the K timed steps (inputs resident in HBM)
  p50/p99         per-request latency of single cc_join calls (hip events on the stream);
                  latency.prepared: the same requests through PreparedJoin; latency.double_join:
                  two-lookup requests (plain and PreparedJoinBatched)
  roofline        algorithmic bytes per launch / mean launch time, against 8 TB/s
  cold            the same step with the caches flushed (1 GiB read) before each launch
  cpu_baseline    the CPU oracle on the host cores, on a bounded sample of the same requests
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--latency-calls", type=int, default=1024)
    ap.add_argument("--cold-steps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=2)
    ap.add_argument("--all-configs", action="store_true",
                    help="also time each of the five workload shapes (adds a 'configs' field)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (known bytes) for counter scaling")
    ap.add_argument("--only-sorts", default="",
                    help="time only the record sorts of these workload shapes (2, 3 and/or 5): "
                         "for counter passes on the sort")
    ap.add_argument("--only-index", action="store_true",
                    help="run only the id-map part (index build, resolve, ingestion batches): for "
                         "counter passes on those kernels")
    ap.add_argument("--only-workloads", default="",
                    help="time only the joins of these workload shapes (e.g. 3,5), without the "
                         "benchmark step, the sort or the id map: for per-workload counter passes")
    return ap.parse_args()


def algorithmic_bytes(torch, st, batch, wd, we, n_lookups=1, author_bytes=8):
    """Bytes the method must move for one launch: per candidate its position, author id (as
    wide as the store keeps it: 4 or 8 bytes), doc row, output row, hit bytes and (second lookup)
    its extra key; per viewer its keys and each distinct edge row that some lookup hits."""
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


def time_launches(torch, fn, iters, warm=5):
    """Median and mean per-launch time (ms) of `fn` on the current stream."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(iters)]
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    return ms[len(ms) // 2], sum(ms) / len(ms)


def calibration_copy(torch, dev):
    """Four plain 256 MiB device-to-device copies: known bytes for scaling traffic counters."""
    src = torch.empty(1 << 28, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def all_configs(torch, P, W, dev, seed, only=(1, 2, 3, 4, 5), joins_only=False, sorts_only=False):
    """Per-launch time and algorithmic bandwidth of each workload shape at full size (only the
    join launches of the listed shapes when joins_only; only their record sorts when
    sorts_only)."""
    res = {}
    st10 = None
    for i in (1, 2, 3, 4, 5):
        if i not in only:
            continue
        s, r = W.SHAPES[i]
        if i == 1:
            st = W.make_store(s, seed, device=dev)
        elif i in (2, 3, 4):
            st10 = st10 or W.make_store(s, seed, device=dev)
            st = st10
        else:
            st10 = None
            torch.cuda.empty_cache()
            st = W.make_store(s, seed, device=dev)
        reqs = W.make_requests(st, r, seed)
        b = W.pack(reqs)
        L = 2 if r.actor else 1
        wd = st.doc_rows.shape[1] * st.doc_rows.element_size()
        we = r.edge_cols * b.edge_rows.element_size()
        store = P.cc_store_create(st.author_id, st.doc_rows)
        alg = algorithmic_bytes(torch, st, b, wd, we, L, P.cc_store_layout(store)[0])
        if i == 5:
            st._by_author = None
            del st
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
        n = b.cand_idx.numel()
        out = torch.empty(n, wd + L * we, dtype=torch.uint8, device=dev)
        hit = torch.empty(n, L, dtype=torch.int8, device=dev)
        if r.n_viewers == 1 and L == 1:
            fn = lambda: P.cc_join(store, b.cand_idx, b.keys, b.edge_rows, out, hit)
            entry = "cc_join"
        else:
            ex = [b.actor] if L == 2 else None
            fn = lambda: P.cc_join_batched(store, b.cand_offsets, b.cand_idx, b.key_offsets,
                                           b.keys, b.edge_rows, out, hit, extra_keys=ex)
            entry = "cc_join_batched"
        if not sorts_only:
            med, mean = time_launches(torch, fn, 100 if n < 500_000 else 30)
        if i == 2 and not joins_only and not sorts_only:
            # The paper's serving batch (b = 8 requests per launch, §6.3.1) of this shape.
            b8 = W.pack(W.make_requests(st10, r, seed, n_viewers=8))
            n8 = b8.cand_idx.numel()
            out8 = torch.empty(n8, wd + we, dtype=torch.uint8, device=dev)
            hit8 = torch.empty(n8, 1, dtype=torch.int8, device=dev)
            fn8 = lambda: P.cc_join_batched(store, b8.cand_offsets, b8.cand_idx, b8.key_offsets,
                                            b8.keys, b8.edge_rows, out8, hit8)
            m8, mean8 = time_launches(torch, fn8, 100)
            alg8 = algorithmic_bytes(torch, st10, b8, wd, we, 1, P.cc_store_layout(store)[0])
            res["2-batch8"] = {"entry": "cc_join_batched", "viewers": 8, "candidates": n8,
                               "ms_median": m8, "ms_mean": mean8,
                               "candidates_per_s": n8 / (m8 / 1e3), "algorithmic_bytes": alg8,
                               "hbm_gbps": alg8 / (m8 / 1e3) / 1e9,
                               "hbm_frac_of_peak": alg8 / (m8 / 1e3) / 1e9 / PEAK_GBPS}
            del b8, out8, hit8
        if i == 3 and not joins_only and not sorts_only:
            # The same requests written into the padded [B, n_max] layout of the paper's batching
            # (pad rows and the valid mask are extra output bytes).
            n_max = r.n_cand
            slots = b.n_viewers * n_max
            outp = torch.empty(b.n_viewers, n_max, wd + we, dtype=torch.uint8, device=dev)
            hitp = torch.empty(b.n_viewers, n_max, 1, dtype=torch.int8, device=dev)
            valid = torch.empty(b.n_viewers, n_max, dtype=torch.int8, device=dev)
            fnp = lambda: P.cc_join_batched_padded(store, b.cand_offsets, b.cand_idx,
                                                   b.key_offsets, b.keys, b.edge_rows, n_max,
                                                   outp, hitp, valid)
            pm, pmean = time_launches(torch, fnp, 30)
            algp = alg + (slots - n) * (wd + we + 1) + slots
            res["3-padded"] = {"entry": "cc_join_batched_padded", "viewers": r.n_viewers,
                               "candidates": n, "n_max": n_max, "ms_median": pm, "ms_mean": pmean,
                               "candidates_per_s": n / (pm / 1e3), "algorithmic_bytes": algp,
                               "hbm_gbps": algp / (pm / 1e3) / 1e9,
                               "hbm_frac_of_peak": algp / (pm / 1e3) / 1e9 / PEAK_GBPS}
            del outp, hitp, valid
        if i in (2, 3, 5) and not joins_only:
            # Alg. 1 Step 1 on the same records (shuffled within each viewer): the sort that
            # precedes the join when affinity records arrive unsorted.
            bs = b if i != 2 else W.pack(W.make_requests(st10, r, seed, n_viewers=64))
            ko = bs.key_offsets
            nk = bs.keys.numel()
            perm = torch.argsort(torch.rand(nk, device=dev) + 2.0 * torch.repeat_interleave(
                torch.arange(ko.numel() - 1, device=dev), ko[1:] - ko[:-1]))
            k_in, r_in = bs.keys[perm].contiguous(), bs.edge_rows[perm].contiguous()
            k_out, r_out = torch.empty_like(k_in), torch.empty_like(r_in)
            ws = torch.empty(P.cc_sort_workspace_bytes(nk, ko.numel() - 1), dtype=torch.uint8,
                             device=dev)
            mk = int((ko[1:] - ko[:-1]).max())
            fns = lambda: P.cc_sort_affinity(ko, k_in, r_in, k_out, r_out, ws, max_keys=mk)
            sm, smean = time_launches(torch, fns, 30)
            alg_s = nk * (16 + 2 * we)
            res[f"{i}-sort"] = {"entry": "cc_sort_affinity", "viewers": ko.numel() - 1,
                                "records": nk, "row_bytes": we, "ms_median": sm,
                                "ms_mean": smean, "records_per_s": nk / (sm / 1e3),
                                "algorithmic_bytes": alg_s, "hbm_gbps": alg_s / (sm / 1e3) / 1e9,
                                "hbm_frac_of_peak": alg_s / (sm / 1e3) / 1e9 / PEAK_GBPS}
            del k_in, r_in, k_out, r_out, ws
        P.cc_store_destroy(store)
        if not sorts_only:
            res[str(i)] = {"entry": entry, "viewers": r.n_viewers, "candidates": n,
                           "keys": b.keys.numel(), "lookups": L, "ms_median": med,
                           "ms_mean": mean, "candidates_per_s": n / (med / 1e3),
                           "algorithmic_bytes": alg, "hbm_gbps": alg / (med / 1e3) / 1e9,
                           "hbm_frac_of_peak": alg / (med / 1e3) / 1e9 / PEAK_GBPS}
        del out, hit, b, reqs
        torch.cuda.empty_cache()
    if not joins_only and not sorts_only:
        res.update(index_workloads(torch, P, W, dev, seed))
    return res


def index_workloads(torch, P, W, dev, seed):
    """The document-id map (§6.3.1, Eq. 6) and ingestion (§6.2) on the one-shard index: build it
    by ingestion, resolve b x tens-of-thousands ids, and apply ingestion batches."""
    import time
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
    med, mean = time_launches(torch, lambda: P.cc_resolve_ids(store, q, pos), 200)
    m = q.numel()
    alg = m * (8 + 8 + 64)            # id in, position out, one 64-byte probe group
    res["resolve"] = {"entry": "cc_resolve_ids", "index": n, "ids": m, "requests": spec.batch,
                      "ms_median": med, "ms_mean": mean, "ids_per_s": m / (med / 1e3),
                      "algorithmic_bytes": alg, "hbm_gbps": alg / (med / 1e3) / 1e9,
                      "hbm_frac_of_peak": alg / (med / 1e3) / 1e9 / PEAK_GBPS}
    # One request end to end on the same index: 50,000 ids resolved (Eq. 6), then joined (Eq. 1)
    # against one viewer's 5,000 keys; eagerly, and replayed from a captured HIP graph (the two
    # launches without their host-side launch cost).
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


def kernel_hash():
    return hashlib.sha256(KERNEL_SRC.read_bytes()).hexdigest()[:16]


def load_traffic():
    """HBM bytes per launch from committed rocprofv3 counter runs, if they match this kernel."""
    if not TRAFFIC.exists():
        return None
    t = json.loads(TRAFFIC.read_text())
    return t.get("bytes_per_launch") if t.get("kernel_sha") == kernel_hash() else None


def cpu_baseline(st_cpu, reqs_cpu, seconds):
    import oracle
    lib = oracle.load()
    cores = len(os.sched_getaffinity(0))
    threads = max(1, min(cores, 16))
    author, rows = st_cpu
    done = [0]

    def one(q):
        oracle.join_single(author, rows, q.cand_idx, q.keys, q.edge_rows, lib=lib)
        return q.cand_idx.numel()

    t0 = time.perf_counter()
    n_req = 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        while time.perf_counter() - t0 < seconds:
            for c in ex.map(one, reqs_cpu[:threads]):
                done[0] += c
                n_req += 1
    dt = time.perf_counter() - t0
    # The same oracle on one thread, for the per-core rate.
    t1, n1, c1 = time.perf_counter(), 0, 0
    while time.perf_counter() - t1 < min(3.0, seconds):
        c1 += one(reqs_cpu[n1 % len(reqs_cpu)])
        n1 += 1
    dt1 = time.perf_counter() - t1
    return {"value": done[0] / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_req} single-viewer requests of the benchmark workload "
                      f"({reqs_cpu[0].cand_idx.numel()} candidates each), lower-bound oracle, "
                      f"one request per thread, {dt:.1f} s wall; one thread: "
                      f"{c1 / dt1 / 1e6:.1f} M candidates/s ({n1} requests, {dt1:.1f} s); "
                      f"host CPU: {cpu_model()}"}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
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
    if args.only_index:
        res = index_workloads(torch, P, W, dev, args.seed)
        if args.calibration_copy:
            calibration_copy(torch, dev)
        print(json.dumps({"metric": METRIC, "only_index": True, "configs": res}), flush=True)
        return
    if args.only_workloads or args.only_sorts:
        ids = tuple(int(x) for x in (args.only_workloads or args.only_sorts).split(","))
        res = all_configs(torch, P, W, dev, args.seed, only=ids,
                          joins_only=bool(args.only_workloads), sorts_only=bool(args.only_sorts))
        if args.calibration_copy:
            calibration_copy(torch, dev)
        key = "only_workloads" if args.only_workloads else "only_sorts"
        print(json.dumps({"metric": METRIC, key: list(ids), "configs": res}), flush=True)
        return
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
    author_bytes = P.cc_store_layout(store)[0]
    alg = [algorithmic_bytes(torch, st, b, wd, we, 1, author_bytes) for _, b in batches]
    torch.cuda.synchronize()

    def step(i):
        b = batches[i % N_BATCHES][1]
        P.cc_join_batched(store, b.cand_offsets, b.cand_idx, b.key_offsets, b.keys, b.edge_rows,
                          out, hit)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / args.steps
    cands_per_s = total * args.steps / (ms_total / 1e3)
    alg_per_launch = sum(alg[i % N_BATCHES] for i in range(args.steps)) / args.steps
    achieved = alg_per_launch / (ms_step / 1e3) / 1e9

    # Cold caches: read 1 GiB before each launch (more than L2 and the 256 MB Infinity Cache
    # hold), then time the launch alone. A read leaves the caches full of clean lines; a write
    # would leave dirty lines whose write-back the launch would then pay for.
    cold = None
    if args.cold_steps:
        flush = torch.ones(1 << 27, dtype=torch.int64, device=dev)
        ts = []
        for i in range(args.cold_steps):
            flush.amax()
            a, bb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            step(i)
            bb.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(bb))
        del flush
        ms_cold = sorted(ts)[len(ts) // 2]
        alg_cold = sum(alg[i % N_BATCHES] for i in range(args.cold_steps)) / args.cold_steps
        cold = {"steps": args.cold_steps, "ms_per_step_median": ms_cold,
                "candidates_per_s": total / (ms_cold / 1e3),
                "hbm_gbps": alg_cold / (ms_cold / 1e3) / 1e9,
                "hbm_frac_of_peak": alg_cold / (ms_cold / 1e3) / 1e9 / PEAK_GBPS}

    # Per-request latency: one request at a time on an idle stream, cycling through 64
    # distinct requests. Each call is timed twice: HIP events around it on the stream, and host
    # wall time from the call until the stream has finished it.
    lat = None
    if args.latency_calls:
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
                    "wall_p50_ms": pick(wall, 0.50), "wall_p99_ms": pick(wall, 0.99),
                    "calls": n}

        def single(q, o, h):
            return lambda: P.cc_join(store, q.cand_idx, q.keys, q.edge_rows, o, h)
        singles = [single(q, torch.empty(q.cand_idx.numel(), wd + we, dtype=torch.uint8,
                                         device=dev),
                          torch.empty(q.cand_idx.numel(), 1, dtype=torch.int8, device=dev))
                   for q in batches[0][0]]
        timed_calls(singles, 32)                            # warm-up
        lat = timed_calls(singles, args.latency_calls)
        lat["candidates_per_request"] = batches[0][0][0].cand_idx.numel()
        # The same requests through PreparedJoin: buffers checked once, then only counts per call
        # (a serving loop that reuses its buffers).
        prepared = [P.PreparedJoin(store, q.cand_idx, q.keys, q.edge_rows,
                                   torch.empty(q.cand_idx.numel(), wd + we, dtype=torch.uint8,
                                               device=dev),
                                   torch.empty(q.cand_idx.numel(), 1, dtype=torch.int8,
                                               device=dev))
                    for q in batches[0][0]]
        timed_calls(prepared, 32)
        lat["prepared"] = timed_calls(prepared, args.latency_calls)
        del prepared
        # The second-degree double join (100,000 candidates, 20,000 keys, two lookups), one
        # request per launch on the same store.
        _, r4 = W.SHAPES[4]
        dj, dj_args = [], []
        for q in W.make_requests(st, r4, args.seed, n_viewers=16):
            b1 = W.pack([q])
            o = torch.empty(q.cand_idx.numel(), wd + 2 * we, dtype=torch.uint8, device=dev)
            h = torch.empty(q.cand_idx.numel(), 2, dtype=torch.int8, device=dev)
            dj_args.append((b1, o, h))
            dj.append((lambda b1=b1, o=o, h=h: P.cc_join_batched(
                store, b1.cand_offsets, b1.cand_idx, b1.key_offsets, b1.keys, b1.edge_rows, o,
                h, extra_keys=[b1.actor])))
        timed_calls(dj, 16)
        lat["double_join"] = timed_calls(dj, min(args.latency_calls, 512))
        lat["double_join"]["candidates_per_request"] = r4.n_cand
        djp = [P.PreparedJoinBatched(store, b1.cand_offsets, b1.cand_idx, b1.key_offsets, b1.keys,
                                     b1.edge_rows, o, h, extra_keys=[b1.actor])
               for b1, o, h in dj_args]
        timed_calls(djp, 16)
        lat["double_join"]["prepared"] = timed_calls(djp, min(args.latency_calls, 512))
        del dj, djp, dj_args

    if args.calibration_copy:
        calibration_copy(torch, dev)

    cpu = None
    if not args.no_cpu_baseline:
        reqs_cpu = [W.Request(q.keys.cpu(), q.edge_rows.cpu(), q.cand_idx.cpu(), None)
                    for q in batches[0][0][:16]]
        cpu = cpu_baseline((st.author_id.cpu(), st.doc_rows.cpu()), reqs_cpu, args.cpu_seconds)

    P.cc_store_destroy(store)
    configs = None
    if args.all_configs:
        del batches, out, hit, st
        torch.cuda.empty_cache()
        configs = all_configs(torch, P, W, dev, args.seed)
    line = {
        "metric": METRIC,
        "value": cands_per_s,
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
                        "of 64 requests",
            "requests_per_step": REQS_PER_STEP,
            "candidates_per_step": total,
            "payload": "bf16 rows copied bit-exact",
            "distinct_batches": N_BATCHES,
        },
        "hbm_gbps": achieved,
        "hbm_frac_of_peak": achieved / PEAK_GBPS,
        "latency": lat,
        "p99_ms": None if lat is None else lat["p99_ms"],
        "cold": cold,
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_GBPS, "unit": "GB/s",
            "frac": achieved / PEAK_GBPS, "traffic": load_traffic(),
            "kernel": "join_kernel<8, 4, 1, true, true>", "algorithmic_bytes_per_launch": alg_per_launch,
        },
        "cpu_baseline": cpu,
        "wall_s_timed_region": wall,
        "configs": configs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
