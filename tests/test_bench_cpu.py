"""bench.py on the CPU: its algorithmic-byte count (the numerator of the roofline) against an
independent count, and its refusal of more than one GPU."""
import subprocess
import sys
from pathlib import Path

import torch

import bench
import workload as W

ROOT = Path(__file__).resolve().parent.parent


def independent_bytes(st, b, wd, we, n_lookups, author_bytes):
    """Per candidate: position, author id, doc row read, output row written, hit bytes and the
    extra keys; per viewer: its keys and each distinct edge row some lookup hits."""
    author = st.author_id.tolist()
    co, ko = b.cand_offsets.tolist(), b.key_offsets.tolist()
    cand, keys = b.cand_idx.tolist(), b.keys.tolist()
    actor = b.actor.tolist() if n_lookups == 2 else None
    n = len(cand)
    total = n * (8 + author_bytes + wd + (wd + n_lookups * we) + n_lookups + 8 * (n_lookups - 1))
    total += 8 * len(keys)
    for v in range(len(co) - 1):
        vkeys = set(keys[ko[v]:ko[v + 1]])
        hit = set()
        for j in range(co[v], co[v + 1]):
            looked = [author[cand[j]]] + ([actor[j]] if actor is not None else [])
            hit.update(k for k in looked if k in vkeys)
        total += we * len(hit)
    return total


def test_algorithmic_bytes_match_an_independent_count():
    for i, lookups in ((2, 1), (4, 2)):
        s, r = W.shape(i, store_n_docs=20_000, store_n_authors=50_000, req_k=300,
                       req_n_cand=2_000, req_n_viewers=3)
        st = W.make_store(s, 7)
        b = W.pack(W.make_requests(st, r, 7))
        wd = st.doc_rows.shape[1] * st.doc_rows.element_size()
        we = r.edge_cols * b.edge_rows.element_size()
        for ab in (4, 8):
            got = bench.algorithmic_bytes(torch, st, b, wd, we, lookups, ab)
            assert got == independent_bytes(st, b, wd, we, lookups, ab), (i, ab)


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


def test_cpu_threads_follow_the_job_share(monkeypatch):
    import os
    avail = len(os.sched_getaffinity(0))
    monkeypatch.delenv("OMP_NUM_THREADS", raising=False)
    assert bench.cpu_threads() == (avail, avail, "affinity mask")
    if avail > 1:
        monkeypatch.setenv("OMP_NUM_THREADS", "1")
        assert bench.cpu_threads() == (1, avail, "OMP_NUM_THREADS")
    monkeypatch.setenv("OMP_NUM_THREADS", str(avail + 5))
    assert bench.cpu_threads()[0] == avail


def test_cpu_baseline_reports_both_thread_counts(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "2")
    calls = []

    def task(n):
        def run():
            calls.append(n)
            return n
        return run
    tasks = {"1": [task(10)], "2": [task(50), task(60)], "4": [task(7)], "4x64": [task(7)]}
    res = bench.cpu_baseline(tasks, 0.01)
    threads = res["threads"]
    assert res["cores"] == threads and threads <= 2
    assert set(res["per_workload"]) == {"1", "2", "4"}
    for leg in res["per_workload"].values():
        assert set(leg) == {"threads_1", f"threads_{threads}"}
        assert all(x["candidates_per_s"] > 0 and x["requests"] >= 1 for x in leg.values())
    assert res["value"] == res["per_workload"]["2"][f"threads_{threads}"]["candidates_per_s"]
    assert res["value_1_thread"] == res["per_workload"]["2"]["threads_1"]["candidates_per_s"]
    assert res["host_cpus_in_affinity"] >= threads
