"""Helpers shared by the GPU parity tests: run the HIP library and the oracle on the same inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2609_22441_amd as P

FILL = 0xCD          # prefill of output buffers, so unwritten bytes are visible


def note(msg: str) -> None:
    """Name the case about to run on the GPU (flushed, so it survives a lost box)."""
    sys.stderr.write(f"[gpu] {msg}\n")
    sys.stderr.flush()


def row_bytes(t) -> int:
    return int(np.prod(t.shape[1:])) * t.element_size()


def gpu_join(store, author_dev, batch, wd, we, n_lookups, default_row=None, stride=None,
             tuning=None, single=False, stream=None):
    """Run the library on device tensors; returns (out uint8 [total, stride], hit int8 [total, L])."""
    dev = batch.cand_idx.device
    total = batch.cand_idx.numel()
    stride = stride or wd + n_lookups * we
    out = torch.full((total, stride), FILL, dtype=torch.uint8, device=dev)
    hit = torch.full((total, n_lookups), -7, dtype=torch.int8, device=dev)
    if single:
        assert n_lookups == 1 and tuning is None
        P.cc_join(store, batch.cand_idx, batch.keys, batch.edge_rows, out, hit,
                  default_row=default_row, stream=stream)
    else:
        P.cc_join_batched(store, batch.cand_offsets, batch.cand_idx, batch.key_offsets,
                          batch.keys, batch.edge_rows, out, hit, default_row=default_row,
                          extra_keys=[batch.actor] if n_lookups == 2 else None, tuning=tuning,
                          stream=stream)
    torch.cuda.synchronize()
    return out.cpu().numpy(), hit.cpu().numpy()


def oracle_join(author_cpu, doc_cpu, batch_cpu, n_lookups, default_row=None, stride=None):
    return oracle.join(author_cpu, doc_cpu, batch_cpu.cand_offsets, batch_cpu.cand_idx,
                       batch_cpu.key_offsets, batch_cpu.keys, batch_cpu.edge_rows,
                       default_row=None if default_row is None else default_row.cpu(),
                       n_lookups=n_lookups,
                       extra_keys=[batch_cpu.actor] if n_lookups == 2 else None,
                       out_stride=stride, fill=FILL)


def assert_same(got, want, what=""):
    go, gh = got
    wo, wh = want[0], want[1]
    assert go.shape == wo.shape, f"{what}: shape {go.shape} vs {wo.shape}"
    if not np.array_equal(go, wo):
        bad = np.argwhere((go != wo).any(axis=1)).ravel()
        raise AssertionError(f"{what}: {bad.size} rows differ, first {bad[:8].tolist()}")
    if not np.array_equal(gh, wh):
        bad = np.argwhere((gh != wh).any(axis=1)).ravel()
        raise AssertionError(f"{what}: {bad.size} hit rows differ, first {bad[:8].tolist()}")
