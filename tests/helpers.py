"""Shared test plumbing: run a workload through the C-ABI, and the oracle's view of it."""
from __future__ import annotations

import numpy as np

from oracle import attention as OA

TOL = {"bf16": 2e-2, "f32": 1e-4}


def query_layout(query):
    return OA.layout(query.prefix.n, [f.n for f in query.frags], query.cross.n)


def query_rows(query) -> np.ndarray:
    """Caller rows of S = prefix | fragments in this query's order | cross."""
    parts = [np.arange(query.prefix.row, query.prefix.row + query.prefix.n)]
    parts += [np.arange(f.row, f.row + f.n) for f in query.frags]
    parts.append(np.arange(query.cross.row, query.cross.row + query.cross.n))
    return np.concatenate(parts).astype(np.int64)


def oracle_rows(wl, query, want_rows=None):
    """Oracle outputs for one query: {caller row: [Hq, d] float64} for the requested caller rows
    (default: every row of the query)."""
    rows = query_rows(query)
    lay = query_layout(query)
    if want_rows is None:
        sel = np.arange(lay.n)
    else:
        want = set(int(r) for r in want_rows)
        sel = np.array([i for i, r in enumerate(rows) if int(r) in want], np.int64)
    if sel.size == 0:
        return {}
    out = OA.attention_rows(wl.q[rows], wl.k[rows], wl.v[rows], lay, sel, wl.rope_theta)
    return {int(rows[i]): out[j] for j, i in enumerate(sel)}


class GpuRun:
    """A pool on cuda:0 holding a workload's activations; runs batches through the library."""

    def __init__(self, wl, num_pages=None, kernel="auto", num_layers=1):
        import torch

        import paper_2511_02749_amd as spanq
        self.torch = torch
        self.wl = wl
        if num_pages is None:
            num_pages = 64 + sum(
                (q.prefix.n + 15) // 16 + sum((f.n + 15) // 16 for f in q.frags) + (q.cross.n + 15) // 16
                for b in wl.batches for q in b)
        self.pool = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                               num_pages=num_pages, dtype=wl.dtype, rope_theta=wl.rope_theta, kernel=kernel,
                               num_layers=num_layers, device=0)
        qa, ka, va = wl.device_arrays()
        conv = (lambda a: torch.from_numpy(a.view(np.int16))) if wl.dtype == "bf16" else torch.from_numpy
        self.q, self.k, self.v = (conv(np.ascontiguousarray(a)).cuda() for a in (qa, ka, va))
        tdt = torch.int16 if wl.dtype == "bf16" else torch.float32
        self.out = torch.zeros(self.q.shape, dtype=tdt, device="cuda")

    def run_batch(self, batch, layer=0, commit=True):
        plan = self.pool.plan(batch)
        plan.prefill(layer, self.q, self.k, self.v, self.out)
        plan.cross(layer, self.q, self.k, self.v, self.out)
        self.torch.cuda.synchronize()
        if commit:
            plan.commit()
        return plan

    def out_rows(self, rows) -> np.ndarray:
        o = self.out[self.torch.as_tensor(np.asarray(rows, np.int64), device="cuda")].cpu().numpy()
        if self.wl.dtype == "bf16":
            return (o.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
        return o

    def close(self):
        self.pool.close()


def max_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(gpu.astype(np.float64) - ref))) if gpu.size else 0.0
