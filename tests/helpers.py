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

    def __init__(self, wl, num_pages=None, kernel="auto", num_layers=1, materialize=False, nan_pool=False):
        import torch

        import paper_2511_02749_amd as spanq
        self.torch = torch
        self.wl = wl
        if num_pages is None:
            num_pages = 64 + sum(
                (q.prefix.n + 15) // 16 + sum((f.n + 15) // 16 for f in q.frags) + (q.cross.n + 15) // 16
                for b in wl.batches for q in b)
        buf = None
        if nan_pool:  # page memory full of NaN bit patterns, as memory reused from other work may be
            elem = 2 if wl.dtype == "bf16" else 4
            n = num_layers * num_pages * 2 * wl.n_kv_heads * 16 * wl.head_dim
            buf = (torch.full((n,), 0x7FC0, dtype=torch.int16, device="cuda") if elem == 2 else
                   torch.full((n,), 0x7FC00000, dtype=torch.int32, device="cuda"))
        self.pool = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                               num_pages=num_pages, dtype=wl.dtype, rope_theta=wl.rope_theta, kernel=kernel,
                               num_layers=num_layers, materialize=materialize, device=0, device_buf=buf)
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


def computed_rows(plan) -> np.ndarray:
    """Caller rows a plan computes: new prefix/fragment rows, then cross rows."""
    pre, cross = plan.rows()
    return np.concatenate([pre, cross])


# Whole-batch checks of bf16 pools (every computed row of the full-size batches):
# max abs error 2e-2 + 2^-8 |oracle| per element, and at most this fraction of
# elements past the plain 2e-2.  The relative term is one unit of bf16's relative
# precision; at |O| of 2 to 5 the bf16 rounding of the cached rotated keys and of the
# rotated query alone moves a few of 1.2e8 outputs past 2e-2 (DESIGN, Z12).
BF16_RTOL = 2.0 ** -8
BF16_OVER_FRAC = 1e-6


def check_rows(run, batch, rows, tol, limit=None, progress=None, rtol=0.0, over_frac=None):
    """Compare GPU output rows with the oracle; each row is evaluated in the first
    query of the batch that contains it.  ``limit`` samples evenly spaced rows.
    Every element must satisfy |gpu - oracle| <= tol + rtol |oracle|; with
    ``over_frac``, at most that fraction of elements may exceed plain ``tol``."""
    rows = np.asarray(rows, np.int64)
    if limit is not None and rows.size > limit:
        rows = rows[np.linspace(0, rows.size - 1, limit).astype(np.int64)]
    remaining = set(int(r) for r in rows)
    worst, where = 0.0, ""
    n_el, n_over, worst_mixed = 0, 0, 0.0
    for qi, q in enumerate(batch):
        mine = [r for r in query_rows(q) if int(r) in remaining]
        if not mine:
            continue
        ref = oracle_rows(run.wl, q, mine)
        got = run.out_rows(mine)
        cross0 = q.cross.row
        for i, r in enumerate(mine):
            e = np.abs(got[i].astype(np.float64) - ref[int(r)])
            n_el += e.size
            n_over += int(np.count_nonzero(e > tol))
            if e.size:
                worst_mixed = max(worst_mixed, float(np.max(e - rtol * np.abs(ref[int(r)]))))
            if e.size and e.max() > worst:
                h, d = np.unravel_index(int(np.argmax(e)), e.shape)
                worst = float(e.max())
                kind = "cross" if cross0 <= int(r) < cross0 + q.cross.n else "prefill"
                where = (f"query {qi} row {int(r)} ({kind}) head {h} dim {d}: gpu {float(got[i][h, d]):.5f} "
                         f"oracle {float(ref[int(r)][h, d]):.5f}")
            remaining.discard(int(r))
        if progress:
            print(f"{progress}: query {qi}: {len(mine)} rows, max abs err so far {worst:.3g}", flush=True)
    assert not remaining
    if over_frac is None and rtol == 0.0:
        assert worst <= tol, f"max abs err {worst} > {tol} at {where}"
    else:
        if progress:
            print(f"{progress}: {n_el} elements, max abs err {worst:.4g} at {where}; {n_over} past {tol}", flush=True)
        assert worst_mixed <= tol, f"|err| - {rtol}|oracle| reaches {worst_mixed} > {tol}; max abs err {worst} at {where}"
        if over_frac is not None:
            assert n_over <= over_frac * n_el, f"{n_over} of {n_el} elements past {tol}"
    return worst


def replay_queries(batch):
    """A batch in the oracle pool replay's form: (prefix, [fragments], cross) token lists."""
    return [(list(map(int, q.prefix.tokens)), [list(map(int, f.tokens)) for f in q.frags],
             list(map(int, q.cross.tokens))) for q in batch]


def assert_tables_match(plan, res, batch):
    """Block tables, hit counts and evictions of a library plan equal the oracle replay's."""
    for qi, q in enumerate(batch):
        qr = res.queries[qi]
        assert plan.block_table(qi, -1) == (qr.prefix.page_ids, qr.prefix.n_hit)
        for c in range(len(q.frags)):
            assert plan.block_table(qi, c) == (qr.frags[c].page_ids, qr.frags[c].n_hit)
        ids, nh = plan.block_table(qi, len(q.frags))
        assert ids == qr.cross.page_ids and nh == 0
    assert plan.evicted() == res.evicted


# ---------------------------------------------------------------- decoder stacks

class _Bf16Layers:
    """Per-layer bf16 bit arrays seen as float32 one layer at a time (the oracle
    converts each to float64 when it uses it)."""

    def __init__(self, arrs):
        self.arrs = arrs

    def __len__(self):
        return len(self.arrs)

    def __getitem__(self, l):
        return (self.arrs[l].astype(np.uint32) << 16).view(np.float32)


def oracle_weights(sw):
    from oracle import stack as OS
    f = lambda a: (a.astype(np.uint32) << 16).view(np.float32)  # noqa: E731
    return OS.Weights(embed=f(sw.embed), attn_norm=_Bf16Layers(sw.attn_norm), w_qkv=_Bf16Layers(sw.w_qkv),
                      w_o=_Bf16Layers(sw.w_o), ffn_norm=_Bf16Layers(sw.ffn_norm), w_gate_up=_Bf16Layers(sw.w_gate_up),
                      w_down=_Bf16Layers(sw.w_down), final_norm=f(sw.final_norm), lm_head=f(sw.lm_head),
                      n_q_heads=sw.n_q_heads, n_kv_heads=sw.n_kv_heads, head_dim=sw.head_dim)


def stack_oracle(swl, query, keep, rows=None, Wt=None):
    """Oracle hidden states of one query: {layer count: {caller row: [hidden]}} for the
    counts in keep, and the float64 logits of its last cross row when the last count
    is the whole stack and the query has a cross segment."""
    from oracle import attention as OA
    from oracle import stack as OS
    Wt = Wt if Wt is not None else oracle_weights(swl.weights)
    toks = OS.query_tokens(query.prefix.tokens, [f.tokens for f in query.frags], query.cross.tokens)
    lay = OA.layout(query.prefix.n, [f.n for f in query.frags], query.cross.n)
    hs = OS.stack_forward(toks, lay, Wt, max(keep), swl.rope_theta, swl.rms_eps, storage="bf16", keep=list(keep))
    qrows = query_rows(query)
    want = set(int(r) for r in (qrows if rows is None else rows))
    out = {L: {int(r): hs[L][i] for i, r in enumerate(qrows) if int(r) in want} for L in keep}
    logits = None
    if max(keep) == swl.weights.n_layers and query.cross.n > 0:
        logits = OS.final_logits(hs[max(keep)][-1], Wt, swl.rms_eps, storage="bf16")
    return out, logits


class StackRun:
    """A pool and a decoder stack on cuda:0 for a stack workload."""

    def __init__(self, swl, num_pages=None, timing=False, kernel="auto"):
        import torch

        import paper_2511_02749_amd as spanq
        self.torch = torch
        self.swl = swl
        sw = swl.weights
        if num_pages is None:
            num_pages = 64 + sum(
                (q.prefix.n + 15) // 16 + sum((f.n + 15) // 16 for f in q.frags) + (q.cross.n + 15) // 16
                for b in swl.batches for q in b)
        self.pool = spanq.Pool(num_q_heads=sw.n_q_heads, num_kv_heads=sw.n_kv_heads, head_dim=sw.head_dim,
                               num_pages=num_pages, dtype="bf16", rope_theta=swl.rope_theta, num_layers=sw.n_layers,
                               timing=timing, kernel=kernel, device=0)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()  # noqa: E731
        self.w = dict(embed=dev(sw.embed), final_norm=dev(sw.final_norm), lm_head=dev(sw.lm_head),
                      attn_norm=[dev(a) for a in sw.attn_norm], w_qkv=[dev(a) for a in sw.w_qkv],
                      w_o=[dev(a) for a in sw.w_o], ffn_norm=[dev(a) for a in sw.ffn_norm],
                      w_gate_up=[dev(a) for a in sw.w_gate_up], w_down=[dev(a) for a in sw.w_down])
        self.model = spanq.Model(self.pool, hidden=sw.hidden, ffn=sw.ffn, vocab=sw.vocab, rms_eps=swl.rms_eps,
                                 **self.w)
        self.n_rows = int(swl.row_tokens.shape[0])
        self.hidden = torch.zeros((self.n_rows, sw.hidden), dtype=torch.int16, device="cuda")

    def run(self, batch, n_layers=None, commit=True, logits=True):
        """Plan a batch and run it through the stack; returns (plan, first tokens,
        logits [queries with cross][vocab] float32 or None)."""
        torch = self.torch
        plan = self.pool.plan(batch)
        n_cross = sum(1 for q in batch if q.cross.n > 0)
        lg = None
        full = n_layers is None or n_layers == self.swl.weights.n_layers
        if logits and full and n_cross:
            lg = torch.zeros((n_cross, self.swl.weights.vocab), dtype=torch.float32, device="cuda")
        toks = self.model.forward(plan, self.swl.row_tokens, n_layers=n_layers, hidden_out=self.hidden,
                                  logits_out=lg, first_tokens=full)
        torch.cuda.synchronize()
        if commit:
            plan.commit()
        return plan, toks, (lg.cpu().numpy() if lg is not None else None)

    def hidden_rows(self, rows) -> np.ndarray:
        h = self.hidden[self.torch.as_tensor(np.asarray(rows, np.int64), device="cuda")].cpu().numpy()
        return (h.view(np.uint16).astype(np.uint32) << 16).view(np.float32)

    def close(self):
        self.model.close()
        self.pool.close()
