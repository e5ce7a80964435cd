#!/usr/bin/env python3
"""Span-prefill attention throughput and cache-hit TTFT on one MI355X.

Workload (default): one Llama-3-8B-shaped attention layer in bf16 (32 query
heads, 8 kv heads, head_dim 128, hidden 4096, random weights N(0, 0.02^2)),
a 256-token shared prefix, a pool of 64 fragments x 512 tokens, 8 queries each
drawing 16 fragments in random order, a 128-token cross segment (question) per
query.  Synthetic, seeded inputs (no dataset, no trained weights).

A timed step is one cold batch through the whole hot path: pool reset, span
planning (hashing, lookup, dedup, allocation), page writes, span-prefill
attention, cross attention with repositioning, KV-split merge and commit.
q/k/v of every row are resident in HBM before timing starts.

Printed JSON (last stdout line):
  value      algorithmic attention TFLOP/s of the cold batch step
             (4 * head_dim * q_heads * allowed (query, key) pairs / step time)
  ttft       single-query time to first token of the attention layer (plan call to
             stream sync after cross attention): cold, warm (all fragments cached, new
             order) and a dense causal run of the same sequence, p50/p99
  roofline   span-prefill attention kernel: algorithmic FLOPs per launch / mean launch
             duration (HIP events on the launch stream) against the bf16 dense MFMA peak
  kv_gather  cross attention with 1/4/16 rows per query over eight distinct
             judge-shaped contexts (335 MB of K/V): GB/s of distinct pages read
             against the 8 TB/s HBM peak
  measured_peaks  what this GPU attains with an MFMA-only loop and a streaming HBM read
             (library probes), with the prefill kernel's and the gathers' rates against them
  cpu_baseline  the float64 oracle on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "span-prefill attention TFLOP/s + cache-hit TTFT (ms), 16×512-tok fragments"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0

# Measured HBM traffic of the span-prefill kernel lives in a profile summary, tagged
# with a digest of the sources that decide it (kernel, tiling, planner); once any of
# them changes the figure is stale and `traffic` is reported as null.
TRAFFIC_FILE = {"c2": "profiles/span_prefill_attention_c2_traffic.md",
                "c3": "profiles/span_prefill_attention_c3_traffic.md"}
TRAFFIC_SOURCES = ["paper_2511_02749_amd/csrc/prefill_mfma.hip", "paper_2511_02749_amd/csrc/mfma_common.h",
                   "paper_2511_02749_amd/csrc/planner.cpp", "paper_2511_02749_amd/csrc/planner.h",
                   "paper_2511_02749_amd/csrc/work.h"]


def sources_digest():
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(config):
    """HBM bytes per launch of the span-prefill kernel from the committed counter
    summary, or None if it is missing or was taken on other sources."""
    path = os.path.join(ROOT, TRAFFIC_FILE[config])
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-json:"):
                rec = json.loads(line.split(":", 1)[1])
                if rec.get("sources") == sources_digest():
                    return rec["traffic_bytes"]
    return None


def copy_calibration(mib, reps=5):
    """A plain streaming copy (y = x * 1, float32) of `mib` MiB, for scaling the HBM
    byte counters: each launch reads and writes exactly mib MiB."""
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read": n * 4, "bytes_written": n * 4, "launches": reps}}),
          flush=True)


def _pct(xs, p):
    import numpy as np
    return float(np.percentile(np.asarray(xs), p)) if xs else None


def _flops(wl, pairs):
    return 4.0 * wl.head_dim * wl.n_q_heads * pairs


def cpu_baseline(wl, query, max_seconds):
    """The oracle on this host's cores over every row of one query (float64), with
    the BLAS and torch thread counts set to the cores this process may use.  Stops
    early, on whole row blocks, if it runs past max_seconds."""
    import numpy as np

    from oracle import attention as OA
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # pragma: no cover
        limiter = None
    try:
        import torch
        torch.set_num_threads(cores)
    except Exception:  # pragma: no cover
        pass
    lay = OA.layout(query.prefix.n, [f.n for f in query.frags], query.cross.n)
    rows = np.concatenate([np.arange(query.prefix.row, query.prefix.row + query.prefix.n)] +
                          [np.arange(f.row, f.row + f.n) for f in query.frags] +
                          [np.arange(query.cross.row, query.cross.row + query.cross.n)])
    q, k, v = wl.q[rows], wl.k[rows], wl.v[rows]
    done, pairs = 0, 0
    t0 = time.perf_counter()
    for b0 in range(0, lay.n, 512):
        sel = np.arange(b0, min(lay.n, b0 + 512))
        OA.attention_rows(q, k, v, lay, sel, wl.rope_theta)
        pairs += int(OA.mask_rows(lay, sel).sum())
        done += sel.size
        if time.perf_counter() - t0 > max_seconds:
            break
    dt = time.perf_counter() - t0
    if limiter is not None:
        limiter.unregister()
    return {"value": _flops(wl, pairs) / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{done} of {lay.n} rows of one C2 query (all rows unless cut at {max_seconds:.0f} s), "
                      f"float64, {dt:.1f} s, {cores} threads"}


def kv_gather(spanq, W, torch, np, reps, rows_list=(1, 4, 16), n_queries=8):
    """Cross attention with few query rows over many cached pages: the KV page-gather
    regime.  Eight independent judge-shaped queries (prompt 2048 + 32 x 256, all
    pages distinct: 8 x 41.9 MB of K/V, more than the 256 MB Infinity Cache) are
    prefilled once; each timed pass then plans all eight (every page a hit) and runs
    only the cross step for Q cross rows per query.  Bytes = every distinct K/V page
    the pass reads, once."""
    hq, hkv, d = 32, 8, 128
    queries, n_rows = W.gather_queries(n_queries=n_queries, cross_len=max(rows_list))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(20251102)
    q, k, v = (torch.randn(n_rows, h, d, generator=gen, device="cuda").to(torch.bfloat16).view(torch.int16)
               for h in (hq, hkv, hkv))
    out = torch.zeros_like(q)
    pages = sum((s.n + 15) // 16 for x in queries for s in [x.prefix, *x.frags, x.cross]) + 64
    pool = spanq.Pool(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=pages, dtype="bf16",
                      rope_theta=1e4, timing=True, device=0)
    stream = torch.cuda.current_stream()
    p = pool.plan(queries, stream)
    p.prefill(0, q, k, v, out)
    p.cross(0, q, k, v, out)
    p.commit()
    p.destroy()
    page_bytes = 2 * hkv * 16 * d * 2
    res = {}
    for nq in rows_list:
        qs = [W.Query(prefix=x.prefix, frags=x.frags, cross=W.Span(tokens=x.cross.tokens[:nq], row=x.cross.row))
              for x in queries]
        times, merged, st = [], [], None
        for r in range(reps + 2):
            p = pool.plan(qs, stream)
            p.cross(0, q, k, v, out)
            p.commit()
            kt = p.kernel_times()
            st = p.stats()
            p.destroy()
            if r >= 2:
                times.append(kt["cross_attention_ms"])
                merged.append(kt["cross_attention_ms"] + kt["combine_ms"])
        assert st["pages_new"] == 0
        nbytes = (st["pages_hit"] + st["pages_cross"]) * page_bytes
        ms = float(np.mean(times))
        ms_merged = float(np.mean(merged))
        gbs = nbytes / (ms * 1e-3) / 1e9
        res[f"q{nq}"] = {"cross_rows_per_query": nq, "bytes": int(nbytes), "ms": ms, "gbs": gbs,
                         "frac": gbs / PEAK_HBM_GBS, "kv_splits": st["kv_splits"],
                         "ms_with_merge": ms_merged, "gbs_with_merge": nbytes / (ms_merged * 1e-3) / 1e9,
                         "frac_with_merge": nbytes / (ms_merged * 1e-3) / 1e9 / PEAK_HBM_GBS}
    pool.close()
    return {"kernel": "cross_attention", "bound": "hbm", "peak_gbs": PEAK_HBM_GBS, "queries": n_queries,
            "kv_per_query_mb": (640 * page_bytes) / 1e6, "by_rows": res}


def reposition_ab(spanq, W, torch, np, reps):
    """Read-time rotation against materialised repositioning (every shifted page copied,
    keys rotated to the final positions, as CIDRA does in place) on warm queries: the
    RAG query with its 16 cached fragments reversed (15 shifted, 480 pages) and the
    judge query with its 32 cached candidates reversed (31 shifted, 496 pages).  Both
    pools plan the same query; a timed pass is plan + cross step (every fragment a hit),
    wall time to stream sync, and kernel times from HIP events on the launch stream.
    The move kernel's algorithmic bytes: each copied page read once and written once."""
    res = {}
    for name, wl in (("c2", W.config_c2()), ("c3", W.config_c3())):
        q0 = wl.batches[0][0]
        rev = W.Query(prefix=q0.prefix, frags=q0.frags[::-1], cross=q0.cross)
        qa, ka, va = wl.device_arrays()
        q, k, v = (torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda() for a in (qa, ka, va))
        out = torch.zeros_like(q)
        pages = 2 * sum((s.n + 15) // 16 for s in [q0.prefix, *q0.frags, q0.cross]) + 64
        page_bytes = 2 * wl.n_kv_heads * 16 * wl.head_dim * 2
        stream = torch.cuda.current_stream()
        entry = {"query": f"prefix {q0.prefix.n} + {len(q0.frags)} x {q0.frags[0].n} (cached, reversed) + "
                          f"cross {q0.cross.n}"}
        for mode in ("read_time_rotation", "materialized"):
            pool = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                              num_pages=pages, dtype=wl.dtype, rope_theta=wl.rope_theta, timing=True,
                              materialize=mode == "materialized", device=0)
            p = pool.plan([q0], stream)
            p.prefill(0, q, k, v, out)
            p.cross(0, q, k, v, out)
            p.commit()
            p.destroy()
            walls, kts, st = [], [], None
            for r in range(reps + 2):
                torch.cuda.synchronize()
                t = time.perf_counter()
                p = pool.plan([rev], stream)
                p.prefill(0, q, k, v, out)
                p.cross(0, q, k, v, out)
                torch.cuda.synchronize()
                dt = (time.perf_counter() - t) * 1e3
                p.commit()
                kt, st = p.kernel_times(), p.stats()
                p.destroy()
                if r >= 2:
                    walls.append(dt)
                    kts.append(kt)
            pool.close()
            assert st["tokens_new"] == 0
            mean = {n: float(np.mean([x[n] for x in kts])) for n in spanq._lib.TIME_FIELDS}
            e = {"warm_ms_p50": _pct(walls, 50),
                 "cross_attention_ms": mean["cross_attention_ms"], "combine_ms": mean["combine_ms"],
                 "cross_gpu_ms": mean["page_write_cross_ms"] + mean["page_move_ms"] + mean["cross_attention_ms"] +
                 mean["combine_ms"]}
            if mode == "materialized":
                ms = mean["page_move_ms"]
                nbytes = 2 * st["pages_moved"] * page_bytes
                gbs = nbytes / (ms * 1e-3) / 1e9
                e["page_move"] = {"kernel": "move_pages", "bound": "hbm", "ms": ms, "pages": st["pages_moved"],
                                  "tokens": st["tokens_moved"], "algorithmic_bytes": nbytes, "gbs": gbs,
                                  "frac": gbs / PEAK_HBM_GBS,
                                  "tokens_per_ms_one_layer": st["tokens_moved"] / ms,
                                  "tokens_per_ms_32_layers": st["tokens_moved"] / ms / 32}
            entry[mode] = e
        entry["materialized_over_read_time"] = {
            "cross_gpu": entry["materialized"]["cross_gpu_ms"] / entry["read_time_rotation"]["cross_gpu_ms"],
            "warm_ttft": entry["materialized"]["warm_ms_p50"] / entry["read_time_rotation"]["warm_ms_p50"]}
        res[name] = entry
        del q, k, v, out
    res["paper_context"] = "CIDRA (section 5.5) repositions at most 500 tokens/ms on the paper's hardware"
    return res


def _percentiles(xs):
    return {"p50": _pct(xs, 50), "p99": _pct(xs, 99), "mean": float(sum(xs) / len(xs)) if xs else None}


def attention_batch(spanq, wl, torch, np, steps, warmup):
    """One cold batch of a single-layer workload, repeated: step time and the two
    attention kernels' rates (HIP events on the launch stream)."""
    qa, ka, va = wl.device_arrays()
    q, k, v = (torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda() for a in (qa, ka, va))
    out = torch.zeros_like(q)
    batch = wl.batches[0]
    pages = sum((s.n + 15) // 16 for s in {id(x): x for qq in batch for x in [qq.prefix, *qq.frags, qq.cross]}.values())
    pool = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                      num_pages=pages + 256, dtype=wl.dtype, rope_theta=wl.rope_theta, timing=True, device=0)
    stream = torch.cuda.current_stream()

    def step():
        pool.reset()
        p = pool.plan(batch, stream)
        p.prefill(0, q, k, v, out)
        p.cross(0, q, k, v, out)
        p.commit()
        return p

    for _ in range(warmup):
        step().destroy()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    plans = [step() for _ in range(steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = plans[0].stats()
    kt = [p.kernel_times() for p in plans]
    for p in plans:
        p.destroy()
    pool.close()
    k1 = float(np.mean([t["prefill_attention_ms"] for t in kt]))
    k2 = float(np.mean([t["cross_attention_ms"] for t in kt]))
    return {"ms_per_step": wall * 1e3 / steps,
            "tflops_step": _flops(wl, st["prefill_pairs"] + st["cross_pairs"]) / (wall / steps) / 1e12,
            "span_prefill_attention": {"ms": k1, "tflops": _flops(wl, st["prefill_pairs"]) / (k1 * 1e-3) / 1e12},
            "cross_attention": {"ms": k2, "tflops": _flops(wl, st["cross_pairs"]) / (k2 * 1e-3) / 1e12},
            "tokens_new": st["tokens_new"], "tokens_cross": st["tokens_cross"]}


def _upload_stack(torch, np, sw):
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()  # noqa: E731
    return dict(embed=dev(sw.embed), final_norm=dev(sw.final_norm), lm_head=dev(sw.lm_head),
                attn_norm=[dev(a) for a in sw.attn_norm], w_qkv=[dev(a) for a in sw.w_qkv],
                w_o=[dev(a) for a in sw.w_o], ffn_norm=[dev(a) for a in sw.ffn_norm],
                w_gate_up=[dev(a) for a in sw.w_gate_up], w_down=[dev(a) for a in sw.w_down])


def stack_flops(sw, rows, pairs_per_layer, queries_with_cross):
    """Model FLOPs of a prefill: the four GEMMs per layer for every computed row,
    attention over the allowed pairs in every layer, the LM head per query."""
    d, hq, hkv, H, F = sw.head_dim, sw.n_q_heads, sw.n_kv_heads, sw.hidden, sw.ffn
    per_row = 2 * (H * (hq + 2 * hkv) * d + hq * d * H + H * 2 * F + F * H)
    return (per_row * rows + 4 * d * hq * pairs_per_layer) * sw.n_layers + 2 * H * sw.vocab * queries_with_cross


def c4_ttft(spanq, W, torch, np, reps, decode_steps=16):
    """C4: a 32-layer 2B-class decoder (hidden 2048, 32/8 heads x 64, SwiGLU 8192) over
    one RAG span query (prefix 512 + 32 fragments x 1024 + question 256).  Time to
    first token from the span_plan call to the first token on the host: cold (fresh
    pool), warm (every fragment cached by the previous query, in reversed order), and
    the same tokens as one causal span (no span sparsity, nothing cached)."""
    t0 = time.perf_counter()
    swl = W.config_c4()
    sw = swl.weights
    wts = _upload_stack(torch, np, sw)
    gen_s = time.perf_counter() - t0
    q = swl.batches[0][0]
    rev = W.Query(prefix=q.prefix, frags=q.frags[::-1], cross=q.cross)
    n_tok = q.prefix.n + sum(f.n for f in q.frags) + q.cross.n
    pool = spanq.Pool(num_q_heads=sw.n_q_heads, num_kv_heads=sw.n_kv_heads, head_dim=sw.head_dim,
                      num_pages=(n_tok + 15) // 16 + 3 * 64 + 64, dtype="bf16", rope_theta=swl.rope_theta,
                      num_layers=sw.n_layers, device=0)
    model = spanq.Model(pool, hidden=sw.hidden, ffn=sw.ffn, vocab=sw.vocab, rms_eps=swl.rms_eps, **wts)

    def one(query, row_tokens):
        torch.cuda.synchronize()
        t = time.perf_counter()
        p = pool.plan([query])
        tok = model.forward(p, row_tokens)
        dt = (time.perf_counter() - t) * 1e3
        st = p.stats()
        p.commit()
        p.destroy()
        return dt, tok[0], st

    cold, warm, dense = [], [], []
    toks = {}
    st_cold = st_warm = None
    for r in range(reps + 1):
        pool.reset()
        c = one(q, swl.row_tokens)
        w = one(rev, swl.row_tokens)
        if r:
            cold.append(c[0])
            warm.append(w[0])
        toks = {"cold_order": c[1], "warm_reversed": w[1]}
        st_cold, st_warm = c[2], w[2]
    # nested generation: the warm query's first token, then greedy decode steps through
    # all 32 layers (span_model_decode), each timed from the call to its token on the host
    p = pool.plan([rev])
    cur = model.forward(p, swl.row_tokens)
    step_ms = []
    for i in range(decode_steps + 2):
        torch.cuda.synchronize()
        t = time.perf_counter()
        cur = model.decode(p, cur)
        if i >= 2:
            step_ms.append((time.perf_counter() - t) * 1e3)
    ctx_pages = sum(len(p.block_table(0, s)[0]) for s in range(-1, len(rev.frags) + 1))
    p.commit()
    p.destroy()
    page_bytes = 2 * sw.n_kv_heads * 16 * sw.head_dim * 2
    w_bytes = sum(a.nbytes for a in [*sw.w_qkv, *sw.w_o, *sw.w_gate_up, *sw.w_down]) + sw.lm_head.nbytes
    kv_bytes = ctx_pages * page_bytes * sw.n_layers
    dstep = _percentiles(step_ms)
    decode = {"steps": len(step_ms), "ms_per_token_p50": dstep["p50"], "ms_per_token_p99": dstep["p99"],
              "context_tokens": n_tok + decode_steps + 2, "weight_bytes": int(w_bytes), "kv_bytes": int(kv_bytes),
              "hbm_gbs_p50": (w_bytes + kv_bytes) / (dstep["p50"] * 1e-3) / 1e9,
              "note": "one query; per step every weight matrix and every cached K/V page of the context is read "
                      "once (the bytes above), plus the host round trip for the token"}
    S = np.concatenate([s.tokens for s in [q.prefix, *q.frags, q.cross]]).astype(np.int32)
    whole = W.Query(prefix=W.Span(tokens=S[:-q.cross.n], row=0), frags=[],
                    cross=W.Span(tokens=S[-q.cross.n:], row=S.size - q.cross.n))
    for r in range(3):
        pool.reset()
        d = one(whole, S)
        if r:
            dense.append(d[0])
    model.close()
    pool.close()
    del wts
    torch.cuda.empty_cache()
    f_cold = stack_flops(sw, st_cold["tokens_new"] + st_cold["tokens_cross"],
                         st_cold["prefill_pairs"] + st_cold["cross_pairs"], 1)
    f_warm = stack_flops(sw, st_warm["tokens_new"] + st_warm["tokens_cross"],
                         st_warm["prefill_pairs"] + st_warm["cross_pairs"], 1)
    c, w_, dd = _percentiles(cold), _percentiles(warm), _percentiles(dense)
    return {"workload": "C4: 32 layers, hidden 2048, 32/8 heads x 64, SwiGLU 8192, vocab 128256, bf16; prefix 512 + "
                        "32 x 1024 fragments + question 256 (33,536 tokens)",
            "cold_ms_p50": c["p50"], "cold_ms_p99": c["p99"], "warm_ms_p50": w_["p50"], "warm_ms_p99": w_["p99"],
            "dense_causal_ms_p50": dd["p50"], "warm_speedup_vs_cold": c["p50"] / w_["p50"],
            "warm_speedup_vs_dense": dd["p50"] / w_["p50"], "reps": len(cold),
            "cold_model_tflops": f_cold / (c["p50"] * 1e-3) / 1e12, "cold_model_tflop": f_cold / 1e12,
            "warm_model_tflop": f_warm / 1e12, "first_tokens": toks, "decode": decode,
            "weights_gen_and_upload_s": gen_s}


def c5_stream(spanq, W, torch, np, n_queries):
    """C5: the 32-layer Llama-3-8B-shaped decoder (random init, bf16) over an agentic
    stream of span queries (1024 fragments of 128..2048 tokens, Zipf 1.1 popularity,
    4-24 per query, shared 256-token prefix, 128-token question), one query at a time,
    with a 200 GB KV pool (95,367 pages of 2 MiB: no eviction) and with a 48 GB cap
    (22,888 pages: LRU eviction), the latter also in the order span_bulk_order gives the
    whole stream as one bulk (section 5.8).  Per query: time to first token (span_plan
    call to the token on the host)."""
    t0 = time.perf_counter()
    sw = W.llama3_8b_weights(threads=len(os.sched_getaffinity(0)))
    print(f"[bench] c5 weights {sw.nbytes() / 1e9:.1f} GB drawn in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)
    wts = _upload_stack(torch, np, sw)
    stream = W.c5_stream(n_queries=n_queries)
    res = {}
    for name, pages, bulk in (("pool_200GB", 95_367, False), ("cap_48GB", 22_888, False),
                              ("cap_48GB_bulk_clustered", 22_888, True)):
        pool = spanq.Pool(num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=pages, dtype="bf16",
                          rope_theta=1e4, num_layers=32, device=0)
        model = spanq.Model(pool, hidden=4096, ffn=14336, vocab=W.VOCAB, rms_eps=1e-5, **wts)
        ttft, hit, tot, flops, evicted, new_tok = [], 0, 0, 0.0, 0, 0
        # the whole stream as one bulk: executed in the order span_bulk_order gives
        t_order = time.perf_counter()
        order = pool.bulk_order([sq.query for sq in stream]) if bulk else list(range(len(stream)))
        order_ms = (time.perf_counter() - t_order) * 1e3
        t_run = time.perf_counter()
        for i, sq in enumerate(stream[j] for j in order):
            torch.cuda.synchronize()
            t = time.perf_counter()
            p = pool.plan([sq.query])
            model.forward(p, sq.row_tokens)
            ttft.append((time.perf_counter() - t) * 1e3)
            st = p.stats()
            p.commit()
            p.destroy()
            hit += st["tokens_hit"]
            tot += st["tokens_hit"] + st["tokens_new"]
            new_tok += st["tokens_new"]
            evicted += st["pages_evicted"]
            flops += stack_flops(sw, st["tokens_new"] + st["tokens_cross"], st["prefill_pairs"] + st["cross_pairs"], 1)
            if i % 32 == 31:
                print(f"[bench] c5 {name}: {i + 1} queries, hit rate {hit / tot:.3f}, "
                      f"ttft p50 {_pct(ttft, 50):.1f} ms", file=sys.stderr, flush=True)
        wall = time.perf_counter() - t_run
        pr = _percentiles(ttft)
        res[name] = {"pages": pages, "pool_gb": pages * 2 * 1024 * 1024 / 1e9, "queries": len(stream),
                     "hit_rate": hit / tot, "evicted_pages": evicted, "new_tokens": new_tok,
                     "ttft_ms_p50": pr["p50"], "ttft_ms_p99": pr["p99"], "ttft_ms_mean": pr["mean"],
                     "stream_s": wall, "prefill_tflops": flops / (sum(ttft) * 1e-3) / 1e12,
                     "model_tflop": flops / 1e12, "order": "bulk clustered (span_bulk_order)" if bulk else "given",
                     "bulk_order_ms": order_ms if bulk else 0.0}
        model.close()
        pool.close()
        torch.cuda.synchronize()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c2", choices=["c2", "c3", "c4", "c5", "repos"],
                    help="c2: the headline run (with C3, C4 and repositioning extras); c3: the judge pattern as "
                         "the main workload; c4: only the 2B-class decoder's TTFT and decode steps; c5: only the "
                         "agentic stream over the 8B-shaped decoder; repos: only the read-time vs materialised "
                         "repositioning comparison")
    ap.add_argument("--c5-queries", type=int, default=256)
    ap.add_argument("--no-extras", action="store_true", help="skip the C3 and C4 extras of the default run")
    ap.add_argument("--kernel", default="auto", choices=["auto", "generic", "mfma"])
    ap.add_argument("--ttft-reps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=60.0,
                    help="upper bound on the oracle baseline's time (it runs every row of one C2 query)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peak-probes", action="store_true",
                    help="skip the MFMA-only and streaming-read probes of the attainable peaks")
    ap.add_argument("--gather-reps", type=int, default=10,
                    help="timed passes of the KV page-gather measurement (0 skips it)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy of MIB MiB (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the span-query path here is a single-GPU build "
              "(no sharding or collectives); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2511_02749_amd as spanq
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)
        return
    if args.config == "c5":
        res = c5_stream(spanq, W, torch, np, args.c5_queries)
        print(json.dumps({"metric": "C5 agentic stream: time to first token per span query (ms) and KV hit rate",
                          "unit": "ms", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic (seeded tokens, random-init weights)",
                          "config": {"workload": "C5: Llama-3-8B-shaped 32-layer decoder, 256 span queries over 1024 "
                                                 "fragments (128..2048 tokens, Zipf 1.1, 4-24 per query), prefix 256, "
                                                 "question 128"},
                          "c5": res}), flush=True)
        return
    if args.config == "c4":
        res = c4_ttft(spanq, W, torch, np, reps=max(5, args.ttft_reps))
        print(json.dumps({"metric": "C4 decoder: time to first token (ms), cold / warm / dense, and decode steps",
                          "unit": "ms", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic (seeded tokens, random-init weights)",
                          "config": {"workload": res["workload"]}, "c4": res}), flush=True)
        return
    if args.config == "repos":
        res = reposition_ab(spanq, W, torch, np, reps=max(5, args.ttft_reps))
        print(json.dumps({"metric": "repositioning: read-time rotation vs materialised copies, warm cross pass",
                          "unit": "ms", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16",
                          "data": "synthetic (seeded tokens and activations)",
                          "config": {"workload": "C2 and C3 first queries, fragments cached, reversed order"},
                          "reposition": res}), flush=True)
        return
    t_gen = time.perf_counter()
    wl = W.config_c2() if args.config == "c2" else W.config_c3()
    batch = wl.batches[0]
    print(f"[bench] workload {wl.name}: {wl.rows} rows generated in {time.perf_counter() - t_gen:.1f} s",
          file=sys.stderr, flush=True)
    qa, ka, va = wl.device_arrays()
    q, k, v = (torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda() for a in (qa, ka, va))
    out = torch.zeros_like(q)
    per_query_pages = max((qq.prefix.n + 15) // 16 + sum((f.n + 15) // 16 for f in qq.frags) +
                          (qq.cross.n + 15) // 16 for qq in batch)
    distinct_pages = sum((s.n + 15) // 16 for s in {id(x): x for qq in batch for x in [qq.prefix, *qq.frags]}.values())
    num_pages = distinct_pages + len(batch) * 64 + 4 * per_query_pages
    pool = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                      num_pages=num_pages, dtype=wl.dtype, rope_theta=wl.rope_theta, kernel=args.kernel,
                      timing=True, device=0)
    stream = torch.cuda.current_stream()

    def step():
        pool.reset()
        plan = pool.plan(batch, stream)
        plan.prefill(0, q, k, v, out)
        plan.cross(0, q, k, v, out)
        plan.commit()
        return plan

    for _ in range(args.warmup):
        step().destroy()
    torch.cuda.synchronize()
    plans = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        plans.append(step())
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = plans[0].stats()
    host_plan_us = float(np.mean([p.stats()["host_plan_us"] for p in plans]))
    host_upload_us = float(np.mean([p.stats()["host_upload_us"] for p in plans]))
    times = [p.kernel_times() for p in plans]
    for p in plans:
        p.destroy()
    ms_step = wall * 1e3 / args.steps
    flops_step = _flops(wl, st["prefill_pairs"] + st["cross_pairs"])
    k1_flops = _flops(wl, st["prefill_pairs"])
    k2_flops = _flops(wl, st["cross_pairs"])
    mean = {n: float(np.mean([t[n] for t in times])) for n in spanq._lib.TIME_FIELDS}
    k1_tflops = k1_flops / (mean["prefill_attention_ms"] * 1e-3) / 1e12
    k2_tflops = k2_flops / (mean["cross_attention_ms"] * 1e-3) / 1e12
    kv_bytes_page = 2 * wl.n_kv_heads * 16 * wl.head_dim * 2
    # least HBM bytes one span-prefill launch must move: its query rows in, its output
    # rows out (bf16), every newly written K/V page read once
    k1_bytes = 2 * st["tokens_new"] * wl.n_q_heads * wl.head_dim * 2 + st["pages_new"] * kv_bytes_page
    print(f"[bench] step {ms_step:.3f} ms; K1 {mean['prefill_attention_ms']:.3f} ms {k1_tflops:.1f} TFLOP/s; "
          f"K2 {mean['cross_attention_ms']:.3f} ms {k2_tflops:.1f} TFLOP/s; combine {mean['combine_ms']:.3f} ms; "
          f"host plan {host_plan_us:.0f} us upload {host_upload_us:.0f} us", file=sys.stderr, flush=True)

    # ---------------- single-query TTFT: cold, warm (cached fragments, new order), dense causal.
    # The wall-clock figures come from a pool without timing events (as a serving
    # process runs it); the per-phase breakdown from the same queries on the timed pool.
    ttft = {}
    if args.ttft_reps > 0:
        q0 = batch[0]
        rev = W.Query(prefix=q0.prefix, frags=q0.frags[::-1], cross=q0.cross)
        plain = spanq.Pool(num_q_heads=wl.n_q_heads, num_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                           num_pages=num_pages, dtype=wl.dtype, rope_theta=wl.rope_theta, kernel=args.kernel,
                           timing=False, device=0)

        host = {"cold": [], "warm": [], "dense": []}

        def one(pl, query, qq, kk, vv, oo, kind):
            torch.cuda.synchronize()
            t = time.perf_counter()
            p = pl.plan([query], stream)
            p.prefill(0, qq, kk, vv, oo)
            p.cross(0, qq, kk, vv, oo)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t) * 1e3
            p.commit()
            if pl is pool:
                s1 = p.stats()
                kt = p.kernel_times()
                host[kind].append((s1["host_plan_us"], s1["host_upload_us"],
                                   kt["prefill_attention_ms"] + kt["page_write_prefill_ms"],
                                   kt["cross_attention_ms"] + kt["page_write_cross_ms"] + kt["combine_ms"]))
            p.destroy()
            return dt

        cold, warm, dense = [], [], []
        for _ in range(args.ttft_reps + 2):
            plain.reset()
            cold.append(one(plain, q0, q, k, v, out, "cold"))
            warm.append(one(plain, rev, q, k, v, out, "warm"))
        for _ in range(max(3, args.ttft_reps // 4)):
            pool.reset()
            one(pool, q0, q, k, v, out, "cold")
            one(pool, rev, q, k, v, out, "warm")
        rows = np.concatenate([np.arange(s.row, s.row + s.n) for s in [q0.prefix, *q0.frags, q0.cross]])
        ridx = torch.as_tensor(rows, device="cuda")
        qd, kd, vd = q[ridx].contiguous(), k[ridx].contiguous(), v[ridx].contiguous()
        od = torch.zeros_like(qd)
        toks = np.concatenate([s.tokens for s in [q0.prefix, *q0.frags, q0.cross]])
        whole = W.Query(prefix=W.Span(tokens=toks, row=0), frags=[], cross=W.Span(tokens=toks[:0], row=0))
        for _ in range(max(3, args.ttft_reps // 4) + 1):
            plain.reset()
            dense.append(one(plain, whole, qd, kd, vd, od, "dense"))
            pool.reset()
            one(pool, whole, qd, kd, vd, od, "dense")
        plain.close()
        cold, warm, dense = cold[2:], warm[2:], dense[1:]
        ttft = {"cold_ms_p50": _pct(cold, 50), "cold_ms_p99": _pct(cold, 99), "warm_ms_p50": _pct(warm, 50),
                "warm_ms_p99": _pct(warm, 99), "dense_causal_ms_p50": _pct(dense, 50),
                "warm_speedup_vs_cold": _pct(cold, 50) / _pct(warm, 50),
                "warm_speedup_vs_dense": _pct(dense, 50) / _pct(warm, 50), "reps": len(cold),
                "query": f"prefix {q0.prefix.n} + {len(q0.frags)} x {q0.frags[0].n} + cross {q0.cross.n}",
                "wall_clock": "pool without timing events; breakdown_us from the same queries on a timed pool",
                "breakdown_us": {kind: dict(zip(("host_plan", "host_upload", "prefill_gpu", "cross_gpu"),
                                                [float(np.median([x[i] for x in v])) * (1 if i < 2 else 1e3)
                                                 for i in range(4)]))
                                 for kind, v in host.items() if v}}
        print(f"[bench] ttft {json.dumps(ttft)}", file=sys.stderr, flush=True)
    pool.close()

    gather = None
    if args.gather_reps > 0:
        gather = kv_gather(spanq, W, torch, np, args.gather_reps)
        print(f"[bench] kv gather {json.dumps(gather)}", file=sys.stderr, flush=True)

    peaks = None
    if not args.no_peak_probes:
        mfma_peak = spanq.probe_mfma_peak(iters=20000, reps=5)
        buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
        read_peak = spanq.probe_read_peak(buf, reps=10)
        del buf
        peaks = {"mfma_bf16_tflops": mfma_peak, "hbm_read_gbs": read_peak,
                 "span_prefill_attention_frac": k1_tflops / mfma_peak,
                 "kv_gather_frac": ({k: v["gbs"] / read_peak for k, v in gather["by_rows"].items()}
                                    if gather else None),
                 "method": "MFMA-only loop: two waves per SIMD on every CU, four independent "
                           "v_mfma_f32_32x32x16_bf16 chains; streaming read: 2 GiB device buffer, "
                           "16-byte non-temporal loads, 10 launches"}
        print(f"[bench] measured peaks {json.dumps(peaks)}", file=sys.stderr, flush=True)

    extras = {}
    if not args.no_extras and args.config == "c2":
        extras["c3"] = attention_batch(spanq, W.config_c3(), torch, np, steps=10, warmup=2)
        extras["c3"]["workload"] = "C3 judge pattern: prompt 2048 + 32 candidates x 256 + judge 256, one query, cold"
        print(f"[bench] c3 {json.dumps(extras['c3'])}", file=sys.stderr, flush=True)
        extras["c4"] = c4_ttft(spanq, W, torch, np, reps=max(5, args.ttft_reps))
        print(f"[bench] c4 {json.dumps(extras['c4'])}", file=sys.stderr, flush=True)
        extras["reposition"] = reposition_ab(spanq, W, torch, np, reps=10)
        print(f"[bench] reposition {json.dumps(extras['reposition'])}", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, batch[0], args.cpu_seconds)
        print(f"[bench] cpu baseline {json.dumps(cpu)}", file=sys.stderr, flush=True)

    result = {
        "metric": METRIC,
        "value": flops_step / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded tokens, random-init projection weights)",
        "config": {
            "workload": ("C2 span-query batch: Llama-3-8B-shaped attention layer (32/8 heads, d 128, hidden 4096), "
                         "prefix 256 + 16 of 64 fragments x 512 in random order + cross 128, 8 queries, cold"
                         if args.config == "c2" else
                         "C3 judge pattern: prompt 2048 + 32 candidates x 256 + judge 256, one query, cold"),
            "queries": len(batch),
            "tokens_new": st["tokens_new"],
            "tokens_cross": st["tokens_cross"],
            "allowed_pairs": st["prefill_pairs"] + st["cross_pairs"],
            "kernel": args.kernel,
        },
        "kernels": {
            "span_prefill_attention": {"ms": mean["prefill_attention_ms"], "tflops": k1_tflops},
            "cross_attention": {"ms": mean["cross_attention_ms"], "tflops": k2_tflops,
                                "kv_splits": st["kv_splits"]},
            "page_write_prefill": {"ms": mean["page_write_prefill_ms"],
                                   "gbs": (st["pages_new"] * kv_bytes_page * 2) / (mean["page_write_prefill_ms"] * 1e-3) / 1e9
                                   if mean["page_write_prefill_ms"] > 0 else None},
            "page_write_cross_ms": mean["page_write_cross_ms"],
            "combine_ms": mean["combine_ms"],
            "host_plan_us": host_plan_us,
            "host_upload_us": host_upload_us,
        },
        "roofline": {"kernel": "span_prefill_attention", "bound": "mfma", "achieved": k1_tflops,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": k1_tflops / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic(args.config) if args.kernel != "generic" else None,
                     "algorithmic_bytes": k1_bytes, "launch_flops": k1_flops},
        "headline": {"span_prefill_attention_tflops": k1_tflops,
                     "span_prefill_attention_frac_of_2.5PF": k1_tflops / PEAK_BF16_TFLOPS,
                     "cache_hit_ttft_ms_p50": ttft.get("warm_ms_p50"),
                     "cold_ttft_ms_p50": ttft.get("cold_ms_p50"),
                     "model_cache_hit_ttft_ms_p50": extras.get("c4", {}).get("warm_ms_p50"),
                     "model_cold_ttft_ms_p50": extras.get("c4", {}).get("cold_ms_p50")},
        "ttft": ttft,
        "kv_gather": gather,
        **extras,
        "measured_peaks": peaks,
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
