"""Seeded synthetic span-query workloads.

This module only *draws inputs*: token ids, the span structure of each query
(shared prefix, commuting fragments, trailing cross segment) and the per-row
q/k/v activations that a projection of random hidden states produces.  It holds
none of the attention method's arithmetic (no masks, positions, RoPE, hashing
or softmax), so both the HIP path and the oracle can consume it without
sharing any of the method's code.

Row convention: every span owns a contiguous run of rows in the q/k/v arrays,
starting at ``Span.row``.  A fragment that several queries draw owns one run
of rows, shared by all of them (the same content always has the same
activations, as it would in the first layer of a model).

Randomness: numpy ``Generator(PCG64)`` seeded through ``SeedSequence`` with a
spawn key ``(kind, index)`` per object, so every object (a fragment's tokens,
a token's hidden state, a weight matrix, a query's draw) is reproducible on
its own.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

KIND_PREFIX = 1
KIND_FRAG = 2
KIND_CROSS = 3
KIND_EMBED = 4
KIND_WEIGHT = 5
KIND_DRAW = 6
KIND_DIRECT = 7
KIND_LEN = 8

VOCAB = 128256


def rng(seed: int, kind: int, index: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(kind, index))))


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (storage format only)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Span:
    tokens: np.ndarray  # int32
    row: int            # first row of this span's q/k/v/out rows

    @property
    def n(self) -> int:
        return int(self.tokens.shape[0])


@dataclass
class Query:
    prefix: Span
    frags: List[Span]
    cross: Span


@dataclass
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16"
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    page_size: int
    batches: List[List[Query]]  # each batch is one span_plan call
    q: np.ndarray              # [rows, Hq, d] float32 (exactly representable in dtype)
    k: np.ndarray              # [rows, Hkv, d]
    v: np.ndarray              # [rows, Hkv, d]
    q_bits: Optional[np.ndarray] = None  # bf16 bit patterns when dtype == "bf16"
    k_bits: Optional[np.ndarray] = None
    v_bits: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)

    @property
    def rows(self) -> int:
        return int(self.q.shape[0])

    def device_arrays(self):
        """The arrays a GPU caller uploads: bf16 bit patterns or fp32 values."""
        if self.dtype == "bf16":
            return self.q_bits, self.k_bits, self.v_bits
        return self.q, self.k, self.v


def _tokens(seed: int, kind: int, index: int, n: int) -> np.ndarray:
    return rng(seed, kind, index).integers(0, VOCAB, size=n, dtype=np.int64).astype(np.int32)


class _RowBook:
    """Assigns contiguous row runs to distinct spans."""

    def __init__(self):
        self.next = 0
        self.token_runs: List[np.ndarray] = []

    def add(self, tokens: np.ndarray) -> Span:
        s = Span(tokens=tokens, row=self.next)
        self.next += tokens.shape[0]
        self.token_runs.append(tokens)
        return s

    def all_tokens(self) -> np.ndarray:
        if not self.token_runs:
            return np.zeros((0,), np.int32)
        return np.concatenate(self.token_runs)


def _project(seed: int, tokens: np.ndarray, hidden: int, hq: int, hkv: int, d: int,
             x_std: float, w_std: float, mode: str):
    """Per-row q/k/v (float32) for the given token ids.

    mode "proj": x = E[token] ~ N(0, x_std^2) per distinct token id, weights
    W_q, W_k, W_v ~ N(0, w_std^2); rows = x @ W.
    mode "direct": q/k/v drawn directly ~ N(0, 1) per distinct token id.
    """
    uniq, inv = np.unique(tokens, return_inverse=True)
    width = (hq + 2 * hkv) * d
    out = np.empty((uniq.shape[0], width), np.float32)
    if mode == "direct":
        for i, t in enumerate(uniq):
            out[i] = rng(seed, KIND_DIRECT, int(t)).standard_normal(width, dtype=np.float32)
    else:
        w = rng(seed, KIND_WEIGHT, 0).standard_normal((hidden, width), dtype=np.float32) * np.float32(w_std)
        chunk = 4096
        for c0 in range(0, uniq.shape[0], chunk):
            c1 = min(uniq.shape[0], c0 + chunk)
            x = np.empty((c1 - c0, hidden), np.float32)
            for i in range(c0, c1):
                x[i - c0] = rng(seed, KIND_EMBED, int(uniq[i])).standard_normal(hidden, dtype=np.float32)
            x *= np.float32(x_std)
            out[c0:c1] = x @ w
    rows = out[inv]
    q = rows[:, : hq * d].reshape(-1, hq, d)
    k = rows[:, hq * d: (hq + hkv) * d].reshape(-1, hkv, d)
    v = rows[:, (hq + hkv) * d:].reshape(-1, hkv, d)
    return np.ascontiguousarray(q), np.ascontiguousarray(k), np.ascontiguousarray(v)


def _finish(name, dtype, hq, hkv, d, theta, batches, book, seed, hidden, x_std, w_std, mode, meta):
    q, k, v = _project(seed, book.all_tokens(), hidden, hq, hkv, d, x_std, w_std, mode)
    wl = Workload(name=name, dtype=dtype, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                  rope_theta=theta, page_size=16, batches=batches, q=q, k=k, v=v, meta=meta)
    if dtype == "bf16":
        wl.q_bits, wl.k_bits, wl.v_bits = (round_to_bf16_bits(a) for a in (q, k, v))
        wl.q, wl.k, wl.v = (bf16_bits_to_f32(b) for b in (wl.q_bits, wl.k_bits, wl.v_bits))
    return wl


def rag_workload(name: str = "rag", *, seed: int = 0, dtype: str = "bf16", n_q_heads: int = 32,
                 n_kv_heads: int = 8, head_dim: int = 128, hidden: int = 4096,
                 prefix_len: int = 256, pool_size: int = 64, frag_lens: Sequence[int] | int = 512,
                 frags_per_query: int = 16, n_queries: int = 8, cross_len: int = 128,
                 x_std: float = 1.0, w_std: float = 0.02, mode: str = "proj",
                 rope_theta: float = 1e4, batch_split: Optional[Sequence[int]] = None,
                 orders: Optional[Sequence[Sequence[int]]] = None,
                 frag_tokens: Optional[Sequence[Optional[np.ndarray]]] = None) -> Workload:
    """A shared prefix, a pool of fragments, queries drawing fragments in random order.

    ``orders`` overrides the random draw with explicit fragment orders per query.
    ``batch_split`` groups queries into successive span_plan calls (default: one batch).
    ``frag_tokens[f]``, where given, replaces fragment f's drawn tokens (its length
    then overrides ``frag_lens[f]``).
    """
    book = _RowBook()
    prefix = book.add(_tokens(seed, KIND_PREFIX, 0, prefix_len))
    if isinstance(frag_lens, int):
        frag_lens = [frag_lens] * pool_size
    frags = []
    for f in range(pool_size):
        given = frag_tokens[f] if frag_tokens is not None and f < len(frag_tokens) else None
        toks = (np.ascontiguousarray(given, dtype=np.int32) if given is not None
                else _tokens(seed, KIND_FRAG, f, int(frag_lens[f])))
        frags.append(book.add(toks))
    queries = []
    for qi in range(n_queries):
        if orders is not None:
            order = [int(x) for x in orders[qi]]
        else:
            order = [int(x) for x in rng(seed, KIND_DRAW, qi).choice(pool_size, size=frags_per_query, replace=False)]
        cross = book.add(_tokens(seed, KIND_CROSS, qi, cross_len))
        queries.append(Query(prefix=prefix, frags=[frags[f] for f in order], cross=cross))
    if batch_split is None:
        batches = [queries]
    else:
        batches, at = [], 0
        for n in batch_split:
            batches.append(queries[at: at + n])
            at += n
    meta = dict(prefix_len=prefix_len, pool_size=pool_size, frags_per_query=frags_per_query,
                n_queries=n_queries, cross_len=cross_len, hidden=hidden, mode=mode, seed=seed)
    return _finish(name, dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, batches, book,
                   seed, hidden, x_std, w_std, mode, meta)


def config_c1(seed: int = 0, mode: str = "proj") -> Workload:
    """fp32 MHA 4x64, hidden 256, prefix 32 + 4 fragments x 64 + cross 16.

    Batch 0: query A, fragments in order (0,1,2,3), cold.  Batch 1: query B,
    a seeded permutation of the same fragments (every fragment page a hit).
    Projection: hidden N(0, 0.02^2), weights N(0, 1).  ``mode="direct"``
    draws q/k/v ~ N(0,1) instead, so the softmax is far from flat.
    """
    perm = [int(x) for x in rng(seed, KIND_DRAW, 1000).permutation(4)]
    if perm == [0, 1, 2, 3]:
        perm = [3, 2, 1, 0]
    wl = rag_workload("c1", seed=seed, dtype="f32", n_q_heads=4, n_kv_heads=4, head_dim=64, hidden=256,
                      prefix_len=32, pool_size=4, frag_lens=64, frags_per_query=4, n_queries=2,
                      cross_len=16, x_std=0.02, w_std=1.0, mode=mode, orders=[[0, 1, 2, 3], perm],
                      batch_split=[1, 1])
    return wl


def config_c2(seed: int = 0, n_queries: int = 8, mode: str = "proj") -> Workload:
    """Llama-3-8B attention layer shape, bf16, GQA 32/8, d 128, hidden 4096.

    Prefix 256 + 16 fragments x 512 drawn from a pool of 64 in random order,
    cross (question) 128 per query, 8 queries in one batch.
    """
    return rag_workload("c2", seed=seed, dtype="bf16", n_q_heads=32, n_kv_heads=8, head_dim=128,
                        hidden=4096, prefix_len=256, pool_size=64, frag_lens=512, frags_per_query=16,
                        n_queries=n_queries, cross_len=128, x_std=1.0, w_std=0.02, mode=mode)


def config_c3(seed: int = 0, mode: str = "proj") -> Workload:
    """Judge pattern: 2048-token shared prompt, 32 candidates x 256, judge cross 256."""
    return rag_workload("c3", seed=seed, dtype="bf16", n_q_heads=32, n_kv_heads=8, head_dim=128,
                        hidden=4096, prefix_len=2048, pool_size=32, frag_lens=256, frags_per_query=32,
                        n_queries=1, cross_len=256, x_std=1.0, w_std=0.02, mode=mode,
                        orders=[list(range(32))])


def small_workload(name: str = "small", *, seed: int = 0, dtype: str = "bf16", n_q_heads: int = 8,
                   n_kv_heads: int = 2, head_dim: int = 128, prefix_len: int = 40,
                   frag_lens: Sequence[int] = (37, 64, 5, 100), n_queries: int = 3,
                   frags_per_query: int = 3, cross_len: int = 23, mode: str = "direct",
                   orders=None, batch_split=None, frag_tokens=None) -> Workload:
    """Small ragged case for parity: lengths off page boundaries, several tiles."""
    return rag_workload(name, seed=seed, dtype=dtype, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                        head_dim=head_dim, hidden=64, prefix_len=prefix_len, pool_size=len(frag_lens),
                        frag_lens=list(frag_lens), frags_per_query=frags_per_query, n_queries=n_queries,
                        cross_len=cross_len, mode=mode, orders=orders, batch_split=batch_split,
                        frag_tokens=frag_tokens)


def shared_head_tokens(seed: int, base_len: int, shares: Sequence[int], lens: Sequence[int]) -> List[np.ndarray]:
    """Fragment token arrays for cache-reuse cases: fragment 0 is ``base_len`` drawn
    tokens; fragment i >= 1 repeats the first ``shares[i-1]`` tokens of fragment 0 and
    continues with ``lens[i-1] - shares[i-1]`` tokens of its own draw."""
    base = _tokens(seed, KIND_FRAG, 0, base_len)
    out = [base]
    for i, (share, n) in enumerate(zip(shares, lens)):
        tail = _tokens(seed, KIND_FRAG, 10_000 + i, int(n) - int(share))
        out.append(np.concatenate([base[:share], tail]).astype(np.int32))
    return out


def gather_queries(seed: int = 0, n_queries: int = 8, prefix_len: int = 2048, n_frags: int = 32,
                   frag_len: int = 256, cross_len: int = 16):
    """Independent judge-shaped queries (C3 layout: prompt 2048 + 32 candidates x 256)
    whose KV pages are all distinct (each query has its own prompt), followed by a
    short cross segment: the KV page-gather regime, where cross attention reads
    many pages for few query rows.  Returns (queries, n_rows); the activations
    are left to the caller (seeded device draws), since the timing does not
    depend on their values and projecting 80K rows on the host would be slow.
    """
    book = _RowBook()
    queries = []
    for qi in range(n_queries):
        prefix = book.add(_tokens(seed, KIND_PREFIX, 1000 + qi, prefix_len))
        frags = [book.add(_tokens(seed, KIND_FRAG, 1000 * (qi + 1) + f, frag_len)) for f in range(n_frags)]
        cross = book.add(_tokens(seed, KIND_CROSS, 1000 + qi, cross_len))
        queries.append(Query(prefix=prefix, frags=frags, cross=cross))
    return queries, book.next


# ---------------------------------------------------------------- decoder stacks

KIND_STACK_W = 9
KIND_STACK_TOK = 10


@dataclass
class StackWeights:
    """Random-init weights of a Llama-shaped decoder, as bf16 bit patterns (uint16).

    x @ W convention (W is [in, out]).  w_qkv[l] holds the q, k and v projections side
    by side ([hidden, (Hq + 2 Hkv) d]); w_gate_up[l] the gate then the up projection
    ([hidden, 2 ffn]).  Projection and embedding entries are N(0, std^2); norm gains
    are 1 + N(0, norm_std^2), so that a missing gain shows in parity.
    """
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    embed: np.ndarray
    attn_norm: List[np.ndarray]
    w_qkv: List[np.ndarray]
    w_o: List[np.ndarray]
    ffn_norm: List[np.ndarray]
    w_gate_up: List[np.ndarray]
    w_down: List[np.ndarray]
    final_norm: np.ndarray
    lm_head: np.ndarray

    def f32(self, a: np.ndarray) -> np.ndarray:
        return bf16_bits_to_f32(a)

    def nbytes(self) -> int:
        arrs = [self.embed, self.final_norm, self.lm_head, *self.attn_norm, *self.w_qkv, *self.w_o,
                *self.ffn_norm, *self.w_gate_up, *self.w_down]
        return int(sum(a.nbytes for a in arrs))


def stack_weights(seed: int, n_layers: int, hidden: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                  ffn: int, vocab: int, std: float = 0.02, norm_std: float = 0.1,
                  threads: int = 8) -> StackWeights:
    """Seeded weights, one PCG64 stream per matrix (drawn in parallel threads)."""
    from concurrent.futures import ThreadPoolExecutor

    qkv = (n_q_heads + 2 * n_kv_heads) * head_dim
    specs = [("embed", 0, (vocab, hidden), std, 0.0), ("final_norm", 0, (hidden,), norm_std, 1.0),
             ("lm_head", 0, (hidden, vocab), std, 0.0)]
    for l in range(n_layers):
        specs += [("attn_norm", l, (hidden,), norm_std, 1.0), ("w_qkv", l, (hidden, qkv), std, 0.0),
                  ("w_o", l, (n_q_heads * head_dim, hidden), std, 0.0), ("ffn_norm", l, (hidden,), norm_std, 1.0),
                  ("w_gate_up", l, (hidden, 2 * ffn), std, 0.0), ("w_down", l, (ffn, hidden), std, 0.0)]
    names = ["embed", "final_norm", "lm_head", "attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down"]

    # a matrix is drawn in chunks of at most 2^22 entries of whole rows, chunk c from
    # its own stream (matrix, layer, c), so large matrices draw in parallel too
    chunk_elems = 1 << 22
    jobs = []
    outs = []
    for name, l, shape, s, mean in specs:
        out = np.empty(shape, np.uint16)
        outs.append(out)
        rows = shape[0]
        per = max(1, chunk_elems // max(1, int(np.prod(shape[1:], dtype=np.int64))))
        for c, r0 in enumerate(range(0, rows, per)):
            jobs.append((name, l, c, out, r0, min(rows, r0 + per), s, mean))

    def draw(job):
        name, l, c, out, r0, r1, s, mean = job
        g = rng(seed, KIND_STACK_W, (1000 * names.index(name) + l) * 4096 + c)
        a = g.standard_normal((r1 - r0,) + out.shape[1:], dtype=np.float32)
        a *= np.float32(s)
        if mean:
            a += np.float32(mean)
        out[r0:r1] = round_to_bf16_bits(a)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(draw, jobs))
    arrs = outs
    got = {n: [None] * n_layers for n in names[3:]}
    top = {}
    for (name, l, _, _, _), a in zip(specs, arrs):
        if name in got:
            got[name][l] = a
        else:
            top[name] = a
    return StackWeights(n_layers=n_layers, hidden=hidden, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                        head_dim=head_dim, ffn=ffn, vocab=vocab, embed=top["embed"], final_norm=top["final_norm"],
                        lm_head=top["lm_head"], **got)


@dataclass
class StackWorkload:
    """Span queries over token ids for a decoder stack.  Every distinct span owns a
    run of caller rows; ``row_tokens[r]`` is the token id at caller row r."""
    name: str
    weights: StackWeights
    batches: List[List[Query]]
    row_tokens: np.ndarray
    rope_theta: float = 1e4
    rms_eps: float = 1e-5
    meta: dict = field(default_factory=dict)


def stack_queries(seed: int, vocab: int, prefix_len: int, frag_lens: Sequence[int], cross_len: int,
                  orders: Sequence[Sequence[int]], batch_split: Optional[Sequence[int]] = None):
    """A shared prefix, a pool of fragments (token ids uniform over [0, vocab)) and one
    query per entry of ``orders`` (fragment indices in this query's order), each with a
    cross segment of its own.  Returns (batches, row_tokens)."""
    book = _RowBook()
    tok = lambda kind, i, n: rng(seed, KIND_STACK_TOK, 100_000 * kind + i).integers(  # noqa: E731
        0, vocab, size=n, dtype=np.int64).astype(np.int32)
    prefix = book.add(tok(KIND_PREFIX, 0, prefix_len))
    frags = [book.add(tok(KIND_FRAG, f, int(n))) for f, n in enumerate(frag_lens)]
    queries = []
    for qi, order in enumerate(orders):
        cross = book.add(tok(KIND_CROSS, qi, cross_len))
        queries.append(Query(prefix=prefix, frags=[frags[int(f)] for f in order], cross=cross))
    if batch_split is None:
        batches = [queries]
    else:
        batches, at = [], 0
        for n in batch_split:
            batches.append(queries[at: at + n])
            at += n
    return batches, book.all_tokens()


def stack_small(seed: int = 0, head_dim: int = 64, n_layers: int = 3, orders=((0, 1, 2), (2, 0, 3)),
                batch_split=None) -> StackWorkload:
    """A small stack for whole-output parity: hidden 4 heads x head_dim, one kv head
    (four query heads per kv head), SwiGLU 2 x hidden, vocab 1000; prefix 40, ragged
    fragments (37, 64, 100, 5), cross 23."""
    hq, hkv = 4, 1
    hidden = hq * head_dim
    w = stack_weights(seed, n_layers, hidden, hq, hkv, head_dim, 2 * hidden, 1000)
    batches, rt = stack_queries(seed, 1000, 40, (37, 64, 100, 5), 23, orders, batch_split)
    return StackWorkload(name=f"stack_small_d{head_dim}", weights=w, batches=batches, row_tokens=rt)


def config_c4(seed: int = 0, n_layers: int = 32) -> StackWorkload:
    """2B-class decoder: 32 layers, hidden 2048, 32 query / 8 kv heads x 64, SwiGLU 8192,
    vocab 128256, RMSNorm eps 1e-5, rotary theta 1e4, bf16.  One RAG query: prefix 512 +
    32 fragments x 1024 + question 256."""
    w = stack_weights(seed, n_layers, 2048, 32, 8, 64, 8192, VOCAB)
    batches, rt = stack_queries(seed, VOCAB, 512, [1024] * 32, 256, [list(range(32))])
    return StackWorkload(name="c4", weights=w, batches=batches, row_tokens=rt,
                         meta=dict(prefix_len=512, n_frags=32, frag_len=1024, cross_len=256))


KIND_C5 = 11


@dataclass
class StreamQuery:
    """One query of a stream: its spans (rows numbered from 0 within the query:
    prefix, fragments in order, cross) and the token id at each of those rows."""
    query: Query
    row_tokens: np.ndarray
    frag_ids: List[int]


def c5_stream(seed: int = 0, n_queries: int = 256, pool_size: int = 1024, len_lo: int = 128, len_hi: int = 2048,
              zipf_s: float = 1.1, k_lo: int = 4, k_hi: int = 24, prefix_len: int = 256, cross_len: int = 128,
              vocab: int = VOCAB) -> List[StreamQuery]:
    """Agentic stream: a pool of fragments with lengths uniform on [len_lo, len_hi];
    fragment popularity Zipf(zipf_s) over ranks, ranks mapped to fragments by a seeded
    permutation; each query draws k ~ U{k_lo..k_hi} distinct fragments with
    probability proportional to popularity (without replacement; draw order = the
    query's order), behind one shared prefix, with its own cross segment."""
    g = rng(seed, KIND_C5, 0)
    lens = g.integers(len_lo, len_hi + 1, size=pool_size)
    perm = rng(seed, KIND_C5, 1).permutation(pool_size)
    pop = np.empty(pool_size, np.float64)
    pop[perm] = np.arange(1, pool_size + 1, dtype=np.float64) ** -zipf_s
    pop /= pop.sum()
    tok = lambda kind, i, n: rng(seed, KIND_C5, 1_000_000 * kind + i).integers(  # noqa: E731
        0, vocab, size=int(n), dtype=np.int64).astype(np.int32)
    prefix_tokens = tok(KIND_PREFIX, 0, prefix_len)
    frag_tokens = {}
    out = []
    for qi in range(n_queries):
        gq = rng(seed, KIND_C5, 2_000_000 + qi)
        k = int(gq.integers(k_lo, k_hi + 1))
        ids = [int(x) for x in gq.choice(pool_size, size=k, replace=False, p=pop)]
        at = 0
        prefix = Span(tokens=prefix_tokens, row=at)
        at += prefix_len
        frags = []
        for f in ids:
            if f not in frag_tokens:
                frag_tokens[f] = tok(KIND_FRAG, f, lens[f])
            frags.append(Span(tokens=frag_tokens[f], row=at))
            at += frag_tokens[f].shape[0]
        cross = Span(tokens=tok(KIND_CROSS, qi, cross_len), row=at)
        at += cross_len
        rt = np.concatenate([prefix.tokens] + [s.tokens for s in frags] + [cross.tokens]).astype(np.int32)
        out.append(StreamQuery(query=Query(prefix=prefix, frags=frags, cross=cross), row_tokens=rt, frag_ids=ids))
    return out


def llama3_8b_weights(seed: int = 0, n_layers: int = 32, threads: int = 16) -> StackWeights:
    """Llama-3-8B-shaped random-init weights: hidden 4096, 32 query / 8 kv heads x 128,
    SwiGLU 14336, vocab 128256."""
    return stack_weights(seed, n_layers, 4096, 32, 8, 128, 14336, VOCAB, threads=threads)
