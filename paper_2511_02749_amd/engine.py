"""Greedy execution of span queries on a pool and a decoder stack.

The generate callbacks that ``spanquery.expand_generates`` takes, backed by the
library: a batch of lowered span queries is laid out in one row space, planned
(``span_plan``: hashing, lookup, allocation), run through the stack for its first
token (``span_model_forward``), then decoded greedily one token per step
(``span_model_decode`` over the plan's block tables), and committed, so that the
prefixes and fragments it computed stay cached for the queries after it.  Every
step of the path runs in the native library; this module only lays out rows and
loops over steps.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence

import numpy as np

from . import spanquery as sq


@dataclass
class CallStats:
    """What one generate call planned: pages and tokens served from the cache or computed."""
    queries: int
    pages_hit: int
    tokens_hit: int
    tokens_new: int
    decode_steps: int


@dataclass
class Engine:
    pool: object                       # paper_2511_02749_amd.Pool (device, bf16)
    model: object                      # paper_2511_02749_amd.Model on that pool
    stream: object = None
    calls: List[CallStats] = field(default_factory=list)

    def generate_many(self, spans: Sequence[sq.Spans], max_tokens: int) -> List[List[int]]:
        """Up to max_tokens greedy tokens for each query (one plan, one batch).  Every
        query needs a cross segment: its first token is read at the last cross row."""
        if max_tokens < 1:
            raise ValueError("max_tokens must be at least 1")
        queries, rows, at = [], [], 0
        for sp in spans:
            if not sp.cross:
                raise ValueError("a generate needs a cross segment to read its first token at")
            queries.append(sq.to_query(sp, row0=at))
            toks = list(sp.prefix) + [t for f in sp.fragments for t in f] + list(sp.cross)
            rows.extend(toks)
            at += len(toks)
        plan = self.pool.plan(queries, self.stream)
        try:
            cur = self.model.forward(plan, np.asarray(rows, np.int32), stream=self.stream)
            out = [[t] for t in cur]
            for _ in range(max_tokens - 1):
                cur = self.model.decode(plan, cur, stream=self.stream)
                for o, t in zip(out, cur):
                    o.append(t)
            st = plan.stats()
            self.calls.append(CallStats(queries=len(queries), pages_hit=st["pages_hit"], tokens_hit=st["tokens_hit"],
                                        tokens_new=st["tokens_new"], decode_steps=st["decode_steps"]))
            plan.commit()
        finally:
            plan.destroy()
        return out

    def generate(self, tokens: Sequence[int], max_tokens: int) -> List[int]:
        """A generate over plain messages: the tokens are the cross segment."""
        return self.generate_many([sq.Spans(prefix=[], fragments=[], cross=list(tokens))], max_tokens)[0]

    def generate_join(self, spans: sq.Spans, max_tokens: int) -> List[int]:
        return self.generate_many([spans], max_tokens)[0]

    def run(self, tree: sq.Node) -> List[int]:
        """Run an optimized tree: its inner generates innermost first, then the root."""
        ex = sq.expand_generates(tree, self.generate, self.generate_join)
        root = sq.to_spans(ex)
        return self.generate_join(root, max(1, root.max_tokens))
