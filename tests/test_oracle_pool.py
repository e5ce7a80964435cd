"""Pins of the hashing and page-cache replay oracle.

* SplitMix64 against its published output streams (tests/golden).
* The paper's chat example (section 2.1, block size 2): after "Hello" and the
  generated "How are you ?", two blocks are cached and the next request finds
  4 of its 5 context tokens cached.
* The paper's RAG example (section 3.1): presenting the same fragments in the
  reverse order gets no fragment hits under stock prefix caching, and all of
  them with span hashing (section 5.4).
* LRU consequences checked by brute force on random streams: the surviving
  pages of every span form a prefix of it; the pages a plan touched are never
  evicted while older evictable pages exist; allocation takes the lowest free
  id; a plan fails exactly when it needs more pages than are free or
  evictable, and then changes nothing.
"""
import os
import random

import pytest

from oracle import hashing as H
from oracle.pool import PoolFull, PoolReplay

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_streams():
    with open(os.path.join(GOLDEN, "splitmix64.txt")) as f:
        rows = [l.split("\t") for l in f if l.strip() and not l.startswith("#")]
    assert rows
    for seed, outs in rows:
        s = int(seed)
        for want in outs.split():
            assert H.splitmix64(s) == int(want)
            s = (s + H.GOLDEN_GAMMA) & H.MASK64


def test_chain_depends_on_everything_before():
    toks = list(range(40))
    a = H.chain(H.ROOT_SEED, toks, 16)
    b = H.chain(H.ROOT_SEED, [99] + toks[1:], 16)
    assert len(a) == 3 and all(x != y for x, y in zip(a, b))
    # partial tail page hashed with its true length
    assert H.chain(H.ROOT_SEED, toks[:33], 16)[2] != H.chain(H.ROOT_SEED, toks[:34], 16)[2]
    assert len(H.chain(H.ROOT_SEED, toks[:33], 16, include_partial=False)) == 2


def test_fragment_chain_independent_of_left_siblings():
    prefix = [5, 6, 7]
    f1, f2 = list(range(100, 120)), list(range(200, 237))
    _, fa = H.query_hashes(prefix, [f1, f2], 16)
    _, fb = H.query_hashes(prefix, [f2, f1], 16)
    assert fa[0] == fb[1] and fa[1] == fb[0]
    # but it does depend on the prefix the fragment attends to
    _, fc = H.query_hashes([5, 6, 8], [f1], 16)
    assert fc[0] != fa[0]


def test_paper_chat_example():
    HELLO, HOW, ARE, YOU, Q, I, AM, FINE = range(1, 9)
    pool = PoolReplay(num_pages=16, page_size=2, stock=True)
    r1 = pool.plan([([HELLO, HOW, ARE, YOU, Q], [], [])])
    pool.commit(r1)
    assert pool.cached_pages() == 2                 # [Hello How] [are you]; "?" sits on a partial block
    r2 = pool.plan([([HELLO, HOW, ARE, YOU, Q, I, AM, FINE], [], [])])
    hit_tokens = r2.queries[0].prefix.n_hit * 2
    assert hit_tokens == 4                          # 4 of the 5 context tokens (80%)
    assert r2.queries[0].prefix.page_ids[:2] == r1.queries[0].prefix.page_ids[:2]


def _rag_queries(order):
    prefix = list(range(1000, 1037))
    frags = [list(range(2000 + 100 * f, 2000 + 100 * f + 40 + 9 * f)) for f in range(3)]
    return [(prefix, [frags[i] for i in order], list(range(5000, 5019)))]


def test_paper_rag_example_stock_vs_span():
    stock = PoolReplay(num_pages=64, page_size=16, stock=True)
    a = stock.plan([(p + [t for f in fs for t in f], [], []) for p, fs, _ in _rag_queries([0, 1, 2])])
    stock.commit(a)
    b = stock.plan([(p + [t for f in fs for t in f], [], []) for p, fs, _ in _rag_queries([2, 1, 0])])
    assert b.queries[0].prefix.n_hit == 37 // 16     # only whole prefix pages before the first fragment

    span = PoolReplay(num_pages=64, page_size=16)
    a = span.plan(_rag_queries([0, 1, 2]))
    span.commit(a)
    b = span.plan(_rag_queries([2, 1, 0]))
    qa, qb = a.queries[0], b.queries[0]
    assert qb.prefix.n_hit == len(qb.prefix.page_ids)
    for child_b, f in enumerate([2, 1, 0]):
        assert qb.frags[child_b].n_hit == len(qb.frags[child_b].page_ids)
        assert qb.frags[child_b].page_ids == qa.frags[f].page_ids
    # cross pages are fresh every time, never cached
    assert set(qb.cross.page_ids).isdisjoint(span.index.values())


def test_dedup_inside_one_plan():
    pool = PoolReplay(num_pages=64, page_size=16)
    qs = _rag_queries([0, 1, 2]) + _rag_queries([1, 2, 0])
    r = pool.plan(qs)
    a, b = r.queries
    assert b.prefix.page_ids == a.prefix.page_ids and b.prefix.n_hit == len(b.prefix.page_ids)
    assert b.frags[0].page_ids == a.frags[1].page_ids
    # distinct pages: prefix 3 + fragments (3 + 4 + 4) + 2 x cross 2
    assert len(r.new_pages) == 3 + 3 + 4 + 4 + 2 + 2
    assert len(set(r.new_pages)) == len(r.new_pages)
    assert r.new_pages == sorted(r.new_pages) == list(range(len(r.new_pages)))


def _survivors_are_prefixes(pool):
    # walk every published page back to its span start: each parent must be published too
    hashes = {p.hash for p in pool.pages.values() if p.published}
    for p in pool.pages.values():
        if p.published and p.idx > 0:
            assert p.parent in hashes, "a cached page whose predecessor was evicted"


@pytest.mark.parametrize("seed", range(6))
def test_lru_stream_properties(seed):
    rnd = random.Random(seed)
    ps = 4
    prefixes = [[rnd.randrange(50) for _ in range(rnd.randrange(0, 9))] for _ in range(2)]
    frags = [[rnd.randrange(50) for _ in range(rnd.randrange(1, 14))] for _ in range(8)]
    pool = PoolReplay(num_pages=rnd.randrange(8, 30), page_size=ps)
    for step in range(40):
        qs = []
        for _ in range(rnd.randrange(1, 3)):
            pre = prefixes[rnd.randrange(2)]
            chosen = rnd.sample(range(8), rnd.randrange(0, 4))
            qs.append((pre, [frags[i] for i in chosen], [rnd.randrange(50) for _ in range(rnd.randrange(0, 6))]))
        before = (dict(pool.index), list(pool.free), pool.tick,
                  {k: (v.pins, v.last_use) for k, v in pool.pages.items()})
        evictable_before = [p for p in pool.pages.values() if p.published and p.pins == 0]
        try:
            r = pool.plan(qs)
        except PoolFull:
            after = (dict(pool.index), list(pool.free), pool.tick,
                     {k: (v.pins, v.last_use) for k, v in pool.pages.items()})
            assert before == after
            continue
        # capacity rule: the plan fitted into free + evictable pages
        assert len(r.new_pages) <= len(before[1]) + len(evictable_before)
        # evictions happen only once the free list is empty, oldest tick first
        if r.evicted:
            assert len(r.new_pages) > len(before[1])
            ticks = [before[3][pid][1] for pid in r.evicted]
            survivors = [p.last_use for p in evictable_before
                         if p.page_id not in r.evicted and p.page_id not in r.hits]
            assert max(ticks) <= min(survivors + [10 ** 9])
        # pages touched by this plan are pinned and stamped with its tick
        for pid in r.hits + r.new_pages:
            assert pool.pages[pid].last_use == r.tick and pool.pages[pid].pins >= 1
        if rnd.random() < 0.85:
            pool.commit(r)
        else:
            pool.destroy(r)
        _survivors_are_prefixes(pool)
        assert len(pool.free) + len(pool.pages) == pool.num_pages


@pytest.mark.parametrize("seed", range(6))
def test_heap_victims_equal_brute_force(seed):
    """The heap-based victim search returns what the rule's definition (the minimum
    key over all evictable pages) returns, on streams with many evictions."""
    rnd = random.Random(100 + seed)
    ps = 4
    prefixes = [[rnd.randrange(40) for _ in range(rnd.randrange(0, 9))] for _ in range(3)]
    frags = [[rnd.randrange(40) for _ in range(rnd.randrange(1, 18))] for _ in range(12)]
    n_pages = rnd.randrange(10, 24)
    fast, slow = PoolReplay(n_pages, ps), PoolReplay(n_pages, ps, brute_force=True)
    evictions = 0
    for step in range(120):
        qs = []
        for _ in range(rnd.randrange(1, 3)):
            chosen = rnd.sample(range(12), rnd.randrange(0, 4))
            qs.append((prefixes[rnd.randrange(3)], [frags[i] for i in chosen],
                       [rnd.randrange(40) for _ in range(rnd.randrange(0, 6))]))
        outs = []
        for pool in (fast, slow):
            try:
                outs.append(pool.plan(qs))
            except PoolFull:
                outs.append(None)
        a, b = outs
        assert (a is None) == (b is None)
        if a is None:
            continue
        assert a.evicted == b.evicted and a.new_pages == b.new_pages and a.hits == b.hits
        for qa, qb in zip(a.queries, b.queries):
            assert qa == qb
        evictions += len(a.evicted)
        if rnd.random() < 0.85:
            fast.commit(a)
            slow.commit(b)
        else:
            fast.destroy(a)
            slow.destroy(b)
    assert evictions > 20
