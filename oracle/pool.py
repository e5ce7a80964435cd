"""Replay of the page cache's bookkeeping (lookup, dedup, allocation, LRU).

Rules, from the paper where it speaks and from the stated readings where it
does not:

* Lookup (section 2): walk a span's pages in order and stop at the first page
  whose hash is not cached (prefix-only lookup), applied per span (section
  5.4), so a fragment hits whatever position it takes in a query.  A hash hit
  also compares the stored page content (tokens, length, index, parent hash);
  a mismatch is a miss.
* Dedup: inside one plan, a page already scheduled for computation by an
  earlier span (earlier query, then earlier child) is a hit for later spans.
* Allocation: the lowest free page id.  With no free page, evict the cached,
  unpinned page with the smallest (last use, -index in span, page id): least
  recently used first and, inside a span, tail pages first, so the surviving
  pages of a span always form a prefix of it.
* Capacity is checked before anything changes: a plan that needs more pages
  than are free or evictable fails with no effect.
* Every successful plan is one LRU tick; pages it hits or allocates take that
  tick as last use.  Pages a plan uses stay pinned until commit (cache pages)
  or destroy (cross pages, which are never published).
* Commit publishes new cache pages (a hash that is already published is not
  published again and its new page is freed), then unpins.
* Stock mode (section 2, the chat example): one chain over the whole prompt,
  trailing partial page never cached.

Parity unpinned: the eviction order is this library's choice (the paper does
not fix one); pinned by brute-force LRU checks and the paper's chat example.
"""
from __future__ import annotations

import heapq
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

from . import hashing


class PoolFull(Exception):
    pass


@dataclass
class PageInfo:
    page_id: int
    hash: int
    parent: int
    tokens: tuple
    idx: int
    last_use: int = 0
    pins: int = 0
    published: bool = False
    cacheable: bool = True


@dataclass
class SpanResult:
    page_ids: List[int]
    n_hit: int


@dataclass
class QueryResult:
    prefix: SpanResult
    frags: List[SpanResult]
    cross: SpanResult


@dataclass
class PlanResult:
    queries: List[QueryResult]
    evicted: List[int]
    new_pages: List[int]          # allocation order (cache pages and cross pages)
    cross_pages: List[int]
    tick: int
    hits: List[int] = field(default_factory=list)
    committed: bool = False
    destroyed: bool = False


class PoolReplay:
    """Replay of the page cache.  The eviction victim is the evictable page with the
    smallest key (last use, -index in span, page id).  ``brute_force`` takes that
    minimum over every evictable page at each eviction (the rule as stated); the
    default pops it from a heap of keys with stale entries skipped, which gives the
    same victims (pinned against brute force in the tests) in time fit for long
    streams."""

    def __init__(self, num_pages: int, page_size: int = 16, stock: bool = False, brute_force: bool = False):
        self.num_pages = num_pages
        self.page_size = page_size
        self.stock = stock
        self.brute_force = brute_force
        self.free: List[int] = list(range(num_pages))
        heapq.heapify(self.free)
        self.index: Dict[int, int] = {}
        self.pages: Dict[int, PageInfo] = {}
        self.tick = 0
        self.evictable_keys: Dict[int, tuple] = {}   # published, unpinned pages -> their key
        self._heap: List[tuple] = []

    # --- helpers -------------------------------------------------------
    def _evictable(self):
        return [self.pages[pid] for pid in self.evictable_keys]

    def _refresh(self, p: PageInfo):
        """Record whether p is evictable (published and unpinned), with its current key."""
        if p.published and p.pins == 0:
            key = (p.last_use, -p.idx, p.page_id)
            if self.evictable_keys.get(p.page_id) != key:
                self.evictable_keys[p.page_id] = key
                heapq.heappush(self._heap, key)
        else:
            self.evictable_keys.pop(p.page_id, None)

    def _victim(self) -> int:
        if self.brute_force:
            return min(self.evictable_keys.values())[2]
        while True:
            key = self._heap[0]
            if self.evictable_keys.get(key[2]) == key:
                return key[2]
            heapq.heappop(self._heap)

    def _lookup(self, h: int, parent: int, toks: tuple, idx: int) -> Optional[int]:
        pid = self.index.get(h)
        if pid is None:
            return None
        p = self.pages[pid]
        if p.tokens != toks or p.idx != idx or p.parent != parent:
            return None
        return pid

    def _span_pages(self, seed: int, tokens: Sequence[int], include_partial: bool):
        """[(hash, parent, tokens, idx, cacheable)] for the pages of a span."""
        ps = self.page_size
        out, h = [], seed
        n = len(tokens)
        for p in range((n + ps - 1) // ps):
            toks = tuple(int(t) for t in tokens[p * ps: (p + 1) * ps])
            full = len(toks) == ps
            nh = hashing.page_hash(h, toks, p)
            out.append((nh, h, toks, p, full or include_partial))
            h = nh
        return out

    # --- plan ----------------------------------------------------------
    def plan(self, queries) -> PlanResult:
        """queries: list of (prefix_tokens, [fragment tokens...], cross_tokens)."""
        tick = self.tick + 1
        pending: Dict[int, int] = {}          # hash -> pending slot
        walk = []                             # per query: list of spans; span = list of ("hit", pid) / ("new", slot)
        new_specs = []                        # slot -> (hash, parent, toks, idx, cacheable, is_cross)
        for prefix, frags, cross in queries:
            if self.stock:
                spans_in = [(hashing.ROOT_SEED, list(prefix) + [t for f in frags for t in f] + list(cross), False)]
            else:
                ph = hashing.chain(hashing.ROOT_SEED, prefix, self.page_size)
                fs = hashing.fragment_seed(ph)
                spans_in = [(hashing.ROOT_SEED, prefix, True)] + [(fs, f, True) for f in frags]
            spans = []
            for seed, toks, partial_ok in spans_in:
                entries, missed = [], False
                for (h, parent, pt, idx, cacheable) in self._span_pages(seed, toks, partial_ok):
                    if not missed and cacheable:
                        if h in pending:
                            spec = new_specs[pending[h]]
                            if spec[2] == pt and spec[3] == idx and spec[1] == parent:
                                entries.append(("new", pending[h], True))
                                continue
                        pid = self._lookup(h, parent, pt, idx)
                        if pid is not None:
                            entries.append(("hit", pid, True))
                            continue
                    missed = True
                    slot = len(new_specs)
                    new_specs.append((h, parent, pt, idx, cacheable, False))
                    if cacheable and h not in pending:
                        pending[h] = slot
                    entries.append(("new", slot, False))
                spans.append(entries)
            ncross = (len(cross) + self.page_size - 1) // self.page_size if not self.stock else 0
            cross_slots = []
            for p in range(ncross):
                slot = len(new_specs)
                new_specs.append((0, 0, (), p, False, True))
                cross_slots.append(slot)
            walk.append((spans, cross_slots))

        hit_pids = []
        for spans, _ in walk:
            for entries in spans:
                for kind, x, _ in entries:
                    if kind == "hit" and x not in hit_pids:
                        hit_pids.append(x)
        need = len(new_specs)
        n_evictable = len(self.evictable_keys) - sum(1 for pid in hit_pids if pid in self.evictable_keys)
        if need > len(self.free) + n_evictable:
            raise PoolFull(f"need {need} pages, {len(self.free)} free, {n_evictable} evictable")

        # mutate
        self.tick = tick
        for pid in hit_pids:
            p = self.pages[pid]
            p.pins += 1
            p.last_use = tick
            self._refresh(p)
        evicted = []
        slot_pid: Dict[int, int] = {}
        order = []
        for spans, cross_slots in walk:
            for entries in spans:
                for kind, x, dup in entries:
                    if kind == "new" and not dup:
                        order.append(x)
            order.extend(cross_slots)
        for slot in order:
            if not self.free:
                v = self.pages[self._victim()]
                del self.evictable_keys[v.page_id]
                del self.index[v.hash]
                del self.pages[v.page_id]
                evicted.append(v.page_id)
                heapq.heappush(self.free, v.page_id)
            pid = heapq.heappop(self.free)
            h, parent, pt, idx, cacheable, is_cross = new_specs[slot]
            self.pages[pid] = PageInfo(page_id=pid, hash=h, parent=parent, tokens=pt, idx=idx,
                                       last_use=tick, pins=1, published=False,
                                       cacheable=cacheable and not is_cross)
            slot_pid[slot] = pid

        qres = []
        for spans, cross_slots in walk:
            srs = []
            for entries in spans:
                ids = [x if kind == "hit" else slot_pid[x] for kind, x, _ in entries]
                nhit = 0
                for kind, x, dup in entries:
                    if kind == "hit" or dup:
                        nhit += 1
                    else:
                        break
                srs.append(SpanResult(page_ids=ids, n_hit=nhit))
            if self.stock:
                prefix_res, frag_res = srs[0], []
            else:
                prefix_res, frag_res = srs[0], srs[1:]
            qres.append(QueryResult(prefix=prefix_res, frags=frag_res,
                                    cross=SpanResult(page_ids=[slot_pid[s] for s in cross_slots], n_hit=0)))
        cross_pages = [slot_pid[s] for _, cs in walk for s in cs]
        return PlanResult(queries=qres, evicted=evicted, new_pages=[slot_pid[s] for s in order],
                          cross_pages=cross_pages, tick=tick, hits=hit_pids)

    def commit(self, plan: PlanResult):
        cross = set(plan.cross_pages)
        for pid in plan.new_pages:
            p = self.pages[pid]
            if pid in cross or not p.cacheable or p.hash in self.index:
                continue
            self.index[p.hash] = pid
            p.published = True
        for pid in plan.new_pages:
            p = self.pages[pid]
            p.pins -= 1
            if not p.published:
                del self.pages[pid]
                heapq.heappush(self.free, pid)
            else:
                self._refresh(p)
        for pid in plan.hits:
            self.pages[pid].pins -= 1
            self._refresh(self.pages[pid])
        plan.committed = True

    def destroy(self, plan: PlanResult):
        """Release a plan that was never committed."""
        if plan.committed:
            return
        for pid in plan.new_pages:
            del self.pages[pid]
            heapq.heappush(self.free, pid)
        for pid in plan.hits:
            self.pages[pid].pins -= 1
            self._refresh(self.pages[pid])
        plan.destroyed = True

    def cached_pages(self) -> int:
        return len(self.index)
