"""The C5 agentic stream through the library's planner on the CPU (host-only pools),
bit for bit against the oracle's pool replay.

256 span queries over a 1024-fragment pool (lengths uniform on 128..2048, Zipf 1.1
popularity, 4 to 24 fragments per query, one shared 256-token prefix, 128-token
cross segments), planned one query at a time, at the two pool sizes the GPU run
uses: 200 GB (95,367 pages of 2 MiB, all 32 layers: nothing is evicted) and a 48 GB
cap (22,888 pages: LRU eviction, tail pages first).  Block tables, hit counts and
eviction lists must match for every query; the hit rate (hit prefix and fragment
tokens over all prefix and fragment tokens) is reported.
"""
import numpy as np
import pytest

import workloads as W
from oracle.pool import PoolReplay
from tests.helpers import assert_tables_match, replay_queries

spanq = pytest.importorskip("paper_2511_02749_amd")

PAGES_200GB = 95_367
PAGES_48GB = 22_888


@pytest.fixture(scope="module")
def stream():
    return W.c5_stream()


@pytest.mark.slow
@pytest.mark.parametrize("num_pages", [PAGES_200GB, PAGES_48GB], ids=["200GB", "48GB"])
def test_c5_stream_plans_match_oracle(stream, num_pages):
    try:
        spanq.load()
    except FileNotFoundError:
        pytest.skip("libspanq.so not built")
    pool = spanq.Pool(num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=num_pages, dtype="bf16",
                      num_layers=32, device=-1)
    replay = PoolReplay(num_pages)
    hit = total = evicted = 0
    for sq in stream:
        batch = [sq.query]
        plan = pool.plan(batch)
        res = replay.plan(replay_queries(batch))
        assert_tables_match(plan, res, batch)
        st = plan.stats()
        hit += st["tokens_hit"]
        total += st["tokens_hit"] + st["tokens_new"]
        evicted += len(res.evicted)
        plan.commit()
        replay.commit(res)
        plan.destroy()
    info = pool.info()
    assert info["cached_pages"] == replay.cached_pages() and info["total_evictions"] == evicted
    print(f"{num_pages} pages: hit rate {hit / total:.4f}, evictions {evicted}, cached {info['cached_pages']}")
    if num_pages == PAGES_200GB:
        assert evicted == 0
    else:
        assert evicted > 0
    pool.close()
