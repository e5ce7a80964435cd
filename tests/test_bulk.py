"""Bulk scheduling (section 5.8): span_bulk_order clusters the queries of a bulk so
that fragment reuse is close in time.  Checked: the order is a permutation and
deterministic; on a bulk that alternates two fragment sets with room for one, it
groups them; on the C5 stream at the 48 GB cap it raises the planner's hit rate
over the given order (the reordered stream is still planned bit for bit like the
oracle's replay)."""
import numpy as np
import pytest

import workloads as W
from oracle.pool import PoolReplay
from tests.helpers import assert_tables_match, replay_queries

spanq = pytest.importorskip("paper_2511_02749_amd")


def _pool(pages, layers=1):
    try:
        spanq.load()
    except FileNotFoundError:
        pytest.skip("libspanq.so not built")
    return spanq.Pool(num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=pages, dtype="bf16", num_layers=layers,
                      device=-1)


def _q(prefix, frags, cross_seed):
    rng = np.random.default_rng(cross_seed)
    return W.Query(prefix=W.Span(tokens=prefix, row=0), frags=[W.Span(tokens=f, row=0) for f in frags],
                   cross=W.Span(tokens=rng.integers(0, 1000, 8).astype(np.int32), row=0))


def _run(pool, queries, order, replay=None):
    hit = tot = 0
    for i in order:
        plan = pool.plan([queries[i]])
        if replay is not None:
            res = replay.plan(replay_queries([queries[i]]))
            assert_tables_match(plan, res, [queries[i]])
            replay.commit(res)
        st = plan.stats()
        hit += st["tokens_hit"]
        tot += st["tokens_hit"] + st["tokens_new"]
        plan.commit()
        plan.destroy()
    return hit / tot


def test_groups_alternating_fragment_sets():
    rng = np.random.default_rng(1)
    prefix = rng.integers(0, 1000, 16).astype(np.int32)
    a, b, c, d = (rng.integers(0, 1000, 64).astype(np.int32) for _ in range(4))
    qs = [_q(prefix, [a, b], i) if i % 2 == 0 else _q(prefix, [c, d], i) for i in range(8)]
    pool = _pool(1 + 8 + 2)   # prefix + one pair of fragments + the cross page
    order = pool.bulk_order(qs)
    assert sorted(order) == list(range(8)) and order == pool.bulk_order(qs)
    assert order == [0, 2, 4, 6, 1, 3, 5, 7]
    given = _run(pool, qs, range(8))
    pool.reset()
    clustered = _run(pool, qs, order)
    assert clustered > given
    pool.close()


@pytest.mark.slow
def test_c5_stream_bulk_order_raises_hit_rate():
    stream = W.c5_stream()
    qs = [s.query for s in stream]
    pages = 22_888
    pool = _pool(pages, layers=32)
    given = _run(pool, qs, range(len(qs)))
    pool.close()
    pool = _pool(pages, layers=32)
    order = pool.bulk_order(qs)
    assert sorted(order) == list(range(len(qs)))
    whole = _run(pool, qs, order, replay=PoolReplay(pages))
    pool.close()
    # bulks of 32 queries, each ordered against the pool as the previous bulks left it
    pool = _pool(pages, layers=32)
    hit = tot = 0
    for b0 in range(0, len(qs), 32):
        chunk = qs[b0: b0 + 32]
        for i in pool.bulk_order(chunk):
            plan = pool.plan([chunk[i]])
            st = plan.stats()
            hit += st["tokens_hit"]
            tot += st["tokens_hit"] + st["tokens_new"]
            plan.commit()
            plan.destroy()
    pool.close()
    print(f"C5 at 48 GB: hit rate given order {given:.4f}, bulks of 32 {hit / tot:.4f}, whole stream {whole:.4f}")
    assert whole > given and hit / tot >= given
