"""Materialised repositioning, the alternative to rotating cached keys at read time.

Section 5.5 uses a cached block at another position by rotating its keys again:
CIDRA writes such re-rotated blocks into the cache before attention, in place,
duplicating a block that concurrent requests need at two positions.  A pool
created with SPAN_FLAG_MATERIALIZE does the same, out of place: each page that a
query's cross rows read at a shifted position (final minus canonical position of a
fragment) gets one transient copy per distinct shift, its keys rotated to the final
positions, its values copied; the cross rows then read the copies unrotated.

Host logic (no GPU): the copies the planner makes are exactly the distinct
(page, shift != 0) pairs of the cross rows' block tables, they are fresh pages,
freed at commit and destroy, counted in the capacity check, and they change nothing
else the planner decides.
GPU (marked gpu): the copies hold the oracle's keys at the final positions and the
values unchanged; the cross rows match the oracle, as with read-time rotation.
"""
import dataclasses
import random
from types import SimpleNamespace

import numpy as np
import pytest

import paper_2511_02749_amd as spanq
import workloads as W
from oracle import attention as OA
from tests.helpers import TOL, GpuRun, check_rows, query_layout, query_rows


def _span(tokens, row=0):
    return SimpleNamespace(tokens=np.asarray(tokens, np.int32), row=row)


def _host_pool(n_pages, materialize=True):
    return spanq.Pool(num_q_heads=8, num_kv_heads=2, head_dim=128, num_pages=n_pages, device=-1,
                      materialize=materialize)


def _expected_moves(plan, queries):
    """Distinct (page, shift) pairs, in query / fragment / page order, of fragments that
    cross rows read at a shifted position."""
    want, seen = [], set()
    for qi, q in enumerate(queries):
        if q.cross.tokens.size == 0:
            continue
        shift = 0
        for c, f in enumerate(q.frags):
            ids, _ = plan.block_table(qi, c)
            if shift:
                for pg, pid in enumerate(ids):
                    if (pid, shift) not in seen:
                        seen.add((pid, shift))
                        want.append((pid, shift, min(16, f.tokens.size - 16 * pg)))
            shift += f.tokens.size
    return want


def _random_batch(rng, frags, prefixes, n_queries):
    qs = []
    for _ in range(n_queries):
        pre = prefixes[rng.randrange(len(prefixes))]
        k = rng.randrange(0, 5)
        chosen = [frags[rng.randrange(len(frags))] for _ in range(k)]
        cross = list(range(7000, 7000 + rng.choice([0, 1, 9, 16, 40])))
        qs.append(SimpleNamespace(prefix=_span(pre), frags=[_span(f) for f in chosen], cross=_span(cross)))
    return qs


def _stream(seed):
    rng = random.Random(seed)
    frags = [list(range(1000 * (i + 1), 1000 * (i + 1) + rng.choice([1, 15, 16, 17, 40, 64]))) for i in range(8)]
    prefixes = [[], list(range(500, 520)), list(range(600, 632))]
    return [_random_batch(rng, frags, prefixes, rng.randrange(1, 4)) for _ in range(25)]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_moves_are_the_shifted_pages_of_cross_reads(seed):
    pool = _host_pool(4096)
    for batch in _stream(seed):
        before = pool.info()
        plan = pool.plan(batch)
        moves = plan.moves()
        want = _expected_moves(plan, batch)
        assert [(m[0], m[2], m[3]) for m in moves] == want
        st = plan.stats()
        assert st["pages_moved"] == len(moves) and st["tokens_moved"] == sum(m[3] for m in moves)
        dst = [m[1] for m in moves]
        assert len(set(dst)) == len(dst)
        used = set()
        for qi, q in enumerate(batch):
            for c in range(-1, len(q.frags) + 1):
                used.update(plan.block_table(qi, c)[0])
        assert not used & set(dst)                          # fresh pages, not in any block table
        info = pool.info()
        assert before["free_pages"] - info["free_pages"] == st["pages_new"] + st["pages_cross"] + len(moves)
        assert info["pinned_pages"] >= len(moves)
        plan.commit()
        plan.destroy()
        after = pool.info()
        assert after["pinned_pages"] == 0
        assert after["free_pages"] == after["num_pages"] - after["cached_pages"]   # copies were freed
    pool.close()


@pytest.mark.parametrize("seed", [3, 4])
def test_materialize_changes_no_other_decision(seed):
    """The same stream on a roomy pool with and without the flag: the same block tables,
    hit counts and cached pages (the copies are allocated last and freed at commit)."""
    pools = [_host_pool(4096, materialize=m) for m in (False, True)]
    for batch in _stream(seed):
        plans = [p.plan(batch) for p in pools]
        for qi, q in enumerate(batch):
            for c in range(-1, len(q.frags) + 1):
                assert plans[0].block_table(qi, c) == plans[1].block_table(qi, c)
        assert plans[0].moves() == []
        for p in plans:
            p.commit()
            p.destroy()
        assert pools[0].info()["cached_pages"] == pools[1].info()["cached_pages"]
    for p in pools:
        p.close()


def test_no_moves_without_a_shift_or_a_cross_segment():
    pool = _host_pool(256)
    a, b = list(range(100, 140)), list(range(200, 233))
    one = SimpleNamespace(prefix=_span(range(20)), frags=[_span(a)], cross=_span([9] * 5))
    no_cross = SimpleNamespace(prefix=_span(range(20)), frags=[_span(a), _span(b)], cross=_span([]))
    p = pool.plan([one, no_cross])
    assert p.moves() == []                                  # first fragment: final == canonical
    p.commit(); p.destroy()
    two = SimpleNamespace(prefix=_span(range(20)), frags=[_span(b), _span(a), _span(b)], cross=_span([9]))
    p = pool.plan([two, two])                               # the same query twice: copies shared
    mv = p.moves()
    ids_a, _ = p.block_table(0, 1)
    ids_b, _ = p.block_table(0, 2)
    assert [(m[0], m[2]) for m in mv] == [(x, 33) for x in ids_a] + [(x, 73) for x in ids_b]
    p.destroy()
    pool.close()


def test_a_page_at_two_shifts_is_copied_twice():
    pool = _host_pool(256)
    a, b, c = list(range(100, 132)), list(range(200, 216)), list(range(300, 348))
    q1 = SimpleNamespace(prefix=_span([]), frags=[_span(b), _span(a)], cross=_span([1]))
    q2 = SimpleNamespace(prefix=_span([]), frags=[_span(c), _span(a)], cross=_span([1]))
    p = pool.plan([q1, q2])
    ids_a, _ = p.block_table(0, 1)
    assert p.block_table(1, 1)[0] == ids_a                   # one cached copy of fragment a
    assert [(m[0], m[2]) for m in p.moves()] == [(x, 16) for x in ids_a] + [(x, 48) for x in ids_a]
    p.destroy()
    pool.close()


def test_copies_count_in_the_capacity_check():
    a, b = list(range(100, 164)), list(range(200, 264))      # 4 pages each
    q = SimpleNamespace(prefix=_span([]), frags=[_span(a), _span(b)], cross=_span([5] * 16))
    for materialize, fits in ((False, True), (True, False)):
        pool = _host_pool(9, materialize=materialize)        # 4 + 4 + 1 cross; + 4 copies of b
        before = pool.info()
        if fits:
            pool.plan([q]).destroy()
        else:
            with pytest.raises(spanq.SpanError) as ei:
                pool.plan([q])
            assert ei.value.code == -2 and pool.info() == before
        pool.close()
    pool = _host_pool(13)
    p = pool.plan([q])
    assert len(p.moves()) == 4 and pool.info()["free_pages"] == 0
    p.destroy()
    pool.close()


# ---------------------------------------------------------------------------- GPU


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(flush=True)
    return torch


def _page(run, layer, page_id):
    raw = run.pool.read_page(layer, page_id)
    if run.wl.dtype == "bf16":
        raw = (raw.astype(np.uint32) << 16).view(np.float32)
    hkv, d = run.wl.n_kv_heads, run.wl.head_dim
    k = raw[: hkv * 16 * d].reshape(hkv, 16, d)
    vt = raw[hkv * 16 * d:].reshape(hkv, d, 16)
    vpos = [(s & 3) | ((s & 4) << 1) | ((s & 8) >> 1) for s in range(16)]
    return k, vt[:, :, vpos].transpose(0, 2, 1)


def _check_copies(run, plan, batch, layer=0):
    """Every copy against the oracle: keys rotated at the final positions, within two
    roundings to the pool's type of the pair's norm (the cached key was rounded once at
    its canonical position, the copy once more); values equal; unfilled slots zero."""
    moves = {m[1]: m for m in plan.moves()}
    seen = set()
    bf16 = run.wl.dtype == "bf16"
    for qi, q in enumerate(batch):
        if q.cross.n == 0:
            continue
        lay = query_layout(q)
        rows = query_rows(q)
        for c, f in enumerate(q.frags):
            sel = np.nonzero(lay.seg == c)[0]
            if lay.pos_final[sel[0]] == lay.pos_canon[sel[0]]:
                continue
            kf = OA.rope(np.asarray(run.wl.k[rows[sel]], np.float64), lay.pos_final[sel], run.wl.rope_theta)
            vf = np.asarray(run.wl.v[rows[sel]], np.float64)
            ids, _ = plan.block_table(qi, c)
            shift = int(lay.pos_final[sel[0]] - lay.pos_canon[sel[0]])
            copies = [d for d, m in moves.items() if m[2] == shift and m[0] in ids]
            assert len(copies) == len(ids)
            for pg, pid in enumerate(ids):
                dst = next(d for d in copies if moves[d][0] == pid)
                seen.add(dst)
                k, v = _page(run, layer, dst)
                n = min(16, f.n - 16 * pg)
                kr = kf[16 * pg: 16 * pg + n].transpose(1, 0, 2)          # [hkv, n, d]
                h = kr.shape[-1] // 2
                norm = np.sqrt(kr[..., :h] ** 2 + kr[..., h:] ** 2)
                norm = np.concatenate([norm, norm], axis=-1)
                rtol = 2.0 ** -7 if bf16 else 2.0 ** -20
                assert np.all(np.abs(k[:, :n] - kr) <= rtol * norm + 1e-6)
                np.testing.assert_array_equal(v[:, :n], vf[16 * pg: 16 * pg + n].transpose(1, 0, 2))
                assert not np.any(k[:, n:]) and not np.any(v[:, n:])
    assert seen == set(moves)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,kernel", [("bf16", "auto"), ("bf16", "generic"), ("f32", "generic")])
def test_materialized_cross_matches_oracle(dtype, kernel):
    _need_gpu()
    wl = W.small_workload(dtype=dtype, orders=[[0, 1, 2, 3], [3, 1, 0, 2], [2, 0, 3, 1]], n_queries=3,
                          frags_per_query=4, batch_split=[1, 2])
    run = GpuRun(wl, kernel=kernel, materialize=True)
    read = GpuRun(wl, kernel=kernel)
    for bi, batch in enumerate(wl.batches):
        plan = run.run_batch(batch, commit=False)
        ref = read.run_batch(batch)
        if bi == 1:
            assert plan.stats()["tokens_new"] == 0 and plan.stats()["pages_moved"] > 0
        _check_copies(run, plan, batch)
        _, cross = plan.rows()
        check_rows(run, batch, cross, TOL[dtype])
        print(f"{dtype} {kernel} batch {bi}: {len(plan.moves())} copies; materialised vs read-time rotation "
              f"max |diff| {float(np.max(np.abs(run.out_rows(cross) - read.out_rows(cross)))):.3g}", flush=True)
        plan.commit()
        plan.destroy()
    run.close()
    read.close()


@pytest.mark.gpu
def test_materialized_per_layer_copies():
    """A two-layer pool: the same activations at both layers give the same copies in
    both slabs and the same cross rows."""
    torch = _need_gpu()
    wl = W.small_workload(orders=[[0, 1, 2, 3], [3, 2, 1, 0]], n_queries=2, frags_per_query=4, batch_split=[1, 1])
    run = GpuRun(wl, num_layers=2, materialize=True)
    outs = []
    for bi, batch in enumerate(wl.batches):
        plan = run.pool.plan(batch)
        per_layer = []
        for layer in (0, 1):
            plan.prefill(layer, run.q, run.k, run.v, run.out)
            plan.cross(layer, run.q, run.k, run.v, run.out)
            torch.cuda.synchronize()
            _, cross = plan.rows()
            per_layer.append(run.out_rows(cross))
        assert np.array_equal(per_layer[0], per_layer[1])
        for _, dst, _, _ in plan.moves():
            assert np.array_equal(run.pool.read_page(0, dst), run.pool.read_page(1, dst))
        if bi == 1:
            _check_copies(run, plan, batch, layer=1)
            check_rows(run, batch, cross, TOL["bf16"])
        plan.commit()
        plan.destroy()
    run.close()


@pytest.mark.gpu
def test_c2_warm_query_materialized():
    """The RAG batch's first query with its 16 cached fragments in reverse order: 15
    fragments shifted, 480 copies.  Copies and every cross row against the oracle."""
    _need_gpu()
    wl = W.config_c2()
    q0 = wl.batches[0][0]
    rev = W.Query(prefix=q0.prefix, frags=q0.frags[::-1], cross=q0.cross)
    run = GpuRun(dataclasses.replace(wl, batches=[[q0], [rev]]), materialize=True)
    run.run_batch([q0])
    plan = run.run_batch([rev], commit=False)
    st = plan.stats()
    assert st["tokens_new"] == 0 and st["pages_moved"] == 15 * 32
    _check_copies(run, plan, [rev])
    _, cross = plan.rows()
    check_rows(run, [rev], cross, TOL["bf16"])
    plan.destroy()
    run.close()
