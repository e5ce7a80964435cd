"""GPU parity: the HIP path through the C-ABI against the oracle, element by element.

Tolerances (max abs error against the float64 oracle run on the same rounded
inputs): 2e-2 for bf16 pools, 1e-4 for fp32 pools.  Page ids / hits are
checked bit-exactly elsewhere (host tests); here the page *contents* and the
attention outputs are checked, plus the two bit-identity invariants: a
fragment's cached KV does not depend on the order it was first seen in, and
cross output over reused pages equals a cold recompute.
"""
import numpy as np
import pytest

import workloads as W
from oracle import attention as OA
from tests.helpers import (TOL, GpuRun, check_rows, computed_rows, max_err, oracle_rows, query_layout,
                           query_rows)

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(flush=True)


_computed_rows = computed_rows
_check_rows = check_rows


@pytest.mark.parametrize("mode", ["proj", "direct"])
def test_c1_cold_then_permuted_hits(mode):
    wl = W.config_c1(mode=mode)
    run = GpuRun(wl)
    a = run.run_batch(wl.batches[0])
    sa = a.stats()
    assert sa["tokens_hit"] == 0 and sa["tokens_new"] == 32 + 4 * 64
    _check_rows(run, wl.batches[0], _computed_rows(a), TOL["f32"])
    b = run.run_batch(wl.batches[1])
    sb = b.stats()
    assert sb["tokens_new"] == 0 and sb["tokens_hit"] == 32 + 4 * 64 and sb["tokens_cross"] == 16
    pre, cross = b.rows()
    assert pre.size == 0 and cross.size == 16
    _check_rows(run, wl.batches[1], cross, TOL["f32"])
    run.close()


SMALL = [
    dict(name="ragged", head_dim=128, n_q_heads=8, n_kv_heads=2),
    dict(name="d64", head_dim=64, n_q_heads=8, n_kv_heads=2),
    dict(name="mha", head_dim=128, n_q_heads=4, n_kv_heads=4),
    dict(name="g2", head_dim=128, n_q_heads=8, n_kv_heads=4),
    dict(name="g8", head_dim=128, n_q_heads=16, n_kv_heads=2),
    dict(name="g8d64", head_dim=64, n_q_heads=16, n_kv_heads=2, cross_len=70),
    dict(name="noprefix", prefix_len=0, frag_lens=(16, 1, 77, 130), cross_len=40),
    dict(name="nocross", cross_len=0),
    dict(name="bigtiles", prefix_len=100, frag_lens=(300, 129, 64), frags_per_query=3, cross_len=150),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kernel", ["generic", "auto"])
@pytest.mark.parametrize("case", SMALL, ids=[c["name"] for c in SMALL])
def test_small_ragged(case, dtype, kernel):
    case = dict(case)
    case.pop("name")
    wl = W.small_workload(dtype=dtype, **case)
    run = GpuRun(wl, kernel=kernel)
    plan = run.run_batch(wl.batches[0])
    _check_rows(run, wl.batches[0], _computed_rows(plan), TOL[dtype])
    run.close()


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("cross_len", [1, 9, 16])
def test_few_row_cross_tiles(head_dim, cross_len):
    """Cross segments of at most 16 rows take the 16-row kernel (four query heads per
    kv head); ragged fragments make partial pages, and every fragment is read at a
    position other than the one it was written at."""
    wl = W.small_workload(head_dim=head_dim, cross_len=cross_len, n_queries=3)
    run = GpuRun(wl)
    plan = run.run_batch(wl.batches[0])
    assert plan.stats()["kv_splits"] >= 1
    _check_rows(run, wl.batches[0], _computed_rows(plan), TOL["bf16"])
    run.close()


@pytest.mark.parametrize("head_dim", [128, 64])
@pytest.mark.parametrize("cross_len", [40, 9])
def test_running_max_raised_mid_row(cross_len, head_dim):
    """Scores that jump by more than 2^16 between key blocks: every query row gets a
    bias along the lowest-frequency rotary pair (dims d/2 - 1 and d - 1, which rotate
    by at most about 0.1 rad over these distances), and the first three 32-key blocks
    of the prefix are pushed down by about 49, 24 and 0 in log2 units at d = 128
    (69, 35, 0 at d = 64).  In the prefill kernel each
    row past the prefix's first block raises its running max twice after its first
    block (the block max climbs from about -40 to -18 to +4), once in an odd and once
    in an even block of the key loop; the cross kernels (40 rows: 32-row tiles, 9 rows:
    the 16-row kernel) take their max on a whole first tile (about -18) and raise it
    on the next.  The result must not depend on any of it."""
    wl = W.small_workload(head_dim=head_dim, prefix_len=96, frag_lens=(300, 129, 64, 200), frags_per_query=3,
                          cross_len=cross_len)
    q, k = wl.q.copy(), wl.k.copy()
    low = head_dim // 2 - 1
    q[:, :, low] += 8.0
    for batch in wl.batches:
        for query in batch:
            r0 = query.prefix.row
            k[r0:r0 + 32, :, low] = -48.0
            k[r0 + 32:r0 + 64, :, low] = -24.0
    wl.q_bits, wl.k_bits = W.round_to_bf16_bits(q), W.round_to_bf16_bits(k)
    wl.q, wl.k = W.bf16_bits_to_f32(wl.q_bits), W.bf16_bits_to_f32(wl.k_bits)
    run = GpuRun(wl)
    plan = run.run_batch(wl.batches[0])
    _check_rows(run, wl.batches[0], _computed_rows(plan), TOL["bf16"])
    run.close()


def test_duplicate_fragment_in_one_query():
    wl = W.small_workload(orders=[[0, 1, 0], [2, 1, 3], [1, 1, 2]], n_queries=3)
    run = GpuRun(wl)
    plan = run.run_batch(wl.batches[0])
    st = plan.stats()
    assert st["tokens_new"] == 40 + 37 + 64 + 5 + 100
    _check_rows(run, wl.batches[0], _computed_rows(plan), TOL["bf16"])
    run.close()


def _page_kv(run, page_id, wl):
    raw = run.pool.read_page(0, page_id)
    if wl.dtype == "bf16":
        raw = (raw.astype(np.uint32) << 16).view(np.float32)
    hkv, d = wl.n_kv_heads, wl.head_dim
    k = raw[: hkv * 16 * d].reshape(hkv, 16, d)
    vt = raw[hkv * 16 * d:].reshape(hkv, d, 16)
    # slot s of a page sits at position s with bits 2 and 3 swapped
    vpos = [(s & 3) | ((s & 4) << 1) | ((s & 8) >> 1) for s in range(16)]
    v = vt[:, :, vpos].transpose(0, 2, 1)
    return k, v


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pages_hold_canonical_kv(dtype):
    wl = W.small_workload(dtype=dtype)
    run = GpuRun(wl)
    q0 = wl.batches[0][0]
    plan = run.run_batch([q0])
    lay = query_layout(q0)
    rows = query_rows(q0)
    for child, f in enumerate(q0.frags):
        ids, _ = plan.block_table(0, child)
        kc, vc = OA.cached_fragment_kv(wl.k[rows], wl.v[rows], lay, child, wl.rope_theta)
        for p, pid in enumerate(ids):
            k, v = _page_kv(run, pid, wl)
            n = min(16, f.n - 16 * p)
            kr, vr = kc[16 * p: 16 * p + n].transpose(1, 0, 2), vc[16 * p: 16 * p + n].transpose(1, 0, 2)
            rtol = 2.0 ** -8 if dtype == "bf16" else 1e-6
            np.testing.assert_allclose(k[:, :n], kr, rtol=rtol, atol=1e-5)
            np.testing.assert_array_equal(v[:, :n], vr.astype(np.float32))
            assert not np.any(k[:, n:]) and not np.any(v[:, n:])   # unfilled slots are zero
    run.close()


@pytest.mark.parametrize("dtype,cross_len", [("bf16", 10), ("bf16", 23), ("bf16", 100), ("f32", 23)])
def test_cross_pages_hold_final_kv(dtype, cross_len):
    """The cross segment's pages hold its keys rotated at their final positions and its
    values, unfilled slots zero, whichever launch writes them: the page-write kernel
    (few-row cross tiles, fp32 pools) or the MFMA cross kernel itself (the others)."""
    wl = W.small_workload(dtype=dtype, cross_len=cross_len)
    run = GpuRun(wl)
    batch = wl.batches[0]
    plan = run.run_batch(batch)
    for qi, q in enumerate(batch):
        ids, n_hit = plan.block_table(qi, len(q.frags))
        assert n_hit == 0 and len(ids) == (q.cross.n + 15) // 16
        final0 = q.prefix.n + sum(f.n for f in q.frags)
        rows = np.arange(q.cross.row, q.cross.row + q.cross.n)
        kc = OA.rope(wl.k[rows].astype(np.float64), final0 + np.arange(q.cross.n), wl.rope_theta)
        vc = wl.v[rows].astype(np.float64)
        for p, pid in enumerate(ids):
            k, v = _page_kv(run, pid, wl)
            n = min(16, q.cross.n - 16 * p)
            kr, vr = kc[16 * p: 16 * p + n].transpose(1, 0, 2), vc[16 * p: 16 * p + n].transpose(1, 0, 2)
            rtol = 2.0 ** -8 if dtype == "bf16" else 1e-6
            np.testing.assert_allclose(k[:, :n], kr, rtol=rtol, atol=1e-5)
            np.testing.assert_array_equal(v[:, :n], vr.astype(np.float32))
            assert not np.any(k[:, n:]) and not np.any(v[:, n:])   # unfilled slots are zero
    _check_rows(run, batch, _computed_rows(plan), TOL[dtype])
    run.close()


def test_permutation_keeps_pages_and_rows_bit_identical():
    wl = W.small_workload(orders=[[0, 1, 2, 3], [3, 1, 0, 2]], n_queries=2, frags_per_query=4,
                          batch_split=[1, 1])
    runs = [GpuRun(wl), GpuRun(wl)]
    plans = [runs[0].run_batch(wl.batches[0]), runs[1].run_batch(wl.batches[1])]
    orders = [[0, 1, 2, 3], [3, 1, 0, 2]]
    for f in range(4):
        tabs = [plans[i].block_table(0, orders[i].index(f))[0] for i in range(2)]
        for pa, pb in zip(*tabs):
            assert np.array_equal(runs[0].pool.read_page(0, pa), runs[1].pool.read_page(0, pb))
        frow = wl.batches[0][0].frags[f]
        rows = np.arange(frow.row, frow.row + frow.n)
        assert np.array_equal(runs[0].out_rows(rows), runs[1].out_rows(rows))
    for r in runs:
        r.close()


@pytest.mark.parametrize("kernel", ["generic", "auto"])
def test_cache_hit_equals_recompute(kernel):
    wl = W.small_workload(orders=[[0, 1, 2, 3], [3, 1, 0, 2]], n_queries=2, frags_per_query=4,
                          batch_split=[1, 1])
    warm = GpuRun(wl, kernel=kernel)
    warm.run_batch(wl.batches[0])
    pw = warm.run_batch(wl.batches[1])
    assert pw.stats()["tokens_new"] == 0
    cold = GpuRun(wl, kernel=kernel)
    pc = cold.run_batch(wl.batches[1])
    assert pc.stats()["tokens_hit"] == 0
    _, cross = pw.rows()
    assert np.array_equal(warm.out_rows(cross), cold.out_rows(cross))
    _check_rows(warm, wl.batches[1], cross, TOL["bf16"])
    warm.close()
    cold.close()


def test_c2_full_size_sampled():
    wl = W.config_c2()
    run = GpuRun(wl)
    batch = wl.batches[0]
    plan = run.run_batch(batch)
    st = plan.stats()
    assert st["tokens_cross"] == 8 * 128
    pre, cross = plan.rows()
    _check_rows(run, batch, pre, TOL["bf16"], limit=96)
    _check_rows(run, batch, cross, TOL["bf16"], limit=96)
    # second pass, every query reversed: all prefix/fragment pages hit
    rev = [W.Query(prefix=q.prefix, frags=q.frags[::-1], cross=q.cross) for q in batch]
    p2 = run.run_batch(rev)
    assert p2.stats()["tokens_new"] == 0
    _, cross2 = p2.rows()
    _check_rows(run, rev, cross2, TOL["bf16"], limit=96)
    run.close()


def test_c3_full_size_sampled():
    wl = W.config_c3()
    run = GpuRun(wl)
    batch = wl.batches[0]
    plan = run.run_batch(batch)
    pre, cross = plan.rows()
    _check_rows(run, batch, pre, TOL["bf16"], limit=64)
    _check_rows(run, batch, cross, TOL["bf16"], limit=64)
    run.close()


# (query heads, kv heads, head dim, fragments): enough row tiles that every one of
# the eight per-XCD queues of the span-prefill kernel holds its work-groups' first
# two items, for each chunking (8 / kv heads chunks of the tiles)
XCD_CASES = [(32, 8, 128, 64), (32, 4, 64, 64), (16, 2, 64, 64), (8, 1, 128, 72)]


@pytest.mark.parametrize("hq,hkv,d,nf", XCD_CASES, ids=[f"kv{c[1]}" for c in XCD_CASES])
def test_prefill_per_xcd_queues(hq, hkv, d, nf):
    """The span-prefill kernel's per-XCD queues (one kv head of one group of spans per
    queue, work-groups moving on to other queues when theirs runs dry), against the
    oracle on rows sampled evenly over every query and fragment."""
    per = nf // 8
    wl = W.rag_workload("xcd", seed=5, n_q_heads=hq, n_kv_heads=hkv, head_dim=d, hidden=64, prefix_len=64,
                        pool_size=nf, frag_lens=256, n_queries=8, cross_len=16, mode="direct",
                        orders=[[per * q + i for i in range(per)] for q in range(8)])
    run = GpuRun(wl)
    batch = wl.batches[0]
    plan = run.run_batch(batch)
    assert plan.stats()["prefill_queues"] == 8
    pre, cross = plan.rows()
    _check_rows(run, batch, pre, TOL["bf16"], limit=512)
    _check_rows(run, batch, cross, TOL["bf16"], limit=64)
    run.close()


def test_prefill_small_launch_uses_one_queue():
    wl = W.small_workload()
    run = GpuRun(wl)
    plan = run.run_batch(wl.batches[0])
    assert plan.stats()["prefill_queues"] == 1
    _check_rows(run, wl.batches[0], _computed_rows(plan), TOL["bf16"])
    run.close()


@pytest.mark.parametrize("cross_len", [1, 4, 16])
def test_few_cross_rows_over_many_pages(cross_len):
    """The KV page-gather regime: a handful of cross rows per query over a long
    cached context (split along the keys, merged by the combine kernel)."""
    wl = W.rag_workload("gather", seed=3, prefix_len=256, pool_size=8, frag_lens=256, frags_per_query=8,
                        n_queries=2, cross_len=cross_len, mode="direct",
                        orders=[list(range(8)), list(range(8))[::-1]], batch_split=[1, 1])
    run = GpuRun(wl)
    run.run_batch(wl.batches[0])
    plan = run.run_batch(wl.batches[1])
    st = plan.stats()
    assert st["tokens_new"] == 0 and st["kv_splits"] > 1
    _, cross = plan.rows()
    _check_rows(run, wl.batches[1], cross, TOL["bf16"])
    run.close()


def test_prefill_relaunches_and_concurrent_streams():
    """The bf16 prefill kernel hands out work items from a per-launch counter that
    each launch leaves at zero.  Launch it repeatedly on one plan (both layers of a
    two-layer pool), then twice at once on two streams, and check every launch."""
    wl = W.config_c2()
    run = GpuRun(wl, num_layers=2)
    batch = wl.batches[0]
    plan = run.pool.plan(batch)
    pre, _ = plan.rows()
    rows = pre[np.linspace(0, pre.size - 1, 48).astype(np.int64)]
    ref = {}
    for q in batch:
        mine = [r for r in query_rows(q) if int(r) in set(int(x) for x in rows) and int(r) not in ref]
        ref.update(oracle_rows(wl, q, mine))
    assert len(ref) == rows.size

    def check(out):
        o = out[torch.as_tensor(rows, device="cuda")].cpu().numpy()
        got = (o.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
        worst = max(max_err(got[i], ref[int(r)]) for i, r in enumerate(rows))
        assert worst <= TOL["bf16"], f"max abs err {worst}"

    for layer in (0, 1, 0, 1, 0):
        run.out.zero_()
        plan.prefill(layer, run.q, run.k, run.v, run.out)
        torch.cuda.synchronize()
        check(run.out)
    outs = [torch.zeros_like(run.out) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for layer, (s, o) in enumerate(zip(streams, outs)):
        plan.prefill(layer, run.q, run.k, run.v, o, stream=s)
    torch.cuda.synchronize()
    for o in outs:
        check(o)
    plan.commit()
    run.close()
