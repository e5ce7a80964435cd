"""The no-allocation planning entry point (span_plan_static) against span_plan.

span_plan_static places a plan's device data in a library-held device array
instead of allocating them.  Its outputs must equal those of the allocating entry
point on the same inputs (the same kernels run on the same data, so bit for bit),
on two plans in a row, the second smaller than the first, and stay within the
bf16 tolerance of the oracle.  Oversized plans, host-only pools and a second live
plan of this kind are refused with an error.
"""
import numpy as np
import pytest

import workloads as W
from tests.helpers import TOL, GpuRun, check_rows, computed_rows

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(flush=True)


def _run(run, batch, static):
    plan = run.pool.plan(batch, static=static)
    run.out.zero_()
    plan.prefill(0, run.q, run.k, run.v, run.out)
    plan.cross(0, run.q, run.k, run.v, run.out)
    torch.cuda.synchronize()
    rows = computed_rows(plan)
    out = run.out_rows(rows)
    plan.commit()
    plan.destroy()
    return rows, out


@pytest.mark.parametrize("kernel", ["auto", "generic"])
def test_static_plan_matches_allocating_plan(kernel):
    """Two plans in a row through span_plan_static (three ragged queries with split-KV
    cross tiles, then one smaller query), each against span_plan on a fresh pool."""
    big = W.small_workload(n_queries=3, cross_len=23)
    small = W.small_workload(seed=5, prefix_len=20, frag_lens=(16, 33), n_queries=1, frags_per_query=2,
                             cross_len=9)
    for wl in (big, small):
        ref_run, st_run = GpuRun(wl, kernel=kernel), GpuRun(wl, kernel=kernel)
        torch.cuda.synchronize()
        rows_a, out_a = _run(ref_run, wl.batches[0], static=False)
        rows_b, out_b = _run(st_run, wl.batches[0], static=True)
        assert np.array_equal(rows_a, rows_b)
        assert np.array_equal(out_a, out_b)
        check_rows(st_run, wl.batches[0], rows_b, TOL["bf16"])
        ref_run.close()
        st_run.close()


def test_static_plan_refusals():
    import paper_2511_02749_amd as spanq
    wl = W.small_workload(n_queries=1)
    run = GpuRun(wl)
    # a second live plan of this kind on the same GPU
    p1 = run.pool.plan(wl.batches[0], static=True)
    with pytest.raises(spanq.SpanError) as e:
        run.pool.plan(wl.batches[0], static=True)
    assert e.value.code == spanq._lib.SPAN_ESTATE
    p1.destroy()
    # more device data than the array holds: 64 queries of 16 cross rows over one
    # fragment each make two-key-group partials of 32 x 64 x 130 floats per split
    prefix = W.Span(tokens=np.arange(256, dtype=np.int32), row=0)
    qs = [W.Query(prefix=prefix, frags=[W.Span(tokens=np.arange(1000 + 64 * i, 1064 + 64 * i, dtype=np.int32),
                                               row=0)],
                  cross=W.Span(tokens=np.arange(16, dtype=np.int32), row=0)) for i in range(64)]
    big_pool = spanq.Pool(num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=4096, dtype="bf16", device=0)
    with pytest.raises(spanq.SpanError) as e:
        big_pool.plan(qs, static=True)
    assert e.value.code == spanq._lib.SPAN_EINVAL and "scratch" in str(e.value)
    # the pool is still usable, and a fitting static plan goes through afterwards
    assert big_pool.info()["pinned_pages"] == 0
    big_pool.plan(qs[:1], static=True).destroy()
    big_pool.close()
    # positions past the rotary table a pool starts with (4096)
    long = W.small_workload(frag_lens=(4200,), n_queries=1, frags_per_query=1)
    lrun = GpuRun(long)
    with pytest.raises(spanq.SpanError) as e:
        lrun.pool.plan(long.batches[0], static=True)
    assert e.value.code == spanq._lib.SPAN_EINVAL and "rotary" in str(e.value)
    lrun.close()
    host = spanq.Pool(num_q_heads=8, num_kv_heads=2, head_dim=128, num_pages=64, device=-1)
    with pytest.raises(spanq.SpanError):
        host.plan(wl.batches[0], static=True)
    host.close()
    run.close()
