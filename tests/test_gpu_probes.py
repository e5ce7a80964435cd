"""The machine-peak probes of the library (MFMA-only loop, streaming read) on the GPU:
each returns a rate below the published peak of its resource, and not far below it."""
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(flush=True)


def test_mfma_probe_is_below_the_dense_bf16_peak():
    import paper_2511_02749_amd as spanq
    tflops = spanq.probe_mfma_peak(iters=2000, reps=3)
    # 2.5 PFLOP/s dense bf16 at the 2.4 GHz peak clock; an MFMA-only loop reaches
    # most of it, so a rate far below means the flop count or the launch is off
    assert 1000.0 < tflops <= 2500.0, tflops


def test_read_probe_is_below_the_hbm_peak():
    import paper_2511_02749_amd as spanq
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    gbs = spanq.probe_read_peak(buf, reps=3)
    assert 2000.0 < gbs <= 8000.0, gbs


def test_probes_reject_bad_arguments():
    import paper_2511_02749_amd as spanq
    with pytest.raises(spanq.SpanError):
        spanq.probe_mfma_peak(iters=0, reps=1)
    buf = torch.empty(8, dtype=torch.uint8, device="cuda")
    with pytest.raises(spanq.SpanError):
        spanq.probe_read_peak(buf, reps=1)  # 8 bytes: rounded down to 0, rejected
    big = torch.empty(4096 + 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(spanq.SpanError):
        spanq.probe_read_peak(big[1:], reps=1)  # not 16-byte aligned
