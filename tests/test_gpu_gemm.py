"""GPU parity of the decoder stack's GEMM dispatch (span_probe_gemm), through the C-ABI.

Y = X W (+ Y) with bf16 inputs and output and fp32 accumulation, against the exact
product of the same bf16 inputs in float64.  Bound per element: an fp32 sum of K
products is within K 2^-24 sum_k |x_k w_k| of the exact sum (recursive summation; the
MFMA's own order of additions stays inside it), the residual add adds one fp32
rounding, and the bf16 result is the nearest bf16 to that, within 2^-8 of it
relatively.  So |y - exact| <= 2^-8 (|exact| + e) + e + 2^-24 |exact|, with
e = K 2^-24 (|X| |W|).

Row counts 129..256 with K >= 4 N, N a multiple of 64 and K a multiple of 256 take
the skinny MFMA kernel (K split into slices that add up in a fixed order when N / 64
tiles are few); the test also runs shapes and row counts on either side of it (the
GEMV kernels up to 8 rows, hipBLASLt for the rest).
"""
import numpy as np
import pytest

import paper_2511_02749_amd as spanq

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)


def _run(M, N, K, residual, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    x = _bf16(rng.standard_normal((M, K)) * scale)
    w = _bf16(rng.standard_normal((K, N)) / np.sqrt(K))
    y0 = _bf16(rng.standard_normal((M, N)))
    xd, wd = x.cuda(), w.cuda()
    yd = y0.cuda() if residual else torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    print(f"gemm M={M} N={N} K={K} residual={residual} seed={seed}", flush=True)
    kern, _ = spanq._lib.probe_gemm(xd, wd, yd, residual=residual)
    torch.cuda.synchronize()
    got = yd.cpu().float().numpy().astype(np.float64)
    x64, w64 = x.float().numpy().astype(np.float64), w.float().numpy().astype(np.float64)
    exact = x64 @ w64 + (y0.float().numpy().astype(np.float64) if residual else 0.0)
    e = K * 2.0 ** -24 * (np.abs(x64) @ np.abs(w64))
    bound = 2.0 ** -8 * (np.abs(exact) + e) + e + 2.0 ** -24 * np.abs(exact)
    err = np.abs(got - exact)
    bad = np.argwhere(err > bound)
    assert bad.size == 0, (f"M={M} N={N} K={K}: {len(bad)} elements out of bound, first {tuple(bad[0])}: "
                           f"got {got[tuple(bad[0])]}, exact {exact[tuple(bad[0])]}, bound {bound[tuple(bad[0])]}")
    assert np.isfinite(got).all()
    return kern


@pytest.mark.parametrize("M", [129, 130, 160, 191, 200, 255, 256])
@pytest.mark.parametrize("N,K", [(64, 256), (192, 768), (512, 2048), (1024, 4096)])
def test_skinny_gemm_matches_exact_product(M, N, K):
    assert _run(M, N, K, residual=False, seed=M * 7 + N + K) == 2


@pytest.mark.parametrize("M,N,K", [(256, 2048, 8192), (177, 2048, 8192), (200, 128, 4096), (256, 4096, 16384)])
def test_skinny_gemm_large_shapes_with_residual(M, N, K):
    """The C4 stack's down projection (K split into slices) and other long
    reductions, residual added."""
    assert _run(M, N, K, residual=True, seed=M + N + K) == 2


@pytest.mark.parametrize("M,N,K,kern", [(8, 2048, 8192, 1), (9, 2048, 8192, 0), (128, 2048, 8192, 0),
                                        (257, 2048, 8192, 0), (256, 2048, 2048, 0), (256, 16384, 2048, 0),
                                        (200, 2040, 8192, 0), (200, 512, 2000, 0)])
def test_gemm_dispatch_outside_the_skinny_kernel(M, N, K, kern):
    """Row counts and shapes beyond the skinny kernel go to the GEMV kernels and to
    hipBLASLt, to the same bound."""
    assert _run(M, N, K, residual=True, seed=M + N + K) == kern


def test_skinny_gemm_rows_do_not_depend_on_row_count():
    """A row's result is the same bits whatever the number of rows computed with it
    (the K slices and the order of additions depend on N and K only)."""
    rng = np.random.default_rng(5)
    K, N = 8192, 2048
    x = _bf16(rng.standard_normal((256, K))).cuda()
    w = _bf16(rng.standard_normal((K, N)) / np.sqrt(K)).cuda()
    outs = []
    for M in (129, 200, 256):
        y = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
        assert spanq._lib.probe_gemm(x[:M].contiguous(), w, y)[0] == 2
        outs.append(y[:9].cpu())
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])
