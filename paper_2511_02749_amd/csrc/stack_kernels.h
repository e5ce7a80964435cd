// Launchers of the decoder-stack kernels (stack_kernels.hip).  Activations are
// bf16 bit patterns, row-major; row sizes are multiples of 16 bytes.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace spanq {

// Row copy: dst[i] = src[idx[i]] (gather) or dst[idx[i]] = src[i] (scatter); idx
// null = identity.  row_bytes a multiple of 16.
hipError_t launch_copy_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows, int row_bytes, bool scatter,
                            hipStream_t s);

// Split rows of qkv [n][q_elems + 2 kv_elems] into q [.][q_elems], k and v
// [.][kv_elems] at rows[i].
hipError_t launch_scatter_qkv(const void* qkv, const int32_t* rows, int64_t n, int q_elems, int kv_elems, void* q,
                              void* k, void* v, hipStream_t s);

// y[i] = RMSNorm(x[sel[i]]) * gain (sel null = identity), hidden <= 8192, a multiple of 8.
hipError_t launch_rmsnorm(const void* x, const int32_t* sel, const void* gain, void* y, int64_t n_rows, int hidden,
                          float eps, hipStream_t s);

// act[i] = silu(gu[i][0:ffn]) * gu[i][ffn:2 ffn].
hipError_t launch_swiglu(const void* gu, void* act, int64_t n, int ffn, hipStream_t s);

// Y[M][N] = X[M][K] W[K][N] (+ Y when residual) for 1 <= M <= 8 rows, bf16 row-major
// in and out, fp32 sums in a fixed order; N a multiple of 8.  part: fp32 scratch of
// at least gemv_part_bytes(M, N, K).  HBM-bound (W read once).
size_t gemv_part_bytes(int M, int N, int K);
hipError_t launch_gemv(const void* x, const void* w, void* y, int M, int N, int K, bool residual, float* part,
                       size_t part_bytes, hipStream_t s);
// The same GEMV with the layer's next step fused into its second pass, bit for bit
// what the separate kernels give: q|k|v rows (N = q_elems + 2 kv_elems) written
// straight to caller rows rows[m] of q, k, v (launch_scatter_qkv); gate|up (N = 2 ffn)
// into act = silu(gate) * up (launch_swiglu); a projection added to the residual
// stream y (N = hidden <= 8192) followed by nout = RMSNorm(y) * gain (launch_rmsnorm).
hipError_t launch_gemv_qkv(const void* x, const void* w, int M, int K, const int32_t* rows, int q_elems,
                           int kv_elems, void* q, void* k, void* v, float* part, size_t part_bytes, hipStream_t s);
hipError_t launch_gemv_swiglu(const void* x, const void* w, void* act, int M, int ffn, int K, float* part,
                              size_t part_bytes, hipStream_t s);
hipError_t launch_gemv_residual_norm(const void* x, const void* w, void* y, int M, int N, int K, const void* gain,
                                     void* nout, float eps, float* part, size_t part_bytes, hipStream_t s);

// Y[M][N] = X[M][K] W[K][N] (+ Y when residual) for 129..256 rows and K >= 4 N from
// the transposed weights wt = W^T [N][K] (bf16 row-major), N a multiple of 64, K a
// multiple of 256 (skinny_gemm_fits).  Split-K launches need part: fp32 scratch of at least
// skinny_gemm_part_bytes(M, N, K) bytes (0 when the launch does not split).  The slices
// are summed in a fixed order.
bool skinny_gemm_fits(int64_t M, int64_t N, int64_t K);
int skinny_gemm_slices(int M, int N, int K);
size_t skinny_gemm_part_bytes(int M, int N, int K);
hipError_t launch_skinny_gemm(const void* x, const void* wt, void* y, int M, int N, int K, bool residual, float* part,
                              size_t part_bytes, hipStream_t s);
// The same with the second pass also forming nout = RMSNorm(y) * gain (N <= 8192),
// bit for bit the plain launch followed by launch_rmsnorm, when the launch splits K
// (skinny_gemm_slices > 1); returns hipErrorNotSupported, having done nothing, when it
// does not.
hipError_t launch_skinny_gemm_norm(const void* x, const void* wt, void* y, int M, int N, int K, const void* gain,
                                   void* nout, float eps, float* part, size_t part_bytes, hipStream_t s);
// Second pass over `slices` fp32 partial planes [slices][M][N]: y += their sum in plane
// order (one rounding), then nout = RMSNorm(y) * gain, one work-group per row.
hipError_t launch_reduce_residual_norm(const float* part, int slices, int M, int N, void* y, const void* gain,
                                       void* nout, float eps, hipStream_t s);
// out[c][r] = in[r][c] for an R x C bf16 matrix.
hipError_t launch_transpose_bf16(const void* in, void* out, int64_t R, int64_t C, hipStream_t s);

// LM head over nq (1, 2, 4 or 8) rows of nf [nq][hidden]: partial logits per chunk
// of the hidden dimension into part [lm_head_chunks(hidden)][nq][vocab] (fp32).
// launch_argmax sums the chunks (in chunk order) for the first n_rows rows into
// logits [n_rows][vocab] (optional) and writes their argmax, lowest id on ties,
// to token [n_rows]; scratch holds argmax_scratch_bytes(nq, vocab) of device memory.
int lm_head_chunks(int hidden);
hipError_t launch_lm_head(const void* nf, const void* w, float* part, int nq, int hidden, int vocab, hipStream_t s);
size_t argmax_scratch_bytes(int nq, int vocab);
hipError_t launch_argmax(const float* part, int nq, int n_rows, int hidden, int vocab, float* logits, int32_t* token,
                         void* scratch, hipStream_t s);

}  // namespace spanq
