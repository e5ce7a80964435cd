// Kernels of the decoder stack around span attention (bf16 activations, fp32
// arithmetic).  All of them are HBM-bound element or row operations; they move
// 16-byte vectors of eight bf16 values so that every wave's accesses are whole
// 1 KiB runs.  The GEMMs of the stack go to hipBLASLt (stack.cpp).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "stack_kernels.h"

namespace spanq {
namespace {

using u16 = unsigned short;

__device__ __forceinline__ float bf(u16 b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// float to bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ u16 to_bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<u16>(u >> 16);
}

__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = static_cast<uint32_t>(to_bf(f[2 * i])) | (static_cast<uint32_t>(to_bf(f[2 * i + 1])) << 16);
  return uint4{w[0], w[1], w[2], w[3]};
}

// dst[i] = src[idx[i]] (gather, scatter = false) or dst[idx[i]] = src[i] (scatter), rows
// of vec16 16-byte vectors; idx == nullptr is the identity.
__global__ void copy_rows_kernel(uint4* __restrict__ dst, const uint4* __restrict__ src, const int32_t* __restrict__ idx,
                                 int64_t n_rows, int vec16, bool scatter) {
  const int64_t total = n_rows * vec16;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / vec16;
    const int c = static_cast<int>(e - i * vec16);
    const int64_t r = idx ? static_cast<int64_t>(idx[i]) : i;
    if (scatter) {
      dst[r * vec16 + c] = src[e];
    } else {
      dst[e] = src[r * vec16 + c];
    }
  }
}

// Split each row of qkv [T][(Hq + 2 Hkv) d] into q, k, v at caller row rows[i].
__global__ void scatter_qkv_kernel(const uint4* __restrict__ qkv, const int32_t* __restrict__ rows, int64_t n,
                                   int vq, int vkv, uint4* __restrict__ q, uint4* __restrict__ k,
                                   uint4* __restrict__ v) {
  const int vrow = vq + 2 * vkv;
  const int64_t total = n * vrow;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / vrow;
    const int c = static_cast<int>(e - i * vrow);
    const int64_t r = rows[i];
    const uint4 x = qkv[e];
    if (c < vq) {
      q[r * vq + c] = x;
    } else if (c < vq + vkv) {
      k[r * vkv + (c - vq)] = x;
    } else {
      v[r * vkv + (c - vq - vkv)] = x;
    }
  }
}

constexpr int kNormThreads = 256;
constexpr int kNormVec = 4;  // 16-byte vectors per thread: hidden <= 256 * 4 * 8 = 8192

// y[i] = x[sel[i]] / sqrt(mean(x^2) + eps) * gain, one work-group per row.
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const uint4* __restrict__ x,
                                                               const int32_t* __restrict__ sel,
                                                               const uint4* __restrict__ gain, uint4* __restrict__ y,
                                                               int vec16, float eps) {
  __shared__ float part[kNormThreads / 64];
  const int64_t row = blockIdx.x;
  const int64_t src = sel ? static_cast<int64_t>(sel[row]) : row;
  float f[kNormVec][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kNormVec; ++j) {
    const int c = threadIdx.x + j * kNormThreads;
    if (c < vec16) {
      unpack8(x[src * vec16 + c], f[j]);
#pragma unroll
      for (int t = 0; t < 8; ++t) ss = fmaf(f[j][t], f[j][t], ss);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) tot += part[w];
  const float scale = 1.0f / sqrtf(tot / static_cast<float>(vec16 * 8) + eps);
#pragma unroll
  for (int j = 0; j < kNormVec; ++j) {
    const int c = threadIdx.x + j * kNormThreads;
    if (c < vec16) {
      float g[8], o[8];
      unpack8(gain[c], g);
#pragma unroll
      for (int t = 0; t < 8; ++t) o[t] = f[j][t] * scale * g[t];
      y[row * vec16 + c] = pack8(o);
    }
  }
}

// act[i][j] = silu(gu[i][j]) * gu[i][F + j], silu(z) = z / (1 + e^-z).
__global__ void swiglu_kernel(const uint4* __restrict__ gu, uint4* __restrict__ act, int64_t n, int vf) {
  const int64_t total = n * vf;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / vf;
    const int c = static_cast<int>(e - i * vf);
    float g[8], u[8], o[8];
    unpack8(gu[i * 2 * vf + c], g);
    unpack8(gu[i * 2 * vf + vf + c], u);
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = g[t] / (1.0f + expf(-g[t])) * u[t];
    act[e] = pack8(o);
  }
}

constexpr int kHeadThreads = 256;
constexpr int kHeadCols = kHeadThreads * 8;  // vocab columns per work-group

// Partial logits of nq rows over a chunk of the hidden dimension:
// part[chunk][q][c] = sum over h in the chunk of n[q][h] * w[h][c].  Work-group
// (column block, chunk); each thread owns 8 consecutive columns.
template <int NQ>
__global__ __launch_bounds__(kHeadThreads) void lm_head_kernel(const u16* __restrict__ n, const uint4* __restrict__ w,
                                                               float* __restrict__ part, int hidden, int vocab,
                                                               int chunk_rows) {
  const int col0 = blockIdx.x * kHeadCols + threadIdx.x * 8;
  const int h0 = blockIdx.y * chunk_rows;
  const int h1 = min(hidden, h0 + chunk_rows);
  float acc[NQ][8];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[q][t] = 0.f;
  if (col0 < vocab) {
    const int vrow = vocab / 8;
    auto row = [&](int h, const uint4& wv) {  // weight row h into the sums
      float f[8];
      unpack8(wv, f);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const float a = bf(n[static_cast<int64_t>(q) * hidden + h]);
#pragma unroll
        for (int t = 0; t < 8; ++t) acc[q][t] = fmaf(a, f[t], acc[q][t]);
      }
    };
    int h = h0;
    for (; h + 8 <= h1; h += 8) {  // eight rows of weights in flight, then their sums in row order
      uint4 wv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) wv[u] = w[static_cast<int64_t>(h + u) * vrow + col0 / 8];
#pragma unroll
      for (int u = 0; u < 8; ++u) row(h + u, wv[u]);
    }
    for (; h < h1; ++h) row(h, w[static_cast<int64_t>(h) * vrow + col0 / 8]);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      float* p = part + (static_cast<int64_t>(blockIdx.y) * NQ + q) * vocab + col0;
      *reinterpret_cast<float4*>(p) = float4{acc[q][0], acc[q][1], acc[q][2], acc[q][3]};
      *reinterpret_cast<float4*>(p + 4) = float4{acc[q][4], acc[q][5], acc[q][6], acc[q][7]};
    }
  }
}

// Logits = the chunks' partials summed in chunk order; token = argmax, lowest id on
// ties, in two passes.  Pass 1, one work-group per (block of kArgCols columns, row):
// the sums (stored as logits if asked) and the block's best value with its lowest
// id.  Pass 2, one work-group per row: the best of the blocks' bests, lower block
// first on ties.  A NaN never wins; a row of NaNs gives id 0x7fffffff.
constexpr int kArgThreads = 256;
constexpr int kArgCols = kArgThreads * 4;

__device__ __forceinline__ void better(float& bv, int& bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

__global__ __launch_bounds__(kArgThreads) void argmax_blocks_kernel(const float* __restrict__ part, int n_chunks,
                                                                    int nq, int vocab, float* __restrict__ logits,
                                                                    float* __restrict__ best_v,
                                                                    int* __restrict__ best_i) {
  // nq is the partials' row stride; the grid covers only the rows wanted
  __shared__ float sv[kArgThreads];
  __shared__ int si[kArgThreads];
  const int q = blockIdx.y;
  const int c0 = blockIdx.x * kArgCols + threadIdx.x * 4;
  float best = -INFINITY;
  int arg = 0x7fffffff;
  if (c0 < vocab) {  // vocab is a multiple of 8: four columns are all in or all out
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k = 0; k < n_chunks; ++k) {
      const float4 p = *reinterpret_cast<const float4*>(part + (static_cast<int64_t>(k) * nq + q) * vocab + c0);
      acc.x += p.x;
      acc.y += p.y;
      acc.z += p.z;
      acc.w += p.w;
    }
    if (logits) *reinterpret_cast<float4*>(logits + static_cast<int64_t>(q) * vocab + c0) = acc;
    const float v[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (v[j] > best) {  // columns rise: an equal later value keeps the lower id
        best = v[j];
        arg = c0 + j;
      }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = arg;
  __syncthreads();
  for (int off = kArgThreads / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      float bv = sv[threadIdx.x];
      int bi = si[threadIdx.x];
      better(bv, bi, sv[threadIdx.x + off], si[threadIdx.x + off]);
      sv[threadIdx.x] = bv;
      si[threadIdx.x] = bi;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    best_v[static_cast<int64_t>(q) * gridDim.x + blockIdx.x] = sv[0];
    best_i[static_cast<int64_t>(q) * gridDim.x + blockIdx.x] = si[0];
  }
}

__global__ __launch_bounds__(kArgThreads) void argmax_rows_kernel(const float* __restrict__ best_v,
                                                                  const int* __restrict__ best_i, int n_blocks,
                                                                  int32_t* __restrict__ token) {
  __shared__ float sv[kArgThreads];
  __shared__ int si[kArgThreads];
  const int q = blockIdx.x;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int b = threadIdx.x; b < n_blocks; b += kArgThreads)
    better(bv, bi, best_v[static_cast<int64_t>(q) * n_blocks + b], best_i[static_cast<int64_t>(q) * n_blocks + b]);
  sv[threadIdx.x] = bv;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int off = kArgThreads / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      float v = sv[threadIdx.x];
      int i = si[threadIdx.x];
      better(v, i, sv[threadIdx.x + off], si[threadIdx.x + off]);
      sv[threadIdx.x] = v;
      si[threadIdx.x] = i;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) token[q] = si[0];
}

// GEMV for a few rows (decode steps): Y[M][N] = X[M][K] W[K][N] (+ Y), M <= 8,
// bf16 in and out, fp32 sums.  Pass 1, work-group (64 columns, one of kGemvChunks
// slices of K): thread (row group g = 0..31, column lane) takes rows g, g + 32, ..
// of the slice and 8 consecutive columns (a wave reads 8 whole 128-byte row
// segments per load); the row groups meet in LDS and the work-group writes fp32
// partials for its slice.  Pass 2, one thread per output element: the slices'
// partials summed in slice order, the residual added, rounded once.  (A last
// work-group per column block finishing the sum in pass 1 would need a device-scope
// release per work-group; across this chip's eight L2s that costs more than the
// second launch.)  Bound: HBM (W read once; partials of kGemvChunks x 4 bytes per
// output element).
constexpr int kGemvCols = 64;
constexpr int kGemvChunks = 16;

template <int MP>
__global__ __launch_bounds__(256) void gemv_partial_kernel(const u16* __restrict__ x, const uint4* __restrict__ w,
                                                           float* __restrict__ part, int M, int N, int K,
                                                           int rows_per_chunk) {
  __shared__ float red[32][MP][kGemvCols];
  const int cl = threadIdx.x & 7;
  const int rg = threadIdx.x >> 3;
  const int c0 = blockIdx.x * kGemvCols + cl * 8;
  const int k0 = blockIdx.y * rows_per_chunk;
  const int k1 = min(K, k0 + rows_per_chunk);
  float acc[MP][8];
#pragma unroll
  for (int m = 0; m < MP; ++m)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[m][j] = 0.f;
  if (c0 < N) {
    const int64_t vrow = N / 8;
    int k = k0 + rg;
    for (; k + 96 < k1; k += 128) {  // four rows in flight
      uint4 wv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) wv[u] = w[static_cast<int64_t>(k + 32 * u) * vrow + c0 / 8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float f[8];
        unpack8(wv[u], f);
#pragma unroll
        for (int m = 0; m < MP; ++m) {
          if (m >= M) break;
          const float a = bf(x[static_cast<int64_t>(m) * K + k + 32 * u]);
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[m][j] = fmaf(a, f[j], acc[m][j]);
        }
      }
    }
    for (; k < k1; k += 32) {
      float f[8];
      unpack8(w[static_cast<int64_t>(k) * vrow + c0 / 8], f);
#pragma unroll
      for (int m = 0; m < MP; ++m) {
        if (m >= M) break;
        const float a = bf(x[static_cast<int64_t>(m) * K + k]);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[m][j] = fmaf(a, f[j], acc[m][j]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < MP; ++m)
#pragma unroll
    for (int j = 0; j < 8; ++j) red[rg][m][cl * 8 + j] = acc[m][j];
  __syncthreads();
  // thread t sums column t % 64 of rows t / 64, t / 64 + 4, .. over the row groups
  const int col = threadIdx.x % kGemvCols;
  const int n_t = blockIdx.x * kGemvCols + col;
  if (n_t < N)
    for (int m = threadIdx.x / kGemvCols; m < M; m += 256 / kGemvCols) {
      float sum = 0.f;
#pragma unroll 8
      for (int g = 0; g < 32; ++g) sum += red[g][m][col];
      part[(static_cast<int64_t>(blockIdx.y) * M + m) * N + n_t] = sum;
    }
}

__global__ __launch_bounds__(256) void gemv_reduce_kernel(const float* __restrict__ part, int chunks, int M, int N,
                                                          u16* __restrict__ y, bool residual) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;  // element m * N + n
  const int64_t MN = static_cast<int64_t>(M) * N;
  if (i >= MN) return;
  float sum = 0.f;
#pragma unroll 4
  for (int c = 0; c < chunks; ++c) sum += part[static_cast<int64_t>(c) * MN + i];
  if (residual) sum += bf(y[i]);
  y[i] = to_bf(sum);
}

// Fused second passes for the decode-sized GEMVs.  Each forms every sum exactly as
// gemv_reduce_kernel does (slices in order, one rounding to bf16) and then does the
// next small step of the layer on it, so that the results are the bits the separate
// kernels give:
// - q|k|v: the rounded values go straight to caller row rows[m] of q, k or v;
__global__ __launch_bounds__(256) void gemv_reduce_qkv_kernel(const float* __restrict__ part, int chunks, int M,
                                                              int N, const int32_t* __restrict__ rows, int nq,
                                                              int nkv, u16* __restrict__ q, u16* __restrict__ k,
                                                              u16* __restrict__ v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t MN = static_cast<int64_t>(M) * N;
  if (i >= MN) return;
  float sum = 0.f;
#pragma unroll 4
  for (int c = 0; c < chunks; ++c) sum += part[static_cast<int64_t>(c) * MN + i];
  const u16 b = to_bf(sum);
  const int m = static_cast<int>(i / N), n = static_cast<int>(i - static_cast<int64_t>(m) * N);
  const int64_t r = rows[m];
  if (n < nq) {
    q[r * nq + n] = b;
  } else if (n < nq + nkv) {
    k[r * nkv + (n - nq)] = b;
  } else {
    v[r * nkv + (n - nq - nkv)] = b;
  }
}

// - gate|up: act[m][f] = silu(gate) * up of the two rounded sums, as swiglu_kernel;
__global__ __launch_bounds__(256) void gemv_reduce_swiglu_kernel(const float* __restrict__ part, int chunks, int M,
                                                                 int F, u16* __restrict__ act) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;  // m * F + f
  if (i >= static_cast<int64_t>(M) * F) return;
  const int64_t N = 2 * static_cast<int64_t>(F), MN = static_cast<int64_t>(M) * N;
  const int64_t m = i / F, f = i - m * F;
  float sg = 0.f, su = 0.f;
#pragma unroll 4
  for (int c = 0; c < chunks; ++c) {
    sg += part[static_cast<int64_t>(c) * MN + m * N + f];
    su += part[static_cast<int64_t>(c) * MN + m * N + F + f];
  }
  const float g = bf(to_bf(sg)), u = bf(to_bf(su));
  act[i] = to_bf(g / (1.0f + expf(-g)) * u);
}

// - a projection into the residual stream: y += the rounded sums (one rounding of the
//   sum with the residual, as gemv_reduce_kernel), then the RMSNorm of the new row
//   with `gain`, formed exactly as rmsnorm_kernel forms it; one work-group per row.
__global__ __launch_bounds__(kNormThreads) void gemv_reduce_norm_kernel(const float* __restrict__ part, int chunks,
                                                                        int M, int N, u16* __restrict__ y,
                                                                        const uint4* __restrict__ gain,
                                                                        uint4* __restrict__ nout, float eps) {
  __shared__ float red[kNormThreads / 64];
  const int64_t row = blockIdx.x;
  const int64_t MN = static_cast<int64_t>(M) * N;
  const int vec16 = N / 8;
  float f[kNormVec][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kNormVec; ++j) {
    const int c = threadIdx.x + j * kNormThreads;
    if (c < vec16) {
      const int64_t i0 = row * N + 8 * c;
      float sum[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) sum[t] = 0.f;
#pragma unroll 4
      for (int cc = 0; cc < chunks; ++cc) {
        const float4* pp = reinterpret_cast<const float4*>(part + static_cast<int64_t>(cc) * MN + i0);
        const float4 a = pp[0], b = pp[1];
        sum[0] += a.x;
        sum[1] += a.y;
        sum[2] += a.z;
        sum[3] += a.w;
        sum[4] += b.x;
        sum[5] += b.y;
        sum[6] += b.z;
        sum[7] += b.w;
      }
      float res[8];
      unpack8(reinterpret_cast<const uint4*>(y)[row * vec16 + c], res);
#pragma unroll
      for (int t = 0; t < 8; ++t) f[j][t] = bf(to_bf(sum[t] + res[t]));
      reinterpret_cast<uint4*>(y)[row * vec16 + c] = pack8(f[j]);
#pragma unroll
      for (int t = 0; t < 8; ++t) ss = fmaf(f[j][t], f[j][t], ss);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) tot += red[w];
  const float scale = 1.0f / sqrtf(tot / static_cast<float>(vec16 * 8) + eps);
#pragma unroll
  for (int j = 0; j < kNormVec; ++j) {
    const int c = threadIdx.x + j * kNormThreads;
    if (c < vec16) {
      float g[8], o[8];
      unpack8(gain[c], g);
#pragma unroll
      for (int t = 0; t < 8; ++t) o[t] = f[j][t] * scale * g[t];
      nout[row * vec16 + c] = pack8(o);
    }
  }
}

int grid_for(int64_t items, int threads) {
  int64_t g = (items + threads - 1) / threads;
  if (g > 65536) g = 65536;
  return static_cast<int>(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_copy_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows, int row_bytes, bool scatter,
                            hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const int vec16 = row_bytes / 16;
  copy_rows_kernel<<<grid_for(n_rows * vec16, 256), 256, 0, s>>>(static_cast<uint4*>(dst),
                                                                 static_cast<const uint4*>(src), idx, n_rows, vec16,
                                                                 scatter);
  return hipGetLastError();
}

hipError_t launch_scatter_qkv(const void* qkv, const int32_t* rows, int64_t n, int q_elems, int kv_elems, void* q,
                              void* k, void* v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int vq = q_elems / 8, vkv = kv_elems / 8;
  scatter_qkv_kernel<<<grid_for(n * (vq + 2 * vkv), 256), 256, 0, s>>>(
      static_cast<const uint4*>(qkv), rows, n, vq, vkv, static_cast<uint4*>(q), static_cast<uint4*>(k),
      static_cast<uint4*>(v));
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const void* x, const int32_t* sel, const void* gain, void* y, int64_t n_rows, int hidden,
                          float eps, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  rmsnorm_kernel<<<static_cast<unsigned>(n_rows), kNormThreads, 0, s>>>(
      static_cast<const uint4*>(x), sel, static_cast<const uint4*>(gain), static_cast<uint4*>(y), hidden / 8, eps);
  return hipGetLastError();
}

hipError_t launch_swiglu(const void* gu, void* act, int64_t n, int ffn, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int vf = ffn / 8;
  swiglu_kernel<<<grid_for(n * vf, 256), 256, 0, s>>>(static_cast<const uint4*>(gu), static_cast<uint4*>(act), n, vf);
  return hipGetLastError();
}

int lm_head_chunks(int hidden) { return hidden >= 2048 ? 8 : 1; }

hipError_t launch_lm_head(const void* nf, const void* w, float* part, int nq, int hidden, int vocab, hipStream_t s) {
  const int chunks = lm_head_chunks(hidden);
  const int rows = (hidden + chunks - 1) / chunks;
  const dim3 grid((vocab + kHeadCols - 1) / kHeadCols, chunks);
  const u16* n = static_cast<const u16*>(nf);
  const uint4* wv = static_cast<const uint4*>(w);
  switch (nq) {
    case 1: lm_head_kernel<1><<<grid, kHeadThreads, 0, s>>>(n, wv, part, hidden, vocab, rows); break;
    case 2: lm_head_kernel<2><<<grid, kHeadThreads, 0, s>>>(n, wv, part, hidden, vocab, rows); break;
    case 4: lm_head_kernel<4><<<grid, kHeadThreads, 0, s>>>(n, wv, part, hidden, vocab, rows); break;
    case 8: lm_head_kernel<8><<<grid, kHeadThreads, 0, s>>>(n, wv, part, hidden, vocab, rows); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t gemv_part_bytes(int M, int N, int K) {
  (void)K;
  return static_cast<size_t>(kGemvChunks) * M * N * sizeof(float);
}

namespace {
// Pass 1 of the GEMV; returns the number of K slices (0 on a launch error).
int gemv_pass1(const void* x, const void* w, int M, int N, int K, float* part, hipStream_t s) {
  const int chunks = std::min(kGemvChunks, (K + 31) / 32);
  const int rows = (K + chunks - 1) / chunks;
  const dim3 grid((N + kGemvCols - 1) / kGemvCols, chunks);
  const u16* xx = static_cast<const u16*>(x);
  const uint4* ww = static_cast<const uint4*>(w);
  if (M == 1) gemv_partial_kernel<1><<<grid, 256, 0, s>>>(xx, ww, part, M, N, K, rows);
  else if (M == 2) gemv_partial_kernel<2><<<grid, 256, 0, s>>>(xx, ww, part, M, N, K, rows);
  else if (M <= 4) gemv_partial_kernel<4><<<grid, 256, 0, s>>>(xx, ww, part, M, N, K, rows);
  else gemv_partial_kernel<8><<<grid, 256, 0, s>>>(xx, ww, part, M, N, K, rows);
  return hipGetLastError() == hipSuccess ? chunks : 0;
}

bool gemv_args_ok(int M, int N, int K, size_t part_bytes) {
  return M >= 1 && M <= 8 && N % 8 == 0 && K >= 1 && gemv_part_bytes(M, N, K) <= part_bytes;
}
}  // namespace

hipError_t launch_gemv(const void* x, const void* w, void* y, int M, int N, int K, bool residual, float* part,
                       size_t part_bytes, hipStream_t s) {
  if (!gemv_args_ok(M, N, K, part_bytes)) return hipErrorInvalidValue;
  const int chunks = gemv_pass1(x, w, M, N, K, part, s);
  if (!chunks) return hipGetLastError();
  const int64_t items = static_cast<int64_t>(M) * N;
  gemv_reduce_kernel<<<static_cast<int>((items + 255) / 256), 256, 0, s>>>(part, chunks, M, N, static_cast<u16*>(y),
                                                                           residual);
  return hipGetLastError();
}

hipError_t launch_gemv_qkv(const void* x, const void* w, int M, int K, const int32_t* rows, int q_elems,
                           int kv_elems, void* q, void* k, void* v, float* part, size_t part_bytes, hipStream_t s) {
  const int N = q_elems + 2 * kv_elems;
  if (!gemv_args_ok(M, N, K, part_bytes)) return hipErrorInvalidValue;
  const int chunks = gemv_pass1(x, w, M, N, K, part, s);
  if (!chunks) return hipGetLastError();
  const int64_t items = static_cast<int64_t>(M) * N;
  gemv_reduce_qkv_kernel<<<static_cast<int>((items + 255) / 256), 256, 0, s>>>(
      part, chunks, M, N, rows, q_elems, kv_elems, static_cast<u16*>(q), static_cast<u16*>(k), static_cast<u16*>(v));
  return hipGetLastError();
}

hipError_t launch_gemv_swiglu(const void* x, const void* w, void* act, int M, int ffn, int K, float* part,
                              size_t part_bytes, hipStream_t s) {
  if (!gemv_args_ok(M, 2 * ffn, K, part_bytes)) return hipErrorInvalidValue;
  const int chunks = gemv_pass1(x, w, M, 2 * ffn, K, part, s);
  if (!chunks) return hipGetLastError();
  const int64_t items = static_cast<int64_t>(M) * ffn;
  gemv_reduce_swiglu_kernel<<<static_cast<int>((items + 255) / 256), 256, 0, s>>>(part, chunks, M, ffn,
                                                                                  static_cast<u16*>(act));
  return hipGetLastError();
}

hipError_t launch_gemv_residual_norm(const void* x, const void* w, void* y, int M, int N, int K, const void* gain,
                                     void* nout, float eps, float* part, size_t part_bytes, hipStream_t s) {
  if (!gemv_args_ok(M, N, K, part_bytes) || N > kNormThreads * kNormVec * 8) return hipErrorInvalidValue;
  const int chunks = gemv_pass1(x, w, M, N, K, part, s);
  if (!chunks) return hipGetLastError();
  gemv_reduce_norm_kernel<<<static_cast<unsigned>(M), kNormThreads, 0, s>>>(
      part, chunks, M, N, static_cast<u16*>(y), static_cast<const uint4*>(gain), static_cast<uint4*>(nout), eps);
  return hipGetLastError();
}

hipError_t launch_reduce_residual_norm(const float* part, int slices, int M, int N, void* y, const void* gain,
                                       void* nout, float eps, hipStream_t s) {
  if (M < 1 || N % 8 != 0 || N > kNormThreads * kNormVec * 8 || slices < 1) return hipErrorInvalidValue;
  gemv_reduce_norm_kernel<<<static_cast<unsigned>(M), kNormThreads, 0, s>>>(
      part, slices, M, N, static_cast<u16*>(y), static_cast<const uint4*>(gain), static_cast<uint4*>(nout), eps);
  return hipGetLastError();
}

size_t argmax_scratch_bytes(int nq, int vocab) {
  return static_cast<size_t>(nq) * ((vocab + kArgCols - 1) / kArgCols) * (sizeof(float) + sizeof(int));
}

hipError_t launch_argmax(const float* part, int nq, int n_rows, int hidden, int vocab, float* logits, int32_t* token,
                         void* scratch, hipStream_t s) {
  if (n_rows < 1 || n_rows > nq || vocab % 8 != 0 || !scratch) return hipErrorInvalidValue;
  const int nb = (vocab + kArgCols - 1) / kArgCols;
  float* bv = static_cast<float*>(scratch);
  int* bi = reinterpret_cast<int*>(bv + static_cast<size_t>(nq) * nb);
  argmax_blocks_kernel<<<dim3(nb, n_rows), kArgThreads, 0, s>>>(part, lm_head_chunks(hidden), nq, vocab, logits, bv, bi);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  argmax_rows_kernel<<<n_rows, kArgThreads, 0, s>>>(bv, bi, nb, token);
  return hipGetLastError();
}

}  // namespace spanq
