// Skinny GEMM of the decoder stack: Y[M][N] = X[M][K] W[K][N] (+ Y) for a few hundred
// rows (a cache-hit query computes only its question's rows, section 5.6) and a long
// reduction (K >= 4 N: the FFN's down projection), bf16 in and out, fp32
// accumulation, on v_mfma_f32_32x32x16_bf16.
//
// At these row counts the product is bound by reading W once (2 M flops per weight
// byte: about 300 at M = 256, where HBM and the bf16 MFMA peak meet), so the kernel
// streams each weight exactly once, from a transposed copy Wt[N][K] that the model
// makes once: both MFMA operands are then runs of eight consecutive k per lane.
//
// Work-group: 4 waves, 64 columns n by up to 256 rows, over one slice of K, in chunks
// of 64 k.  Wave w takes rows 64 w .. 64 w + 63 (two 32-row blocks) and both 32-column
// blocks: four 32 x 32 accumulators.  A chunk of Wt (64 x 64, 8 KiB) goes to LDS by
// global-to-LDS DMA (each wave moves a quarter; rows XOR-swizzled at 16 bytes), where
// all four waves read it; a wave's own X rows go straight to registers.  Both streams
// run D chunks ahead (a ring of D + 1 LDS stages and D + 1 register sets), so that
// about D x 8 KiB of weights per work-group are in flight to cover HBM latency: the
// wait before chunk c is a fixed vector-memory count (everything issued for chunks
// c + 1 .. c + D - 1 may still be outstanding).  When N / 64 tiles do not fill the
// chip, K is split and the slices write fp32 partials that a second kernel adds in
// slice order (with the residual), so a result does not depend on timing or on the
// number of rows.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "mfma_common.h"
#include "stack_kernels.h"

namespace spanq {
namespace {

using mfma::block_sync;
using mfma::dma16_m0;
using mfma::lds_byte;
using mfma::wait_vm_all;
using mfma::wait_vmcnt;

constexpr int kSkN = 64;        // columns per work-group
constexpr int kSkKC = 64;       // k per chunk
constexpr int kSkMinM = 129;    // every wave has rows from here on
constexpr int kSkMaxM = 256;    // rows per launch
constexpr int kSkThreads = 256;
constexpr int kSkDepth = 4;     // chunks in flight ahead of the one computed
constexpr int kSkStage = kSkN * kSkKC * 2;  // 8 KiB of Wt per chunk
constexpr int kSkLds = (kSkDepth + 1) * kSkStage;

// 16-byte chunk c of Wt row n (within a stage) sits at chunk c ^ (n & 7).
__device__ __forceinline__ int wswz(int n) { return n & 7; }

// NC: chunks per K slice.  The chunk loop is unrolled whole, so that the compiler's
// own waits for the X registers see one straight sequence of loads (a loop's back
// edge would make them conservative, waiting for everything once per turn).
template <int D, int NC>
__global__ __launch_bounds__(kSkThreads) void skinny_gemm_kernel(const bf16_t* __restrict__ x,
                                                                  const bf16_t* __restrict__ wt,
                                                                  bf16_t* __restrict__ y, float* __restrict__ part,
                                                                  int M, int N, int K, int residual) {
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
  const int lane = static_cast<int>(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int n0 = static_cast<int>(blockIdx.x) * kSkN;
  const int slice = static_cast<int>(blockIdx.y);
  const int k_begin = slice * NC * kSkKC;
  const int half = lane >> 5, l32 = lane & 31;

  // Wt DMA of one chunk: 8 instructions of 1 KiB (8 rows of 128 bytes); wave w issues
  // 2w and 2w + 1.  Lane l of instruction q writes row 8q + l / 8, stored chunk l % 8.
  const int wr0 = 16 * wave + (lane >> 3), wr1 = wr0 + 8;
  const bf16_t* wsrc0 = wt + static_cast<int64_t>(n0 + wr0) * K + k_begin + 8 * ((lane & 7) ^ wswz(wr0));
  const bf16_t* wsrc1 = wt + static_cast<int64_t>(n0 + wr1) * K + k_begin + 8 * ((lane & 7) ^ wswz(wr1));
  // This wave's X rows (clamped into the matrix; rows past M are computed and dropped).
  const bf16_t* xr0 = x + static_cast<int64_t>(min(64 * wave + l32, M - 1)) * K + k_begin + 8 * half;
  const bf16_t* xr1 = x + static_cast<int64_t>(min(64 * wave + 32 + l32, M - 1)) * K + k_begin + 8 * half;

  // D + 1 register sets of X operands: set u holds chunk c with c % (D + 1) == u,
  // [row block][k step].
  bf16x8_t xs[D + 1][2][4];
  // Issue chunk c: its Wt DMA (2 instructions) then its X loads (8).
  auto issue = [&](int c, bf16x8_t (&xv)[2][4]) {
    const int ofs = c * kSkKC;
    unsigned char* st = lds + (c % (D + 1)) * kSkStage;
    dma16_m0(wsrc0 + ofs, lds_byte(st + (2 * wave) * 1024));
    dma16_m0(wsrc1 + ofs, lds_byte(st + (2 * wave + 1) * 1024));
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      xv[0][ks] = *reinterpret_cast<const bf16x8_t*>(xr0 + ofs + 16 * ks);
      xv[1][ks] = *reinterpret_cast<const bf16x8_t*>(xr1 + ofs + 16 * ks);
    }
  };

  f32x16_t acc[2][2];  // [row block][column block]
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

  auto compute = [&](int c, const bf16x8_t (&xv)[2][4]) {
    const unsigned char* st = lds + (c % (D + 1)) * kSkStage;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int cl = 2 * ks + half;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int n = 32 * i + l32;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(st + n * 128 + 16 * (cl ^ wswz(n)));
        acc[0][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xv[0][ks], acc[0][i], 0, 0, 0);
        acc[1][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xv[1][ks], acc[1][i], 0, 0, 0);
      }
    }
  };

#pragma unroll
  for (int c = 0; c < D && c < NC; ++c) issue(c, xs[c]);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    // chunk c is in once everything but the chunks c + 1 .. c + D - 1 issued after it is
    if (c + D - 1 < NC)
      wait_vmcnt<10 * (D - 1)>();
    else
      wait_vm_all();
    block_sync();  // every wave's share of the stage is in; chunk c - 1's stage is free
    if (c + D < NC) issue(c + D, xs[(c + D) % (D + 1)]);
    compute(c, xs[c % (D + 1)]);
  }

  // Accumulator [j][i], element r: row m = 64 wave + 32 j + l32, column n = 32 i +
  // 8 (r / 4) + 4 half + r % 4 of the tile: four runs of four consecutive n per lane.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = 64 * wave + 32 * j + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + 32 * i + 8 * g + 4 * half;
        float v0 = acc[j][i][4 * g], v1 = acc[j][i][4 * g + 1], v2 = acc[j][i][4 * g + 2], v3 = acc[j][i][4 * g + 3];
        if (part) {
          *reinterpret_cast<float4*>(part + (static_cast<int64_t>(slice) * M + m) * N + n) =
              make_float4(v0, v1, v2, v3);
        } else {
          bf16_t* dst = y + static_cast<int64_t>(m) * N + n;
          if (residual) {
            const uint2 r = *reinterpret_cast<const uint2*>(dst);
            v0 += mfma::lo_bf16(r.x);
            v1 += mfma::hi_bf16(r.x);
            v2 += mfma::lo_bf16(r.y);
            v3 += mfma::hi_bf16(r.y);
          }
          *reinterpret_cast<uint2*>(dst) = make_uint2(mfma::pack_bf16x2(v0, v1), mfma::pack_bf16x2(v2, v3));
        }
      }
  }
}

// Y[m][n..n+3] = bf16(sum over slices in order (+ Y)), four columns per thread.
__global__ __launch_bounds__(256) void skinny_reduce_kernel(const float* __restrict__ part, int slices, int M, int N,
                                                            bf16_t* __restrict__ y, int residual) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;  // quad index
  const int64_t quads = static_cast<int64_t>(M) * N / 4;
  if (i >= quads) return;
  const int64_t plane = static_cast<int64_t>(M) * N;
  float4 s = reinterpret_cast<const float4*>(part)[i];
  for (int k = 1; k < slices; ++k) {
    const float4 t = reinterpret_cast<const float4*>(part + k * plane)[i];
    s.x += t.x;
    s.y += t.y;
    s.z += t.z;
    s.w += t.w;
  }
  uint2* dst = reinterpret_cast<uint2*>(y) + i;
  if (residual) {
    const uint2 r = *dst;
    s.x += mfma::lo_bf16(r.x);
    s.y += mfma::hi_bf16(r.x);
    s.z += mfma::lo_bf16(r.y);
    s.w += mfma::hi_bf16(r.y);
  }
  *dst = make_uint2(mfma::pack_bf16x2(s.x, s.y), mfma::pack_bf16x2(s.z, s.w));
}

// out[c][r] = in[r][c], 64 x 64 tiles through LDS (bf16 bit patterns).
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ in, uint16_t* __restrict__ out,
                                                             int64_t R, int64_t C) {
  __shared__ uint16_t tile[64][65];
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64, c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int tx = static_cast<int>(threadIdx.x) & 63, ty = static_cast<int>(threadIdx.x) >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < R && c < C) ? in[r * C + c] : uint16_t{0};
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < C && r < R) out[c * R + r] = tile[tx][i];
  }
}

}  // namespace

// Chunks per K slice the kernel is built for (its loop is unrolled whole).
constexpr int kSkChunkCounts[] = {4, 8, 16, 32, 64};

// K slices: the fewest that give the chip's 256 compute units a work-group each (or
// the most there are), every slice a count of chunks the kernel is built for.
int skinny_gemm_slices(int M, int N, int K) {
  (void)M;
  const int tiles = N / kSkN, chunks = K / kSkKC;
  int best = 0;
  for (int s = 1; s <= chunks; ++s) {
    if (chunks % s != 0) continue;
    const int nc = chunks / s;
    bool built = false;
    for (int c : kSkChunkCounts) built |= c == nc;
    if (!built) continue;
    best = s;
    if (static_cast<int64_t>(tiles) * s >= 256) break;
  }
  return best;
}

// Shapes the kernel takes: besides the row range and tile multiples, a reduction at
// least four times the output width (K >= 4 N, e.g. the FFN's down projection).  Each
// work-group reads all of its K slice of X, so X is read N / 64 times over from L2;
// on wider outputs (q/k/v, output and gate/up projections at 256 rows) that traffic
// makes this kernel slower than hipBLASLt's tiles, while on long reductions with few
// output tiles hipBLASLt leaves most of the chip idle (measured at 256 rows: K 8192,
// N 2048: 28 us against 43 us; K 2048, N 16384: 42 us against 27 us).
bool skinny_gemm_fits(int64_t M, int64_t N, int64_t K) {
  return M >= kSkMinM && M <= kSkMaxM && N >= kSkN && N % kSkN == 0 && N <= (int64_t{1} << 24) && K >= 4 * N &&
         K >= kSkKC &&
         K % kSkKC == 0 && K <= (int64_t{1} << 20) &&
         skinny_gemm_slices(static_cast<int>(M), static_cast<int>(N), static_cast<int>(K)) > 0;
}

size_t skinny_gemm_part_bytes(int M, int N, int K) {
  const int s = skinny_gemm_slices(M, N, K);
  return s > 1 ? static_cast<size_t>(s) * M * N * sizeof(float) : 0;
}

namespace {
// The main kernel for `slices` K slices (partials to part when slices > 1).
hipError_t skinny_main(const void* x, const void* wt, void* y, int M, int N, int K, int slices, bool residual,
                       float* part, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(N / kSkN), static_cast<unsigned>(slices));
  const int nc = K / kSkKC / slices;
  const bf16_t *xb = static_cast<const bf16_t*>(x), *wb = static_cast<const bf16_t*>(wt);
  bf16_t* yb = static_cast<bf16_t*>(y);
  float* pb = slices > 1 ? part : nullptr;
  const int r = residual ? 1 : 0;
  switch (nc) {
    case 4: hipLaunchKernelGGL((skinny_gemm_kernel<kSkDepth, 4>), grid, dim3(kSkThreads), kSkLds, s, xb, wb, yb, pb, M, N, K, r); break;
    case 8: hipLaunchKernelGGL((skinny_gemm_kernel<kSkDepth, 8>), grid, dim3(kSkThreads), kSkLds, s, xb, wb, yb, pb, M, N, K, r); break;
    case 16: hipLaunchKernelGGL((skinny_gemm_kernel<kSkDepth, 16>), grid, dim3(kSkThreads), kSkLds, s, xb, wb, yb, pb, M, N, K, r); break;
    case 32: hipLaunchKernelGGL((skinny_gemm_kernel<kSkDepth, 32>), grid, dim3(kSkThreads), kSkLds, s, xb, wb, yb, pb, M, N, K, r); break;
    case 64: hipLaunchKernelGGL((skinny_gemm_kernel<kSkDepth, 64>), grid, dim3(kSkThreads), kSkLds, s, xb, wb, yb, pb, M, N, K, r); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_skinny_gemm(const void* x, const void* wt, void* y, int M, int N, int K, bool residual, float* part,
                              size_t part_bytes, hipStream_t s) {
  if (!skinny_gemm_fits(M, N, K)) return hipErrorInvalidValue;
  const int slices = skinny_gemm_slices(M, N, K);
  if (slices > 1 && (!part || part_bytes < skinny_gemm_part_bytes(M, N, K))) return hipErrorInvalidValue;
  hipError_t e = skinny_main(x, wt, y, M, N, K, slices, residual, part, s);
  if (e != hipSuccess || slices == 1) return e;
  const int64_t quads = static_cast<int64_t>(M) * N / 4;
  hipLaunchKernelGGL(skinny_reduce_kernel, dim3(static_cast<unsigned>((quads + 255) / 256)), dim3(256), 0, s, part,
                     slices, M, N, static_cast<bf16_t*>(y), residual ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_skinny_gemm_norm(const void* x, const void* wt, void* y, int M, int N, int K, const void* gain,
                                   void* nout, float eps, float* part, size_t part_bytes, hipStream_t s) {
  if (!skinny_gemm_fits(M, N, K)) return hipErrorInvalidValue;
  const int slices = skinny_gemm_slices(M, N, K);
  if (slices == 1) return hipErrorNotSupported;
  if (!part || part_bytes < skinny_gemm_part_bytes(M, N, K)) return hipErrorInvalidValue;
  hipError_t e = skinny_main(x, wt, y, M, N, K, slices, true, part, s);
  if (e != hipSuccess) return e;
  return launch_reduce_residual_norm(part, slices, M, N, y, gain, nout, eps, s);
}

hipError_t launch_transpose_bf16(const void* in, void* out, int64_t R, int64_t C, hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((C + 63) / 64), static_cast<unsigned>((R + 63) / 64));
  hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t*>(in),
                     static_cast<uint16_t*>(out), R, C);
  return hipGetLastError();
}

}  // namespace spanq
