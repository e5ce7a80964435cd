// Machine-peak probes: an MFMA-only loop and a streaming HBM read.  They measure what
// this chip attains for the two resources the attention kernels are bound by, so that
// the kernels' rates can be read against it as well as against the published peaks.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "mfma_common.h"

namespace spanq {

// Written only under a condition the compiler cannot decide, so that the work that
// feeds it is kept (external linkage: the stores cannot be dropped); nothing reads them.
__device__ float g_probe_sink_f;
__device__ uint32_t g_probe_sink_u;

namespace {

using namespace mfma;

constexpr int kMfmaChains = 4;  // independent accumulator chains per wave

// Every wave runs iters rounds of kMfmaChains independent 32x32x16 bf16 MFMAs, with
// operands held in registers: no memory traffic, no other arithmetic in the loop.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void mfma_peak_kernel(int iters) {
  const uint32_t lane = threadIdx.x & 63;
  // small bf16 values that depend on the lane (0x3C00 + lane is about 2^-7 .. 2^-6)
  const uint32_t wa = (0x3C00u + lane) * 0x00010001u, wb = (0x3C40u + (lane ^ 5)) * 0x00010001u;
  const bf16x8_t a = __builtin_bit_cast(bf16x8_t, u32x4_t{wa, wa, wa, wa});
  const bf16x8_t b = __builtin_bit_cast(bf16x8_t, u32x4_t{wb, wb, wb, wb});
  f32x16_t acc[kMfmaChains];
#pragma unroll
  for (int c = 0; c < kMfmaChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int c = 0; c < kMfmaChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kMfmaChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[c][i];
  if (s == -1.f) g_probe_sink_f = s;
}

// Grid-stride read of n16 16-byte words with four loads in flight per lane, folded
// by xor into one word per lane.
__global__ __launch_bounds__(256) void read_peak_kernel(const u32x4_t* __restrict__ src, int64_t n16) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  uint32_t x = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4_t v0 = __builtin_nontemporal_load(src + i);
    const u32x4_t v1 = __builtin_nontemporal_load(src + i + stride);
    const u32x4_t v2 = __builtin_nontemporal_load(src + i + 2 * stride);
    const u32x4_t v3 = __builtin_nontemporal_load(src + i + 3 * stride);
    x ^= (v0[0] ^ v0[1] ^ v0[2] ^ v0[3]) ^ (v1[0] ^ v1[1] ^ v1[2] ^ v1[3]) ^ (v2[0] ^ v2[1] ^ v2[2] ^ v2[3]) ^
         (v3[0] ^ v3[1] ^ v3[2] ^ v3[3]);
  }
  for (; i < n16; i += stride) {
    const u32x4_t v = __builtin_nontemporal_load(src + i);
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (x == 0x9E3779B9u) g_probe_sink_u = x;
}

}  // namespace

double probe_mfma_flops(int iters, int n_cu) {
  constexpr int kWavesPerCu = 8;
  return 2.0 * 32 * 32 * 16 * kMfmaChains * static_cast<double>(iters) * kWavesPerCu * n_cu;
}

hipError_t launch_probe_mfma(int iters, int n_cu, hipStream_t s) {
  // two 4-wave work-groups per compute unit: two waves on each SIMD
  mfma_peak_kernel<<<2 * n_cu, 256, 0, s>>>(iters);
  return hipGetLastError();
}

hipError_t launch_probe_read(const void* buf, int64_t bytes, int n_cu, hipStream_t s) {
  read_peak_kernel<<<8 * n_cu, 256, 0, s>>>(static_cast<const u32x4_t*>(buf), bytes / 16);
  return hipGetLastError();
}

}  // namespace spanq
