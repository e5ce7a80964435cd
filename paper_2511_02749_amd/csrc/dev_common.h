// Device helpers shared by the HIP kernels: bf16 storage and rotary angles.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace spanq {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float(static_cast<uint32_t>(x) << 16); }

// float -> bfloat16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>(0x7fc0u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f32_to_bf16(x); }

// A split-KV partial of one (row, head), written by the attention kernels and merged
// by the combine pass, with (m, l) in fp32 beside it.  bf16 pools store O / l in fp16:
// a convex combination of V rows, so bounded by the largest |V| (fp16 holds up to
// 65504), with 11 significant bits against the output's 8, at half the bytes of fp32.
// fp32 pools store the unnormalised O in fp32.
typedef _Float16 f16_t;
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
template <typename T>
struct PartOf;
template <>
struct PartOf<bf16_t> {
  using type = f16_t;
  static constexpr bool normalized = true;
};
template <>
struct PartOf<float> {
  using type = float;
  static constexpr bool normalized = false;
};

// Position of key slot s (0..15) inside a page's transposed V rows: bits 2 and 3
// swapped, i.e. quads ordered {0-3, 8-11, 4-7, 12-15}.  A P.V operand of the MFMA
// kernel then covers 8 consecutive positions (one 16-byte LDS read).
__host__ __device__ __forceinline__ int v_pos(int s) { return (s & 3) | ((s & 4) << 1) | ((s & 8) >> 1); }

// cos and sin of position `pos` at frequency index i (rotary pair (i, i + d/2)),
// read from the pool's table of (cos, sin) pairs laid out [position][d/2]; the
// table is computed on the host in double precision and rounded once.
__device__ __forceinline__ void rope_cs(const float2* __restrict__ tab, int half, int pos, int i, float* sn,
                                        float* cs) {
  const float2 v = tab[static_cast<int64_t>(pos) * half + i];
  *cs = v.x;
  *sn = v.y;
}

}  // namespace spanq
