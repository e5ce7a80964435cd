// The page write of new keys and values (K3), shared by the page-write kernel and
// the cross kernel that writes its cross-segment pages itself: one page, kv heads
// [hb, he).  K goes to [kv_head][slot][d] rotated at its position; V goes
// transposed to [kv_head][d][v_pos(slot)].  Unfilled slots are zeroed so that
// masked keys never feed a NaN into the P.V product.  Every global access is a
// 16-byte chunk; the V transpose goes through `tile` (32 KiB of LDS), a group of kv
// heads at a time.  All nth threads of the work-group call it (it has barriers).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dev_common.h"
#include "work.h"

namespace spanq {

template <typename T>
struct Chunk16 {
  static constexpr int E = 16 / static_cast<int>(sizeof(T));  // elements per chunk
  T x[E];
};

template <typename T>
__device__ __forceinline__ Chunk16<T> load16(const T* p) {
  return __builtin_bit_cast(Chunk16<T>, *reinterpret_cast<const uint4*>(p));
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const Chunk16<T>& c) {
  *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, c);
}

constexpr int kPageWriteLds = 32768;

// Eight LDS rows of four bf16 each (the slots of eight consecutive positions, dims
// d .. d + 3) regrouped into four 16-byte chunks, chunk j holding dim d + j of the
// eight positions in order.
__device__ __forceinline__ void regroup_8x4(const uint2 (&in)[8], uint4 (&out)[4]) {
  uint32_t w[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint2 a = in[2 * k], b = in[2 * k + 1];
    w[0][k] = (a.x & 0xffffu) | (b.x << 16);
    w[1][k] = (a.x >> 16) | (b.x & 0xffff0000u);
    w[2][k] = (a.y & 0xffffu) | (b.y << 16);
    w[3][k] = (a.y >> 16) | (b.y & 0xffff0000u);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) out[j] = uint4{w[j][0], w[j][1], w[j][2], w[j][3]};
}

template <typename T, int D>
__device__ __forceinline__ void write_page_heads(const NewPage& pg, int hb, int he, const T* __restrict__ k,
                                                 const T* __restrict__ v, T* __restrict__ pool, int64_t layer_off,
                                                 int hkv, const float2* __restrict__ rope, T* tile, int tid,
                                                 int nth) {
  constexpr int E = Chunk16<T>::E;
  constexpr int H = D / 2;
  constexpr int HG = kPageWriteLds / (kPage * D * static_cast<int>(sizeof(T)));  // kv heads per LDS pass
  const int64_t page_elems = 2ll * hkv * kPage * D;
  T* kp = pool + layer_off + static_cast<int64_t>(pg.page_id) * page_elems;
  T* vp = kp + static_cast<int64_t>(hkv) * kPage * D;

  // K: item (slot, chunk of E rotary pairs (i, i + H), group of up to KH heads): the
  // pairs' (cos, sin) are read once for the item's heads
  constexpr int KH = 4;
  const int hgroups = (he - hb + KH - 1) / KH;
  for (int e = tid; e < hgroups * kPage * (H / E); e += nth) {
    const int q = e % (H / E);
    const int s = (e / (H / E)) % kPage;
    const int h0 = hb + KH * (e / (H / E * kPage));
    const int h1 = min(he, h0 + KH);
    float cs[E], sn[E];
    if (s < pg.n_valid) {
      const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(pg.pos0 + s) * H + q * E);
#pragma unroll
      for (int u2 = 0; u2 < E / 2; ++u2) {
        const float4 w = cs4[u2];  // (cos, sin) of pairs q*E + 2u2 and + 1
        cs[2 * u2] = w.x;
        sn[2 * u2] = w.y;
        cs[2 * u2 + 1] = w.z;
        sn[2 * u2 + 1] = w.w;
      }
    }
    for (int h = h0; h < h1; ++h) {
      Chunk16<T> y0, y1;
      if (s < pg.n_valid) {
        const T* src = k + (static_cast<int64_t>(pg.src_row + s) * hkv + h) * D + q * E;
        const Chunk16<T> x0 = load16(src), x1 = load16(src + H);
#pragma unroll
        for (int u = 0; u < E; ++u) {
          const float a0 = to_f32(x0.x[u]), a1 = to_f32(x1.x[u]);
          y0.x[u] = from_f32<T>(a0 * cs[u] - a1 * sn[u]);
          y1.x[u] = from_f32<T>(a1 * cs[u] + a0 * sn[u]);
        }
      } else {
#pragma unroll
        for (int u = 0; u < E; ++u) y0.x[u] = y1.x[u] = from_f32<T>(0.f);
      }
      T* dst = kp + (static_cast<int64_t>(h) * kPage + s) * D + q * E;
      store16(dst, y0);
      store16(dst + H, y1);
    }
  }

  // V: rows [slot][d] of a group of heads into LDS, then transposed rows out
  for (int h0 = hb; h0 < he; h0 += HG) {
    const int hn = min(HG, he - h0);
    for (int e = tid; e < kPage * hn * (D / E); e += nth) {
      const int qd = e % (D / E);
      const int sh = e / (D / E);
      const int hh = sh % hn;
      const int s = sh / hn;
      Chunk16<T> val;
      if (s < pg.n_valid) {
        val = load16(v + (static_cast<int64_t>(pg.src_row + s) * hkv + h0 + hh) * D + qd * E);
      } else {
#pragma unroll
        for (int u = 0; u < E; ++u) val.x[u] = from_f32<T>(0.f);
      }
      store16(tile + (s * HG + hh) * D + qd * E, val);
    }
    __syncthreads();
    // row (head, d) holds 16 positions; position p carries slot v_pos(p) (an involution)
    if constexpr (sizeof(T) == 2) {
      // item (head, four dims, half of the positions): eight 8-byte reads, four chunks out
      for (int e = tid; e < hn * (D / 4) * 2; e += nth) {
        const int pc = e & 1;
        const int d4 = (e >> 1) % (D / 4);
        const int hh = (e >> 1) / (D / 4);
        uint2 in[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          in[u] = *reinterpret_cast<const uint2*>(tile + (v_pos(8 * pc + u) * HG + hh) * D + 4 * d4);
        uint4 out[4];
        regroup_8x4(in, out);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<uint4*>(vp + (static_cast<int64_t>(h0 + hh) * D + 4 * d4 + j) * kPage + 8 * pc) = out[j];
      }
    } else {
      for (int e = tid; e < hn * D * (kPage / E); e += nth) {
        const int pc = e % (kPage / E);
        const int hd = e / (kPage / E);
        const int d = hd % D;
        const int hh = hd / D;
        Chunk16<T> out;
#pragma unroll
        for (int u = 0; u < E; ++u) out.x[u] = tile[(v_pos(pc * E + u) * HG + hh) * D + d];
        store16(vp + (static_cast<int64_t>(h0 + hh) * D + d) * kPage + pc * E, out);
      }
    }
    __syncthreads();
  }
}

// The same write for n pages (pages[0 .. n)) and one kv head h, the pages in groups
// that fill `tile`: the K chunks and V rows of a whole group are in flight at once,
// with two barriers per group (a cross segment's 8 pages at head dim 128 are one
// group).
template <typename T, int D>
__device__ __forceinline__ void write_pages_one_head(const NewPage* __restrict__ pages, int n, int h,
                                                     const T* __restrict__ k, const T* __restrict__ v,
                                                     T* __restrict__ pool, int64_t layer_off, int hkv,
                                                     const float2* __restrict__ rope, T* tile, int tid, int nth) {
  constexpr int E = Chunk16<T>::E;
  constexpr int H = D / 2;
  constexpr int PG = kPageWriteLds / (kPage * D * static_cast<int>(sizeof(T)));  // pages per LDS pass
  const int64_t page_elems = 2ll * hkv * kPage * D;
  auto kbase = [&](const NewPage& pg) {
    return pool + layer_off + static_cast<int64_t>(pg.page_id) * page_elems + static_cast<int64_t>(h) * kPage * D;
  };
  for (int p0 = 0; p0 < n; p0 += PG) {
    const int pn = min(PG, n - p0);
    // K: item (page, slot, chunk of E rotary pairs)
    for (int e = tid; e < pn * kPage * (H / E); e += nth) {
      const int q = e % (H / E);
      const int ps = e / (H / E);
      const int s = ps % kPage;
      const NewPage pg = pages[p0 + ps / kPage];
      Chunk16<T> y0, y1;
      if (s < pg.n_valid) {
        const T* src = k + (static_cast<int64_t>(pg.src_row + s) * hkv + h) * D + q * E;
        const Chunk16<T> x0 = load16(src), x1 = load16(src + H);
        const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(pg.pos0 + s) * H + q * E);
#pragma unroll
        for (int u2 = 0; u2 < E / 2; ++u2) {
          const float4 w = cs4[u2];  // (cos, sin) of pairs q*E + 2u2 and + 1
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const int u = 2 * u2 + b;
            const float cs = b ? w.z : w.x, sn = b ? w.w : w.y;
            const float a0 = to_f32(x0.x[u]), a1 = to_f32(x1.x[u]);
            y0.x[u] = from_f32<T>(a0 * cs - a1 * sn);
            y1.x[u] = from_f32<T>(a1 * cs + a0 * sn);
          }
        }
      } else {
#pragma unroll
        for (int u = 0; u < E; ++u) y0.x[u] = y1.x[u] = from_f32<T>(0.f);
      }
      T* dst = kbase(pg) + s * D + q * E;
      store16(dst, y0);
      store16(dst + H, y1);
    }
    // V: rows [page][slot][d] into LDS, then rows [d][16 positions] out
    for (int e = tid; e < pn * kPage * (D / E); e += nth) {
      const int qd = e % (D / E);
      const int ps = e / (D / E);
      const int s = ps % kPage;
      const NewPage pg = pages[p0 + ps / kPage];
      Chunk16<T> val;
      if (s < pg.n_valid) {
        val = load16(v + (static_cast<int64_t>(pg.src_row + s) * hkv + h) * D + qd * E);
      } else {
#pragma unroll
        for (int u = 0; u < E; ++u) val.x[u] = from_f32<T>(0.f);
      }
      store16(tile + ps * D + qd * E, val);
    }
    __syncthreads();
    if constexpr (sizeof(T) == 2) {
      for (int e = tid; e < pn * (D / 4) * 2; e += nth) {
        const int pc = e & 1;
        const int d4 = (e >> 1) % (D / 4);
        const int pi = (e >> 1) / (D / 4);
        uint2 in[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          in[u] = *reinterpret_cast<const uint2*>(tile + (pi * kPage + v_pos(8 * pc + u)) * D + 4 * d4);
        uint4 out[4];
        regroup_8x4(in, out);
        T* vrow = kbase(pages[p0 + pi]) + static_cast<int64_t>(hkv) * kPage * D;
#pragma unroll
        for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(vrow + (4 * d4 + j) * kPage + 8 * pc) = out[j];
      }
    } else {
      for (int e = tid; e < pn * D * (kPage / E); e += nth) {
        const int pc = e % (kPage / E);
        const int pd = e / (kPage / E);
        const int d = pd % D;
        const int pi = pd / D;
        Chunk16<T> out;
#pragma unroll
        for (int u = 0; u < E; ++u) out.x[u] = tile[(pi * kPage + v_pos(pc * E + u)) * D + d];
        store16(kbase(pages[p0 + pi]) + static_cast<int64_t>(hkv) * kPage * D + d * kPage + pc * E, out);
      }
    }
    __syncthreads();
  }
}

}  // namespace spanq
