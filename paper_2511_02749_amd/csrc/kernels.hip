// Page writer (K3), generic span attention and KV-split combine for gfx950.
//
// Rotary encoding (section 5.5 cites RoFormer): rotate-half pairs (i, i + d/2)
// at angle pos * theta^(-2i/d); cos/sin come from the pool's position table.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"
#include "page_write.h"

namespace spanq {

// ------------------------------------------------------------------ K3
// One work-group per new page (per page and group of kv heads when pages are few);
// the write itself is write_page_heads (page_write.h).
template <typename T, int D>
__global__ __launch_bounds__(256) void rope_write_kernel(const NewPage* __restrict__ pages,
                                                         const T* __restrict__ k, const T* __restrict__ v,
                                                         T* __restrict__ pool, int64_t layer_off, int hkv,
                                                         int heads_per_group, const float2* __restrict__ rope) {
  __shared__ uint4 lds_raw[kPageWriteLds / 16];
  const NewPage pg = pages[blockIdx.x];
  // this work-group's kv heads (all of them, or one group when the pages are few)
  const int hb = blockIdx.y * heads_per_group;
  const int he = min(hkv, hb + heads_per_group);
  write_page_heads<T, D>(pg, hb, he, k, v, pool, layer_off, hkv, rope, reinterpret_cast<T*>(lds_raw),
                         static_cast<int>(threadIdx.x), static_cast<int>(blockDim.x));
}

template <typename T, int D>
static hipError_t rope_write_t(const PoolGeom& g, const NewPage* pages, int n, const void* k, const void* v,
                               const float2* rope, hipStream_t s) {
  // few pages (cross segments): a work-group per (page, kv head), so the write is not
  // left to a handful of compute units
  const int hpg = n >= 256 ? g.hkv : 1;
  hipLaunchKernelGGL((rope_write_kernel<T, D>), dim3(n, (g.hkv + hpg - 1) / hpg), dim3(256), 0, s, pages,
                     static_cast<const T*>(k), static_cast<const T*>(v), static_cast<T*>(g.base), g.layer_off, g.hkv,
                     hpg, rope);
  return hipGetLastError();
}

hipError_t launch_rope_write(const PoolGeom& g, const NewPage* pages, int n, const void* k, const void* v,
                             const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (g.dtype == SPAN_BF16) {
    if (g.d == 128) return rope_write_t<bf16_t, 128>(g, pages, n, k, v, rope, s);
    return rope_write_t<bf16_t, 64>(g, pages, n, k, v, rope, s);
  }
  if (g.d == 128) return rope_write_t<float, 128>(g, pages, n, k, v, rope, s);
  return rope_write_t<float, 64>(g, pages, n, k, v, rope, s);
}

// ------------------------------------------------------------------ decode writes
// Decoded tokens into their cross pages: one work-group per SlotWrite.  Keys are
// rotated at their positions into slots slot0 .., values go to the transposed slot
// positions.  A write at slot 0 opens a page fresh from the free list, whatever it
// held before: it also zeroes the slots past its tokens, as K3 does, so that masked
// keys never feed a stale NaN into the P.V product.  Other writes leave the page's
// other slots alone (earlier tokens, and the zeros past the end).
template <typename T, int D>
__global__ __launch_bounds__(256) void append_kv_kernel(const SlotWrite* __restrict__ writes,
                                                        const T* __restrict__ k, const T* __restrict__ v,
                                                        T* __restrict__ pool, int64_t layer_off, int hkv,
                                                        const float2* __restrict__ rope) {
  constexpr int E = Chunk16<T>::E;
  constexpr int H = D / 2;
  const SlotWrite w = writes[blockIdx.x];
  const int64_t page_elems = 2ll * hkv * kPage * D;
  T* kp = pool + layer_off + static_cast<int64_t>(w.page_id) * page_elems;
  T* vp = kp + static_cast<int64_t>(hkv) * kPage * D;
  // K: item (head, token j, chunk of E pairs (i, i + H))
  for (int e = threadIdx.x; e < hkv * w.n * (H / E); e += blockDim.x) {
    const int qc = e % (H / E);
    const int hj = e / (H / E);
    const int j = hj % w.n;
    const int h = hj / w.n;
    const T* src = k + (static_cast<int64_t>(w.src_row + j) * hkv + h) * D + qc * E;
    const Chunk16<T> x0 = load16(src), x1 = load16(src + H);
    const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(w.pos0 + j) * H + qc * E);
    Chunk16<T> y0, y1;
#pragma unroll
    for (int u2 = 0; u2 < E / 2; ++u2) {
      const float4 c = cs4[u2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int u = 2 * u2 + b;
        const float cs = b ? c.z : c.x, sn = b ? c.w : c.y;
        const float a0 = to_f32(x0.x[u]), a1 = to_f32(x1.x[u]);
        y0.x[u] = from_f32<T>(a0 * cs - a1 * sn);
        y1.x[u] = from_f32<T>(a1 * cs + a0 * sn);
      }
    }
    T* dst = kp + (static_cast<int64_t>(h) * kPage + w.slot0 + j) * D + qc * E;
    store16(dst, y0);
    store16(dst + H, y1);
  }
  // V: element (head, d, token j) to [head][d][v_pos(slot0 + j)]
  for (int e = threadIdx.x; e < hkv * D * w.n; e += blockDim.x) {
    const int j = e % w.n;
    const int hd = e / w.n;
    const int d = hd % D;
    const int h = hd / D;
    vp[(static_cast<int64_t>(h) * D + d) * kPage + v_pos(w.slot0 + j)] =
        v[(static_cast<int64_t>(w.src_row + j) * hkv + h) * D + d];
  }
  if (w.slot0 == 0 && w.n < kPage) {
    const int rest = kPage - w.n;  // slots n .. 15
    Chunk16<T> zero;
#pragma unroll
    for (int u = 0; u < E; ++u) zero.x[u] = from_f32<T>(0.f);
    for (int e = threadIdx.x; e < hkv * rest * (D / E); e += blockDim.x) {
      const int c = e % (D / E);
      const int hs = e / (D / E);
      const int h = hs / rest, slot = w.n + hs % rest;
      store16(kp + (static_cast<int64_t>(h) * kPage + slot) * D + c * E, zero);
    }
    for (int e = threadIdx.x; e < hkv * D * rest; e += blockDim.x) {
      const int slot = w.n + e % rest;
      const int hd = e / rest;
      vp[static_cast<int64_t>(hd) * kPage + v_pos(slot)] = from_f32<T>(0.f);
    }
  }
}

template <typename T, int D>
static hipError_t append_kv_t(const PoolGeom& g, const SlotWrite* w, int n, const void* k, const void* v,
                              const float2* rope, hipStream_t s) {
  hipLaunchKernelGGL((append_kv_kernel<T, D>), dim3(n), dim3(256), 0, s, w, static_cast<const T*>(k),
                     static_cast<const T*>(v), static_cast<T*>(g.base), g.layer_off, g.hkv, rope);
  return hipGetLastError();
}

hipError_t launch_append_kv(const PoolGeom& g, const SlotWrite* writes, int n, const void* k, const void* v,
                            const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (g.dtype == SPAN_BF16) {
    if (g.d == 128) return append_kv_t<bf16_t, 128>(g, writes, n, k, v, rope, s);
    return append_kv_t<bf16_t, 64>(g, writes, n, k, v, rope, s);
  }
  if (g.d == 128) return append_kv_t<float, 128>(g, writes, n, k, v, rope, s);
  return append_kv_t<float, 64>(g, writes, n, k, v, rope, s);
}

// ------------------------------------------------------------------ page moves
// Materialised repositioning: two work-groups per MovePage, one for the keys
// (blockIdx.y 0) and one for the values.  Keys of every kv head and slot are
// rotated by the page's delta (rotations in one plane add, so a key stored rotated
// at position p comes out rotated at p + delta); the transposed values are copied
// as they are.  Slots past n_valid hold the zeros K3 wrote and stay zero.  Each
// thread issues all its loads (four key items, eight value chunks) before storing.
template <typename T, int D>
__global__ __launch_bounds__(256) void move_pages_kernel(const MovePage* __restrict__ moves, T* __restrict__ pool,
                                                         int64_t layer_off, int hkv,
                                                         const float2* __restrict__ rope) {
  constexpr int E = Chunk16<T>::E;
  constexpr int H = D / 2;
  constexpr int U = 4;
  const MovePage m = moves[blockIdx.x];
  const int64_t page_elems = 2ll * hkv * kPage * D;
  const T* src = pool + layer_off + static_cast<int64_t>(m.src_page) * page_elems;
  T* dst = pool + layer_off + static_cast<int64_t>(m.dst_page) * page_elems;
  if (blockIdx.y != 0) {
    // V: the [kv head][d][slot] block, copied
    const uint4* vs = reinterpret_cast<const uint4*>(src + static_cast<int64_t>(hkv) * kPage * D);
    uint4* vd = reinterpret_cast<uint4*>(dst + static_cast<int64_t>(hkv) * kPage * D);
    const int n_v = hkv * kPage * D / E;
    for (int e0 = threadIdx.x; e0 < n_v; e0 += 2 * U * blockDim.x) {
      uint4 x[2 * U];
#pragma unroll
      for (int j = 0; j < 2 * U; ++j) {
        const int e = e0 + j * blockDim.x;
        if (e < n_v) x[j] = vs[e];
      }
#pragma unroll
      for (int j = 0; j < 2 * U; ++j) {
        const int e = e0 + j * blockDim.x;
        if (e < n_v) vd[e] = x[j];
      }
    }
    return;
  }
  const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(m.delta) * H);

  // K: item e = (head, slot) row e / (H / E), chunk q = e % (H / E) of E pairs (i, i + H)
  const int n_k = hkv * kPage * (H / E);
  for (int e0 = threadIdx.x; e0 < n_k; e0 += U * blockDim.x) {
    Chunk16<T> x0[U], x1[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int e = e0 + j * blockDim.x;
      if (e < n_k) {
        const int64_t off = static_cast<int64_t>(e / (H / E)) * D + (e % (H / E)) * E;
        x0[j] = load16(src + off);
        x1[j] = load16(src + off + H);
      }
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int e = e0 + j * blockDim.x;
      if (e >= n_k) break;
      const int q = e % (H / E);
      const int64_t off = static_cast<int64_t>(e / (H / E)) * D + q * E;
      Chunk16<T> y0, y1;
#pragma unroll
      for (int u2 = 0; u2 < E / 2; ++u2) {
        const float4 w = cs4[q * (E / 2) + u2];  // (cos, sin) of pairs q*E + 2u2 and + 1
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int u = 2 * u2 + b;
          const float cs = b ? w.z : w.x, sn = b ? w.w : w.y;
          const float a0 = to_f32(x0[j].x[u]), a1 = to_f32(x1[j].x[u]);
          y0.x[u] = from_f32<T>(a0 * cs - a1 * sn);
          y1.x[u] = from_f32<T>(a1 * cs + a0 * sn);
        }
      }
      store16(dst + off, y0);
      store16(dst + off + H, y1);
    }
  }
}

template <typename T, int D>
static hipError_t move_pages_t(const PoolGeom& g, const MovePage* moves, int n, const float2* rope, hipStream_t s) {
  hipLaunchKernelGGL((move_pages_kernel<T, D>), dim3(n, 2), dim3(256), 0, s, moves, static_cast<T*>(g.base), g.layer_off,
                     g.hkv, rope);
  return hipGetLastError();
}

hipError_t launch_move_pages(const PoolGeom& g, const MovePage* moves, int n, const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (g.dtype == SPAN_BF16) {
    if (g.d == 128) return move_pages_t<bf16_t, 128>(g, moves, n, rope, s);
    return move_pages_t<bf16_t, 64>(g, moves, n, rope, s);
  }
  if (g.d == 128) return move_pages_t<float, 128>(g, moves, n, rope, s);
  return move_pages_t<float, 64>(g, moves, n, rope, s);
}

// ------------------------------------------------------------------ generic attention
// One wave per (tile, query head); lane r owns query row r of the tile.  Each
// key page is staged in LDS (rotated by the page's delta when it is read from a
// different position than it was written at), then every lane scores its row
// against the 16 slots and folds them into an online softmax (base 2).
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_generic_kernel(const WorkTile* __restrict__ tiles,
                                                          const KvPage* __restrict__ kv,
                                                          const T* __restrict__ q, T* __restrict__ out,
                                                          const T* __restrict__ pool, int64_t layer_off, int hq,
                                                          int hkv, float scale_log2,
                                                          const float2* __restrict__ rope,
                                                          void* __restrict__ part_o, float* __restrict__ part_ml) {
  constexpr int H = D / 2;
  __shared__ float ks[kPage][D + 1];
  __shared__ float vs[D][kPage + 1];
  const WorkTile t = tiles[blockIdx.x];
  const int h = blockIdx.y;
  const int g = (h * hkv) / hq;
  const int lane = threadIdx.x;
  const bool active = lane < t.n_rows;
  const int qpos = t.q_pos0 + lane;
  const int64_t page_elems = 2ll * hkv * kPage * D;

  float qv[D];
  float acc[D];
#pragma unroll
  for (int i = 0; i < D; ++i) acc[i] = 0.f;
  if (active) {
    const T* qr = q + (static_cast<int64_t>(t.q_row0 + lane) * hq + h) * D;
#pragma unroll
    for (int i = 0; i < H; ++i) {
      float sn, cs;
      rope_cs(rope, D / 2, qpos, i, &sn, &cs);
      const float x0 = to_f32(qr[i]);
      const float x1 = to_f32(qr[i + H]);
      qv[i] = x0 * cs - x1 * sn;
      qv[i + H] = x1 * cs + x0 * sn;
    }
  } else {
#pragma unroll
    for (int i = 0; i < D; ++i) qv[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int pi = t.kv_begin; pi < t.kv_end; ++pi) {
    const KvPage pg = kv[pi];
    const T* kp = pool + layer_off + static_cast<int64_t>(pg.page_id) * page_elems + static_cast<int64_t>(g) * kPage * D;
    const T* vp = pool + layer_off + static_cast<int64_t>(pg.page_id) * page_elems +
                  static_cast<int64_t>(hkv) * kPage * D + static_cast<int64_t>(g) * D * kPage;
    __syncthreads();
    for (int e = lane; e < kPage * H; e += 64) {
      const int s = e / H;
      const int i = e - s * H;
      float x0 = to_f32(kp[s * D + i]);
      float x1 = to_f32(kp[s * D + i + H]);
      if (pg.delta != 0) {
        float sn, cs;
        rope_cs(rope, D / 2, pg.delta, i, &sn, &cs);
        const float y0 = x0 * cs - x1 * sn;
        x1 = x1 * cs + x0 * sn;
        x0 = y0;
      }
      ks[s][i] = x0;
      ks[s][i + H] = x1;
    }
    for (int e = lane; e < D * kPage; e += 64) vs[e / kPage][e % kPage] = to_f32(vp[(e / kPage) * kPage + v_pos(e % kPage)]);
    __syncthreads();
    if (!active) continue;
    float sc[kPage];
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < kPage; ++s) {
      const bool ok = s < pg.n_valid && pg.pos0 + s <= qpos;
      float dot = 0.f;
#pragma unroll
      for (int i = 0; i < D; ++i) dot += qv[i] * ks[s][i];
      sc[s] = ok ? dot * scale_log2 : -INFINITY;
      mx = fmaxf(mx, sc[s]);
    }
    if (mx == -INFINITY) continue;
    const float m_new = fmaxf(m, mx);
    const float corr = exp2f(m - m_new);  // m == -inf gives 0
    l *= corr;
#pragma unroll
    for (int i = 0; i < D; ++i) acc[i] *= corr;
#pragma unroll
    for (int s = 0; s < kPage; ++s) {
      const float p = exp2f(sc[s] - m_new);
      l += p;
#pragma unroll
      for (int i = 0; i < D; ++i) acc[i] += p * vs[i][s];
    }
    m = m_new;
  }
  if (!active) return;
  const int64_t orow = static_cast<int64_t>(t.q_row0 + lane);
  if (t.part < 0) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
    T* o = out + (orow * hq + h) * D;
#pragma unroll
    for (int i = 0; i < D; ++i) o[i] = from_f32<T>(acc[i] * inv);
  } else {
    const int64_t slot = (static_cast<int64_t>(t.part) * hq + h) * kGenericBM + lane;
    using P = typename PartOf<T>::type;
    P* po = static_cast<P*>(part_o) + slot * D;
    const float inv = !PartOf<T>::normalized ? 1.f : (l > 0.f ? 1.f / l : 0.f);
#pragma unroll
    for (int i = 0; i < D; ++i) po[i] = static_cast<P>(acc[i] * inv);
    part_ml[slot * 2 + 0] = m;
    part_ml[slot * 2 + 1] = l;
  }
}

template <typename T, int D>
static hipError_t attn_generic_t(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q,
                                 void* out, void* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  hipLaunchKernelGGL((attn_generic_kernel<T, D>), dim3(n, g.hq), dim3(64), 0, s, tiles, kv,
                     static_cast<const T*>(q), static_cast<T*>(out), static_cast<const T*>(g.base), g.layer_off,
                     g.hq, g.hkv, scale_log2, rope, part_o, part_ml);
  return hipGetLastError();
}

hipError_t launch_attn_generic(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q,
                               void* out, void* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (g.dtype == SPAN_BF16) {
    if (g.d == 128) return attn_generic_t<bf16_t, 128>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
    return attn_generic_t<bf16_t, 64>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
  }
  if (g.d == 128) return attn_generic_t<float, 128>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
  return attn_generic_t<float, 64>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
}

// ------------------------------------------------------------------ K4 combine
// out = sum_p o_p 2^(m_p - M) / sum_p l_p 2^(m_p - M), M = max_p m_p, with o_p the
// unnormalised partial (l_p times the stored O / l for bf16 pools).  One work-group
// per (tile, query head, block of 256 / (D / 8) rows): its threads cover the block's
// (row, 8 output dims) pairs.  With fewer pairs than threads (a few rows over many
// KV splits: decode steps and the page gather), S threads share a pair and each
// takes every S-th part (S a power of two, at most 32 and at most the part count),
// merging as it goes: a running max, the sums so far rescaled when it rises.  The S
// merges then meet in LDS in a tree.  Loads of four parts are in flight at once.  A
// part that saw no key of the row (max -inf) is skipped; a row that no part saw
// comes out 0.
struct Merge {
  float m, l;
  float a[8];
};

__device__ __forceinline__ void merge_into(Merge& x, float m2, float l2, const float* a2) {
  if (m2 == -INFINITY) return;
  if (x.m == -INFINITY) {
    x.m = m2;
    x.l = l2;
#pragma unroll
    for (int i = 0; i < 8; ++i) x.a[i] = a2[i];
    return;
  }
  const float mn = fmaxf(x.m, m2);
  const float f1 = exp2f(x.m - mn), f2 = exp2f(m2 - mn);
  x.m = mn;
  x.l = x.l * f1 + l2 * f2;
#pragma unroll
  for (int i = 0; i < 8; ++i) x.a[i] = x.a[i] * f1 + a2[i] * f2;
}

template <typename T, int D>
__global__ __launch_bounds__(256) void combine_kernel(const CombineTile* __restrict__ tiles,
                                                      const void* __restrict__ part_o,
                                                      const float* __restrict__ part_ml, int bm, int hq, int R,
                                                      T* __restrict__ out) {
  constexpr int C8 = D / 8;  // R: rows per work-group, at most 256 / C8
  __shared__ float sh_m[256], sh_l[256], sh_a[8][256];
  const CombineTile t = tiles[blockIdx.x];
  const int h = blockIdx.y;
  const int row0 = blockIdx.z * R;
  if (row0 >= t.n_rows) return;
  const int pairs = min(R, t.n_rows - row0) * C8;
  int S = 1;
  while (S < 32 && 2 * S * pairs <= 256 && 2 * S <= t.n_parts) S *= 2;
  const int per_pass = 256 / S;
  const int s = threadIdx.x % S;
  for (int base = 0; base < pairs; base += per_pass) {
    const int pi = base + threadIdx.x / S;
    Merge x;
    x.m = -INFINITY;
    x.l = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) x.a[i] = 0.f;
    const int r = row0 + pi / C8, c = pi % C8;
    if (pi < pairs) {
      auto slot_of = [&](int p) { return (static_cast<int64_t>(t.part0 + p) * hq + h) * bm + r; };
      for (int p0 = s; p0 < t.n_parts; p0 += 4 * S) {
        float2 ml[4];
        float a2[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int p = p0 + u * S;
          if (p < t.n_parts) {
            const int64_t sl = slot_of(p);
            ml[u] = *reinterpret_cast<const float2*>(part_ml + sl * 2);
            if constexpr (PartOf<T>::normalized) {  // O / l in fp16: back to O
              typedef f16_t f16x8_t __attribute__((ext_vector_type(8)));
              const f16x8_t v = *reinterpret_cast<const f16x8_t*>(static_cast<const f16_t*>(part_o) + sl * D + 8 * c);
#pragma unroll
              for (int i = 0; i < 8; ++i) a2[u][i] = static_cast<float>(v[i]) * ml[u].y;
            } else {
              const float* po = static_cast<const float*>(part_o) + sl * D + 8 * c;
              const float4 lo = *reinterpret_cast<const float4*>(po), hi = *reinterpret_cast<const float4*>(po + 4);
              a2[u][0] = lo.x, a2[u][1] = lo.y, a2[u][2] = lo.z, a2[u][3] = lo.w;
              a2[u][4] = hi.x, a2[u][5] = hi.y, a2[u][6] = hi.z, a2[u][7] = hi.w;
            }
          } else {
            ml[u] = float2{-INFINITY, 0.f};
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) merge_into(x, ml[u].x, ml[u].y, a2[u]);
      }
    }
    if (S > 1) {  // tree over the S threads of a pair (consecutive threads)
      sh_m[threadIdx.x] = x.m;
      sh_l[threadIdx.x] = x.l;
#pragma unroll
      for (int i = 0; i < 8; ++i) sh_a[i][threadIdx.x] = x.a[i];
      __syncthreads();
      for (int st = S / 2; st >= 1; st /= 2) {
        if (s < st) {
          const int o = threadIdx.x + st;
          float a2[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) a2[i] = sh_a[i][o];
          merge_into(x, sh_m[o], sh_l[o], a2);
          sh_m[threadIdx.x] = x.m;
          sh_l[threadIdx.x] = x.l;
#pragma unroll
          for (int i = 0; i < 8; ++i) sh_a[i][threadIdx.x] = x.a[i];
        }
        __syncthreads();
      }
    }
    if (pi < pairs && s == 0) {
      const float inv = x.l > 0.f ? 1.f / x.l : 0.f;
      T* dst = out + (static_cast<int64_t>(t.q_row0 + r) * hq + h) * D + 8 * c;
#pragma unroll
      for (int i = 0; i < 8; ++i) dst[i] = from_f32<T>(x.a[i] * inv);
    }
    __syncthreads();  // the LDS of this pass is read before the next one writes
  }
}

hipError_t launch_combine(const PoolGeom& g, const CombineTile* tiles, int n, const void* part_o,
                          const float* part_ml, int bm, int max_parts, void* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  // Fewer rows per work-group when tiles have many parts, so that about four parts
  // fall to each thread: one round of loads in flight instead of a chain of rounds.
  int share = 1;
  while (share < 32 && 8 * share <= max_parts) share *= 2;
  const int rows_per_group = std::max(1, 256 / (g.d / 8) / share);
  dim3 grid(n, g.hq, (bm + rows_per_group - 1) / rows_per_group);
  if (g.dtype == SPAN_BF16) {
    if (g.d == 128)
      hipLaunchKernelGGL((combine_kernel<bf16_t, 128>), grid, dim3(256), 0, s, tiles, part_o, part_ml, bm, g.hq, rows_per_group,
                         static_cast<bf16_t*>(out));
    else
      hipLaunchKernelGGL((combine_kernel<bf16_t, 64>), grid, dim3(256), 0, s, tiles, part_o, part_ml, bm, g.hq, rows_per_group,
                         static_cast<bf16_t*>(out));
  } else {
    if (g.d == 128)
      hipLaunchKernelGGL((combine_kernel<float, 128>), grid, dim3(256), 0, s, tiles, part_o, part_ml, bm, g.hq, rows_per_group,
                         static_cast<float*>(out));
    else
      hipLaunchKernelGGL((combine_kernel<float, 64>), grid, dim3(256), 0, s, tiles, part_o, part_ml, bm, g.hq, rows_per_group,
                         static_cast<float*>(out));
  }
  return hipGetLastError();
}

}  // namespace spanq
