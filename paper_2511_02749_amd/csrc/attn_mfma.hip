// bf16 MFMA span attention for gfx950 (CDNA4).
//
// One work-group of four waves per (row tile of 128/G query tokens, kv head).  The
// G query heads that share the kv head are packed into the work-group: wave w
// handles head (w mod G) and token rows 32*(w div G) .. +31, so every K/V tile
// staged in LDS feeds all four waves.  Two work-groups fit a CU (registers: two
// waves per SIMD; LDS: 2 x 68 KB), and having two independent work-groups, each
// with its own barrier, lets one group's softmax overlap the other's MFMAs.
//
// Scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//   A = K tile (32 keys x 16 dims, from LDS), B = Q^T (16 dims x 32 rows, kept in
//   registers for the whole key loop), C = 32 keys x 32 rows.
// In that C layout each lane owns one query row (lane mod 32) and 16 of the 32
// keys, so the running max needs a single exchange between the two half-waves
// and the row sum needs none until the end.  P^T is then already a valid B operand
// of O^T = V^T P^T once the key order inside each 16-key step is permuted the same
// way on the A side: the lane of half h holds keys {4h..4h+3, 8+4h..8+4h+3} (+16 for
// the second step), and reads exactly those keys of V^T from LDS.  V pages are
// stored transposed ([d][slot]) by the page writer for this reason.
//
// Keys are read in tiles of 4 pages (64 keys) through the block table; the next
// tile is fetched into registers while the current one is computed, then written
// to the other LDS buffer (one barrier per tile).  A page read at a position other
// than the one it was written at (cross rows over cached fragments) is rotated by
// its delta while it is staged (rotary composition R(a)R(b) = R(a + b)); cached
// pages are never rewritten.  Masking (causal positions, partial and missing pages)
// runs only on tiles that need it.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"

namespace spanq {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

namespace {

constexpr int kBN = 64;  // keys per tile (4 pages)

// Two floats to packed bfloat16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int D, int G>
struct Cfg {
  static constexpr int RB = 4 / G;           // 32-row blocks per work-group
  static constexpr int BM = 32 * RB;         // query tokens per tile
  static constexpr int NW = 4;               // waves
  static constexpr int NT = 64 * NW;         // threads
  static constexpr int KS = D / 16;          // 16-dim steps of the QK contraction
  static constexpr int DB = D / 32;          // 32-dim blocks of the output
  static constexpr int KROW = D + 8;         // padded LDS row of the K tile (bf16)
  static constexpr int VROW = kBN + 4;       // padded LDS row of the V^T tile (bf16)
  static constexpr int KCH = D / 16;         // 8-dim chunk pairs (i, i + D/2) per key
  static constexpr int KTASK = kBN * KCH;    // K staging tasks per tile
  static constexpr int VTASK = 4 * D * 2;    // V staging tasks per tile (16 B each)
  static constexpr int KPT = (KTASK + NT - 1) / NT;
  static constexpr int VPT = (VTASK + NT - 1) / NT;
  static constexpr int LDS_K = kBN * KROW;
  static constexpr int LDS_V = D * VROW;
};

struct TilePages {
  int id[4];
  int nv[4];
  int pos0[4];
  int delta[4];
};

__device__ __forceinline__ void read_pages(const KvPage* __restrict__ kv, int first, int end, TilePages& tp) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int pi = first + p;
    if (pi < end) {
      const KvPage pg = kv[pi];
      tp.id[p] = pg.page_id;
      tp.nv[p] = pg.n_valid;
      tp.pos0[p] = pg.pos0;
      tp.delta[p] = pg.delta;
    } else {
      tp.id[p] = -1;
      tp.nv[p] = 0;
      tp.pos0[p] = 0;
      tp.delta[p] = 0;
    }
  }
}

// arr[p] for a runtime p in 0..3 without an indexed (scratch) access
__device__ __forceinline__ int pick4(const int (&a)[4], int p) {
  return p == 0 ? a[0] : p == 1 ? a[1] : p == 2 ? a[2] : a[3];
}

template <int D, int G>
struct Stage {
  u32x4_t klo[Cfg<D, G>::KPT];
  u32x4_t khi[Cfg<D, G>::KPT];
  u32x4_t v[Cfg<D, G>::VPT];
};

// Global -> register staging of one key tile.  Every staging task of a wave lies
// in one page (a page holds 16 * D/16 K tasks and 2 * D V tasks, both multiples of
// the wave size), so the page index is made wave-uniform and the page base address
// lives in scalar registers; each lane only adds a fixed 32-bit offset.
template <int D, int G>
__device__ __forceinline__ void fetch(const bf16_t* __restrict__ pool, int64_t layer_off, int hkv, int kvh,
                                      const TilePages& tp, Stage<D, G>& st) {
  using C = Cfg<D, G>;
  const int64_t page_elems = 2ll * hkv * kPage * D;
#pragma unroll
  for (int t = 0; t < C::KPT; ++t) {
    const int task = threadIdx.x + t * C::NT;
    st.klo[t] = u32x4_t{0, 0, 0, 0};
    st.khi[t] = u32x4_t{0, 0, 0, 0};
    if (task < C::KTASK) {
      const int key = task / C::KCH;
      const int c = task - key * C::KCH;
      const int p = __builtin_amdgcn_readfirstlane(key >> 4);
      const int pid = pick4(tp.id, p);
      if (pid >= 0) {
        const bf16_t* base = pool + (layer_off + pid * page_elems + static_cast<int64_t>(kvh) * kPage * D);
        const uint32_t off = static_cast<uint32_t>((key & 15) * D + 8 * c);
        st.klo[t] = *reinterpret_cast<const u32x4_t*>(base + off);
        st.khi[t] = *reinterpret_cast<const u32x4_t*>(base + off + D / 2);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < C::VPT; ++t) {
    const int task = threadIdx.x + t * C::NT;
    st.v[t] = u32x4_t{0, 0, 0, 0};
    if (task < C::VTASK) {
      const int p = __builtin_amdgcn_readfirstlane(task / (2 * D));
      const int rem = task - p * (2 * D);
      const int pid = pick4(tp.id, p);
      if (pid >= 0) {
        const bf16_t* base = pool + (layer_off + pid * page_elems + static_cast<int64_t>(hkv) * kPage * D +
                                     static_cast<int64_t>(kvh) * D * kPage);
        const uint32_t off = static_cast<uint32_t>((rem >> 1) * kPage + 8 * (rem & 1));
        st.v[t] = *reinterpret_cast<const u32x4_t*>(base + off);
      }
    }
  }
}

// Rotate a staged chunk pair (dims 8c..8c+7 and D/2+8c..) by `delta` positions.
template <int D>
__device__ __forceinline__ void rotate_pair(u32x4_t& lo, u32x4_t& hi, int c, int delta,
                                            const float2* __restrict__ rope) {
  const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(delta) * (D / 2) + 8 * c);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float4 v = cs4[w];  // (cos, sin) of frequencies 8c + 2w and 8c + 2w + 1
    const float c0 = v.x, s0 = v.y, c1 = v.z, s1 = v.w;
    const float a0 = lo_bf16(lo[w]), a1 = hi_bf16(lo[w]);
    const float b0 = lo_bf16(hi[w]), b1 = hi_bf16(hi[w]);
    lo[w] = pack_bf16x2(a0 * c0 - b0 * s0, a1 * c1 - b1 * s1);
    hi[w] = pack_bf16x2(b0 * c0 + a0 * s0, b1 * c1 + a1 * s1);
  }
}

template <int D, int G>
__device__ __forceinline__ void store(bf16_t* __restrict__ k_lds, bf16_t* __restrict__ v_lds, const TilePages& tp,
                                      Stage<D, G>& st, const float2* __restrict__ rope) {
  using C = Cfg<D, G>;
#pragma unroll
  for (int t = 0; t < C::KPT; ++t) {
    const int task = threadIdx.x + t * C::NT;
    if (task < C::KTASK) {
      const int key = task / C::KCH;
      const int c = task - key * C::KCH;
      const int delta = pick4(tp.delta, key >> 4);
      if (delta != 0) rotate_pair<D>(st.klo[t], st.khi[t], c, delta, rope);
      *reinterpret_cast<u32x4_t*>(k_lds + key * C::KROW + 8 * c) = st.klo[t];
      *reinterpret_cast<u32x4_t*>(k_lds + key * C::KROW + D / 2 + 8 * c) = st.khi[t];
    }
  }
#pragma unroll
  for (int t = 0; t < C::VPT; ++t) {
    const int task = threadIdx.x + t * C::NT;
    if (task < C::VTASK) {
      const int p = task / (2 * D);
      const int rem = task - p * (2 * D);
      const int drow = rem >> 1;
      const int half = rem & 1;
      bf16_t* dst = v_lds + drow * C::VROW + 16 * p + 8 * half;   // 8-byte aligned rows
      *reinterpret_cast<u32x2_t*>(dst) = u32x2_t{st.v[t][0], st.v[t][1]};
      *reinterpret_cast<u32x2_t*>(dst + 4) = u32x2_t{st.v[t][2], st.v[t][3]};
    }
  }
}

}  // namespace

template <int D, int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_mfma_kernel(const WorkTile* __restrict__ tiles,
                                                            const KvPage* __restrict__ kv,
                                                            const bf16_t* __restrict__ q, bf16_t* __restrict__ out,
                                                            const bf16_t* __restrict__ pool, int64_t layer_off,
                                                            int hq, int hkv, float scale_log2,
                                                            const float2* __restrict__ rope,
                                                            float* __restrict__ part_o, float* __restrict__ part_ml) {
  using C = Cfg<D, G>;
  __shared__ __attribute__((aligned(16))) bf16_t k_lds[2][C::LDS_K];
  __shared__ __attribute__((aligned(16))) bf16_t v_lds[2][C::LDS_V];

  const WorkTile t = tiles[blockIdx.x];
  const int kvh = blockIdx.y;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int head = kvh * G + (wave % G);
  const int rb = wave / G;
  const int h2 = lane >> 5;
  const int r = lane & 31;
  const int row = 32 * rb + r;
  const bool row_ok = row < t.n_rows;
  const int qpos = t.q_pos0 + row;
  const int wave_min_pos = t.q_pos0 + 32 * rb;

  const int n_pages = t.kv_end - t.kv_begin;
  const int n_tiles = (n_pages + 3) >> 2;
  TilePages cur, nxt;
  Stage<D, G> st;
  // first key tile in flight while the query rows are loaded and rotated
  if (n_tiles > 0) {
    read_pages(kv, t.kv_begin, t.kv_end, cur);
    fetch<D, G>(pool, layer_off, hkv, kvh, cur, st);
  }

  // ---- Q^T operand, rotated at the row's position and pre-scaled by log2(e)/sqrt(d)
  bf16x8_t qf[C::KS];
  {
    float x[C::KS][8];
    if (row_ok) {
      const bf16_t* src = q + (static_cast<int64_t>(t.q_row0 + row) * hq + head) * D + 8 * h2;
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        const u32x4_t w = *reinterpret_cast<const u32x4_t*>(src + 16 * s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[s][2 * e] = lo_bf16(w[e]);
          x[s][2 * e + 1] = hi_bf16(w[e]);
        }
      }
#pragma unroll
      for (int s = 0; s < C::KS / 2; ++s) {
        // frequencies 16s + 8h2 .. +7: 8 consecutive (cos, sin) pairs, 64 bytes
        const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(qpos) * (D / 2) + 16 * s + 8 * h2);
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const float4 v = cs4[e2];  // (cos, sin) of frequencies 2*e2 and 2*e2 + 1
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int e = 2 * e2 + u;
            const float cs = u ? v.z : v.x;
            const float sn = u ? v.w : v.y;
            const float a = x[s][e], b = x[s + C::KS / 2][e];
            x[s][e] = (a * cs - b * sn) * scale_log2;
            x[s + C::KS / 2][e] = (b * cs + a * sn) * scale_log2;
          }
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < C::KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[s][e] = 0.f;
    }
#pragma unroll
    for (int s = 0; s < C::KS; ++s) {
      u32x4_t w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(x[s][2 * e], x[s][2 * e + 1]);
      qf[s] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  f32x16_t o[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m = -INFINITY;
  float l = 0.f;

  if (n_tiles > 0) store<D, G>(k_lds[0], v_lds[0], cur, st, rope);
  __syncthreads();

  for (int j = 0; j < n_tiles; ++j) {
    const int buf = j & 1;
    const bool more = j + 1 < n_tiles;
    if (more) {
      read_pages(kv, t.kv_begin + 4 * (j + 1), t.kv_end, nxt);
      fetch<D, G>(pool, layer_off, hkv, kvh, nxt, st);
    }
    const bf16_t* kl = k_lds[buf];
    const bf16_t* vl = v_lds[buf];

    // ---- S^T = K Q^T over 64 keys (two 32-key blocks)
    f32x16_t s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {  // two independent accumulator chains, interleaved
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(kl + (32 * kb + r) * C::KROW + 16 * ks + 8 * h2);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[kb], 0, 0, 0);
      }

    // ---- mask: causal positions, partial pages, missing pages (wave-uniform test)
    bool need = false;
#pragma unroll
    for (int p = 0; p < 4; ++p) need |= (cur.nv[p] < kPage) || (cur.pos0[p] + kPage - 1 > wave_min_pos);
    if (need) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          // key 32kb + 8(i/4) + 4h2 + i%4 lies in page 2kb + i/8, slot 8((i/4)%2) + 4h2 + i%4
          const int p = 2 * kb + (i >> 3);
          const int slot = 8 * ((i >> 2) & 1) + 4 * h2 + (i & 3);
          const bool ok = slot < cur.nv[p] && cur.pos0[p] + slot <= qpos;
          if (!ok) s[kb][i] = -INFINITY;
        }
    }

    // ---- online softmax (base 2; scores already scaled), one max per 64-key tile
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = __builtin_amdgcn_exp2f(m - m_use);
    m = m_new;
    // the running max moves on few tiles once it has settled: rescale only then
    if (__any(corr != 1.f)) {
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
    }
    l *= corr;

    // ---- P = 2^(S - m) to bf16, and O^T += V^T P^T.  Block 0's exponentials are
    // computed first; block 1's are interleaved with block 0's MFMAs, so the
    // transcendental unit and the matrix core work at the same time.
    bf16x8_t pk[2][2];
    auto exp_block = [&](int kb) {
      float psum = 0.f;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        u32x4_t w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(s[kb][8 * half + 2 * e] - m_use);
          const float p1 = __builtin_amdgcn_exp2f(s[kb][8 * half + 2 * e + 1] - m_use);
          psum += p0 + p1;
          w[e] = pack_bf16x2(p0, p1);
        }
        pk[kb][half] = __builtin_bit_cast(bf16x8_t, w);
      }
      l += psum;
    };
    auto pv_block = [&](int kb) {
#pragma unroll
      for (int stp = 0; stp < 2; ++stp)
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {  // DB independent accumulator chains, interleaved
          const bf16_t* vrow = vl + (32 * db + r) * C::VROW + 4 * h2;
          const int k0 = 32 * kb + 16 * stp;
          const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vrow + k0);
          const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vrow + k0 + 8);
          const u32x4_t w = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, w);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pk[kb][stp], o[db], 0, 0, 0);
        }
    };
    exp_block(0);
    pv_block(0);
    exp_block(1);
#pragma unroll
    for (int i = 0; i < 2 * C::DB; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // its two LDS reads (next V operand)
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // block-1 softmax VALU
      __builtin_amdgcn_sched_group_barrier(0x400, 2, 0);  // block-1 exponentials
    }
    pv_block(1);

    if (more) {
      store<D, G>(k_lds[buf ^ 1], v_lds[buf ^ 1], nxt, st, rope);
      cur = nxt;
    }
    __syncthreads();
  }

  // ---- epilogue
  const float l_row = l + __shfl_xor(l, 32);
  if (!row_ok) return;
  const int64_t orow = static_cast<int64_t>(t.q_row0 + row);
  if (t.part < 0) {
    const float inv = l_row > 0.f ? 1.f / l_row : 0.f;
    bf16_t* dst = out + (orow * hq + head) * D;
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = 32 * db + 8 * g4 + 4 * h2;
        const u32x2_t w = u32x2_t{pack_bf16x2(o[db][4 * g4] * inv, o[db][4 * g4 + 1] * inv),
                                  pack_bf16x2(o[db][4 * g4 + 2] * inv, o[db][4 * g4 + 3] * inv)};
        *reinterpret_cast<u32x2_t*>(dst + d0) = w;
      }
  } else {
    const int64_t slot = (static_cast<int64_t>(t.part) * hq + head) * C::BM + row;
    float* po = part_o + slot * D;
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = 32 * db + 8 * g4 + 4 * h2;
        *reinterpret_cast<float4*>(po + d0) =
            float4{o[db][4 * g4], o[db][4 * g4 + 1], o[db][4 * g4 + 2], o[db][4 * g4 + 3]};
      }
    if (h2 == 0) {
      part_ml[slot * 2] = m;
      part_ml[slot * 2 + 1] = l_row;
    }
  }
}

int mfma_bm(int g) { return 128 / g; }

bool mfma_supported(int hq, int hkv, int d, int dtype) {
  if (dtype != SPAN_BF16 || hkv <= 0 || hq % hkv != 0) return false;
  const int g = hq / hkv;
  // g = 8 would need 16 waves per work-group and spill at 128 registers per lane
  return (d == 64 || d == 128) && (g == 1 || g == 2 || g == 4);
}

template <int D, int G>
static hipError_t launch_t(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q, void* out,
                           float* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  hipLaunchKernelGGL((attn_mfma_kernel<D, G>), dim3(n, g.hkv), dim3(256), 0, s, tiles, kv,
                     static_cast<const bf16_t*>(q), static_cast<bf16_t*>(out), static_cast<const bf16_t*>(g.base),
                     g.layer_off, g.hq, g.hkv, scale_log2, rope, part_o, part_ml);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q, void* out,
                           float* po, float* pml, const float2* inv, hipStream_t s) {
  switch (g.hq / g.hkv) {
    case 1: return launch_t<D, 1>(g, tiles, n, kv, q, out, po, pml, inv, s);
    case 2: return launch_t<D, 2>(g, tiles, n, kv, q, out, po, pml, inv, s);
    case 4: return launch_t<D, 4>(g, tiles, n, kv, q, out, po, pml, inv, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_mfma(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q,
                            void* out, float* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!mfma_supported(g.hq, g.hkv, g.d, g.dtype)) return hipErrorInvalidValue;
  if (g.d == 128) return launch_d<128>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
  return launch_d<64>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
}

}  // namespace spanq
