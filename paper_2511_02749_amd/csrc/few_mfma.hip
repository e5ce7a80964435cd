// Cross attention for row tiles of at most 16 rows (the few-row, page-gather regime
// of section 5.5 of the paper: a short cross segment over a long list of cached
// fragment pages), bf16, four query heads per kv head, on 16x16x32 MFMAs.
//
// The kernel takes the work tiles the planner marks for two key groups: waves
// 0..3 (group 0) and 4..7 (group 1) each hold the 4 query heads of the kv head, 16
// rows apiece, and take alternate key tiles of each pair; each group writes its own
// split-KV partial (slots part and part + 1), which the combine pass merges.
//
// Against the 32-row kernel (attn_mfma.hip) a wave holds half the rows, so its
// accumulators, scores and query operands take half the registers, and a 64-key
// tile is 16 QK MFMAs in four independent 4-deep chains (one per 16-key block)
// instead of two 8-deep ones.  Layouts (v_mfma_f32_16x16x32_bf16, lane l, g = l / 16):
//   scores  S^T = K Q^T: A = K[16 keys][32 dims] (key l % 16, dims 8g..8g+7),
//           B = Q^T[32 dims][16 rows] (row l % 16), C: keys 4g..4g+3 of row l % 16;
//   output  O^T = V^T P^T: B = P^T over 32 keys, whose k index 8g + i is key 4g + i
//           of the first 16-key block (i < 4) or 16 + 4g + i - 4 of the second, which
//           is exactly the C layout of two score blocks; A = V^T[16 dims][those keys]:
//           slots 4g..4g+3 of two pages, 8 contiguous bytes of each page's V row
//           (pages store slot s at position s with bits 2 and 3 swapped);
//   C of O^T: dims 4g..4g+3 of row l % 16.
// Rows are reduced over the four lanes l % 16 + 16g with v_permlane16_swap and
// v_permlane32_swap.
//
// Tile stream, DMA, tile records, ring and query rotation (per-tile delta) are those
// of attn_mfma.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"
#include "mfma_common.h"

namespace spanq {

namespace {

using namespace mfma;

typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kFStages = 4;  // LDS ring depth; tiles are fetched in pairs, two ahead
constexpr int kFG = 4;       // query heads per kv head (rows per item: at most 16)

template <int D>
struct FGeo {
  static constexpr int KS = D / 32;          // 32-dim steps of the QK contraction
  static constexpr int DB = D / 16;          // 16-dim blocks of the output
  static constexpr int KBYTES = kBN * D * 2;  // K tile: [64 keys][D]
  static constexpr int VBYTES = D * kBN * 2;  // V tile: [4 pages][D][16 positions]
  static constexpr int RBYTES = 1024;         // cos/sin row of the tile's delta (4D bytes used)
  static constexpr int STAGE = KBYTES + VBYTES + RBYTES;
  static constexpr int KPW = KBYTES / 1024 / kNW;
  static constexpr int VPW = VBYTES / 1024 / kNW;
  static constexpr int RPW = 4 * D / kNW;     // bytes of the cos/sin row per wave
  static constexpr int NDMA = KPW + VPW + 1;
  static constexpr int CH = D / 4;            // 16-byte chunks per rotary row
  static constexpr int RTBYTES = 32 * 4 * D;      // rotary rows of positions 0..31 (0..15 used)
  static constexpr int BRBYTES = kNW * 4 * D;     // one rotary row per wave (its rows' base)
  static constexpr int LDS = kFStages * STAGE + RTBYTES + BRBYTES;
};

template <int NDMA>
__device__ __forceinline__ void wait_tiles_f(int k) {
  if (k >= 2)
    wait_vmcnt<2 * NDMA>();
  else if (k == 1)
    wait_vmcnt<NDMA>();
  else
    wait_vmcnt<0>();
}

// x combined with the values of lanes l ^ 16, l ^ 32 and l ^ 48 (the row's lanes)
__device__ __forceinline__ float row_max4(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row_sum4(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

}  // namespace

template <int D>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(2, 2))) void few_mfma_kernel(
    const WorkTile* __restrict__ tiles, int n_tiles_total, const TileRec* __restrict__ kt,
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ pool, int64_t layer_off, int hq, int hkv, int bm,
    float scale_log2, const float2* __restrict__ rope, f16_t* __restrict__ part_o, float* __restrict__ part_ml) {
  using GE = FGeo<D>;
  constexpr int KS = GE::KS, DB = GE::DB, NDMA = GE::NDMA;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int hsub = wave % kFG;  // head inside the kv head's group
  const int kg = wave / kFG;    // key group: tile kg of every pair
  const int r = lane & 15;      // this lane's row
  const int g = lane >> 4;      // its quarter of the wave
  const int64_t page_elems = 2ll * hkv * kPage * D;
  // Work items are (row tile, kv head); the grid is a multiple of hkv, so a
  // work-group keeps one kv head and walks row tiles t0, t0 + tstride, ...
  const int kvh = blockIdx.x % hkv;
  const int t0 = blockIdx.x / hkv;
  const int tstride = gridDim.x / hkv;
  const int head = kvh * kFG + hsub;

  // ---- DMA side of the tile stream (as in attn_mfma.hip: one page per wave, per-lane
  // offsets, the cos/sin row of the tile's delta with it)
  ItemKeys is;
  int is_t = t0, is_j = 0;
  bool is_ok = is_t < n_tiles_total;
  if (is_ok) load_item_keys(tiles, is_t, is);
  int n_issued = 0;
  constexpr int CPK = D / 8;
  uint32_t dk_ofs[GE::KPW], dv_ofs[GE::VPW];
#pragma unroll
  for (int u = 0; u < GE::KPW; ++u) {
    const int qi = wave * GE::KPW + u;
    const int key = qi * (64 / CPK) + lane / CPK;
    const int c = (lane % CPK) ^ kswz<D>(key);
    dk_ofs[u] = 2u * static_cast<uint32_t>(kvh * kPage * D + (key & 15) * D + 8 * c);
  }
#pragma unroll
  for (int u = 0; u < GE::VPW; ++u) {
    const int qi = wave * GE::VPW + u;
    const int d = 32 * (qi % (D / 32)) + (lane >> 1);
    const int h = (lane & 1) ^ ((d >> 3) & 1);
    dv_ofs[u] = 2u * static_cast<uint32_t>(hkv * kPage * D + kvh * D * kPage + d * kPage + 8 * h);
  }
  const int wpage = wave / 2;
  static_assert(GE::KPW * (64 / CPK) * 2 == 16 && GE::VPW * 2 == D / 32, "one page per wave");
  static_assert(GE::RTBYTES % (1024 * kNW) == 0 && GE::LDS <= 160 * 1024, "LDS plan");
  // This wave's page id and the delta of the next two tiles of the item, loaded by
  // lanes 0..3 at the end of an issue phase (lane 2u + f: tile rc_tile + u, field f)
  // so that the next phase need not wait for a scalar load per tile; the wait of the
  // pair's barrier (all DMA of this wave) also drains this load.
  int rc_val = 0;
  int rc_tile = -2;  // record index held in lanes 0, 1; rc_tile + 1 in lanes 2, 3
  int rc_s[4] = {0, 0, 0, 0};  // the four values, read into scalars right after the barrier
  auto issue_next = [&]() {
    while (is_ok && is_j >= is.n) {
      is_t += tstride;
      is_j = 0;
      is_ok = is_t < n_tiles_total;
      if (is_ok) load_item_keys(tiles, is_t, is);
    }
    if (!is_ok) return;
    const int ti = (is.kv_begin >> 2) + is_j;
    int pid, delta;
    if (ti == rc_tile) {
      pid = rc_s[0];
      delta = rc_s[1];
    } else if (ti == rc_tile + 1) {
      pid = rc_s[2];
      delta = rc_s[3];
    } else {
      const TileRec& rec = kt[ti];
      pid = rec.page_id[wpage];
      delta = rec.delta;
    }
    unsigned char* const stage = lds + (n_issued & 3) * GE::STAGE;
    const unsigned char* pg =
        reinterpret_cast<const unsigned char*>(pool + layer_off) + static_cast<int64_t>(pid) * (page_elems * 2);
#pragma unroll
    for (int u = 0; u < GE::KPW; ++u) dma16_m0(pg + dk_ofs[u], lds_byte(stage + (wave * GE::KPW + u) * 1024));
#pragma unroll
    for (int u = 0; u < GE::VPW; ++u)
      dma16_m0(pg + dv_ofs[u], lds_byte(stage + GE::KBYTES + (wave * GE::VPW + u) * 1024));
    if (lane < GE::RPW / 16)
      dma16_m0(reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(delta) * (D / 2)) + wave * GE::RPW +
                   16 * lane,
               lds_byte(stage + GE::KBYTES + GE::VBYTES + wave * GE::RPW));
    ++is_j;
    ++n_issued;
  };
  for (int k = 0; k < kFStages - 2; ++k) issue_next();

  // ---- compute-side state: query operands (rotated at the item's positions; per
  // tile rotated further by -delta), accumulators
  bf16x8_t qbase[KS], qf[KS];
  f32x4_t o[DB];
  float m = kNoMax, l = 0.f;
  int q_delta = 0;
  int qpos = 0, wave_min_pos = 0;

  // S^T over a 64-key tile: four 16-key blocks, each a chain over the KS dim steps
  auto qk = [&](const unsigned char* stage, f32x4_t (&sc)[4]) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) sc[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int key = 16 * kb + r;
        const int c = (4 * s + g) ^ kswz<D>(key);
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(stage + key * 2 * D + 16 * c);
        sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[s], sc[kb], 0, 0, 0);
      }
  };
  // causal positions and partial/empty pages: element j of block kb is key
  // 16kb + 4g + j of the tile (wave-uniform test)
  auto mask = [&](f32x4_t (&sc)[4], const TilePages& cur) {
    if (cur.nk < kBN || cur.pos0 + kBN - 1 > wave_min_pos) {
      const int lim = min(cur.nk, qpos - cur.pos0 + 1) - 4 * g;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (16 * kb + j >= lim) sc[kb][j] = -INFINITY;
    }
  };
  // O^T += V^T P^T over the tile: two 32-key steps (pages 2t, 2t + 1)
  const int sg = ((g & 1) << 1) | (g >> 1);  // position block of slots 4g..4g+3 in a page row
  auto pv = [&](const unsigned char* stage, const bf16x8_t (&pk)[2]) {
    const unsigned char* vt = stage + GE::KBYTES;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int d = 16 * db + r;
        const int ofs = d * 32 + 16 * ((sg >> 1) ^ ((d >> 3) & 1)) + 8 * (sg & 1);
        const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vt + (2 * t) * D * 32 + ofs);
        const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vt + (2 * t + 1) * D * 32 + ofs);
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pk[t], o[db], 0, 0, 0);
      }
  };
  // qf <- R(-delta) qbase; the cos/sin row of delta came with the tile's DMA.
  // Frequencies 32s + 8g .. +7 of this lane: bytes 256s + 64g .. +63 of the row.
  auto rotate_q = [&](const unsigned char* stage) {
    const float4* row = reinterpret_cast<const float4*>(stage + GE::KBYTES + GE::VBYTES);
#pragma unroll
    for (int s = 0; s < KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qbase[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qbase[s + KS / 2]);
      u32x4_t na, nb;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float4 v = row[16 * s + 4 * g + w];  // (cos, sin) of frequencies 32s + 8g + 2w, +1
        const float a0 = lo_bf16(a4[w]), a1 = hi_bf16(a4[w]);
        const float b0 = lo_bf16(b4[w]), b1 = hi_bf16(b4[w]);
        na[w] = pack_bf16x2(a0 * v.x + b0 * v.y, a1 * v.z + b1 * v.w);
        nb[w] = pack_bf16x2(b0 * v.x - a0 * v.y, b1 * v.z - a1 * v.w);
      }
      qf[s] = __builtin_bit_cast(bf16x8_t, na);
      qf[s + KS / 2] = __builtin_bit_cast(bf16x8_t, nb);
    }
  };

  // ---- query rotation at item start: R(base + r) = R(base) R(r) with R(0..31) in LDS
  // for the whole kernel and R(base) (base = row 0's position) brought by DMA with the
  // item's raw query
  unsigned char* const rt_lds = lds + kFStages * GE::STAGE;
  unsigned char* const br_lds = rt_lds + GE::RTBYTES + wave * 4 * D;
  auto prefetch = [&](int ti, bf16x8_t (&qn)[KS]) {
    const WorkTile tn = tiles[ti];
    if (lane < GE::CH) {
      const unsigned char* src =
          reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(tn.q_pos0) * (D / 2)) + 16 * lane;
      dma16(src, br_lds);
    }
    if (r < tn.n_rows) {
      const bf16_t* src = q + (static_cast<int64_t>(tn.q_row0 + r) * hq + head) * D + 8 * g;
#pragma unroll
      for (int s = 0; s < KS; ++s) qn[s] = *reinterpret_cast<const bf16x8_t*>(src + 32 * s);
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) qn[s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
    }
  };
  // qf <- R(position) qn * log2(e)/sqrt(d), rounded to bf16 once
  auto rotate_next = [&](const bf16x8_t (&qn)[KS]) {
    wait_vm_all();  // this wave's base row and query have landed
    __asm__ volatile("" ::: "memory");
    const float4* br = reinterpret_cast<const float4*>(br_lds);
    const float4* rt = reinterpret_cast<const float4*>(rt_lds + r * 4 * D);
#pragma unroll
    for (int s = 0; s < KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qn[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qn[s + KS / 2]);
      u32x4_t na, nb;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        // frequencies 32s + 8g + 2e2 and +1: one 16-byte chunk of each rotary row
        const int ch = 16 * s + 4 * g + e2;
        const float4 vb = br[ch];
        const float4 vr = rt[ch ^ (r & (GE::CH - 1))];
        float ra[2], rb2[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float cb = u ? vb.z : vb.x, sb = u ? vb.w : vb.y;
          const float cr = u ? vr.z : vr.x, sr = u ? vr.w : vr.y;
          const float cs = cb * cr - sb * sr;
          const float sn = sb * cr + cb * sr;
          const float a = u ? hi_bf16(a4[e2]) : lo_bf16(a4[e2]);
          const float b = u ? hi_bf16(b4[e2]) : lo_bf16(b4[e2]);
          ra[u] = (a * cs - b * sn) * scale_log2;
          rb2[u] = (b * cs + a * sn) * scale_log2;
        }
        na[e2] = pack_bf16x2(ra[0], ra[1]);
        nb[e2] = pack_bf16x2(rb2[0], rb2[1]);
      }
      qf[s] = __builtin_bit_cast(bf16x8_t, na);
      qf[s + KS / 2] = __builtin_bit_cast(bf16x8_t, nb);
    }
  };
  if (t0 < n_tiles_total) {
    // rotary rows 0..31, chunk c of row r stored at chunk c ^ (r mod CH)
    constexpr int RT_PER_WAVE = GE::RTBYTES / 1024 / kNW;
#pragma unroll
    for (int u = 0; u < RT_PER_WAVE; ++u) {
      const int qi = wave * RT_PER_WAVE + u;
      const int pos = qi * 64 + lane;  // 16-byte chunk index in the LDS table
      const int rr = pos / GE::CH, cc = pos % GE::CH;
      const unsigned char* src =
          reinterpret_cast<const unsigned char*>(rope) + rr * 4 * D + 16 * (cc ^ (rr & (GE::CH - 1)));
      dma16(src, rt_lds + qi * 1024);
    }
    bf16x8_t qn[KS];
    prefetch(t0, qn);
    wait_vm_all();
    block_sync();  // every wave's share of the table has landed
    rotate_next(qn);
  }

  int c = 0;  // stream index of the tile being computed
  for (int ct = t0; ct < n_tiles_total;) {
    const WorkTile t = tiles[ct];
    const int n_tiles = (t.kv_end - t.kv_begin) >> 2;
    const bool has_next = ct + tstride < n_tiles_total;
    qpos = t.q_pos0 + r;
    wave_min_pos = t.q_pos0;
#pragma unroll
    for (int s = 0; s < KS; ++s) qbase[s] = qf[s];
    q_delta = 0;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m = kNoMax;
    l = 0.f;
    bool first = true;  // this wave's first tile of the item

    auto compute = [&](int j, int cs) {  // tile j of the item, stream slot cs
      TilePages cur;
      read_tile(kt, (t.kv_begin >> 2) + j, cur);
      __asm__ volatile("" ::"s"(cur.pos0), "s"(cur.nk), "s"(cur.delta));
      const unsigned char* stage = lds + (cs & 3) * GE::STAGE;
      if (cur.delta != q_delta) {
        q_delta = cur.delta;
        rotate_q(stage);
      }
      // online softmax (base 2; scores already scaled) with the lazily raised running
      // max of mfma_common.h: the row max is formed on the wave's first tile of the
      // item and on the rare raise, which forms the scores anew from the tile still in
      // LDS rather than keeping them in registers past the exponentials
      f32x4_t sc[4];
      qk(stage, sc);
      mask(sc, cur);
      auto tile_max = [&]() {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j2 = 0; j2 < 4; ++j2) mx = fmaxf(mx, sc[kb][j2]);
        return row_max4(mx);
      };
      bf16x8_t pk[2];
      // the lane's sum of P by v_dot2 over the packed bf16 values (the weights the
      // P.V MFMAs take), as the 32-row kernel forms it
      auto exps = [&]() {
        const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);
        float ts0 = 0.f, ts1 = 0.f;
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          u32x4_t w;
#pragma unroll
          for (int h = 0; h < 2; ++h)  // block 2t2 + h: elements 4h .. 4h + 3 of the operand
#pragma unroll
            for (int e = 0; e < 2; ++e) {
              const uint32_t pw = pack_bf16x2(__builtin_amdgcn_exp2f(sc[2 * t2 + h][2 * e] - m),
                                              __builtin_amdgcn_exp2f(sc[2 * t2 + h][2 * e + 1] - m));
              w[2 * h + e] = pw;
              if (e)
                ts1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts1, false);
              else
                ts0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts0, false);
            }
          pk[t2] = __builtin_bit_cast(bf16x8_t, w);
        }
        return ts0 + ts1;
      };
      if (first) m = fmaxf(m, tile_max());
      first = false;
      float psum = exps();
      if (__builtin_expect(__any(!(psum <= kSumCap)), 0)) {
        __asm__ volatile("");
        qk(stage, sc);
        mask(sc, cur);
        const float m_new = fmaxf(m, tile_max());
        const float corr = __builtin_amdgcn_exp2f(m - m_new);
        m = m_new;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= corr;
        l *= corr;
        psum = exps();
      }
      l += psum;
      pv(stage, pk);
    };
    for (int j = 0; j < n_tiles;) {
      const int sz = min(2, n_tiles - j);
      // tiles c .. c + sz - 1 have landed for every wave, and every wave is done with
      // the tiles before c, whose stages take the next ones (up to c + 3)
      wait_tiles_f<NDMA>(n_issued - c - sz);
      block_sync();
      // (before this phase issues any DMA: a wait for the load here is no extra wait)
#pragma unroll
      for (int x = 0; x < 4; ++x) rc_s[x] = __builtin_amdgcn_readlane(rc_val, x);
      __asm__ volatile("" ::"s"(rc_s[0]), "s"(rc_s[1]), "s"(rc_s[2]), "s"(rc_s[3]));
#pragma unroll
      for (int u = 0; u < kFStages - 1; ++u)
        if (n_issued < c + kFStages) issue_next();
      // the records of the item's next two tiles, for the next phase
      if (is_ok && is_j < is.n) {
        const int ti = (is.kv_begin >> 2) + is_j;
        const int u = min(lane >> 1, is.n - 1 - is_j);  // past the item's end: repeat its last tile
        const int* rp = reinterpret_cast<const int*>(kt + ti + u);
        rc_val = (lane & 1) ? rp[6] : rp[wpage];  // TileRec: page_id[0..3], pos0, nk, delta, pad
        rc_tile = ti;
      }
      if (kg < sz) compute(j + kg, c + kg);
      c += sz;
      j += sz;
    }

    // ---- epilogue: this group's partial (O / l in fp16, running max, row sum).
    // The next item's query is rotated first, so the stores do not sit in front of
    // that wait.
    const float l_row = row_sum4(l);
    bf16x8_t qn[KS];
    if (has_next) {
      prefetch(ct + tstride, qn);
      rotate_next(qn);
    }
    if (r < t.n_rows && t.part >= 0) {
      const int64_t slot = (static_cast<int64_t>(t.part + kg) * hq + head) * bm + r;
      f16_t* po = part_o + slot * D;
      const float inv = l_row > 0.f ? 1.f / l_row : 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f16x4_t*>(po + 16 * db + 4 * g) =
            f16x4_t{static_cast<f16_t>(o[db][0] * inv), static_cast<f16_t>(o[db][1] * inv),
                    static_cast<f16_t>(o[db][2] * inv), static_cast<f16_t>(o[db][3] * inv)};
      if (g == 0) {  // a row that saw no key: max -inf, as the merge expects
        part_ml[slot * 2] = l_row > 0.f ? m : -INFINITY;
        part_ml[slot * 2 + 1] = l_row;
      }
    }
    if (!has_next) break;
    ct += tstride;
  }
}

bool few_supported(int hq, int hkv, int d, int dtype) {
  return dtype == SPAN_BF16 && hkv > 0 && hq == kFG * hkv && (d == 64 || d == 128);
}

template <int D>
static hipError_t launch_few_d(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q,
                               void* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  const size_t lds = FGeo<D>::LDS;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&few_mfma_kernel<D>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (attr != hipSuccess) return attr;
  int cus = 0;
  const hipError_t e = cu_count(&cus);
  if (e != hipSuccess) return e;
  // one work-group per CU, a multiple of hkv (each keeps one kv head)
  const int64_t items = static_cast<int64_t>(n) * g.hkv;
  const int grid = static_cast<int>(std::min<int64_t>(items, std::max(1, cus / g.hkv) * g.hkv));
  hipLaunchKernelGGL((few_mfma_kernel<D>), dim3(grid), dim3(kNT), lds, s, tiles, n, kt, static_cast<const bf16_t*>(q),
                     static_cast<const bf16_t*>(g.base), g.layer_off, g.hq, g.hkv, mfma_bm(kFG), scale_log2, rope,
                     static_cast<f16_t*>(part_o), part_ml);
  return hipGetLastError();
}

hipError_t launch_few_mfma(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q,
                           void* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!few_supported(g.hq, g.hkv, g.d, g.dtype) || part_o == nullptr || part_ml == nullptr)
    return hipErrorInvalidValue;
  return g.d == 128 ? launch_few_d<128>(g, tiles, n, kt, q, part_o, part_ml, rope, s)
                    : launch_few_d<64>(g, tiles, n, kt, q, part_o, part_ml, rope, s);
}

}  // namespace spanq
