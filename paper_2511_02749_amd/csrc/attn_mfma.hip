// bf16 MFMA span attention for gfx950 (CDNA4).
//
// One work-group of eight waves per (row tile of 256/G query tokens, kv head).  The
// G query heads that share the kv head are packed into the work-group: wave w
// handles head (w mod G) and token rows 32*(w div G) .. +31, so every K/V tile
// staged in LDS feeds all eight waves.
//
// Scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//   A = K tile (32 keys x 16 dims, from LDS), B = Q^T (16 dims x 32 rows, kept in
//   registers for the whole key loop), C = 32 keys x 32 rows.
// In that C layout each lane owns one query row (lane mod 32) and 16 of the 32
// keys, so the running max needs a single exchange between the two half-waves
// and the row sum needs none until the end.  P^T is then already a valid B operand
// of O^T = V^T P^T once the key order inside each 16-key step is permuted the same
// way on the A side: the lane of half h holds keys {4h..4h+3, 8+4h..8+4h+3}.  Pages
// store V transposed with the slots of each page in exactly that order (bits 2 and
// 3 of the slot swapped), so each V operand is one 16-byte LDS read.
//
// Keys are read in tiles of 4 pages (64 keys) through the block table.  Tiles go
// straight from HBM to LDS (global_load_lds_dwordx4, no register staging) into a
// ring of four stages, two tiles ahead of the one being computed; the LDS tiles
// are XOR-swizzled at 16-byte granularity so MFMA operand reads are free of bank
// conflicts.  One barrier per tile: passing it means every wave has finished the
// tile two back, whose stage the next prefetch overwrites.
//
// Repositioning (cross rows over cached fragments): the planner pads each span's
// run of pages to whole tiles, so all keys of a tile share one delta d between the
// position they were rotated at and the position this query gives them.  Instead of
// rotating K, the query operand is rotated by -d when d changes (rotary composition
// R(a)^T R(b) = R(b - a)); the cos/sin row for d rides along with the tile's DMA.
// Cached pages are never rewritten.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"

namespace spanq {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

namespace {

constexpr int kBN = 64;     // keys per tile (4 pages)
constexpr int kNW = 8;      // waves per work-group
constexpr int kNT = 64 * kNW;
constexpr int kStages = 4;  // LDS ring depth; tiles are fetched two ahead

// Two floats to packed bfloat16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int D>
struct Geo {
  static constexpr int KS = D / 16;                // 16-dim steps of the QK contraction
  static constexpr int DB = D / 32;                // 32-dim blocks of the output
  static constexpr int KBYTES = kBN * D * 2;       // K tile: [64 keys][D], rows of 2D bytes
  static constexpr int VBYTES = D * kBN * 2;       // V tile: [D][64 positions], rows of 128 bytes
  static constexpr int RBYTES = 1024;              // cos/sin row of the tile's delta (4D bytes used)
  static constexpr int STAGE = KBYTES + VBYTES + RBYTES;
  static constexpr int KPW = KBYTES / 1024 / kNW;  // K DMA instructions per wave per tile
  static constexpr int VPW = VBYTES / 1024 / kNW;  // V DMA instructions per wave per tile
  static constexpr int RPW = 4 * D / kNW;          // bytes of the cos/sin row per wave
};

// 16-byte chunk swizzles: chunk c of K row `key` sits at c ^ kswz(key); chunk c of
// V row d at c ^ vswz(d).  16 consecutive lanes reading one chunk column then hit
// 16 distinct 16-byte bank groups.
template <int D>
__device__ __forceinline__ int kswz(int key) {
  return D == 128 ? (key & 15) : ((key >> 1) & 7);
}
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

struct TilePages {
  int id[4];
  int nv[4];
  int pos0[4];
  int delta;
};

__device__ __forceinline__ void read_pages(const KvPage* __restrict__ kv, int first, TilePages& tp) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const KvPage pg = kv[first + p];
    tp.id[p] = pg.page_id;
    tp.nv[p] = pg.n_valid;
    tp.pos0[p] = pg.pos0;
  }
  tp.delta = kv[first].delta;
}

__device__ __forceinline__ int pick4(const int (&a)[4], int p) {
  return p == 0 ? a[0] : p == 1 ? a[1] : p == 2 ? a[2] : a[3];
}

// One lane's 16 bytes from global memory to LDS at lds_wave + 16 * lane.
__device__ __forceinline__ void dma16(const void* g, void* lds_wave) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                   (__attribute__((address_space(3))) void*)lds_wave, 16, 0, 0);
}

// Wait until at most n of this wave's vector-memory operations are outstanding.
__device__ __forceinline__ void wait_vm(int n) {
  // s_waitcnt: vmcnt in bits 3:0, expcnt 6:4 and lgkmcnt 11:8 left at their maximum
  switch (n) {
    case 2: __builtin_amdgcn_s_waitcnt(0x0F72); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x0F73); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x0F74); break;
    case 5: __builtin_amdgcn_s_waitcnt(0x0F75); break;
    case 6: __builtin_amdgcn_s_waitcnt(0x0F76); break;
    case 8: __builtin_amdgcn_s_waitcnt(0x0F78); break;
    case 10: __builtin_amdgcn_s_waitcnt(0x0F7A); break;
    default: __builtin_amdgcn_s_waitcnt(0x0F70); break;
  }
}

__device__ __forceinline__ void block_sync() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}

// Issue the DMA of one key tile (4 pages) into an LDS stage.
template <int D, bool ROT>
__device__ __forceinline__ void issue_tile(const bf16_t* __restrict__ pool, int64_t layer_off, int64_t page_elems,
                                           int hkv, int kvh, const TilePages& tp, unsigned char* stage,
                                           const float2* __restrict__ rope, int wave, int lane) {
  using G = Geo<D>;
  // K rows: instruction q covers bytes [1024q, 1024q + 1024), keys of one page
#pragma unroll
  for (int u = 0; u < G::KPW; ++u) {
    const int q = wave * G::KPW + u;
    const int byte = q * 1024 + 16 * lane;
    const int key = byte / (2 * D);
    const int c = ((byte % (2 * D)) >> 4) ^ kswz<D>(key);
    const int pid = pick4(tp.id, __builtin_amdgcn_readfirstlane(key >> 4));
    const bf16_t* src = pool + (layer_off + pid * page_elems + static_cast<int64_t>(kvh) * kPage * D) +
                        ((key & 15) * D + 8 * c);
    dma16(src, stage + q * 1024);
  }
  // V rows: row d holds the 64 key positions of the tile (16 per page)
#pragma unroll
  for (int u = 0; u < G::VPW; ++u) {
    const int q = wave * G::VPW + u;
    const int byte = q * 1024 + 16 * lane;
    const int d = byte >> 7;
    const int c = ((byte & 127) >> 4) ^ vswz(d);
    const int pid = pick4(tp.id, c >> 1);
    const bf16_t* src = pool + (layer_off + pid * page_elems + static_cast<int64_t>(hkv) * kPage * D +
                                static_cast<int64_t>(kvh) * D * kPage) +
                        (d * kPage + 8 * (c & 1));
    dma16(src, stage + G::KBYTES + q * 1024);
  }
  if (ROT) {
    // cos/sin of the tile's delta: each wave brings RPW bytes with its first lanes
    if (lane < G::RPW / 16) {
      const unsigned char* src = reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(tp.delta) * (D / 2)) +
                                 wave * G::RPW + 16 * lane;
      dma16(src, stage + G::KBYTES + G::VBYTES + wave * G::RPW);
    }
  }
}

}  // namespace

template <int D, int G, bool ROT>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_mfma_kernel(
    const WorkTile* __restrict__ tiles, const KvPage* __restrict__ kv, const bf16_t* __restrict__ q,
    bf16_t* __restrict__ out, const bf16_t* __restrict__ pool, int64_t layer_off, int hq, int hkv, float scale_log2,
    const float2* __restrict__ rope, float* __restrict__ part_o, float* __restrict__ part_ml) {
  using GE = Geo<D>;
  constexpr int BM = 32 * (kNW / G);
  constexpr int NDMA = GE::KPW + GE::VPW + (ROT ? 1 : 0);  // DMA instructions per wave per tile
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  const WorkTile t = tiles[blockIdx.x];
  const int kvh = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int head = kvh * G + (wave % G);
  const int rb = wave / G;
  const int h2 = lane >> 5;
  const int r = lane & 31;
  const int row = 32 * rb + r;
  const bool row_ok = row < t.n_rows;
  const int qpos = t.q_pos0 + row;
  const int wave_min_pos = t.q_pos0 + 32 * rb;
  const int64_t page_elems = 2ll * hkv * kPage * D;
  const int n_tiles = (t.kv_end - t.kv_begin) >> 2;

  // ---- first key tiles in flight while the query rows are loaded and rotated
  // (three ahead for the software-pipelined loop, two for the repositioning one)
  constexpr int AHEAD = ROT ? 2 : 3;
  TilePages tp;
  for (int j = 0; j < AHEAD && j < n_tiles; ++j) {
    read_pages(kv, t.kv_begin + 4 * j, tp);
    issue_tile<D, ROT>(pool, layer_off, page_elems, hkv, kvh, tp, lds + j * GE::STAGE, rope, wave, lane);
  }

  // ---- Q^T operand, rotated at the row's position and pre-scaled by log2(e)/sqrt(d)
  bf16x8_t qf[GE::KS];
  {
    float x[GE::KS][8];
    if (row_ok) {
      const bf16_t* src = q + (static_cast<int64_t>(t.q_row0 + row) * hq + head) * D + 8 * h2;
#pragma unroll
      for (int s = 0; s < GE::KS; ++s) {
        const u32x4_t w = *reinterpret_cast<const u32x4_t*>(src + 16 * s);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[s][2 * e] = lo_bf16(w[e]);
          x[s][2 * e + 1] = hi_bf16(w[e]);
        }
      }
#pragma unroll
      for (int s = 0; s < GE::KS / 2; ++s) {
        // frequencies 16s + 8h2 .. +7: 8 consecutive (cos, sin) pairs, 64 bytes
        const float4* cs4 = reinterpret_cast<const float4*>(rope + static_cast<int64_t>(qpos) * (D / 2) + 16 * s + 8 * h2);
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const float4 v = cs4[e2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int e = 2 * e2 + u;
            const float cs = u ? v.z : v.x;
            const float sn = u ? v.w : v.y;
            const float a = x[s][e], b = x[s + GE::KS / 2][e];
            x[s][e] = (a * cs - b * sn) * scale_log2;
            x[s + GE::KS / 2][e] = (b * cs + a * sn) * scale_log2;
          }
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < GE::KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[s][e] = 0.f;
    }
#pragma unroll
    for (int s = 0; s < GE::KS; ++s) {
      u32x4_t w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(x[s][2 * e], x[s][2 * e + 1]);
      qf[s] = __builtin_bit_cast(bf16x8_t, w);
    }
  }
  bf16x8_t qbase[ROT ? GE::KS : 1];  // query at delta 0 (cross rows only)
  if (ROT) {
#pragma unroll
    for (int s = 0; s < GE::KS; ++s) qbase[s] = qf[s];
  }
  int q_delta = 0;

  f32x16_t o[GE::DB];
#pragma unroll
  for (int db = 0; db < GE::DB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m = -INFINITY;
  float l = 0.f;

  const int xor32_addr = (lane ^ 32) << 2;  // ds_bpermute byte address of the other half-wave

  // ---- building blocks of one 64-key tile
  // S^T = K Q^T over the tile (two 32-key blocks, interleaved accumulator chains)
  auto qk = [&](const unsigned char* stage, f32x16_t (&sc)[2]) {
    const bf16_t* kl = reinterpret_cast<const bf16_t*>(stage);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sc[kb][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < GE::KS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int key = 32 * kb + r;
        const int c = (2 * ks + h2) ^ kswz<D>(key);
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(kl + key * D + 8 * c);
        sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sc[kb], 0, 0, 0);
      }
  };
  // causal positions and partial/empty pages; the test is wave-uniform
  auto mask = [&](f32x16_t (&sc)[2], const TilePages& cur) {
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
          if (!ok) sc[kb][i] = -INFINITY;
        }
    }
  };
  // online softmax (base 2; scores already scaled), one running max per tile
  auto softmax_max = [&](const f32x16_t (&sc)[2]) -> float {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[kb][i]);
    mx = fmaxf(mx, __int_as_float(__builtin_amdgcn_ds_bpermute(xor32_addr, __float_as_int(mx))));
    const float m_new = fmaxf(m, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = __builtin_amdgcn_exp2f(m - m_use);
    m = m_new;
    // the running max moves on few tiles once it has settled: rescale only then (a
    // real branch; the empty volatile asm keeps the compiler from if-converting it)
    if (__builtin_expect(__any(corr != 1.f), 0)) {
      __asm__ volatile("");
#pragma unroll
      for (int db = 0; db < GE::DB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
    }
    l *= corr;
    return m_use;
  };
  // P = 2^(S - m) to bf16; step g of the P.V contraction covers page g of the tile
  auto softmax_exp = [&](const f32x16_t (&sc)[2], float m_use, bf16x8_t (&pk)[4]) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int kb = g >> 1, half = g & 1;
      float psum = 0.f;
      u32x4_t w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(sc[kb][8 * half + 2 * e] - m_use);
        const float p1 = __builtin_amdgcn_exp2f(sc[kb][8 * half + 2 * e + 1] - m_use);
        psum += p0 + p1;
        w[e] = pack_bf16x2(p0, p1);
      }
      l += psum;
      pk[g] = __builtin_bit_cast(bf16x8_t, w);
    }
  };
  // O^T += V^T P^T
  auto pv = [&](const unsigned char* stage, const bf16x8_t (&pk)[4]) {
    const bf16_t* vl = reinterpret_cast<const bf16_t*>(stage + GE::KBYTES);
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int db = 0; db < GE::DB; ++db) {  // DB independent accumulator chains, interleaved
        const int d = 32 * db + r;
        const int c = (2 * g + h2) ^ vswz(d);
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(vl + d * kBN + 8 * c);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pk[g], o[db], 0, 0, 0);
      }
  };
  // query at (position - delta) = R(-delta) applied to the query at delta 0
  auto rotate_q = [&](const unsigned char* stage) {
    const float2* row_cs = reinterpret_cast<const float2*>(stage + GE::KBYTES + GE::VBYTES);
#pragma unroll
    for (int s = 0; s < GE::KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qbase[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qbase[s + GE::KS / 2]);
      u32x4_t na, nb;
      const float4* cs4 = reinterpret_cast<const float4*>(row_cs + 16 * s + 8 * h2);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float4 v = cs4[w];  // (cos, sin) of frequencies 16s + 8h2 + 2w and +1
        const float a0 = lo_bf16(a4[w]), a1 = hi_bf16(a4[w]);
        const float b0 = lo_bf16(b4[w]), b1 = hi_bf16(b4[w]);
        na[w] = pack_bf16x2(a0 * v.x + b0 * v.y, a1 * v.z + b1 * v.w);
        nb[w] = pack_bf16x2(b0 * v.x - a0 * v.y, b1 * v.z - a1 * v.w);
      }
      qf[s] = __builtin_bit_cast(bf16x8_t, na);
      qf[s + GE::KS / 2] = __builtin_bit_cast(bf16x8_t, nb);
    }
  };

  if constexpr (!ROT) {
    // ---- software pipeline: scores of tile j+1 are formed (MFMA) while the softmax
    // of tile j runs (VALU / transcendental), then tile j's P.V.  Stages in use during
    // iteration j: j (V), j+1 (K), j+2 and j+3 (in flight).
    // One step consumes the scores `cur` of tile j and forms `nxt` for tile j+1; for
    // the last tile the extra QK reads a stale stage and its result is dropped (that
    // keeps the step free of branches around the MFMAs it interleaves).
    auto step = [&](int j, f32x16_t (&cur)[2], f32x16_t (&nxt)[2]) {
      wait_vm((j + 2 < n_tiles ? 1 : 0) * NDMA);  // tile j+1 landed (only j+2 may be in flight)
      block_sync();                                // ... for every wave; tile j-1 is done
      if (j + 3 < n_tiles) {
        read_pages(kv, t.kv_begin + 4 * (j + 3), tp);
        issue_tile<D, ROT>(pool, layer_off, page_elems, hkv, kvh, tp, lds + ((j + 3) & 3) * GE::STAGE, rope, wave,
                           lane);
      }
      TilePages pg;
      read_pages(kv, t.kv_begin + 4 * j, pg);
      mask(cur, pg);
      const float m_use = softmax_max(cur);
      bf16x8_t pk[4];
      softmax_exp(cur, m_use, pk);
      qk(lds + ((j + 1) & 3) * GE::STAGE, nxt);
      pv(lds + (j & 3) * GE::STAGE, pk);
    };
    f32x16_t sa[2], sb[2];
    if (n_tiles > 0) {
      wait_vm(min(2, n_tiles - 1) * NDMA);
      block_sync();
      qk(lds, sa);
    }
    int j = 0;
    for (; j + 1 < n_tiles; j += 2) {
      step(j, sa, sb);
      step(j + 1, sb, sa);
    }
    if (j < n_tiles) step(j, sa, sb);
  } else {
    for (int j = 0; j < n_tiles; ++j) {
      if (j + 2 < n_tiles) {
        read_pages(kv, t.kv_begin + 4 * (j + 2), tp);
        issue_tile<D, ROT>(pool, layer_off, page_elems, hkv, kvh, tp, lds + ((j + 2) & 3) * GE::STAGE, rope, wave,
                           lane);
      }
      const int ahead = min(2, n_tiles - 1 - j);  // tiles issued after tile j
      wait_vm(ahead * NDMA);
      block_sync();

      TilePages cur;
      read_pages(kv, t.kv_begin + 4 * j, cur);
      const unsigned char* stage = lds + (j & 3) * GE::STAGE;
      if (cur.delta != q_delta) {
        q_delta = cur.delta;
        rotate_q(stage);
      }
      f32x16_t sc[2];
      qk(stage, sc);
      mask(sc, cur);
      const float m_use = softmax_max(sc);
      bf16x8_t pk[4];
      softmax_exp(sc, m_use, pk);
      pv(stage, pk);
    }
  }

  // ---- epilogue
  const float l_row = l + __int_as_float(__builtin_amdgcn_ds_bpermute(xor32_addr, __float_as_int(l)));
  if (!row_ok) return;
  const int64_t orow = static_cast<int64_t>(t.q_row0 + row);
  if (t.part < 0) {
    const float inv = l_row > 0.f ? 1.f / l_row : 0.f;
    bf16_t* dst = out + (orow * hq + head) * D;
#pragma unroll
    for (int db = 0; db < GE::DB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = 32 * db + 8 * g4 + 4 * h2;
        const u32x2_t w = u32x2_t{pack_bf16x2(o[db][4 * g4] * inv, o[db][4 * g4 + 1] * inv),
                                  pack_bf16x2(o[db][4 * g4 + 2] * inv, o[db][4 * g4 + 3] * inv)};
        *reinterpret_cast<u32x2_t*>(dst + d0) = w;
      }
  } else {
    const int64_t slot = (static_cast<int64_t>(t.part) * hq + head) * BM + row;
    float* po = part_o + slot * D;
#pragma unroll
    for (int db = 0; db < GE::DB; ++db)
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

int mfma_bm(int g) { return 32 * (kNW / g); }

bool mfma_supported(int hq, int hkv, int d, int dtype) {
  if (dtype != SPAN_BF16 || hkv <= 0 || hq % hkv != 0) return false;
  const int g = hq / hkv;
  return (d == 64 || d == 128) && (g == 1 || g == 2 || g == 4 || g == 8);
}

template <int D, int G, bool ROT>
static hipError_t launch_t(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q, void* out,
                           float* part_o, float* part_ml, const float2* rope, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  const size_t lds = static_cast<size_t>(kStages) * Geo<D>::STAGE;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_mfma_kernel<D, G, ROT>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((attn_mfma_kernel<D, G, ROT>), dim3(n, g.hkv), dim3(kNT), lds, s, tiles, kv,
                     static_cast<const bf16_t*>(q), static_cast<bf16_t*>(out), static_cast<const bf16_t*>(g.base),
                     g.layer_off, g.hq, g.hkv, scale_log2, rope, part_o, part_ml);
  return hipGetLastError();
}

template <int D, bool ROT>
static hipError_t launch_d(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q, void* out,
                           float* po, float* pml, const float2* rope, hipStream_t s) {
  switch (g.hq / g.hkv) {
    case 1: return launch_t<D, 1, ROT>(g, tiles, n, kv, q, out, po, pml, rope, s);
    case 2: return launch_t<D, 2, ROT>(g, tiles, n, kv, q, out, po, pml, rope, s);
    case 4: return launch_t<D, 4, ROT>(g, tiles, n, kv, q, out, po, pml, rope, s);
    case 8: return launch_t<D, 8, ROT>(g, tiles, n, kv, q, out, po, pml, rope, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_mfma(const PoolGeom& g, const WorkTile* tiles, int n, const KvPage* kv, const void* q,
                            void* out, float* part_o, float* part_ml, const float2* rope, bool reposition,
                            hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!mfma_supported(g.hq, g.hkv, g.d, g.dtype)) return hipErrorInvalidValue;
  if (g.d == 128)
    return reposition ? launch_d<128, true>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s)
                      : launch_d<128, false>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
  return reposition ? launch_d<64, true>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s)
                    : launch_d<64, false>(g, tiles, n, kv, q, out, part_o, part_ml, rope, s);
}

}  // namespace spanq
