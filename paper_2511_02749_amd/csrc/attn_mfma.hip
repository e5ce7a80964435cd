// bf16 MFMA cross attention for gfx950 (CDNA4): rows that attend over cached
// fragment pages at positions other than the ones the pages were written at
// (repositioning, section 5.5 of the paper), optionally with the key list of an
// item split into parts whose partial results a combine pass merges.  Span prefill
// has a software-pipelined kernel of its own (prefill_mfma.hip), and cross tiles of
// at most 16 rows one on 16-row MFMAs (few_mfma.hip).
//
// Work items are (row tile of 256/G query tokens, kv head).  The G query heads that
// share a kv head are packed into one item: wave w of the eight handles head
// (w mod G) and token rows 32*(w div G) .. +31, so every K/V tile staged in LDS
// feeds all eight waves.
//
// The kernel is persistent: one work-group per CU keeps one kv head and walks the
// row tiles t0, t0 + stride, ... in order.  Key tiles of consecutive items form one stream through the LDS ring,
// so the next item's first tiles are already in flight while the current item
// finishes, and no work-group launch or ring refill sits between items.
//
// Scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//   A = K tile (32 keys x 16 dims, from LDS), B = Q^T (16 dims x 32 rows, kept in
//   registers for the whole item), C = 32 keys x 32 rows.
// In that C layout each lane owns one query row (lane mod 32) and 16 of the 32
// keys, so a row max needs a single exchange between the two half-waves (and is
// formed only on an item's first tile and on the rare raise of the lazily raised
// running max, mfma_common.h), and the row sum needs none until the end.  P^T is then already a valid B operand
// of O^T = V^T P^T once the key order inside each 16-key step is permuted the same
// way on the A side: the lane of half h holds keys {4h..4h+3, 8+4h..8+4h+3}.  Pages
// store V transposed with the slots of each page in exactly that order (bits 2 and
// 3 of the slot swapped), so each V operand is one 16-byte LDS read.
//
// Keys are read in tiles of 4 pages (64 keys) through the block table.  Tiles go
// straight from HBM to LDS (global_load_lds_dwordx4, no register staging) into a
// ring of four stages; the LDS tiles are XOR-swizzled at 16-byte granularity so MFMA
// operand reads are free of bank conflicts.  Tiles are taken in pairs, with one wait
// and one barrier per pair: passing it means every wave has finished the previous
// pair, whose stages the next fetches overwrite.
//
// Repositioning (cross rows over cached fragments): the planner pads each span's
// run of pages to whole tiles, so all keys of a tile share one delta d between the
// position they were rotated at and the position this query gives them.  Instead of
// rotating K, the query operand is rotated by -d when d changes (rotary composition
// R(a)^T R(b) = R(b - a)); the cos/sin row for d rides along with the tile's DMA.
// Cached pages are never rewritten.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"
#include "mfma_common.h"
#include "page_write.h"

namespace spanq {

namespace {

using namespace mfma;

constexpr int kStages = 4;  // LDS ring depth; tiles are fetched two ahead

template <int D>
struct Geo {
  static constexpr int KS = D / 16;                // 16-dim steps of the QK contraction
  static constexpr int DB = D / 32;                // 32-dim blocks of the output
  static constexpr int KBYTES = kBN * D * 2;       // K tile: [64 keys][D], rows of 2D bytes
  static constexpr int VBYTES = D * kBN * 2;       // V tile: [4 pages][D][16 positions]
  static constexpr int RBYTES = 1024;              // cos/sin row of the tile's delta (4D bytes used)
  static constexpr int STAGE = KBYTES + VBYTES + RBYTES;
  static constexpr int KPW = KBYTES / 1024 / kNW;  // K DMA instructions per wave per tile
  static constexpr int VPW = VBYTES / 1024 / kNW;  // V DMA instructions per wave per tile
  static constexpr int RPW = 4 * D / kNW;          // bytes of the cos/sin row per wave

  static constexpr int NDMA = KPW + VPW + 1;       // DMA instructions per wave per tile
  // Beyond the ring (query rotation at item start): the rotary rows of positions
  // 0..31 for the whole kernel, and one rotary row per wave (its 32-row block's
  // first position) for the next item.
  static constexpr int CH = D / 4;                     // 16-byte chunks per rotary row
  static constexpr int RTBYTES = 32 * 4 * D;
  static constexpr int BRBYTES = kNW * 4 * D;
  static constexpr int LDS = kStages * STAGE + RTBYTES + BRBYTES;
};

// Wait until at most k tiles (NDMA operations each) of this wave's DMA are in flight.
template <int NDMA>
__device__ __forceinline__ void wait_tiles(int k) {
  if (k >= 2)
    wait_vmcnt<2 * NDMA>();
  else if (k == 1)
    wait_vmcnt<NDMA>();
  else
    wait_vmcnt<0>();
}

}  // namespace

template <int D, int G>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_mfma_kernel(
    const WorkTile* __restrict__ tiles, int n_tiles_total, const TileRec* __restrict__ kt, const bf16_t* __restrict__ q,
    bf16_t* __restrict__ out, bf16_t* __restrict__ pool, int64_t layer_off, int hq, int hkv, float scale_log2,
    const float2* __restrict__ rope, f16_t* __restrict__ part_o, float* __restrict__ part_ml,
    const bf16_t* __restrict__ kin, const bf16_t* __restrict__ vin, const NewPage* __restrict__ wpages) {
  using GE = Geo<D>;
  constexpr int BM = 32 * (kNW / G);
  // Two key groups (cross attention, four query heads per kv head): a few-row item
  // lets its two 32-row wave groups take alternate key tiles of each pair.
  constexpr bool kTwoCapable = kNW / G == 2;
  constexpr int NDMA = GE::NDMA;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int hsub = wave % G;  // head inside the kv head's group
  const int rb = wave / G;    // 32-row block
  const int h2 = lane >> 5;
  const int r = lane & 31;
  const int row = 32 * rb + r;
  const int64_t page_elems = 2ll * hkv * kPage * D;
  const int xor32_addr = (lane ^ 32) << 2;  // ds_bpermute byte address of the other half-wave
  // Work items are (row tile, kv head).  The grid is a multiple of hkv, so a
  // work-group keeps one kv head and walks row tiles t0, t0 + tstride, ...
  const int kvh = blockIdx.x % hkv;
  const int t0 = blockIdx.x / hkv;
  const int tstride = gridDim.x / hkv;
  const int head = kvh * G + hsub;

  // ---- DMA side of the tile stream: item `is_i`, its tile `is_j`
  ItemKeys is;
  int is_t = t0, is_j = 0;
  bool is_ok = is_t < n_tiles_total;
  if (is_ok) load_item_keys(tiles, is_t, is);
  int n_issued = 0;  // tiles of the stream issued so far
  // Per-lane source offsets (bytes, inside a page) of this wave's DMA instructions.
  // K instruction u fills LDS bytes [1024q, 1024q + 1024) of the K tile, q = wave KPW
  // + u: 1024 / 2D keys of one page, chunk c of key k stored at chunk c ^ kswz(k).  V
  // instruction u fills 1024 bytes of the V tile, laid out [page][d][two 16-byte
  // halves] with half h of row d stored at h ^ (d >> 3 & 1): 32 rows of one page.
  // All of a wave's instructions read the same page of the tile (page wave / 2), so
  // a tile's fetch is one page id per wave plus these offsets: the uniform work of
  // the fetch, which all eight waves repeat on the CU's one scalar unit, stays small.
  // (No registers to spare here: the offsets are recomputed for every tile from an
  // opaque copy of the lane id, not hoisted out of the tile loop.)
  constexpr int CPK = D / 8;  // 16-byte chunks per key row
  auto dk_ofs = [&](int ln, int u) __attribute__((always_inline)) {
    const int qi = wave * GE::KPW + u;
    const int key = qi * (64 / CPK) + ln / CPK;
    const int c = (ln % CPK) ^ kswz<D>(key);
    return 2u * static_cast<uint32_t>(kvh * kPage * D + (key & 15) * D + 8 * c);
  };
  auto dv_ofs = [&](int ln, int u) __attribute__((always_inline)) {
    const int qi = wave * GE::VPW + u;
    const int d = 32 * (qi % (D / 32)) + (ln >> 1);
    const int h = (ln & 1) ^ ((d >> 3) & 1);
    return 2u * static_cast<uint32_t>(hkv * kPage * D + kvh * D * kPage + d * kPage + 8 * h);
  };
  const int wpage = wave / 2;  // the page of the tile this wave's instructions read
  static_assert(GE::KPW * (64 / CPK) * 2 == 16 && GE::VPW * 2 == D / 32, "one page per wave");
  auto issue_next = [&]() {
    while (is_ok && is_j >= is.n) {
      is_t += tstride;
      is_j = 0;
      is_ok = is_t < n_tiles_total;
      if (is_ok) load_item_keys(tiles, is_t, is);
    }
    if (!is_ok) return;
    const TileRec& rec = kt[(is.kv_begin >> 2) + is_j];
    const int pid = rec.page_id[wpage];
    const int delta = rec.delta;
    unsigned char* const stage = lds + (n_issued & 3) * GE::STAGE;
    const unsigned char* pg =
        reinterpret_cast<const unsigned char*>(pool + layer_off) + static_cast<int64_t>(pid) * (page_elems * 2);
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
#pragma unroll
    for (int u = 0; u < GE::KPW; ++u) dma16_m0(pg + dk_ofs(ln, u), lds_byte(stage + (wave * GE::KPW + u) * 1024));
#pragma unroll
    for (int u = 0; u < GE::VPW; ++u)
      dma16_m0(pg + dv_ofs(ln, u), lds_byte(stage + GE::KBYTES + (wave * GE::VPW + u) * 1024));
    // cos/sin of the tile's delta: each wave brings RPW bytes with its first lanes
    if (lane < GE::RPW / 16)
      dma16_m0(reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(delta) * (D / 2)) + wave * GE::RPW +
                   16 * lane,
               lds_byte(stage + GE::KBYTES + GE::VBYTES + wave * GE::RPW));
    ++is_j;
    ++n_issued;
  };
  // The cross-segment pages in this work-group's key ranges (wpages given), written
  // here for its kv head before the tile stream starts, while the LDS is still free.
  // Every work-group that reads such a page writes it; their writes agree, and each
  // reads only after its own have completed.
  if (wpages) {
    bool wrote = false;
    for (int ti = t0; ti < n_tiles_total; ti += tstride) {
      const WorkTile* tw = tiles + __builtin_amdgcn_readfirstlane(ti);
      const int cnt = tw->flags >> kWriteShift, w0 = tw->w_first;
      if (cnt > 0)
        write_pages_one_head<bf16_t, D>(wpages + w0, cnt, kvh, kin, vin, pool, layer_off, hkv, rope,
                                        reinterpret_cast<bf16_t*>(lds), static_cast<int>(threadIdx.x), kNT);
      wrote |= cnt > 0;
    }
    if (wrote) {
      wait_vm_all();  // this wave's page stores are done
      block_sync();   // and every other wave's
    }
  }
  for (int k = 0; k < kStages - 2; ++k) issue_next();

  bf16x8_t qf[GE::KS];                // Q^T operand of the current item
  bf16x8_t qbase[GE::KS];             // query at delta 0
  f32x16_t o[GE::DB];
  float m, l;
  int q_delta = 0;
  int qpos = 0, wave_min_pos = 0;

  // ---- building blocks of one 64-key tile
  // S^T = K Q^T over the tile (two 32-key blocks, interleaved accumulator chains)
  // (the K operands of step ks + 1 are read while the MFMAs of step ks run)
  auto qk = [&](const unsigned char* stage, f32x16_t (&sc)[2]) {
    const bf16_t* kl = reinterpret_cast<const bf16_t*>(stage);
    auto kop = [&](int ks, int kb) {
      const int key = 32 * kb + r;
      const int c = (2 * ks + h2) ^ kswz<D>(key);
      return *reinterpret_cast<const bf16x8_t*>(kl + key * D + 8 * c);
    };
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sc[kb][i] = 0.f;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks = 0; ks < GE::KS; ++ks) {
      const bf16x8_t a0 = kop(ks, 0), a1 = kop(ks, 1);
      sc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[ks], sc[0], 0, 0, 0);
      sc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[ks], sc[1], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
    // instruction order: reads of two steps ahead, then per step its two MFMAs and
    // the reads of the step after next
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int ks = 0; ks < GE::KS; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      if (ks + 2 < GE::KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
  };
  // causal positions and partial/empty pages; the test is wave-uniform
  auto mask = [&](f32x16_t (&sc)[2], const TilePages& cur) {
    if (cur.nk < kBN || cur.pos0 + kBN - 1 > wave_min_pos) {
      // key k is kept iff k < nk and pos0 + k <= qpos; element i of block kb is key
      // 32kb + 8(i/4) + 4h2 + i%4, compared as a constant against lim - 4h2
      const int lim = min(cur.nk, qpos - cur.pos0 + 1) - 4 * h2;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (32 * kb + 8 * (i >> 2) + (i & 3) >= lim) sc[kb][i] = -INFINITY;
    }
  };
  // online softmax (base 2; scores already scaled) with the lazily raised running
  // max of mfma_common.h: the row max over a tile (both half-waves) is formed only on
  // an item's first tile and on the rare raise
  auto tile_max = [&](const f32x16_t (&sc)[2]) -> float {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[kb][i]);
    return fmaxf(mx, __int_as_float(__builtin_amdgcn_ds_bpermute(xor32_addr, __float_as_int(mx))));
  };
  // P = 2^(S - m) to bf16 (step g of the P.V contraction covers page g of the tile);
  // returns this lane's sum of P, formed by v_dot2 over the packed bf16 values, i.e.
  // over exactly the weights the P.V MFMAs take (two chains for independent adds)
  auto softmax_exp = [&](const f32x16_t (&sc)[2], bf16x8_t (&pk)[4]) -> float {
    const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);
    float ts0 = 0.f, ts1 = 0.f;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int kb = g >> 1, half = g & 1;
      u32x4_t w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // the dot product takes the packed word itself (not w[e] read back, which
        // hipcc at -O3 has been seen to feed from the vector's element 0)
        const uint32_t pw = pack_bf16x2(__builtin_amdgcn_exp2f(sc[kb][8 * half + 2 * e] - m),
                                        __builtin_amdgcn_exp2f(sc[kb][8 * half + 2 * e + 1] - m));
        w[e] = pw;
        if (e & 1)
          ts1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts1, false);
        else
          ts0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts0, false);
      }
      pk[g] = __builtin_bit_cast(bf16x8_t, w);
    }
    return ts0 + ts1;
  };
  // P of a tile whose scores `scores(sc)` forms (QK and mask); the rare raise sets m
  // to the tile's row max, rescales O and l and takes P again, with the scores formed
  // anew from the tile still in LDS, so that they need not stay in registers past the
  // exponentials (a real branch; the empty volatile asm keeps the compiler from
  // if-converting it)
  auto softmax = [&](auto scores, bf16x8_t (&pk)[4], bool first) {
    f32x16_t sc[2];
    scores(sc);
    if (first) m = fmaxf(m, tile_max(sc));
    float psum = softmax_exp(sc, pk);
    if (__builtin_expect(__any(!(psum <= kSumCap)), 0)) {
      __asm__ volatile("");
      scores(sc);
      const float m_new = fmaxf(m, tile_max(sc));
      const float corr = __builtin_amdgcn_exp2f(m - m_new);
      m = m_new;
#pragma unroll
      for (int db = 0; db < GE::DB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
      l *= corr;
      psum = softmax_exp(sc, pk);
    }
    l += psum;
  };
  // O^T += V^T P^T
  // (the V operand of page g, dims 32db + r: 16 bytes at [g][32db + r][half h2])
  auto pv = [&](const unsigned char* stage, const bf16x8_t (&pk)[4]) {
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
    const uint32_t vofs = 32u * (ln & 31) + 16u * ((ln >> 5) ^ ((ln >> 3) & 1));
    const bf16x8_t* a = reinterpret_cast<const bf16x8_t*>(stage + GE::KBYTES + vofs);
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int db = 0; db < GE::DB; ++db)  // DB independent accumulator chains, interleaved
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(g * D * 32 + db * 1024) / 16], pk[g], o[db], 0, 0, 0);
    __builtin_amdgcn_s_setprio(0);
  };
  // query at (position - delta) = R(-delta) applied to the query at delta 0
  // The cos/sin row came with the tile's DMA, which the tile's wait and barrier
  // already cover; it is read with plain ds_read instructions the compiler does not
  // see, since it would otherwise drain every DMA in flight before reading it.
  auto rotate_q = [&](const unsigned char* stage) {
    const unsigned row_addr = static_cast<unsigned>(reinterpret_cast<uintptr_t>(stage + GE::KBYTES + GE::VBYTES)) +
                              64u * h2;
#pragma unroll
    for (int s = 0; s < GE::KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qbase[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qbase[s + GE::KS / 2]);
      u32x4_t na, nb;
      float4 cs4[4];
      // frequencies 16s + 8h2 .. +7: bytes 128s + 64h2 .. +63 of the row
      __asm__ volatile(
          "ds_read_b128 %0, %4 offset:%5\n"
          "ds_read_b128 %1, %4 offset:%6\n"
          "ds_read_b128 %2, %4 offset:%7\n"
          "ds_read_b128 %3, %4 offset:%8\n"
          "s_waitcnt lgkmcnt(0)"
          : "=v"(cs4[0]), "=v"(cs4[1]), "=v"(cs4[2]), "=v"(cs4[3])
          : "v"(row_addr), "i"(128 * s), "i"(128 * s + 16), "i"(128 * s + 32), "i"(128 * s + 48)
          : "memory");
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

  // ---- query rotation at item start without scattered table reads: the rotary
  // angles of row r (0..31) of a wave's 32-row block come
  // from R(base + r) = R(base) R(r), with R(0..31) kept in LDS for the whole kernel
  // and R(base) (base = the block's first position) brought into LDS by DMA
  // together with the item's raw query.
  unsigned char* const rt_lds = lds + kStages * GE::STAGE;
  unsigned char* const br_lds = rt_lds + GE::RTBYTES + wave * 4 * D;
  // An item in two-key-group mode gives both wave groups rows 0..31 (the group
  // picks key tiles instead); otherwise wave group rb holds rows 32rb .. 32rb + 31.
  auto two_groups = [&](const WorkTile& w) { return kTwoCapable && (w.flags & kTwoKeyGroups) != 0; };
  auto prefetch = [&](int ti, bf16x8_t (&qn)[GE::KS]) {
    const WorkTile tn = tiles[ti];
    const int rbn = two_groups(tn) ? 0 : rb;
    if (32 * rbn < tn.n_rows && lane < GE::CH) {
      const unsigned char* src =
          reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(tn.q_pos0 + 32 * rbn) * (D / 2)) + 16 * lane;
      dma16(src, br_lds);
    }
    if (32 * rbn + r < tn.n_rows) {
      const bf16_t* src = q + (static_cast<int64_t>(tn.q_row0 + 32 * rbn + r) * hq + head) * D + 8 * h2;
#pragma unroll
      for (int s = 0; s < GE::KS; ++s) qn[s] = *reinterpret_cast<const bf16x8_t*>(src + 16 * s);
    } else {
#pragma unroll
      for (int s = 0; s < GE::KS; ++s) qn[s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
    }
  };
  // qf <- R(position) qn * log2(e)/sqrt(d), rounded to bf16 once
  auto rotate_next = [&](const WorkTile& tn, const bf16x8_t (&qn)[GE::KS]) {
    wait_vm_all();  // this wave's base row and query have landed
    __asm__ volatile("" ::: "memory");
    if (32 * (two_groups(tn) ? 0 : rb) >= tn.n_rows) {  // no row of this wave is real
#pragma unroll
      for (int s = 0; s < GE::KS; ++s) qf[s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
      return;
    }
    const float4* br = reinterpret_cast<const float4*>(br_lds);
    const float4* rt = reinterpret_cast<const float4*>(rt_lds + r * 4 * D);
#pragma unroll
    for (int s = 0; s < GE::KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qn[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qn[s + GE::KS / 2]);
      u32x4_t na, nb;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        // frequencies 16s + 8h2 + 2e2 and +1: one 16-byte chunk of each rotary row
        const int ch = 8 * s + 4 * h2 + e2;
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
      qf[s + GE::KS / 2] = __builtin_bit_cast(bf16x8_t, nb);
    }
  };
  {
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
      bf16x8_t qn[GE::KS];
      prefetch(t0, qn);
      wait_vm_all();
      block_sync();  // every wave's share of the table has landed
      rotate_next(tiles[t0], qn);
    }
  }

  int c = 0;  // stream index of the tile being computed
  for (int ct = t0; ct < n_tiles_total;) {
    const WorkTile t = tiles[ct];
    const int n_tiles = (t.kv_end - t.kv_begin) >> 2;
    const bool two = two_groups(t);
    const int grp = two ? rb : 0;          // key group of this wave
    const int irow = two ? r : row;        // this lane's row inside the item
    const int rb0 = two ? 0 : 32 * rb;     // first row of this wave
    const bool row_ok = irow < t.n_rows;
    // a wave whose rows are all past the item's rows only moves tiles (few-row
    // items, e.g. short cross segments, then cost half the compute)
    const bool active = rb0 < t.n_rows;
    const bool has_next = ct + tstride < n_tiles_total;
    qpos = t.q_pos0 + irow;
    wave_min_pos = t.q_pos0 + rb0;

#pragma unroll
    for (int s = 0; s < GE::KS; ++s) qbase[s] = qf[s];
    q_delta = 0;
#pragma unroll
    for (int db = 0; db < GE::DB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
    m = kNoMax;
    l = 0.f;
    bool first = true;  // this wave's first tile of the item

    // ---- key tiles of this item, in groups of two (one for an odd last tile)
    bf16x8_t qn[GE::KS];  // raw query of the next item, loaded after the loop
    auto compute = [&](int j, int cs) {  // tile j of the item, stream slot cs
      // page entries of the tile, consumed here: a scalar-load wait later on would
      // also drain the LDS reads of the QK step (both share one counter)
      TilePages cur;
      read_tile(kt, (t.kv_begin >> 2) + j, cur);
      __asm__ volatile("" ::"s"(cur.pos0), "s"(cur.nk), "s"(cur.delta));
      const unsigned char* stage = lds + (cs & 3) * GE::STAGE;
      if (cur.delta != q_delta) {
        q_delta = cur.delta;
        rotate_q(stage);
      }
      bf16x8_t pk[4];
      softmax(
          [&](f32x16_t (&sc)[2]) {
            qk(stage, sc);
            mask(sc, cur);
          },
          pk, first);
      first = false;
      pv(stage, pk);
    };
    for (int j = 0; j < n_tiles;) {
      const int sz = min(2, n_tiles - j);
      // tiles c .. c + sz - 1 have landed for every wave, and every wave is done with
      // the tiles before c, whose stages take the next ones (up to c + 3)
      wait_tiles<NDMA>(n_issued - c - sz);
      block_sync();
#pragma unroll
      for (int u = 0; u < kStages - 1; ++u)
        if (n_issued < c + kStages) issue_next();
      if (active) {
        // two key groups: this wave takes tile grp of the pair; otherwise both
        const int u1 = two ? min(grp + 1, sz) : sz;
        for (int u = grp; u < u1; ++u) compute(j + u, c + u);
      }
      c += sz;
      j += sz;
    }

    // ---- epilogue of the item.  The next item's query is rotated first, so the
    // output stores do not sit in front of that wait; the loop is only re-entered
    // through that rotation, so no path carries a pending query load around it.
    const float l_row = l + __int_as_float(__builtin_amdgcn_ds_bpermute(xor32_addr, __float_as_int(l)));
    auto store = [&]() {
      if (!row_ok) return;
      const int64_t orow = static_cast<int64_t>(t.q_row0 + irow);
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
        const int64_t slot = (static_cast<int64_t>(t.part + grp) * hq + head) * BM + irow;
        f16_t* po = part_o + slot * D;
        const float inv = l_row > 0.f ? 1.f / l_row : 0.f;  // O / l in fp16
#pragma unroll
        for (int db = 0; db < GE::DB; ++db)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = 32 * db + 8 * g4 + 4 * h2;
            *reinterpret_cast<f16x4_t*>(po + d0) =
                f16x4_t{static_cast<f16_t>(o[db][4 * g4] * inv), static_cast<f16_t>(o[db][4 * g4 + 1] * inv),
                        static_cast<f16_t>(o[db][4 * g4 + 2] * inv), static_cast<f16_t>(o[db][4 * g4 + 3] * inv)};
          }
        if (h2 == 0) {  // a row that saw no key: max -inf, as the merge expects
          part_ml[slot * 2] = l_row > 0.f ? m : -INFINITY;
          part_ml[slot * 2 + 1] = l_row;
        }
      }
    };
    if (!has_next) {
      store();
      break;
    }
    prefetch(ct + tstride, qn);
    rotate_next(tiles[ct + tstride], qn);
    store();
    ct += tstride;
  }
}

int mfma_bm(int g) { return 32 * (kNW / g); }

bool mfma_supported(int hq, int hkv, int d, int dtype) {
  if (dtype != SPAN_BF16 || hkv <= 0 || hq % hkv != 0) return false;
  const int g = hq / hkv;
  return (d == 64 || d == 128) && (g == 1 || g == 2 || g == 4 || g == 8);
}

hipError_t cu_count(int* n) {
  static int cached[64] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && cached[dev] > 0) {
    *n = cached[dev];
    return hipSuccess;
  }
  e = hipDeviceGetAttribute(n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64) cached[dev] = *n;
  return hipSuccess;
}

template <int D, int G>
static hipError_t launch_t(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q, void* out,
                           void* part_o, float* part_ml, const float2* rope, const CrossWrites& w, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  const size_t lds = Geo<D>::LDS;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_mfma_kernel<D, G>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (attr != hipSuccess) return attr;
  int cus = 0;
  hipError_t e = cu_count(&cus);
  if (e != hipSuccess) return e;
  // one work-group per CU, a multiple of hkv (each keeps one kv head)
  const int64_t items = static_cast<int64_t>(n) * g.hkv;
  const int grid = static_cast<int>(std::min<int64_t>(items, std::max(1, cus / g.hkv) * g.hkv));
  hipLaunchKernelGGL((attn_mfma_kernel<D, G>), dim3(grid), dim3(kNT), lds, s, tiles, n, kt,
                     static_cast<const bf16_t*>(q), static_cast<bf16_t*>(out), static_cast<bf16_t*>(g.base),
                     g.layer_off, g.hq, g.hkv, scale_log2, rope, static_cast<f16_t*>(part_o), part_ml,
                     static_cast<const bf16_t*>(w.k), static_cast<const bf16_t*>(w.v), w.pages);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q, void* out,
                           void* po, float* pml, const float2* rope, const CrossWrites& w, hipStream_t s) {
  switch (g.hq / g.hkv) {
    case 1: return launch_t<D, 1>(g, tiles, n, kt, q, out, po, pml, rope, w, s);
    case 2: return launch_t<D, 2>(g, tiles, n, kt, q, out, po, pml, rope, w, s);
    case 4: return launch_t<D, 4>(g, tiles, n, kt, q, out, po, pml, rope, w, s);
    case 8: return launch_t<D, 8>(g, tiles, n, kt, q, out, po, pml, rope, w, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_mfma(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q,
                            void* out, void* part_o, float* part_ml, const float2* rope, const CrossWrites& w,
                            hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!mfma_supported(g.hq, g.hkv, g.d, g.dtype)) return hipErrorInvalidValue;
  if (w.pages && (!w.k || !w.v)) return hipErrorInvalidValue;
  return g.d == 128 ? launch_d<128>(g, tiles, n, kt, q, out, part_o, part_ml, rope, w, s)
                    : launch_d<64>(g, tiles, n, kt, q, out, part_o, part_ml, rope, w, s);
}

}  // namespace spanq
