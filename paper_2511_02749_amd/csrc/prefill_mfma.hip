// Span-prefill attention (rows of new prefix and fragment pages) as a
// software-pipelined bf16 MFMA kernel for gfx950 (CDNA4).
//
// What it computes (span-query prefill, sections 5.1 and 5.6 of the paper): every
// row of a fragment attends causally to the shared prefix and to its own fragment,
// at the fragment's query-independent (canonical) positions; prefix rows attend
// causally to the prefix.  The planner has already laid out, per row tile, the list
// of key pages the tile may see, padded to whole 4-page tiles; keys past a row's own
// position and empty page slots are masked here.
//
// Work items, operand layouts and the query rotation are those of the cross kernel
// (attn_mfma.hip): an item is (row tile of 256/G tokens, kv head), wave w handles
// query head w mod G and rows 32(w div G) .. +31, scores are formed transposed
// (S^T = K Q^T, v_mfma_f32_32x32x16_bf16) so each lane owns one query row, and P^T
// feeds O^T = V^T P^T straight from registers.
//
// The difference is the key loop.  The 64-key tiles of an item are split into
// 32-key blocks, and block u is processed as
//     QK(u + 1)  ||  softmax(u)  ||  PV(u - 1)
// in one fenced instruction sequence: the QK and PV MFMAs of the neighbouring blocks
// run while this wave's vector ALU does the softmax of the block between them,
// instead of every wave alternating between MFMA-only and VALU-only phases.
//
// Softmax uses a lazily raised running max: P = 2^(S - m) is taken against the
// current m, which an item's first block sets to its row max and which is raised
// afterwards only when a block's exponentials, summed per lane, pass 2^16 (or are
// not finite).  After the first block, a block's QK accumulator starts at -m, so the
// MFMAs themselves form S - m; a raise by d shifts the next block's scores (already
// formed) by -d.  The check costs one compare per block and no row max; the rare
// raise (row max, P taken again, rescale of O and of the row sum) is a branch after
// the pipelined block, so the block itself has no data-dependent control.  P stays
// below 2^16, which bf16 and the fp32 accumulators hold with the same relative
// precision as values below 1; the result O / l does not depend on which m was used.
// The row max is reduced with a max3 tree and one v_permlane32_swap (no LDS round
// trip); the row sum comes from v_dot2 over the packed bf16 P, i.e. exactly the
// weights the PV MFMAs use.
//
// K/V stream: the key tiles of a work-group's items form one stream.  Before the
// QK of stream tile x every wave waits for its own DMA of tiles <= x, passes one
// barrier, and prepares the DMA of tile x + 2 (HBM to LDS, global_load_lds from a
// scalar page address, no register staging), whose instructions it issues one per
// chunk of the block that follows, so the eight waves do not queue them at once.
// When the stream enters an item, each wave also touches the query rows it will load
// for it two tiles later, so that load finds them in the caches.  K(x) is read only by QK(x), before the barrier of tile x + 1,
// and V(x) only by PV(x), before the barrier of tile x + 2; so the fetch at the
// barrier of tile x may overwrite the K of tile x - 1 and the V of tile x - 2: a
// 3-slot K ring and a 4-slot V ring (132 KiB of LDS at head dim 128 with the rotary
// rows).  Both tiles' LDS layouts are read conflict-free by 16 consecutive lanes.
//
// Work-groups take items from queue counters (three items ahead), so compute units
// that run slower take fewer; with eight queues, one per XCD, the work-groups of an
// XCD share one kv head of a group of spans, so pages that a span's row tiles all
// read are fetched into that XCD's L2 once.  An item's output rows leave through an
// LDS staging area as whole row segments at the next item's first barrier.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <type_traits>

#include "../../include/spanq.h"
#include "dev_common.h"
#include "kernels.h"
#include "mfma_common.h"

namespace spanq {

namespace {

using namespace mfma;

template <int D>
struct PGeo {
  static constexpr int KS = D / 16;                         // 16-dim steps of the QK contraction
  static constexpr int DB = D / 32;                         // 32-dim blocks of the output
  static constexpr int KBYTES = kBN * D * 2;                // K tile [64 keys][D]
  static constexpr int VBYTES = D * kBN * 2;                // V tile [D][64 positions]
  static constexpr int KPW = KBYTES / 1024 / kNW;         // K DMA instructions per wave per tile
  static constexpr int VPW = VBYTES / 1024 / kNW;         // V DMA instructions per wave per tile
  static constexpr int NDMA = KPW + VPW;
  static constexpr int NK = 3;                              // K ring slots
  static constexpr int NV = 4;                              // V ring slots
  static constexpr int CH = D / 4;                          // 16-byte chunks per rotary row
  static constexpr int RTBYTES = 32 * 4 * D;                // rotary rows of positions 0..31
  static constexpr int BRBYTES = kNW * 4 * D;               // one rotary row per wave (its rows' base)
  static constexpr int VOFF = NK * KBYTES;
  static constexpr int RTOFF = VOFF + NV * VBYTES;
  static constexpr int BROFF = RTOFF + RTBYTES;
  // Output staging, per wave 32 rows of SROW bytes: at head dim 128 the V slot freed
  // by the previous item (16 KiB, one 32-dim block per pass), at 64 a region of its
  // own (whole 128-byte rows in one pass).
  static constexpr bool STAGE_IN_V = D == 128;
  static constexpr int SROW = STAGE_IN_V ? VBYTES / kNW / 32 : 2 * D;
  static constexpr int STOFF = BROFF + BRBYTES;
  static constexpr int SCHOFF = STOFF + (STAGE_IN_V ? 0 : kNW * 32 * SROW);  // schedule words
  static constexpr int TOFF = SCHOFF + 64;  // per wave 256 bytes that cache-warming loads land in
  static constexpr int LDS = TOFF + kNW * 256;
  static_assert(SROW % 64 == 0 && (2 * D) % SROW == 0, "a pass covers whole 32-dim blocks");
};

__device__ __forceinline__ float max3f(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

// Combine a value with the one of the other half-wave (lane ^ 32).
__device__ __forceinline__ float swap_max(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float swap_sum(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}


// s_waitcnt vmcnt(n) for n in {0, N}
template <int N>
__device__ __forceinline__ void wait_group(int n) {
  if (n)
    wait_vmcnt<N>();
  else
    wait_vmcnt<0>();
}

}  // namespace

template <int D, int G>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(2, 2))) void prefill_mfma_kernel(
    const WorkTile* __restrict__ tiles, int n_items, const TileRec* __restrict__ kt, const bf16_t* __restrict__ q,
    bf16_t* __restrict__ out, const bf16_t* __restrict__ pool, int64_t layer_off, int hq, int hkv, float scale_log2,
    const float2* __restrict__ rope, unsigned* __restrict__ sched, const int32_t* __restrict__ xchunks,
    int n_chunks) {
  using GE = PGeo<D>;
  constexpr int KS = GE::KS, DB = GE::DB, NDMA = GE::NDMA;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int hsub = wave % G;  // head inside the kv head's group
  const int rb = wave / G;    // 32-row block
  const int h2 = lane >> 5;
  const int r = lane & 31;
  const int row = 32 * rb + r;  // this lane's row inside an item
  const int64_t page_elems = 2ll * hkv * kPage * D;
  unsigned char* const kring = lds;
  unsigned char* const vring = lds + GE::VOFF;
  unsigned char* const rt_lds = lds + GE::RTOFF;
  unsigned char* const br_lds = lds + GE::BROFF + wave * 4 * D;

  // ---------------- item schedule.  Item e is (row tile e / hkv, kv head e mod hkv).
  // Items come from queues, each with its own counter sched[x]:
  // - one queue (n_chunks == 0): every item, e = r, row tiles longest first;
  // - eight queues, one per XCD (n_chunks == 8 / hkv): queue x holds the tiles of
  //   chunk x / hkv for kv head x mod hkv, e = (chunk start + r) hkv + x mod hkv.
  //   Work-groups are dispatched to the eight XCDs in turn, so work-group b is on
  //   XCD b mod 8 and takes from queue b mod 8: a queue's K/V pages stay in one L2.
  // Work-group b takes the first two items of its queue statically (its position
  // among the queue's work-groups, and that plus their count), then one item at a
  // time from the queue's counter, so compute units that run faster take more items.
  // A work-group whose queue runs dry moves on to the next queue (the XCDs of one
  // chip do not run this kernel equally fast); items are "none" once every queue is
  // dry.  Counters only grow, so a dry queue stays dry.  (The host uses eight queues
  // only when every queue holds at least its two static items per work-group.)
  // The grab for item k + 3 is issued right after the first barrier of item k and
  // its result is first read at the first barrier of item k + 1, after that
  // barrier's full wait: the atomic's latency hides behind a whole item.  Only a
  // move to another queue waits for an atomic.  (The build turns off the compiler's
  // atomic optimizer, whose broadcast of the result would read it, and so wait for
  // it, right after the atomic.)
  const int n_total = n_items * hkv;
  const int grid = gridDim.x;
  const int n_queues = n_chunks > 0 ? 8 : 1;
  const int home = n_chunks > 0 ? static_cast<int>(blockIdx.x & 7) : 0;
  const int q_wgs = n_chunks > 0 ? (grid - home + 7) >> 3 : grid;             // work-groups of the home queue
  const int q_pos = n_chunks > 0 ? static_cast<int>(blockIdx.x >> 3) : static_cast<int>(blockIdx.x);
  int h_tile0 = 0, h_head = 0, h_len = n_total;
  if (n_chunks > 0) {
    const int c = home / hkv;
    h_tile0 = xchunks[c];
    h_len = xchunks[c + 1] - h_tile0;
    h_head = home - c * hkv;
  }
  auto home_item = [&](int r) __attribute__((always_inline)) {
    return n_chunks > 0 ? (h_tile0 + r) * hkv + h_head : r;
  };
  int ec0 = home_item(q_pos);                                          // compute item k
  int ec1 = q_pos + q_wgs < h_len ? home_item(q_pos + q_wgs) : n_total;  // item k + 1
  int ec2 = n_total;                                  // item k + 2, read at item k's first barrier
  unsigned grab_raw = 0;   // thread 0: counter value the last grab returned
  bool grabbed = false;    // the last grab was issued (not skipped as known empty)
  int* const sched_lds = reinterpret_cast<int*>(lds + GE::SCHOFF);  // two slots, by item parity
  // Thread 0's current queue, kept in LDS (only thread 0 touches it), so that it holds
  // no registers across the key loop: index, first tile, kv head, length, first
  // counted item, queue moves so far.
  int* const qs = sched_lds + 4;
  auto set_queue = [&](int x) __attribute__((always_inline)) {  // thread 0
    int tile0 = 0, head = 0, len = n_total, first = 2 * grid;
    if (n_chunks > 0) {
      const int c = x / hkv;
      tile0 = xchunks[c];
      len = xchunks[c + 1] - tile0;
      head = x - c * hkv;
      first = 2 * ((grid - x + 7) >> 3);
    }
    qs[0] = x;
    qs[1] = tile0;
    qs[2] = head;
    qs[3] = len;
    qs[4] = first;
  };
  if (threadIdx.x == 0) {
    set_queue(home);
    qs[5] = 0;
  }
  auto grab = [&](int last_known) __attribute__((always_inline)) {
    grabbed = last_known < n_total;
    if (grabbed && threadIdx.x == 0) grab_raw = atomicAdd(sched + qs[0], 1u);
  };
  auto grabbed_item = [&]() __attribute__((always_inline)) {  // thread 0
    if (!grabbed) return n_total;
    int r = qs[4] + static_cast<int>(grab_raw);
    while (r >= qs[3]) {
      const int moves = qs[5] + 1;
      qs[5] = moves;
      if (moves >= n_queues) return n_total;
      set_queue(qs[0] == 7 ? 0 : qs[0] + 1);
      r = qs[4] + static_cast<int>(atomicAdd(sched + qs[0], 1u));
    }
    return n_chunks > 0 ? (qs[1] + r) * hkv + qs[2] : r;
  };

  // ---------------- DMA side: the stream's next tile is tile dk_j of item dk_e, which
  // is item k + dk_k of the schedule
  ItemKeys dk;
  int dk_k = 0, dk_e = ec0, dk_j = 0;
  bool dk_ok = true;
  load_item_keys(tiles, dk_e / hkv, dk);
  int dk_kvh = dk_e % hkv;
  int fk = 0, fv = 0;  // ring slots of the next fetch
  // Per-lane source offsets (bytes, inside a page) of this wave's DMA instructions.
  // K instruction u fills LDS bytes [1024q, 1024q + 1024) of the K tile, q = wave
  // KPW + u: keys 4q.. (head dim 128) of one page, chunk c of key k stored at chunk
  // c ^ kswz(k).  V instruction u fills 1024 bytes of the V tile, which is laid out
  // [page][d][two 16-byte halves], half h of row d stored at h ^ (d >> 3 & 1): rows
  // 32b .. 32b + 31 of one page.  Every instruction of wave w reads page w / 2 of the
  // tile, so a fetch is one scalar page address plus these 32-bit offsets.
  constexpr int CPK = D / 8;  // 16-byte chunks per key row
  static_assert(GE::KPW * (64 / CPK) * 2 == 16 && GE::VPW * 2 == D / 32, "one page per wave");
  const int wpage = wave / 2;
  uint32_t dk_ofs[GE::KPW], dv_ofs[GE::VPW];
#pragma unroll
  for (int u = 0; u < GE::KPW; ++u) {
    const int qi = wave * GE::KPW + u;
    const int key = qi * (64 / CPK) + lane / CPK;
    const int c = (lane % CPK) ^ kswz<D>(key);
    dk_ofs[u] = 2u * static_cast<uint32_t>((key & 15) * D + 8 * c);
  }
#pragma unroll
  for (int u = 0; u < GE::VPW; ++u) {
    const int qi = wave * GE::VPW + u;
    const int d = 32 * (qi % (D / 32)) + (lane >> 1);
    const int h = (lane & 1) ^ ((d >> 3) & 1);
    dv_ofs[u] = 2u * static_cast<uint32_t>(hkv * kPage * D + d * kPage + 8 * h);
  }
  // (position of key 0, real keys) of stream tiles x, x + 1, x + 2 after the fetch
  // at the barrier of tile x
  int mp0 = 0, mn0 = 0, mp1 = 0, mn1 = 0, mp2 = 0, mn2 = 0;
  // A fetch is prepared at a barrier (tile record, page address, LDS slots) and its
  // NDMA instructions are issued either at once or one per chunk of the block that
  // follows the barrier, so that the eight waves do not all queue their DMA at the
  // same moment.
  const unsigned char* f_base = nullptr;  // the wave's page of the prepared tile
  uint32_t f_mk = 0, f_mv = 0;           // LDS destinations of its K and V instructions
  const unsigned char* const pool_b = reinterpret_cast<const unsigned char*>(pool + layer_off);
  unsigned char* const touch_lds = lds + GE::TOFF + wave * 256;
  auto fetch_prep = [&]() __attribute__((always_inline)) -> int {  // DMA instructions to issue
    if (dk_ok && dk_j >= dk.n) {  // every item has at least one key tile
      ++dk_k;
      dk_e = dk_k == 1 ? ec1 : ec2;
      dk_j = 0;
      dk_ok = dk_e < n_total;
      if (dk_ok) {
        load_item_keys(tiles, dk_e / hkv, dk);
        dk_kvh = dk_e % hkv;
        // the query rows this wave will load for the new item, two tiles from now,
        // brought into the caches now (lines of 128 bytes, D / 64 per row)
        const WorkTile* tn = tiles + __builtin_amdgcn_readfirstlane(dk_e / hkv);
        const int rows = tn->n_rows, row0 = tn->q_row0;
        constexpr int LPR = D / 64;
        const int trow = 32 * rb + lane / LPR;
        if (lane < 32 * LPR && trow < rows)
          touch4_m0(q + (static_cast<int64_t>(row0 + trow) * hq + dk_kvh * G + hsub) * D + 64 * (lane % LPR),
                    lds_byte(touch_lds));
      }
    }
    mp0 = mp1;
    mn0 = mn1;
    mp1 = mp2;
    mn1 = mn2;
    if (!dk_ok) return 0;
    TilePages tp;
    read_tile(kt, (dk.kv_begin >> 2) + dk_j, tp);
    mp2 = tp.pos0;
    mn2 = tp.nk;
    // the kv head's K rows of a page start kvh * 16 * D elements in, its V rows as many
    // elements past the page's V half
    f_base = pool_b + (static_cast<int64_t>(pick4(tp.id, wpage)) * page_elems + dk_kvh * kPage * D) * 2;
    f_mk = lds_byte(kring + fk * GE::KBYTES + wave * GE::KPW * 1024);
    f_mv = lds_byte(vring + fv * GE::VBYTES + wave * GE::VPW * 1024);
    ++dk_j;
    fk = (fk == GE::NK - 1) ? 0 : fk + 1;
    fv = (fv == GE::NV - 1) ? 0 : fv + 1;
    return NDMA;
  };
  int last_ops = 0;  // DMA instructions of the most recent fetch group
  auto issue_dma = [&](int u) __attribute__((always_inline)) {  // instruction u of the prepared fetch
    if (u < GE::KPW)
      dma16_s(f_base, dk_ofs[u], f_mk + u * 1024);
    else
      dma16_s(f_base, dv_ofs[u - GE::KPW], f_mv + (u - GE::KPW) * 1024);
  };
  auto fetch_next = [&]() __attribute__((always_inline)) -> int {  // prepared and issued at once
    const int n = fetch_prep();
    if (n) {
#pragma unroll
      for (int u = 0; u < NDMA; ++u) issue_dma(u);
    }
    return n;
  };

  // ---------------- compute-side state
  bf16x8_t qf[KS];  // Q^T operand of the current item (rotated, scaled by log2(e)/sqrt(d))
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m = kNoMax, l = 0.f;
  // -m in all 16 places: the initial value of a block's QK accumulator, so that the
  // MFMAs form S - m (every block but an item's first, whose scores are raw)
  f32x16_t mneg;
#pragma unroll
  for (int i = 0; i < 16; ++i) mneg[i] = 0.f;
  auto set_mneg = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 16; ++i) mneg[i] = -m;
  };
  int qpos = 0, wave_min_pos = 0;

  // Per-lane LDS byte offsets of the MFMA operand reads inside a ring slot: K step
  // ks of key block 0 (block 1 is 32 rows further, a constant), and the V operand of
  // page 0, dims 0..31 (other pages and dim blocks are constant offsets).
  uint32_t kofs[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) kofs[ks] = 2u * (r * D + 8 * ((2 * ks + h2) ^ kswz<D>(r)));
  const uint32_t vofs = 32u * r + 16u * (h2 ^ ((r >> 3) & 1));
  auto lds_at = [&](uint32_t base, uint32_t ofs) __attribute__((always_inline)) {
    return reinterpret_cast<const bf16x8_t*>(lds + base + ofs);
  };

  // ---- building blocks of one 32-key block (block kb of a 64-key tile)
  // S^T = K Q^T over the block
  auto qk = [&](uint32_t kbase, int kb, f32x16_t& sc) __attribute__((always_inline)) {
    kbase += kb * 32 * D * 2;
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*lds_at(kbase, kofs[ks]), qf[ks], sc, 0, 0, 0);
  };
  // causal positions and partial/empty pages, for block kb of a tile whose key 0 is
  // at pos0 with nk real keys; the test is wave-uniform.  Element i is key
  // 32kb + 8(i/4) + 4h2 + i%4 of the tile, kept iff it is a real key (< nk) at a
  // position <= the row's.
  auto mask = [&](f32x16_t& sc, int kb, int pos0, int nk) __attribute__((always_inline)) {
    if (nk < 32 * kb + 32 || pos0 + 32 * kb + 31 > wave_min_pos) {
      const int lim = min(nk, qpos - pos0 + 1) - 32 * kb - 4 * h2;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (8 * (i >> 2) + (i & 3) >= lim) sc[i] = -INFINITY;
    }
  };
  // the block's row max (both half-waves)
  auto row_max = [&](const f32x16_t& sc) __attribute__((always_inline)) -> float {
    const float a0 = max3f(sc[0], sc[1], sc[2]), a1 = max3f(sc[3], sc[4], sc[5]);
    const float a2 = max3f(sc[6], sc[7], sc[8]), a3 = max3f(sc[9], sc[10], sc[11]);
    const float a4 = max3f(sc[12], sc[13], sc[14]);
    return swap_max(max3f(max3f(a0, a1, a2), max3f(a3, a4, sc[15]), -INFINITY));
  };
  // O^T += V^T P^T over block kb of a tile (its pages 2kb, 2kb + 1); the V operand of
  // page g, dims 32db.. is 16 bytes at [g][32db + r][half h2]
  auto pv = [&](uint32_t vbase, int kb, const bf16x8_t (&pk)[2]) __attribute__((always_inline)) {
    vbase += kb * 2 * D * 32;
    const bf16x8_t* a = lds_at(vbase, vofs);
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int db = 0; db < DB; ++db)  // DB independent accumulator chains
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(half * D * 32 + db * 1024) / 16], pk[half], o[db], 0, 0, 0);
  };
  // P = 2^(sc - d) of a block's 16 (offset) scores in this lane, packed to bf16 in w;
  // the row sums of the packed values in ts0, ts1
  auto exp_block = [&](const f32x16_t& sc, float d, u32x4_t (&w)[2], float& ts0, float& ts1) __attribute__((always_inline)) {
    const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);
    ts0 = 0.f;
    ts1 = 0.f;
#pragma unroll
    for (int wd = 0; wd < 8; ++wd) {
      const int half = wd >> 2, e = wd & 3;
      const uint32_t pw = pack_bf16x2(__builtin_amdgcn_exp2f(sc[8 * half + 2 * e] - d),
                                      __builtin_amdgcn_exp2f(sc[8 * half + 2 * e + 1] - d));
      w[half][e] = pw;
      if (e & 1)
        ts1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts1, false);
      else
        ts0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts0, false);
    }
  };
  // The rare raise of the running max, after a block whose exponentials (taken
  // against the current m; its scores sc are S - m) summed past kSumCap in some lane
  // or were not finite: m moves up by d to the block's row max, the block's P is
  // taken again, and corr = 2^-d rescales what was accumulated.  Returns d.
  auto raise_max = [&](const f32x16_t& sc, u32x4_t (&w)[2], float& ts0, float& ts1, float& corr)
                       __attribute__((always_inline)) -> float {
    const float d = fmaxf(0.f, row_max(sc));
    corr = __builtin_amdgcn_exp2f(-d);
    m += d;
    exp_block(sc, d, w, ts0, ts1);
    set_mneg();
    return d;
  };
  // after the block (whose PV MFMAs still added terms taken against the old m): the
  // rare rescale of O and l, then the block's row sum
  auto rescale = [&](bool up, float corr, float tsum) __attribute__((always_inline)) {
    if (__builtin_expect(up, 0)) {
      __asm__ volatile("");
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
      l *= corr;
    }
    l += tsum;
  };

  // Operands of a block's chunks 0 and 1, read during the block before it.
  struct Pre {
    bf16x8_t k[2], v[2];
  };
  // One pipelined block, in a fixed instruction order: the softmax of scores s_in
  // (lazily raised max, P = 2^(S - m) packed into pk_out, its row sum) runs in KS
  // chunks; chunk t also issues the QK MFMA of step t of the next key block (WQK, K
  // tile at byte kaddr) and the PV MFMA t of the previous block (WPV, V of pages
  // vaddr.., operand pk_prev), the LDS reads of the operands two chunks ahead and,
  // in the block after a barrier (WDMA), one DMA instruction of the fetch prepared
  // there.  The operands of chunks 0 and 1 come from the previous block (pre.v always;
  // pre.k if PREK, else K is read here, right after the barrier that made it
  // valid), and the last two chunks read those of the next block (K at nkaddr if
  // NXK, V at nvaddr if NXV), so the MFMAs of chunk 0 need not wait for LDS.  Chunk
  // 0 issues its MFMAs before the row max, which they do not depend on.  The chunks
  // are fenced, so the compiler keeps this order and at most four operand reads (16
  // registers) are in flight.
  auto block = [&](auto wqk, auto wpv, auto prek, auto nxk, auto nxv, auto wdma, const f32x16_t& s_in,
                   bf16x8_t (&pk_out)[2], uint32_t kaddr, f32x16_t& s_out, uint32_t vaddr,
                   const bf16x8_t (&pk_prev)[2], Pre& pre, uint32_t nkaddr, uint32_t nvaddr, float& corr,
                   float& tsum) __attribute__((always_inline)) -> bool {
    constexpr bool WQK = decltype(wqk)::value, WPV = decltype(wpv)::value, PREK = decltype(prek)::value;
    constexpr bool NXK = decltype(nxk)::value, NXV = decltype(nxv)::value, WDMA = decltype(wdma)::value;
    constexpr int WPC = 8 / KS;  // packed words of P per chunk (8 words per block)
    auto rdk = [&](uint32_t base, int t) __attribute__((always_inline)) { return *lds_at(base, kofs[t]); };
    auto rdv = [&](uint32_t base, int t) __attribute__((always_inline)) {
      return lds_at(base, vofs)[((t / DB) * D * 32 + (t % DB) * 1024) / 16];
    };
    bf16x8_t ak[KS], av[KS];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if constexpr (WQK) ak[t] = PREK ? pre.k[t] : rdk(kaddr, t);
      if constexpr (WPV) av[t] = pre.v[t];
    }
    auto qk_mfma = [&](int t) __attribute__((always_inline)) {
      s_out = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[t], qf[t], t == 0 ? mneg : s_out, 0, 0, 0);
    };
    const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);
    float ts0 = 0.f, ts1 = 0.f;
    u32x4_t w[2];
    bool up = false;
#pragma unroll
    for (int t = 0; t < KS; ++t) {
      if constexpr (WQK) {
        if (PREK || t > 0) qk_mfma(t);
      }
      if constexpr (WPV) o[t % DB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[t], pk_prev[t / DB], o[t % DB], 0, 0, 0);
      if constexpr (WDMA) {  // one DMA instruction of the fetch prepared at the barrier
        if (t < NDMA && last_ops) issue_dma(t);
      }
      if (t + 2 < KS) {
        if constexpr (WQK) ak[t + 2] = rdk(kaddr, t + 2);
        if constexpr (WPV) av[t + 2] = rdv(vaddr, t + 2);
      } else {
        if constexpr (NXK) pre.k[t + 2 - KS] = rdk(nkaddr, t + 2 - KS);
        if constexpr (NXV) pre.v[t + 2 - KS] = rdv(nvaddr, t + 2 - KS);
      }
      if (t == 0) {
        __builtin_amdgcn_sched_barrier(0);
        // an item's first block (the only one without PV work; its scores are raw) sets
        // m to its row max (every row of an item sees its list's first key; a row that
        // saw none would start from m = 0, with nothing accumulated yet)
        if constexpr (!WPV) {
          m = fmaxf(m, row_max(s_in));
          m = m == kNoMax ? 0.f : m;
          set_mneg();
        }
        if constexpr (WQK && !PREK) qk_mfma(0);
      }
#pragma unroll
      for (int x = 0; x < WPC; ++x) {
        const int wd = t * WPC + x, half = wd >> 2, e = wd & 3;
        // scores are S - m already, except an item's first block's
        const float p0 = __builtin_amdgcn_exp2f(WPV ? s_in[8 * half + 2 * e] : s_in[8 * half + 2 * e] - m);
        const float p1 = __builtin_amdgcn_exp2f(WPV ? s_in[8 * half + 2 * e + 1] : s_in[8 * half + 2 * e + 1] - m);
        // the dot product takes the packed word itself, not w[.][e] read back: with
        // the read-back form, hipcc 7.2 at -O3 feeds every fdot2 the vector's element 0
        const uint32_t pw = pack_bf16x2(p0, p1);
        w[half][e] = pw;
        if (e & 1)
          ts1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts1, false);
        else
          ts0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw), ones, ts0, false);
      }
      // the chunk's exponentials end here: without this, the optimizer moves every
      // one of them behind the block's last MFMA
      __asm__ volatile("" : "+v"(ts0), "+v"(ts1));
      __builtin_amdgcn_sched_barrier(0);
    }
    tsum = ts0 + ts1;
    corr = 1.f;
    if (WPV && __builtin_expect(__any(!(tsum <= kSumCap)), 0)) {
      up = true;
      const float d = raise_max(s_in, w, ts0, ts1, corr);
      tsum = ts0 + ts1;
      if constexpr (WQK) {  // the next block's scores were formed against the old m
#pragma unroll
        for (int i = 0; i < 16; ++i) s_out[i] -= d;
      }
    }
    pk_out[0] = __builtin_bit_cast(bf16x8_t, w[0]);
    pk_out[1] = __builtin_bit_cast(bf16x8_t, w[1]);
    return up;
  };

  // ---------------- query rotation at item start: the rotary angles of row r (0..31)
  // of a wave's 32-row block come from R(base + r) = R(base) R(r), with R(0..31)
  // kept in LDS for the whole kernel and R(base) (base = the block's first
  // position) brought into LDS by DMA together with the item's raw query.
  // (these helpers run once per item; their per-lane address parts are derived
  // from an opaque copy of the lane id so that none of them is hoisted out of the
  // item loop into registers held across the tile loop)
  auto prefetch = [&](int e, bf16x8_t (&qn)[KS]) __attribute__((always_inline)) {
    const WorkTile tn = tiles[e / hkv];
    const int head = (e % hkv) * G + hsub;
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
    const int lrow = 32 * rb + (ln & 31), lh2 = ln >> 5;
    if (32 * rb < tn.n_rows && ln < GE::CH) {
      const unsigned char* src =
          reinterpret_cast<const unsigned char*>(rope + static_cast<int64_t>(tn.q_pos0 + 32 * rb) * (D / 2)) +
          16 * ln;
      dma16(src, br_lds);
    }
    if (lrow < tn.n_rows) {
      const bf16_t* src = q + (static_cast<int64_t>(tn.q_row0 + lrow) * hq + head) * D + 8 * lh2;
#pragma unroll
      for (int s = 0; s < KS; ++s) qn[s] = *reinterpret_cast<const bf16x8_t*>(src + 16 * s);
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) qn[s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
    }
  };
  // qf <- R(position) qn * log2(e)/sqrt(d), rounded to bf16 once (the loads of qn
  // and of the base row must have landed; the scale rides on the rotary rows 0..31)
  auto rotate = [&](const WorkTile& tn, const bf16x8_t (&qn)[KS]) __attribute__((always_inline)) {
    __asm__ volatile("" ::: "memory");
    if (32 * rb >= tn.n_rows) {  // no row of this wave is real
#pragma unroll
      for (int s = 0; s < KS; ++s) qf[s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0u, 0u, 0u, 0u});
      return;
    }
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
    const int lr = ln & 31, lh2 = ln >> 5;
    const float4* br = reinterpret_cast<const float4*>(br_lds);
    const float4* rt = reinterpret_cast<const float4*>(rt_lds + lr * 4 * D);
#pragma unroll
    for (int s = 0; s < KS / 2; ++s) {
      const u32x4_t a4 = __builtin_bit_cast(u32x4_t, qn[s]);
      const u32x4_t b4 = __builtin_bit_cast(u32x4_t, qn[s + KS / 2]);
      u32x4_t na, nb;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        // frequencies 16s + 8h2 + 2e2 and +1: one 16-byte chunk of each rotary row
        const int ch = 8 * s + 4 * lh2 + e2;
        const float4 vb = br[ch];
        const float4 vr = rt[ch ^ (lr & (GE::CH - 1))];
        float ra[2], rb2[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float cb = u ? vb.z : vb.x, sb = u ? vb.w : vb.y;
          const float cr = u ? vr.z : vr.x, sr = u ? vr.w : vr.y;
          const float cs = cb * cr - sb * sr;
          const float sn = sb * cr + cb * sr;
          const float a = u ? hi_bf16(a4[e2]) : lo_bf16(a4[e2]);
          const float b = u ? hi_bf16(b4[e2]) : lo_bf16(b4[e2]);
          ra[u] = a * cs - b * sn;  // cs, sn carry the scale (rotary rows 0..31 do)
          rb2[u] = b * cs + a * sn;
        }
        na[e2] = pack_bf16x2(ra[0], ra[1]);
        nb[e2] = pack_bf16x2(rb2[0], rb2[1]);
      }
      qf[s] = __builtin_bit_cast(bf16x8_t, na);
      qf[s + KS / 2] = __builtin_bit_cast(bf16x8_t, nb);
      // one frequency block at a time: its rotary rows are 8 LDS reads, all of them
      // at once would need 128 registers next to O and both queries
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---------------- output of the previous item, stored at the next item's first
  // barrier so the stores sit behind no DMA wait (st_rows = 0: nothing pending;
  // the call then only clears O).  A lane holds one row and 4 of every 8
  // consecutive dims, so stored straight from registers each instruction would
  // touch 32 rows 16 bytes at a time; instead the rows pass through this wave's
  // LDS staging area and leave as 16-byte pieces of whole 64- or 128-byte row
  // segments.  `stage` must not be read or written by any other wave meanwhile.
  int st_row0 = 0, st_rows = 0, st_head = 0;
  float st_inv = 0.f;
  auto store_out = [&](uint32_t stage) __attribute__((always_inline)) {
    constexpr int SROW = GE::SROW;
    constexpr int CPR = SROW / 16;     // 16-byte chunks per staged row
    constexpr int RPG = 256 / SROW;    // staged rows per 256 bytes (one pass of the banks)
    constexpr int DBP = SROW / 64;     // 32-dim blocks per pass
    constexpr int RPI = 64 / CPR;      // rows per store instruction
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
    const int lr = ln & 31, lh2 = ln >> 5;
    if (st_rows > 0) {
#pragma unroll
      for (int ps = 0; ps < DB / DBP; ++ps) {
        // chunk c of staged row x sits at chunk c ^ ((x / RPG) mod CPR): the 32
        // rows of one 8-byte write then spread over every bank pair twice
#pragma unroll
        for (int dd = 0; dd < DBP; ++dd)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int db = ps * DBP + dd;
            const int c = (4 * dd + g4) ^ ((lr / RPG) & (CPR - 1));
            const u32x2_t w = u32x2_t{pack_bf16x2(o[db][4 * g4] * st_inv, o[db][4 * g4 + 1] * st_inv),
                                      pack_bf16x2(o[db][4 * g4 + 2] * st_inv, o[db][4 * g4 + 3] * st_inv)};
            *reinterpret_cast<u32x2_t*>(lds + stage + lr * SROW + 16 * c + 8 * lh2) = w;
          }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int k = 0; k < 32 / RPI; ++k) {
          const int x = k * RPI + ln / CPR, c = ln % CPR;
          const u32x4_t v = *reinterpret_cast<const u32x4_t*>(lds + stage + x * SROW + 16 * (c ^ ((x / RPG) & (CPR - 1))));
          const int lrow = 32 * rb + x;
          if (lrow < st_rows)
            *reinterpret_cast<u32x4_t*>(out + (static_cast<int64_t>(st_row0 + lrow) * hq + st_head) * D +
                                        32 * DBP * ps + 8 * c) = v;
        }
        __builtin_amdgcn_wave_barrier();
      }
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
    st_rows = 0;
  };
  // ---------------- kernel prologue: rotary rows 0..31, stream tiles 0 and 1, first query
  // raw query rows of the next item: loaded during an item's last block and rotated
  // at the next item's first barrier, after the previous item's rows are stored
  bf16x8_t qn[KS];
  {
    constexpr int RT_PER_WAVE = GE::RTBYTES / 1024 / kNW;
#pragma unroll
    for (int u = 0; u < RT_PER_WAVE; ++u) {  // chunk c of row r stored at chunk c ^ (r mod CH)
      const int qi = wave * RT_PER_WAVE + u;
      const int pos = qi * 64 + lane;
      const int rr = pos / GE::CH, cc = pos % GE::CH;
      const unsigned char* src =
          reinterpret_cast<const unsigned char*>(rope) + rr * 4 * D + 16 * (cc ^ (rr & (GE::CH - 1)));
      dma16(src, rt_lds + qi * 1024);
    }
    fetch_next();
    fetch_next();
    prefetch(ec0, qn);
    grab(ec1);  // item 2
    wait_vm_all();
    block_sync();
    // fold log2(e)/sqrt(d) into the rotary rows of positions 0..31, so that the query
    // rotation, whose angles compose them with a base row, need not multiply by it
    float4* rt4 = reinterpret_cast<float4*>(rt_lds);
    for (int i = threadIdx.x; i < GE::RTBYTES / 16; i += kNT) {
      float4 v = rt4[i];
      v.x *= scale_log2;
      v.y *= scale_log2;
      v.z *= scale_log2;
      v.w *= scale_log2;
      rt4[i] = v;
    }
    block_sync();
  }

  int ck = 0, cv = 0;  // ring slots of the compute tile
  auto kslot = [&](int k) __attribute__((always_inline)) { return static_cast<uint32_t>(k * GE::KBYTES); };
  auto vslot = [&](int v) __attribute__((always_inline)) { return static_cast<uint32_t>(GE::VOFF + v * GE::VBYTES); };
  auto next3 = [](int k) __attribute__((always_inline)) { return k == 2 ? 0 : k + 1; };
  auto next4 = [](int v) __attribute__((always_inline)) { return (v + 1) & 3; };
  // this wave's output staging: at head dim 128 in V slot cv - 1, which holds the
  // tile consumed last; it is refilled only by the fetch after the next barrier
  auto stage_at = [&](int v) __attribute__((always_inline)) {
    return static_cast<uint32_t>((GE::STAGE_IN_V ? GE::VOFF + ((v + 3) & 3) * GE::VBYTES : GE::STOFF) +
                                 wave * 32 * GE::SROW);
  };

  int kpar = 0;  // parity of the compute item: its schedule slot
  while (ec0 < n_total) {
    const WorkTile t = tiles[ec0 / hkv];
    const int head = (ec0 % hkv) * G + hsub;
    const int n = (t.kv_end - t.kv_begin) >> 2;  // at least 1: a row tile sees its own first page
    const bool has_next = ec1 < n_total;
    qpos = t.q_pos0 + row;
    wave_min_pos = t.q_pos0 + 32 * rb;
    m = kNoMax;
    l = 0.f;

    // the barrier before the QK of a stream tile, then the fetch of the tile two ahead
    // (its DMA instructions go out one per chunk of the block after the barrier)
    auto sync_fetch = [&]() __attribute__((always_inline)) {
      wait_group<NDMA>(last_ops);
      block_sync();
      last_ops = fetch_prep();
    };

    // Key blocks u = 0 .. 2n-1 of the item (block u&1 of tile u/2), processed as
    //   QK(u + 1) || softmax(u) || PV(u - 1);
    // the barrier and fetch come before the QK that opens a tile (u + 1 even).
    f32x16_t S[2];
    bf16x8_t P[2][2];
    Pre pre;
    using T_ = std::true_type;
    using F_ = std::false_type;
    // u = 2j: QK(2j + 1) (same tile) || softmax(2j) || PV(2j - 1) (previous tile); reads
    // the V operands of the next block (block 0 of the V tile at vnext)
    auto step_even = [&](auto with_pv, auto prek, uint32_t kslot0, uint32_t vprev,
                         uint32_t vnext) __attribute__((always_inline)) {
      float corr, tsum;
      const bool up = block(T_{}, with_pv, prek, F_{}, T_{}, F_{}, S[0], P[0], kslot0 + 32 * D * 2, S[1],
                            vprev + 2 * D * 32, P[1], pre, 0u, vnext, corr, tsum);
      rescale(up, corr, tsum);
      mask(S[1], 1, mp0, mn0);
    };
    // u = 2j + 1 (not the last): barrier; QK(2j + 2) (next tile) || softmax(2j + 1) || PV(2j);
    // reads the operands of the block after it (block 1 of the same K and V tiles)
    auto step_odd = [&](uint32_t knext, uint32_t vcur) __attribute__((always_inline)) {
      sync_fetch();
      __builtin_amdgcn_sched_barrier(0);
      float corr, tsum;
      const bool up = block(T_{}, T_{}, F_{}, T_{}, T_{}, T_{}, S[1], P[1], knext, S[0], vcur, P[0], pre,
                            knext + 32 * D * 2, vcur + 2 * D * 32, corr, tsum);
      rescale(up, corr, tsum);
      mask(S[0], 0, mp0, mn0);
    };
    // u = 2n - 1: softmax(2n - 1) || PV(2n - 2), then PV(2n - 1)
    auto last_odd = [&](uint32_t vcur) __attribute__((always_inline)) {
      if (has_next) prefetch(ec1, qn);  // the next item's query rows
      float corr, tsum;
      const bool up = block(F_{}, T_{}, F_{}, F_{}, F_{}, F_{}, S[1], P[1], 0u, S[0], vcur, P[0], pre, 0u, 0u, corr, tsum);
      rescale(up, corr, tsum);
      pv(vcur, 1, P[1]);
    };

    // ---- the barrier of tile 0 (its wait also covers the query rows loaded during
    // the previous item's last block and the previous grab): publish item k + 2, grab
    // item k + 3, store the previous item's rows, rotate this item's query, fetch
    wait_vm_all();
    if (threadIdx.x == 0) sched_lds[kpar] = grabbed_item();
    block_sync();
    ec2 = __builtin_amdgcn_readfirstlane(sched_lds[kpar]);
    kpar ^= 1;
    grab(ec2);
    store_out(stage_at(cv));
    rotate(t, qn);
    last_ops = fetch_next();
    qk(kslot(ck), 0, S[0]);
    mask(S[0], 0, mp0, mn0);
    step_even(F_{}, F_{}, kslot(ck), 0u, vslot(cv));
    for (int j = 0; j + 1 < n; ++j) {
      const int ck1 = next3(ck), cv1 = next4(cv);
      step_odd(kslot(ck1), vslot(cv));
      step_even(T_{}, T_{}, kslot(ck1), vslot(cv), vslot(cv1));
      ck = ck1;
      cv = cv1;
    }
    last_odd(vslot(cv));
    ck = next3(ck);
    cv = next4(cv);

    // ---- this item's rows are stored at the next barrier
    const float l_row = swap_sum(l);
    st_row0 = t.q_row0;
    st_rows = t.n_rows;
    st_head = head;
    st_inv = l_row > 0.f ? 1.f / l_row : 0.f;
    ec0 = ec1;  // next item
    ec1 = ec2;
    --dk_k;
  }
  block_sync();  // every wave is done with the last V tile
  store_out(stage_at(cv));
  // The work-group that finishes last leaves the counters at zero for the next
  // launch; the fence orders this work-group's grabs before its count.
  if (threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(sched + kQueueDone, 1u) == gridDim.x - 1) {
      for (int x = 0; x < n_queues; ++x) atomicExch(sched + x, 0u);
      atomicExch(sched + kQueueDone, 0u);
    }
  }
}

template <int D, int G>
static hipError_t launch_t(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q, void* out,
                           const float2* rope, unsigned* sched, const int32_t* chunks_host,
                           const int32_t* chunks_dev, int n_chunks, int cus, int* queues, hipStream_t s) {
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  const size_t lds = PGeo<D>::LDS;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_mfma_kernel<D, G>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (attr != hipSuccess) return attr;
  // one work-group per CU; items are scheduled dynamically
  const int64_t items = static_cast<int64_t>(n) * g.hkv;
  if (items >= (1ll << 30)) return hipErrorInvalidValue;
  const int grid = static_cast<int>(std::min<int64_t>(items, std::max(1, cus)));
  // per-XCD queues only if each holds the two static items of each of its work-groups
  bool xcd = n_chunks > 0 && n_chunks * g.hkv == 8 && grid >= 8 && chunks_host && chunks_dev &&
             chunks_host[0] == 0 && chunks_host[n_chunks] == n;
  for (int x = 0; xcd && x < 8; ++x) {
    const int c = x / g.hkv;
    xcd = chunks_host[c + 1] - chunks_host[c] >= 2 * ((grid - x + 7) / 8);
  }
  if (queues) *queues = xcd ? 8 : 1;
  hipLaunchKernelGGL((prefill_mfma_kernel<D, G>), dim3(grid), dim3(kNT), lds, s, tiles, n, kt,
                     static_cast<const bf16_t*>(q), static_cast<bf16_t*>(out), static_cast<const bf16_t*>(g.base),
                     g.layer_off, g.hq, g.hkv, scale_log2, rope, sched, chunks_dev, xcd ? n_chunks : 0);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q, void* out,
                           const float2* rope, unsigned* sched, const int32_t* ch, const int32_t* cd, int nc, int cus,
                           int* queues, hipStream_t s) {
  switch (g.hq / g.hkv) {
    case 1: return launch_t<D, 1>(g, tiles, n, kt, q, out, rope, sched, ch, cd, nc, cus, queues, s);
    case 2: return launch_t<D, 2>(g, tiles, n, kt, q, out, rope, sched, ch, cd, nc, cus, queues, s);
    case 4: return launch_t<D, 4>(g, tiles, n, kt, q, out, rope, sched, ch, cd, nc, cus, queues, s);
    case 8: return launch_t<D, 8>(g, tiles, n, kt, q, out, rope, sched, ch, cd, nc, cus, queues, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill_mfma(const PoolGeom& g, const WorkTile* tiles, int n, const TileRec* kt, const void* q,
                               void* out, const float2* rope, unsigned* sched, const int32_t* chunks_host,
                               const int32_t* chunks_dev, int n_chunks, int* queues, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (!mfma_supported(g.hq, g.hkv, g.d, g.dtype) || sched == nullptr) return hipErrorInvalidValue;
  int cus = 0;
  const hipError_t e = cu_count(&cus);
  if (e != hipSuccess) return e;
  return g.d == 128 ? launch_d<128>(g, tiles, n, kt, q, out, rope, sched, chunks_host, chunks_dev, n_chunks, cus,
                                    queues, s)
                    : launch_d<64>(g, tiles, n, kt, q, out, rope, sched, chunks_host, chunks_dev, n_chunks, cus,
                                   queues, s);
}

}  // namespace spanq
