// Device pieces shared by the two bf16 MFMA attention kernels (attn_mfma.hip,
// prefill_mfma.hip): operand types, LDS swizzles, the key-tile page record, the
// global-to-LDS DMA of one key tile and the wait/barrier primitives.
//
// A key tile is 4 pages (64 keys) of one kv head.  In LDS its K rows are
// [64 keys][D] and its V rows [4 pages][D][16 positions], both XOR-swizzled at
// 16-byte granularity so that the MFMA operand reads of 16 consecutive lanes hit 16
// distinct bank groups.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dev_common.h"
#include "work.h"

namespace spanq {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

namespace mfma {

constexpr int kBN = 64;  // keys per tile (4 pages)
constexpr int kNW = 8;   // waves per work-group
constexpr int kNT = 64 * kNW;

// Lazily raised running max of the online softmax, in all MFMA kernels: P = 2^(S - m)
// is taken against the current m, and m is raised (P taken again, the accumulated O
// and row sum rescaled) only when a lane's P over a block of keys sums past kSumCap or
// is not finite.  kNoMax, the max before any key, is finite: a masked score gives
// 2^(-inf - m) = 0 and a real one 2^(S - kNoMax) = inf, which forces the first raise.
constexpr float kSumCap = 65536.f;
constexpr float kNoMax = -1e30f;

// Two floats to packed bfloat16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 16-byte chunk swizzle of the K rows: chunk c of row `key` sits at c ^ kswz(key).
template <int D>
__device__ __forceinline__ int kswz(int key) {
  return D == 128 ? (key & 15) : ((key >> 1) & 7);
}

// A tile's four pages come from one span: consecutive positions, and only the
// span's last page may be partial (then followed by empty padding pages).  So key k
// of the tile (0..63) is a real key iff k < nk, at position pos0 + k.
struct TilePages {
  int id[4];
  int pos0;   // position of key 0
  int nk;     // real keys in the tile
  int delta;  // reposition delta of every key of the tile
};

// Tile `ti` of the tiled key lists (scalar loads: `kt` is read-only for the kernel).
__device__ __forceinline__ void read_tile(const TileRec* __restrict__ kt, int ti, TilePages& tp) {
  const TileRec& r = kt[ti];
#pragma unroll
  for (int p = 0; p < 4; ++p) tp.id[p] = r.page_id[p];
  tp.nk = r.nk;
  tp.pos0 = r.pos0;
  tp.delta = r.delta;
}

// a[p] for p in 0..3, as two levels of selects (no branches, no indexed access)
__device__ __forceinline__ int pick4(const int (&a)[4], int p) {
  const int lo = (p & 1) ? a[1] : a[0];
  const int hi = (p & 1) ? a[3] : a[2];
  return (p & 2) ? hi : lo;
}

// One lane's 16 bytes from global memory to LDS at lds_wave + 16 * lane.  Issued as
// inline assembly with the LDS address in M0, so that the compiler's wait-count
// model does not see the LDS write in flight: with it visible, every later LDS
// operand read would wait for all LDS traffic (lgkmcnt(0)), DMA included.  The
// kernels order every read of DMA'd data themselves (vmcnt waits and barriers).
__device__ __forceinline__ uint32_t lds_byte(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}
__device__ __forceinline__ void dma16_m0(const void* g, uint32_t lds_wave) {
  __asm__ volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds_wave) : "memory");
}
__device__ __forceinline__ void dma16(const void* g, void* lds_wave) { dma16_m0(g, lds_byte(lds_wave)); }
// The same from a wave-uniform base (scalar registers) plus a 32-bit per-lane byte
// offset: no 64-bit address arithmetic on the vector ALU.
__device__ __forceinline__ void dma16_s(const void* base, uint32_t ofs, uint32_t lds_wave) {
  __asm__ volatile("global_load_lds_dwordx4 %0, %1" ::"v"(ofs), "s"(base), "{m0}"(lds_wave) : "memory");
}
// Four bytes per lane to LDS at lds_wave + 4 * lane: used only to bring lines into the
// caches ahead of a later load (the LDS bytes are never read).
__device__ __forceinline__ void touch4_m0(const void* g, uint32_t lds_wave) {
  __asm__ volatile("global_load_lds_dword %0, off" ::"v"(g), "{m0}"(lds_wave) : "memory");
}

// s_waitcnt with vmcnt = N (bits 3:0 and 15:14); expcnt and lgkmcnt left at their
// maximum, so only vector-memory operations are waited for.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
__device__ __forceinline__ void wait_vm_all() { wait_vmcnt<0>(); }

__device__ __forceinline__ void block_sync() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}

// The DMA side of an item only needs where its key list starts and its tile count.
struct ItemKeys {
  int kv_begin;
  int n;  // key tiles
};

__device__ __forceinline__ void load_item_keys(const WorkTile* __restrict__ tiles, int ti, ItemKeys& it) {
  const WorkTile* tile = tiles + __builtin_amdgcn_readfirstlane(ti);  // a scalar load
  it.kv_begin = tile->kv_begin;
  it.n = (tile->kv_end - tile->kv_begin) >> 2;
}

}  // namespace mfma
}  // namespace spanq
