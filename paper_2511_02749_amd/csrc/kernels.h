// Launchers of the HIP kernels (kernels.hip, attn_mfma.hip, few_mfma.hip, prefill_mfma.hip,
// probes.hip).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "work.h"

namespace spanq {

struct PoolGeom {
  void* base;          // page memory
  int64_t layer_off;   // element offset of the layer slab
  int32_t hq, hkv, d;
  int32_t dtype;       // SPAN_F32 / SPAN_BF16
};

// K3: rotate keys at their positions and write keys/values of new pages.
hipError_t launch_rope_write(const PoolGeom& g, const NewPage* pages, int n_pages, const void* k,
                             const void* v, const float2* rope, hipStream_t s);

// Nested generation: write decoded tokens' keys (rotated at their positions) and
// values into slots of their cross pages, leaving the pages' other slots as they are.
hipError_t launch_append_kv(const PoolGeom& g, const SlotWrite* writes, int n_writes, const void* k, const void* v,
                            const float2* rope, hipStream_t s);

// Materialised repositioning: copy each move's source page to its destination
// page with the keys rotated by the move's delta (values copied unchanged).
hipError_t launch_move_pages(const PoolGeom& g, const MovePage* moves, int n_moves, const float2* rope,
                             hipStream_t s);

// Generic (vector ALU) span attention over work tiles of up to 64 rows.
constexpr int kGenericBM = 64;
hipError_t launch_attn_generic(const PoolGeom& g, const WorkTile* tiles, int n_tiles, const KvPage* kv,
                               const void* q, void* out, void* part_o, float* part_ml,
                               const float2* rope, hipStream_t s);

// bf16 MFMA attention kernels: eight waves per work-group, work items (row tile,
// kv head); a row tile has mfma_bm(g) = 256 / g query tokens (g = query heads per
// kv head).  Key lists come in whole 4-page tiles with one delta per tile, given as
// tile records: a work tile's keys are kt[kv_begin / 4 .. kv_end / 4).
bool mfma_supported(int hq, int hkv, int d, int dtype);
int mfma_bm(int g);
// Compute units of the current device (the persistent kernels run one work-group
// on each).
hipError_t cu_count(int* n);

// Cross attention: the query is rotated by each tile's delta; tiles with
// part >= 0 write partials (fp16 O / l and fp32 (m, l)) for the combine pass.
// With w.pages given, the kernel also writes the cross-segment pages that each tile
// names (WorkTile::w_first, flags >> kWriteShift) from the caller's k, v rows, as
// launch_rope_write would, before reading them: the separate page-write launch and
// its gap disappear from the cross pass.
struct CrossWrites {
  const NewPage* pages = nullptr;
  const void* k = nullptr;
  const void* v = nullptr;
};
hipError_t launch_attn_mfma(const PoolGeom& g, const WorkTile* tiles, int n_tiles, const TileRec* kt,
                            const void* q, void* out, void* part_o, float* part_ml,
                            const float2* rope, const CrossWrites& w, hipStream_t s);

// Cross attention for two-key-group tiles of at most 16 rows (four query heads per
// kv head, bf16, d 64 or 128) on 16x16x32 MFMAs; writes partial slots part and
// part + 1 of each tile, like the two-key-group mode of launch_attn_mfma.
bool few_supported(int hq, int hkv, int d, int dtype);
hipError_t launch_few_mfma(const PoolGeom& g, const WorkTile* tiles, int n_tiles, const TileRec* kt, const void* q,
                           void* part_o, float* part_ml, const float2* rope, hipStream_t s);

// Span prefill (no repositioning, no key splits), the software-pipelined kernel.
// Every tile must have at least one key tile.  `sched` is kSchedWords zeroed device
// words, the launch's queue counters (words 0..7) and finish count (word
// kQueueDone); the kernel leaves them at zero when it ends, so launches that run
// one after another may share them and overlapping ones may not.  chunks_host /
// chunks_dev: the n_chunks + 1 offsets of the per-XCD tile chunks (n_chunks = 8 /
// kv heads), or n_chunks = 0 for one queue; the launch falls back to one queue when
// a chunk is too short for the grid.  *queues (if given) receives the queue count
// the launch used (8 or 1).
constexpr int kQueueDone = 8;
constexpr int kSchedWords = 16;
hipError_t launch_prefill_mfma(const PoolGeom& g, const WorkTile* tiles, int n_tiles, const TileRec* kt,
                               const void* q, void* out, const float2* rope, unsigned* sched,
                               const int32_t* chunks_host, const int32_t* chunks_dev, int n_chunks, int* queues,
                               hipStream_t s);

// Split-KV partial buffers: n_parts x H_q x bm slots of D elements (O / l in fp16
// for bf16 pools, the unnormalised O in fp32 for fp32 pools), then the slots' (m, l)
// as fp32 pairs.  Bytes of one O element:
constexpr int part_elem_bytes(bool bf16_pool) { return bf16_pool ? 2 : 4; }

// K4: merge KV-split partials (bm = rows per tile of the producing kernel).
hipError_t launch_combine(const PoolGeom& g, const CombineTile* tiles, int n_tiles, const void* part_o,
                          const float* part_ml, int bm, int max_parts, void* out, hipStream_t s);

// Machine-peak probes (probes.hip): an MFMA-only loop on every compute unit (two
// waves per SIMD, probe_mfma_flops(iters, n_cu) flops per launch) and a streaming
// read of `bytes` (a multiple of 16) at buf.
hipError_t launch_probe_mfma(int iters, int n_cu, hipStream_t s);
double probe_mfma_flops(int iters, int n_cu);
hipError_t launch_probe_read(const void* buf, int64_t bytes, int n_cu, hipStream_t s);

}  // namespace spanq
