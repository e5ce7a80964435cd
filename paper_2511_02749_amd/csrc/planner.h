// Host-side page cache index and span planner (no HIP dependency).
#pragma once
#include <cstdint>
#include <set>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "work.h"

namespace spanq {

uint64_t mix64(uint64_t x);
uint64_t page_hash(uint64_t prev, const int32_t* tok, int32_t n, int32_t page_idx);
uint64_t fragment_seed(uint64_t prefix_last_or_root);

struct PageRec {
  uint64_t hash = 0;
  uint64_t parent = 0;
  int32_t idx = 0;
  int32_t n_tok = 0;
  int64_t last_use = 0;
  int32_t pins = 0;
  bool used = false;
  bool published = false;
  bool cacheable = false;
  int64_t seen_stamp = 0;  // last plan() call that listed this page among its hits
};

struct SpanIn {
  const int32_t* tok;
  int32_t n;
  int64_t row;
};

struct QueryIn {
  SpanIn prefix;
  std::vector<SpanIn> frags;
  SpanIn cross;
};

// Planned span of one query.
struct SpanPlan {
  int kind = 0;  // 0 prefix, 1 fragment, 2 cross
  int query = 0;
  int child = 0;
  int32_t n_tok = 0;
  int64_t row = 0;
  int32_t canon0 = 0;  // canonical position of token 0
  int32_t final0 = 0;  // final position of token 0 in its query
  std::vector<int32_t> pages;
  int32_t n_hit = 0;
  std::vector<int32_t> moved;  // materialised repositioning: copy of each page at
                               // final positions (empty if the span is not shifted)
};

struct Tiling {
  int bm_prefill = 64;   // rows per prefill tile
  int bm_cross = 64;     // rows per cross tile
  int kv_heads = 1;      // work items per tile (one per kv head)
  int target_items = 512;     // work-groups the cross launch aims for (KV splits x tiles x heads)
  int min_split_pages = 16;   // at least 256 keys per KV split
  bool pad4 = false;          // pad span runs to 4-page tiles (MFMA kernel)
  int two_group_rows = 0;     // cross tiles of at most this many rows use kTwoKeyGroups
  int few_rows = 0;           // two-key-group tiles of at most this many rows go last
                              // in the cross list (the 16-row kernel takes them)
  bool materialize = false;   // cross rows read re-rotated copies of shifted pages
                              // (delta 0) instead of rotating at read time
};

// Work-list shape for the attention kernels.  The MFMA kernel is persistent, one
// 8-wave work-group per CU walking (row tile, kv head) items: the cross launch aims
// at one item per CU (splitting the keys further only adds partials to merge).
// The generic kernel (one wave per row tile and query head) is latency-bound and
// wants more work-groups.
// Few-row cross tiles (a short question over a long context) let the MFMA
// kernel's two wave groups work on alternate key tiles; that needs four query
// heads per kv head (two 32-row groups of four waves).
inline Tiling tiling_for(bool mfma, int bm, int hq, int hkv) {
  Tiling t;
  t.bm_prefill = bm;
  t.bm_cross = bm;
  t.kv_heads = mfma ? hkv : hq;
  t.target_items = mfma ? 256 : 1024;
  t.pad4 = mfma;
  t.two_group_rows = (mfma && hq == 4 * hkv) ? 32 : 0;
  t.few_rows = t.two_group_rows > 0 ? 16 : 0;
  return t;
}

class PoolIndex;

struct Plan {
  PoolIndex* pool = nullptr;
  int64_t tick = 0;
  std::vector<SpanPlan> spans;
  std::vector<std::vector<int>> query_spans;  // per query: prefix, fragments..., cross
  std::vector<int32_t> evicted, new_pages, cross_pages, hits;
  std::vector<MovePage> moves;  // materialised repositioning copies, one per distinct
                                // (page, delta != 0) that cross rows read
  bool committed = false;

  // work lists
  std::vector<KvPage> kv;
  std::vector<TileRec> kv_tiles;  // pad4 plans: kv in tiles of four pages
  std::vector<NewPage> k3_prefill, k3_cross;
  std::vector<WorkTile> t_prefill, t_cross;
  std::vector<int32_t> prefill_chunks;  // MFMA prefill: offsets of the 8 / H_kv tile chunks of
                                        // the per-XCD queues (empty: one queue)
  std::vector<CombineTile> combine;
  struct RowRun {
    int64_t row0;
    int32_t n;
  };
  std::vector<RowRun> rows_prefill, rows_cross;  // one run per row tile, in work order
  int32_t n_parts = 0;
  int32_t n_cross_few = 0;  // the last n_cross_few cross tiles: two key groups, <= few_rows rows
  int32_t kv_splits = 1;
  int32_t max_pos = 0;  // every position (and reposition delta) used is below this
  int bm_cross = 64;

  int64_t pages_hit = 0, pages_new = 0, tokens_hit = 0, tokens_new = 0, tokens_cross = 0;
  int64_t prefill_pairs = 0, cross_pairs = 0, cross_kv_pages = 0;

  // Nested generation: the work of the last decode step (tokens appended to each
  // query's cross segment), and totals over all steps.
  struct DecodeStep {
    std::vector<SlotWrite> writes;
    std::vector<KvPage> kv;
    std::vector<TileRec> kv_tiles;
    std::vector<WorkTile> tiles;
    std::vector<CombineTile> combine;
    std::vector<RowRun> rows;
    int32_t n_parts = 0, n_few = 0, kv_splits = 1;
    int64_t tokens = 0, pages_new = 0, pairs = 0;
  } dec;
  int64_t decode_steps = 0, decode_tokens = 0, decode_pages = 0;
};

class PoolIndex {
 public:
  PoolIndex(int64_t num_pages, int32_t page_size, int32_t hash_mode);

  // Returns 0, or -2 (pool full, unchanged), -1 (bad input) with msg set.
  int plan(const std::vector<QueryIn>& qs, bool build_work, const Tiling& tiling, Plan* out,
           std::string* msg);
  // Append n_new[q] decoded tokens (caller rows rows[q] ..) to each query's cross
  // segment: pages for them (transient, like cross pages) and the decode step's
  // work lists in p->dec.  Returns 0, -2 (pool full; plan and pool unchanged) or -1.
  int decode(Plan* p, const std::vector<int32_t>& n_new, const std::vector<int64_t>& rows, const Tiling& tiling,
             std::string* msg);
  void commit(Plan* p);
  void release(Plan* p);  // destroy without commit
  void reset();
  int64_t lookup(uint64_t h) const;  // page id or -1

  int64_t num_pages() const { return num_pages_; }
  int64_t free_count() const { return static_cast<int64_t>(freed_.size()) + (num_pages_ - watermark_); }
  int64_t cached_count() const { return static_cast<int64_t>(index_.size()); }
  int64_t evictable_count() const { return n_evictable_; }
  int64_t pinned_count() const;
  int64_t tick() const { return tick_; }
  int64_t total_evictions() const { return total_evictions_; }
  int32_t page_size() const { return page_size_; }
  int live_plans = 0;

 private:
  struct Spec {
    uint64_t hash, parent;
    int32_t idx, n_tok;
    const int32_t* tok;
    bool cacheable, cross;
  };
  // Working storage of plan(), kept from call to call so that planning a batch does
  // not allocate it again: the page specs, and the batch's own pages by hash (open
  // addressing; a slot is live iff its stamp is the current call's).
  std::vector<Spec> specs_;
  std::vector<uint64_t> pend_key_;
  std::vector<int32_t> pend_val_;
  std::vector<uint32_t> pend_stamp_;
  uint32_t pend_gen_ = 0;
  size_t pend_mask_ = 0;
  void pending_begin(size_t n);
  int32_t pending_find(uint64_t h) const;
  void pending_insert(uint64_t h, int32_t v);  // keeps an existing entry
  // Page-hash chains of spans planned before, by (tokens address, length, seed), each
  // with a copy of its tokens: a span given again (same address, same tokens, checked
  // in full) takes its chain from here instead of hashing its tokens again.  Part of
  // the pool's state: cleared by reset(), and whenever it would hold more than
  // kChainCacheTokens tokens or kChainCacheSpans spans.  Open addressing over flat arenas whose storage is kept
  // when cleared (a slot is live iff its stamp is the current one), so that filling it
  // again after a reset allocates nothing.
  struct ChainSlot {
    const int32_t* tok = nullptr;
    int32_t n = 0;
    uint64_t seed = 0;
    uint32_t stamp = 0;
    size_t tok_off = 0, chain_off = 0, chain_n = 0;
  };
  static constexpr size_t kChainCacheTokens = size_t{1} << 22;
  static constexpr size_t kChainCacheSpans = size_t{1} << 16;
  std::vector<ChainSlot> chain_slots_;
  std::vector<int32_t> chain_tok_;
  std::vector<uint64_t> chain_hash_;
  uint32_t chain_stamp_ = 1;
  size_t chain_live_ = 0;
  void clear_chain_cache();
  size_t chain_slot(const int32_t* tok, int32_t n, uint64_t seed) const;  // its slot or the empty one to use
  const uint64_t* cached_chain(const int32_t* tok, int32_t n, uint64_t seed) const;
  void remember_chain(const int32_t* tok, int32_t n, uint64_t seed, const std::vector<uint64_t>& chain);
  bool content_equal(int32_t pid, const Spec& s) const;
  bool spec_equal(const Spec& a, const Spec& b) const;
  int32_t pop_free();
  void push_free(int32_t pid);
  void evict_one(Plan* p);
  void build_work(Plan* p, const Tiling& tiling);

  int64_t num_pages_;
  int32_t page_size_;
  int32_t hash_mode_;
  std::vector<PageRec> pages_;
  std::vector<int32_t> page_tokens_;
  std::unordered_map<uint64_t, int32_t> index_;
  // Free page ids: every id >= watermark_, plus the ids in freed_ (all < watermark_).
  std::set<int32_t> freed_;
  int64_t watermark_ = 0;
  // Evictable pages (published, unpinned) in LRU order: a binary min-heap of
  // (last_use, -idx, id) entries with lazy deletion.  An entry is current iff its
  // page is still published and unpinned and the page's generation (bumped each
  // time the page becomes evictable) matches; pinning a page just leaves its entry
  // stale.  Victims come out in the same order as from an ordered set.
  struct LruEntry {
    int64_t last_use;
    int32_t neg_idx;
    int32_t pid;
    uint32_t gen;
  };
  std::vector<LruEntry> lru_;
  std::vector<uint32_t> gen_;   // per page; survives the page being freed
  int64_t n_evictable_ = 0;
  void make_evictable(int32_t pid);
  bool lru_current(const LruEntry& e) const;
  int64_t tick_ = 0;
  int64_t stamp_ = 0;  // counts plan() calls, successful or not
  int64_t total_evictions_ = 0;
};

}  // namespace spanq
