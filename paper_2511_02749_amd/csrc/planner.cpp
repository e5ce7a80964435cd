// Page cache index and span planner.
//
// Hashing follows sections 2 and 5.4 of the paper: pages are hashed in chains
// (each page folds in the previous page's hash), a lookup stops at a chain's
// first miss, and at each commuting child the chain restarts from a seed that
// depends on the shared prefix only.  Allocation, deduplication and eviction
// rules are this library's (the paper leaves them to vLLM's block pool):
// lowest free page id; a span already scheduled in the same plan is a hit;
// LRU victim by (last use, -index in span, page id), so tail pages go first.
#include "planner.h"

#include <algorithm>
#include <cstring>
#include <limits>

#include "../../include/spanq.h"

namespace spanq {

uint64_t mix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// A page hash as the index stores it.  Test builds of the host code may define
// SPANQ_TEST_HASH_BITS to keep only that many low bits, so that unrelated pages
// collide often and the content check behind every index hit is exercised; the
// library is never built so.
static inline uint64_t stored_hash(uint64_t h) {
#ifdef SPANQ_TEST_HASH_BITS
  return h & ((1ull << SPANQ_TEST_HASH_BITS) - 1);
#else
  return h;
#endif
}

uint64_t page_hash(uint64_t prev, const int32_t* tok, int32_t n, int32_t page_idx) {
  uint64_t h = prev;
  for (int32_t i = 0; i < n; ++i) h = mix64(h ^ static_cast<uint64_t>(static_cast<uint32_t>(tok[i])));
  return stored_hash(mix64(h ^ (static_cast<uint64_t>(static_cast<uint32_t>(n)) << 32) ^
                           static_cast<uint64_t>(static_cast<uint32_t>(page_idx))));
}

uint64_t fragment_seed(uint64_t prefix_last_or_root) { return mix64(prefix_last_or_root ^ SPAN_HASH_FRAG_TAG); }

namespace {
// The page-hash chains of up to kLanes spans, advanced in lockstep: the chains are
// independent, so their multiply latencies overlap (one chain leaves the multiplier
// idle most of the time; eight keep it busy).  out[c] is exactly the chain page_hash
// gives for span c from seeds[c].
constexpr int kLanes = 8;
// Lanes beyond k hash lane 0's tokens and their results are dropped, so that the
// pages every span has in full take one loop without per-lane conditions.
void chains(const uint64_t* seeds, const SpanIn* const* spans, int k, int32_t ps, std::vector<uint64_t>* const* out) {
  uint64_t h[kLanes];
  int32_t n[kLanes];
  const int32_t* t[kLanes];
  int32_t nmax = 0, nmin = spans[0]->n;
  for (int c = 0; c < kLanes; ++c) {
    h[c] = c < k ? seeds[c] : 0;
    n[c] = c < k ? spans[c]->n : 0;
    t[c] = c < k ? spans[c]->tok : spans[0]->tok;
    nmax = std::max(nmax, n[c]);
    if (c < k) {
      nmin = std::min(nmin, n[c]);
      out[c]->clear();
      out[c]->reserve(static_cast<size_t>((n[c] + ps - 1) / ps));
    }
  }
  int32_t p = 0;
  for (; (p + 1) * ps <= nmin; ++p) {
    const int32_t base = p * ps;
    for (int32_t i = 0; i < ps; ++i)
      for (int c = 0; c < kLanes; ++c) h[c] = mix64(h[c] ^ static_cast<uint64_t>(static_cast<uint32_t>(t[c][base + i])));
    for (int c = 0; c < kLanes; ++c) {
      h[c] = stored_hash(mix64(h[c] ^ (static_cast<uint64_t>(static_cast<uint32_t>(ps)) << 32) ^
                               static_cast<uint64_t>(static_cast<uint32_t>(p))));
      if (c < k) out[c]->push_back(h[c]);
    }
  }
  for (; p * ps < nmax; ++p) {
    const int32_t base = p * ps;
    for (int32_t i = 0; i < ps; ++i)
      for (int c = 0; c < kLanes; ++c)
        if (base + i < n[c]) h[c] = mix64(h[c] ^ static_cast<uint64_t>(static_cast<uint32_t>(t[c][base + i])));
    for (int c = 0; c < kLanes; ++c)
      if (base < n[c]) {
        const int32_t m = std::min(ps, n[c] - base);
        h[c] = stored_hash(mix64(h[c] ^ (static_cast<uint64_t>(static_cast<uint32_t>(m)) << 32) ^
                                 static_cast<uint64_t>(static_cast<uint32_t>(p))));
        out[c]->push_back(h[c]);
      }
  }
}
}  // namespace

PoolIndex::PoolIndex(int64_t num_pages, int32_t page_size, int32_t hash_mode)
    : num_pages_(num_pages), page_size_(page_size), hash_mode_(hash_mode) {
  pages_.resize(static_cast<size_t>(num_pages));
  gen_.assign(static_cast<size_t>(num_pages), 0u);
  page_tokens_.resize(static_cast<size_t>(num_pages) * page_size);
  index_.reserve(static_cast<size_t>(std::min<int64_t>(num_pages, 1 << 20)));
  reset();
}

void PoolIndex::clear_chain_cache() {
  chain_tok_.clear();
  chain_hash_.clear();
  chain_live_ = 0;
  if (++chain_stamp_ == 0) {  // stamps wrapped: clear them all
    for (ChainSlot& c : chain_slots_) c.stamp = 0;
    chain_stamp_ = 1;
  }
}

size_t PoolIndex::chain_slot(const int32_t* tok, int32_t n, uint64_t seed) const {
  const size_t mask = chain_slots_.size() - 1;
  size_t i = static_cast<size_t>(mix64(reinterpret_cast<uintptr_t>(tok) ^ mix64(seed ^ static_cast<uint32_t>(n)))) & mask;
  for (;; i = (i + 1) & mask) {
    const ChainSlot& c = chain_slots_[i];
    if (c.stamp != chain_stamp_ || (c.tok == tok && c.n == n && c.seed == seed)) return i;
  }
}

const uint64_t* PoolIndex::cached_chain(const int32_t* tok, int32_t n, uint64_t seed) const {
  if (chain_live_ == 0) return nullptr;
  const ChainSlot& c = chain_slots_[chain_slot(tok, n, seed)];
  if (c.stamp != chain_stamp_ ||
      (n > 0 && std::memcmp(chain_tok_.data() + c.tok_off, tok, sizeof(int32_t) * static_cast<size_t>(n)) != 0))
    return nullptr;
  return chain_hash_.data() + c.chain_off;
}

void PoolIndex::remember_chain(const int32_t* tok, int32_t n, uint64_t seed, const std::vector<uint64_t>& chain) {
  if (static_cast<size_t>(n) > kChainCacheTokens) return;
  if (chain_tok_.size() + static_cast<size_t>(n) > kChainCacheTokens || chain_live_ >= kChainCacheSpans)
    clear_chain_cache();
  if (2 * (chain_live_ + 1) > chain_slots_.size()) {  // keep the table at most half full
    std::vector<ChainSlot> old;
    old.swap(chain_slots_);
    chain_slots_.assign(std::max<size_t>(64, 2 * old.size()), ChainSlot{});
    const uint32_t st = chain_stamp_;
    chain_stamp_ = 1;
    for (ChainSlot& c : chain_slots_) c.stamp = 0;
    for (const ChainSlot& c : old)
      if (c.stamp == st) {
        ChainSlot d = c;
        d.stamp = chain_stamp_;
        chain_slots_[chain_slot(c.tok, c.n, c.seed)] = d;
      }
  }
  ChainSlot& c = chain_slots_[chain_slot(tok, n, seed)];
  if (c.stamp != chain_stamp_) ++chain_live_;
  c.tok = tok;
  c.n = n;
  c.seed = seed;
  c.stamp = chain_stamp_;
  c.tok_off = chain_tok_.size();
  c.chain_off = chain_hash_.size();
  c.chain_n = chain.size();
  chain_tok_.insert(chain_tok_.end(), tok, tok + n);
  chain_hash_.insert(chain_hash_.end(), chain.begin(), chain.end());
}

void PoolIndex::reset() {
  clear_chain_cache();
  // Records of ids >= watermark_ are rewritten when they are allocated again.
  for (int64_t i = 0; i < watermark_; ++i) pages_[i] = PageRec{};
  index_.clear();
  lru_.clear();
  n_evictable_ = 0;
  freed_.clear();
  watermark_ = 0;
}

int64_t PoolIndex::pinned_count() const {
  int64_t n = 0;
  for (int64_t i = 0; i < watermark_; ++i) n += (pages_[i].used && pages_[i].pins > 0) ? 1 : 0;
  return n;
}

int64_t PoolIndex::lookup(uint64_t h) const {
  auto it = index_.find(h);
  return it == index_.end() ? -1 : it->second;
}

bool PoolIndex::content_equal(int32_t pid, const Spec& s) const {
  const PageRec& p = pages_[pid];
  if (p.idx != s.idx || p.n_tok != s.n_tok || p.parent != s.parent) return false;
  return std::memcmp(&page_tokens_[static_cast<size_t>(pid) * page_size_], s.tok,
                     sizeof(int32_t) * s.n_tok) == 0;
}

void PoolIndex::pending_begin(size_t n) {
  size_t cap = 64;
  while (cap < 2 * n) cap *= 2;
  if (cap > pend_key_.size()) {
    pend_key_.assign(cap, 0);
    pend_val_.assign(cap, 0);
    pend_stamp_.assign(cap, 0);
    pend_gen_ = 0;
  }
  pend_mask_ = pend_key_.size() - 1;
  if (++pend_gen_ == 0) {  // stamps wrapped: clear them all
    std::fill(pend_stamp_.begin(), pend_stamp_.end(), 0u);
    pend_gen_ = 1;
  }
}

int32_t PoolIndex::pending_find(uint64_t h) const {
  for (size_t i = static_cast<size_t>(h ^ (h >> 29)) & pend_mask_;; i = (i + 1) & pend_mask_) {
    if (pend_stamp_[i] != pend_gen_) return -1;
    if (pend_key_[i] == h) return pend_val_[i];
  }
}

void PoolIndex::pending_insert(uint64_t h, int32_t v) {
  for (size_t i = static_cast<size_t>(h ^ (h >> 29)) & pend_mask_;; i = (i + 1) & pend_mask_) {
    if (pend_stamp_[i] != pend_gen_) {
      pend_stamp_[i] = pend_gen_;
      pend_key_[i] = h;
      pend_val_[i] = v;
      return;
    }
    if (pend_key_[i] == h) return;
  }
}

bool PoolIndex::spec_equal(const Spec& a, const Spec& b) const {
  return a.idx == b.idx && a.n_tok == b.n_tok && a.parent == b.parent &&
         (a.tok == b.tok || std::memcmp(a.tok, b.tok, sizeof(int32_t) * a.n_tok) == 0);
}

int32_t PoolIndex::pop_free() {
  if (!freed_.empty()) {
    auto it = freed_.begin();
    int32_t pid = *it;
    freed_.erase(it);
    return pid;
  }
  return static_cast<int32_t>(watermark_++);
}

void PoolIndex::push_free(int32_t pid) {
  pages_[pid] = PageRec{};
  if (pid + 1 == watermark_) {
    --watermark_;
    while (!freed_.empty() && *freed_.rbegin() + 1 == watermark_) {
      freed_.erase(std::prev(freed_.end()));
      --watermark_;
    }
  } else {
    freed_.insert(pid);
  }
}

namespace {
// min-heap order of LRU entries: (last_use, -idx, id) ascending
template <typename E>
bool lru_after(const E& a, const E& b) {
  if (a.last_use != b.last_use) return a.last_use > b.last_use;
  if (a.neg_idx != b.neg_idx) return a.neg_idx > b.neg_idx;
  return a.pid > b.pid;
}
}  // namespace

bool PoolIndex::lru_current(const LruEntry& e) const {
  const PageRec& r = pages_[e.pid];
  return r.published && r.pins == 0 && gen_[e.pid] == e.gen;
}

void PoolIndex::make_evictable(int32_t pid) {
  const PageRec& r = pages_[pid];
  const uint32_t g = ++gen_[pid];
  lru_.push_back(LruEntry{r.last_use, -r.idx, pid, g});
  std::push_heap(lru_.begin(), lru_.end(), lru_after<LruEntry>);
  ++n_evictable_;
  // drop stale entries once they outnumber the live ones
  if (lru_.size() > 2 * static_cast<size_t>(n_evictable_) + 1024) {
    std::vector<LruEntry> keep;
    keep.reserve(static_cast<size_t>(n_evictable_));
    for (const LruEntry& e : lru_)
      if (lru_current(e)) keep.push_back(e);
    std::make_heap(keep.begin(), keep.end(), lru_after<LruEntry>);
    lru_.swap(keep);
  }
}

void PoolIndex::evict_one(Plan* p) {
  while (!lru_current(lru_.front())) {
    std::pop_heap(lru_.begin(), lru_.end(), lru_after<LruEntry>);
    lru_.pop_back();
  }
  const int32_t pid = lru_.front().pid;
  std::pop_heap(lru_.begin(), lru_.end(), lru_after<LruEntry>);
  lru_.pop_back();
  --n_evictable_;
  index_.erase(pages_[pid].hash);
  p->evicted.push_back(pid);
  ++total_evictions_;
  push_free(pid);
}

namespace {
struct Entry {
  bool hit;     // page served by a published page
  bool dup;     // page scheduled earlier in this plan
  int32_t x;    // page id (hit) or slot (new)
};
}  // namespace

int PoolIndex::plan(const std::vector<QueryIn>& qs, bool build, const Tiling& tiling, Plan* out,
                    std::string* msg) {
  const int32_t ps = page_size_;
  std::vector<Spec>& specs = specs_;
  specs.clear();
  {
    size_t pages_in = 0;
    for (const QueryIn& q : qs) {
      pages_in += (q.prefix.n + ps - 1) / ps + (q.cross.n + ps - 1) / ps;
      for (const SpanIn& f : q.frags) pages_in += (f.n + ps - 1) / ps;
    }
    specs.reserve(pages_in);
    pending_begin(pages_in);  // at most half full: every probe ends
  }
  struct SpanWalk {
    int kind, query, child;
    SpanIn in;
    std::vector<Entry> entries;
  };
  std::vector<SpanWalk> walk;
  std::vector<std::vector<int>> query_spans(qs.size());
  // A span given twice in one call (same tokens pointer, length and chain seed) has
  // the same page chain: hash it once.
  struct MemoKey {
    const int32_t* tok;
    int32_t n;
    uint64_t seed;
    bool operator==(const MemoKey& o) const { return tok == o.tok && n == o.n && seed == o.seed; }
  };
  struct MemoHash {
    size_t operator()(const MemoKey& k) const {
      return static_cast<size_t>(mix64(reinterpret_cast<uintptr_t>(k.tok) ^ mix64(k.seed ^ static_cast<uint32_t>(k.n))));
    }
  };
  std::unordered_map<MemoKey, std::vector<uint64_t>, MemoHash> memo;
  auto chain_of = [&](uint64_t seed, const SpanIn& in) -> const std::vector<uint64_t>& {
    auto it = memo.find(MemoKey{in.tok, in.n, seed});
    if (it != memo.end()) return it->second;
    if (const uint64_t* c = cached_chain(in.tok, in.n, seed))
      return memo.emplace(MemoKey{in.tok, in.n, seed}, std::vector<uint64_t>(c, c + (in.n + ps - 1) / ps))
          .first->second;
    std::vector<uint64_t> hs;
    uint64_t h = seed;
    for (int32_t p = 0; p * ps < in.n; ++p) {
      const int32_t n = std::min(ps, in.n - p * ps);
      h = page_hash(h, in.tok + p * ps, n, p);
      hs.push_back(h);
    }
    remember_chain(in.tok, in.n, seed, hs);
    return memo.emplace(MemoKey{in.tok, in.n, seed}, std::move(hs)).first->second;
  };

  // Every fragment chain of the batch first, kLanes at a time: a fragment's chain
  // starts from a seed its query's prefix chain gives.
  std::vector<uint64_t> frag_seed(qs.size(), SPAN_HASH_ROOT);
  if (hash_mode_ != SPAN_HASH_STOCK) {
    struct Todo {
      const SpanIn* in;
      uint64_t seed;
      std::vector<uint64_t>* out;
    };
    std::vector<Todo> todo;
    for (size_t qi = 0; qi < qs.size(); ++qi) {
      const std::vector<uint64_t>& ph = chain_of(SPAN_HASH_ROOT, qs[qi].prefix);
      const uint64_t fs = fragment_seed(ph.empty() ? SPAN_HASH_ROOT : ph.back());
      frag_seed[qi] = fs;
      for (const SpanIn& f : qs[qi].frags) {
        auto ins = memo.try_emplace(MemoKey{f.tok, f.n, fs});
        if (!ins.second) continue;
        if (const uint64_t* c = cached_chain(f.tok, f.n, fs))
          ins.first->second.assign(c, c + (f.n + ps - 1) / ps);
        else
          todo.push_back({&f, fs, &ins.first->second});  // node values stay put
      }
    }
    for (size_t i = 0; i < todo.size(); i += kLanes) {
      const int k = static_cast<int>(std::min<size_t>(kLanes, todo.size() - i));
      uint64_t seeds[kLanes];
      const SpanIn* in[kLanes];
      std::vector<uint64_t>* out[kLanes];
      for (int c = 0; c < k; ++c) {
        seeds[c] = todo[i + c].seed;
        in[c] = todo[i + c].in;
        out[c] = todo[i + c].out;
      }
      chains(seeds, in, k, ps, out);
      for (int c = 0; c < k; ++c) remember_chain(in[c]->tok, in[c]->n, seeds[c], *out[c]);
    }
  }
  for (size_t qi = 0; qi < qs.size(); ++qi) {
    const QueryIn& q = qs[qi];
    struct Src { uint64_t seed; SpanIn in; int kind, child; bool partial_ok; };
    std::vector<Src> srcs;
    if (hash_mode_ == SPAN_HASH_STOCK) {
      srcs.push_back({SPAN_HASH_ROOT, q.prefix, 0, 0, false});
    } else {
      srcs.push_back({SPAN_HASH_ROOT, q.prefix, 0, 0, true});
      for (size_t c = 0; c < q.frags.size(); ++c)
        srcs.push_back({frag_seed[qi], q.frags[c], 1, static_cast<int>(c), true});
    }
    for (const Src& s : srcs) {
      SpanWalk w{s.kind, static_cast<int>(qi), s.child, s.in, {}};
      const std::vector<uint64_t>& hs = chain_of(s.seed, s.in);
      w.entries.reserve(hs.size());
      bool missed = false;
      for (int32_t p = 0; p * ps < s.in.n; ++p) {
        int32_t n = std::min(ps, s.in.n - p * ps);
        Spec sp{hs[p], p == 0 ? s.seed : hs[p - 1], p, n, s.in.tok + p * ps, n == ps || s.partial_ok, false};
        if (!missed && sp.cacheable) {
          const int32_t pj = pending_find(sp.hash);
          if (pj >= 0 && spec_equal(specs[pj], sp)) {
            w.entries.push_back({false, true, pj});
            continue;
          }
          auto jt = index_.find(sp.hash);
          if (jt != index_.end() && content_equal(jt->second, sp)) {
            w.entries.push_back({true, false, jt->second});
            continue;
          }
        }
        missed = true;
        int32_t slot = static_cast<int32_t>(specs.size());
        specs.push_back(sp);
        if (sp.cacheable) pending_insert(sp.hash, slot);
        w.entries.push_back({false, false, slot});
      }
      query_spans[qi].push_back(static_cast<int>(walk.size()));
      walk.push_back(std::move(w));
    }
    // cross segment: transient pages, never looked up
    SpanWalk w{2, static_cast<int>(qi), 0, q.cross, {}};
    if (hash_mode_ != SPAN_HASH_STOCK) {
      for (int32_t p = 0; p * ps < q.cross.n; ++p) {
        int32_t n = std::min(ps, q.cross.n - p * ps);
        int32_t slot = static_cast<int32_t>(specs.size());
        specs.push_back(Spec{0, 0, p, n, q.cross.tok + p * ps, false, true});
        w.entries.push_back({false, false, slot});
      }
    }
    query_spans[qi].push_back(static_cast<int>(walk.size()));
    walk.push_back(std::move(w));
  }

  // Materialised repositioning (the alternative to rotating at read time: section
  // 5.5 re-rotates cached blocks into place, CIDRA in place): every page
  // of a fragment that a query's cross rows read at a shifted position gets a
  // transient copy whose keys sit at the final positions.  A page read at the same
  // shift by several queries of the batch is copied once; a page read at two
  // shifts is copied twice (the duplication of a block with two targets).  Source
  // pages are never rewritten, so the moves have no dependencies among them.
  // Page identity: a hit's page id, or -1 - slot for a page this plan computes
  // (a batch duplicate names the slot of its first occurrence).
  struct MoveSrc {
    int64_t page;
    int32_t delta, n_valid;
  };
  std::vector<MoveSrc> moves;
  std::vector<std::vector<int32_t>> move_of(walk.size());
  if (tiling.materialize && hash_mode_ != SPAN_HASH_STOCK) {
    std::unordered_map<uint64_t, int32_t> seen;
    for (size_t qi = 0; qi < qs.size(); ++qi) {
      if (qs[qi].cross.n == 0) continue;
      const auto& ids = query_spans[qi];
      int32_t shift = 0;  // final minus canonical position of the fragment's tokens
      for (size_t c = 1; c + 1 < ids.size(); ++c) {
        const SpanWalk& w = walk[ids[c]];
        if (shift != 0) {
          auto& mv = move_of[ids[c]];
          for (size_t pg = 0; pg < w.entries.size(); ++pg) {
            const Entry& e = w.entries[pg];
            const int64_t page = e.hit ? e.x : -1 - static_cast<int64_t>(e.x);
            const uint64_t key = (static_cast<uint64_t>(page) << 32) ^ static_cast<uint32_t>(shift);
            auto it = seen.find(key);
            if (it == seen.end()) {
              it = seen.emplace(key, static_cast<int32_t>(moves.size())).first;
              moves.push_back({page, shift, std::min(ps, w.in.n - static_cast<int32_t>(pg) * ps)});
            }
            mv.push_back(it->second);
          }
        }
        shift += w.in.n;
      }
    }
  }

  // distinct published pages this plan hits, in walk order
  std::vector<int32_t> hit_pids;
  const int64_t stamp = ++stamp_;
  for (const auto& w : walk)
    for (const auto& e : w.entries)
      if (e.hit && pages_[e.x].seen_stamp != stamp) {
        pages_[e.x].seen_stamp = stamp;
        hit_pids.push_back(e.x);
      }
  int64_t need = static_cast<int64_t>(specs.size() + moves.size());
  int64_t evictable = n_evictable_;
  for (int32_t pid : hit_pids)
    if (pages_[pid].published && pages_[pid].pins == 0) --evictable;
  if (need > free_count() + evictable) {
    *msg = "pool exhausted: plan needs " + std::to_string(need) + " pages, " +
           std::to_string(free_count()) + " free, " + std::to_string(evictable) + " evictable";
    return SPAN_ENOMEM;
  }

  // ---- mutate
  Plan& P = *out;
  P.pool = this;
  P.tick = ++tick_;
  for (int32_t pid : hit_pids) {
    PageRec& r = pages_[pid];
    if (r.published && r.pins == 0) --n_evictable_;  // its heap entry goes stale
    r.pins += 1;
    r.last_use = P.tick;
  }
  P.hits = hit_pids;
  std::vector<int32_t> slot_pid(specs.size(), -1);
  P.new_pages.reserve(static_cast<size_t>(need));
  auto alloc = [&](int32_t slot) {
    if (free_count() == 0) evict_one(&P);
    int32_t pid = pop_free();
    const Spec& s = specs[slot];
    PageRec& r = pages_[pid];
    r = PageRec{};
    r.hash = s.hash;
    r.parent = s.parent;
    r.idx = s.idx;
    r.n_tok = s.n_tok;
    r.last_use = P.tick;
    r.pins = 1;
    r.used = true;
    r.published = false;
    r.cacheable = s.cacheable && !s.cross;
    std::memcpy(&page_tokens_[static_cast<size_t>(pid) * ps], s.tok, sizeof(int32_t) * s.n_tok);
    slot_pid[slot] = pid;
    P.new_pages.push_back(pid);
    if (s.cross) P.cross_pages.push_back(pid);
  };
  for (size_t qi = 0; qi < qs.size(); ++qi)
    for (int wi : query_spans[qi])
      for (const Entry& e : walk[wi].entries)
        if (!e.hit && !e.dup) alloc(e.x);
  // repositioned copies last: transient like cross pages, never published
  for (const MoveSrc& m : moves) {
    if (free_count() == 0) evict_one(&P);
    const int32_t pid = pop_free();
    PageRec& r = pages_[pid];
    r = PageRec{};
    r.last_use = P.tick;
    r.pins = 1;
    r.used = true;
    P.new_pages.push_back(pid);
    const int32_t src = m.page >= 0 ? static_cast<int32_t>(m.page) : slot_pid[-1 - m.page];
    P.moves.push_back(MovePage{src, pid, m.delta, m.n_valid});
  }

  P.query_spans = query_spans;
  P.spans.resize(walk.size());
  for (size_t wi = 0; wi < walk.size(); ++wi) {
    const SpanWalk& w = walk[wi];
    SpanPlan& sp = P.spans[wi];
    sp.kind = w.kind;
    sp.query = w.query;
    sp.child = w.child;
    sp.n_tok = w.in.n;
    sp.row = w.in.row;
    sp.n_hit = 0;
    for (int32_t m : move_of[wi]) sp.moved.push_back(P.moves[m].dst_page);
    sp.pages.reserve(w.entries.size());
    bool leading = true;
    for (const Entry& e : w.entries) {
      sp.pages.push_back(e.hit ? e.x : slot_pid[e.x]);
      if (leading && (e.hit || e.dup)) {
        ++sp.n_hit;
      } else {
        leading = false;
      }
    }
    if (w.kind != 2) {
      int64_t np = static_cast<int64_t>(sp.pages.size());
      P.pages_hit += sp.n_hit;
      int64_t new_here = 0;
      for (size_t i = sp.n_hit; i < w.entries.size(); ++i) new_here += (!w.entries[i].dup) ? 1 : 0;
      P.pages_new += new_here;
      int64_t hit_tok = std::min<int64_t>(w.in.n, static_cast<int64_t>(sp.n_hit) * ps);
      P.tokens_hit += hit_tok;
      P.tokens_new += (np > sp.n_hit) ? (w.in.n - hit_tok) : 0;
    } else {
      P.tokens_cross += w.in.n;
    }
  }
  if (build) build_work(&P, tiling);
  ++live_plans;
  return SPAN_OK;
}

namespace {
// Append the pages of one span to a key list.  Page pg holds tokens 16pg.. at
// positions pos_base + 16pg.. in the reader's frame; `delta` is the rotation the
// reader still has to apply.  With pad4 the span's run is padded to a multiple of
// four pages with empty (n_valid = 0, fully masked) copies of its last page, so a
// 4-page tile never mixes spans (one delta per tile).
void append_span(std::vector<KvPage>& kv, const std::vector<int32_t>& pages, int32_t n_tok, int32_t ps,
                 int32_t pos_base, int32_t delta, bool pad4) {
  const int32_t np = static_cast<int32_t>(pages.size());
  const int32_t padded = (pad4 && np > 0) ? (np + 3) / 4 * 4 : np;
  const size_t at = kv.size();
  kv.resize(at + padded);
  KvPage* out = kv.data() + at;
  for (int32_t pg = 0; pg < np; ++pg)
    out[pg] = KvPage{pages[pg], std::min(ps, n_tok - pg * ps), pos_base + pg * ps, delta};
  for (int32_t pg = np; pg < padded; ++pg) out[pg] = KvPage{pages[np - 1], 0, pos_base + (np - 1) * ps, delta};
}

// One past the last page of kv[kv0, kv1) whose first position is <= last_pos
// (positions are non-decreasing along a list); rounded up to whole 4-page tiles
// with pad4 (the extra pages are masked by position or are empty).
int32_t list_end(const std::vector<KvPage>& kv, int32_t kv0, int32_t kv1, int32_t last_pos, bool pad4) {
  const int32_t end = static_cast<int32_t>(
      std::upper_bound(kv.begin() + kv0, kv.begin() + kv1, last_pos,
                       [](int32_t pos, const KvPage& k) { return pos < k.pos0; }) - kv.begin());
  return pad4 ? std::min(kv1, kv0 + ((end - kv0 + 3) / 4) * 4) : end;
}

// Order of the prefill row tiles.
// Generic kernel: longest key lists first, so the launch ends on short tiles.
// MFMA kernel with 1, 2, 4 or 8 kv heads: queues for the chip's eight L2 domains
// (XCDs).  The tiles are cut into R = 8 / kv_heads chunks; queue x serves chunk
// x / kv_heads for kv head x mod kv_heads, so the work-groups of one XCD read the
// K/V of one kv head of one group of spans and find the pages the span's other row
// tiles fetched in their L2.  In a chunk the long tiles come span by span (a span's
// tiles together, longest first), then its share of the shortest tiles (an eighth
// of the work), longest first, so that a queue ends on short items.  chunks receives
// the R + 1 chunk offsets (empty for the generic order).
void order_prefill(std::vector<WorkTile>& tiles, const std::vector<int32_t>& span_of, const Tiling& t,
                   std::vector<int32_t>* chunks) {
  chunks->clear();
  auto work = [](const WorkTile& w) { return static_cast<int64_t>(w.kv_end - w.kv_begin); };
  const int hkv = t.kv_heads;
  if (!t.pad4 || !(hkv == 1 || hkv == 2 || hkv == 4 || hkv == 8) || tiles.empty()) {
    std::stable_sort(tiles.begin(), tiles.end(),
                     [&](const WorkTile& a, const WorkTile& b) { return work(a) > work(b); });
    return;
  }
  const int R = 8 / hkv;
  const size_t n = tiles.size();
  int64_t total = 0;
  for (const WorkTile& w : tiles) total += work(w);
  // the shortest tiles, an eighth of the work
  std::vector<size_t> by_work(n);
  for (size_t i = 0; i < n; ++i) by_work[i] = i;
  std::stable_sort(by_work.begin(), by_work.end(), [&](size_t a, size_t b) { return work(tiles[a]) < work(tiles[b]); });
  std::vector<char> is_short(n, 0);
  int64_t short_work = 0;
  for (size_t i : by_work) {
    if (8 * short_work >= total) break;
    is_short[i] = 1;
    short_work += work(tiles[i]);
  }
  // long tiles span by span (spans with more long work first), longest first in a span
  std::vector<int64_t> span_work(static_cast<size_t>(*std::max_element(span_of.begin(), span_of.end())) + 1, 0);
  for (size_t i = 0; i < n; ++i)
    if (!is_short[i]) span_work[span_of[i]] += work(tiles[i]);
  std::vector<size_t> long_list;
  long_list.reserve(n);
  for (size_t i = 0; i < n; ++i)
    if (!is_short[i]) long_list.push_back(i);
  std::stable_sort(long_list.begin(), long_list.end(), [&](size_t a, size_t b) {
    const int64_t wa = span_work[span_of[a]], wb = span_work[span_of[b]];
    if (wa != wb) return wa > wb;
    if (span_of[a] != span_of[b]) return span_of[a] < span_of[b];
    return work(tiles[a]) > work(tiles[b]);
  });
  std::vector<std::vector<size_t>> part(R);
  const int64_t long_work = total - short_work;
  int64_t acc = 0;
  int rho = 0;
  for (size_t i : long_list) {
    while (rho + 1 < R && acc * R >= long_work * (rho + 1)) ++rho;
    part[rho].push_back(i);
    acc += work(tiles[i]);
  }
  // the short tiles, longest first, dealt to the chunk with the least work so far
  std::vector<int64_t> part_work(R, 0);
  for (int c = 0; c < R; ++c)
    for (size_t i : part[c]) part_work[c] += work(tiles[i]);
  for (auto it = by_work.rbegin(); it != by_work.rend(); ++it) {
    if (!is_short[*it]) continue;
    const int c = static_cast<int>(std::min_element(part_work.begin(), part_work.end()) - part_work.begin());
    part[c].push_back(*it);
    part_work[c] += work(tiles[*it]);
  }
  std::vector<WorkTile> out;
  out.reserve(n);
  chunks->push_back(0);
  for (int c = 0; c < R; ++c) {
    for (size_t i : part[c]) out.push_back(tiles[i]);
    chunks->push_back(static_cast<int32_t>(out.size()));
  }
  tiles.swap(out);
}
}  // namespace

namespace {
// Row tiles of cross attention (cross and decode rows) before the KV split.
struct CrossTile {
  int32_t row0, n, pos0, kv0, kv1;
  // the query's cross-segment pages: key-list entries wkv0 .. wkv0 + wn, cross page
  // writes wk3 .. wk3 + wn (wn = 0: none to write, e.g. decode rows)
  int32_t wkv0 = 0, wk3 = 0, wn = 0;
};

// The key list a query's cross (and decode) rows read: the prefix, each fragment
// at its final positions (its repositioned copies at delta 0 when it has them, else
// its pages with the delta still to apply) and the cross segment's pages.
// Returns the key-list index where the cross segment's pages begin.
int32_t append_query_keys(const Plan& p, const std::vector<int>& ids, int32_t ps, bool pad4, std::vector<KvPage>& kv) {
  for (int c = 0; c + 1 < static_cast<int>(ids.size()); ++c) {
    const SpanPlan& s = p.spans[ids[c]];
    if (!s.moved.empty())
      append_span(kv, s.moved, s.n_tok, ps, s.final0, 0, pad4);  // copies at final positions
    else
      append_span(kv, s.pages, s.n_tok, ps, s.final0, s.final0 - s.canon0, pad4);
  }
  const SpanPlan& cross = p.spans[ids.back()];
  const int32_t at = static_cast<int32_t>(kv.size());
  append_span(kv, cross.pages, cross.n_tok, ps, cross.final0, 0, pad4);
  return at;
}

// Split the keys of the row tiles into the same number of parts (enough work items
// for the launch, at least min_split_pages per part), tiles with more than one part
// (or two key groups) writing partials that a combine tile merges; few-row
// two-key-group tiles go last.
void tile_cross(const std::vector<CrossTile>& ct, int32_t max_pages, const Tiling& t, std::vector<WorkTile>* tiles,
                std::vector<CombineTile>* combine, int32_t* n_parts, int32_t* n_few, int32_t* kv_splits) {
  int32_t splits = 1;
  if (!ct.empty()) {
    int64_t items = static_cast<int64_t>(ct.size()) * t.kv_heads;
    int64_t want = (t.target_items + items - 1) / items;
    int64_t cap = std::max<int64_t>(1, max_pages / t.min_split_pages);
    splits = static_cast<int32_t>(std::max<int64_t>(1, std::min(want, cap)));
  }
  *kv_splits = splits;
  const int32_t align = t.pad4 ? 4 : 1;
  for (const CrossTile& c : ct) {
    int32_t n_pages = c.kv1 - c.kv0;
    int32_t chunk = (n_pages + splits - 1) / splits;
    chunk = ((chunk + align - 1) / align) * align;   // splits cut at whole tiles
    int32_t parts = (chunk > 0) ? (n_pages + chunk - 1) / chunk : 1;
    const bool two = c.n <= t.two_group_rows;     // each split writes two partials
    // the cross pages among key-list entries [b, e): (first write, count << kWriteShift)
    auto writes = [&](int32_t b, int32_t e, int32_t* first) {
      const int32_t lo = std::max(b, c.wkv0), hi = std::min(e, c.wkv0 + c.wn);
      *first = hi > lo ? c.wk3 + (lo - c.wkv0) : 0;
      return hi > lo ? (hi - lo) << kWriteShift : 0;
    };
    if (parts <= 1 && !two) {
      int32_t wf = 0;
      const int32_t wfl = writes(c.kv0, c.kv1, &wf);
      tiles->push_back(WorkTile{c.row0, c.n, c.pos0, c.kv0, c.kv1, -1, wfl, wf});
      continue;
    }
    int32_t part0 = *n_parts;
    for (int32_t s = 0; s < parts; ++s) {
      int32_t b = c.kv0 + s * chunk;
      int32_t e = std::min(c.kv1, b + chunk);
      int32_t wf = 0;
      const int32_t wfl = writes(b, e, &wf);
      tiles->push_back(WorkTile{c.row0, c.n, c.pos0, b, e, *n_parts, (two ? kTwoKeyGroups : 0) | wfl, wf});
      *n_parts += two ? 2 : 1;
    }
    combine->push_back(CombineTile{c.row0, c.n, part0, *n_parts - part0});
  }
  // Few-row two-key-group tiles last, for the kernel that takes them.
  *n_few = 0;
  if (t.few_rows > 0) {
    auto few = [&](const WorkTile& w) { return (w.flags & kTwoKeyGroups) != 0 && w.n_rows <= t.few_rows; };
    std::stable_partition(tiles->begin(), tiles->end(), [&](const WorkTile& w) { return !few(w); });
    *n_few = static_cast<int32_t>(std::count_if(tiles->begin(), tiles->end(), few));
  }
}

// Tiled key lists: every list (and every split of one) starts at a multiple of four
// pages, so kv[4i .. 4i + 3] is a tile.
void tile_records(const std::vector<KvPage>& kv, bool pad4, std::vector<TileRec>* out) {
  out->clear();
  if (!pad4) return;
  out->reserve(kv.size() / 4);
  for (size_t i = 0; i + 3 < kv.size(); i += 4) {
    const KvPage* k = &kv[i];
    out->push_back(TileRec{{k[0].page_id, k[1].page_id, k[2].page_id, k[3].page_id}, k[0].pos0,
                           k[0].n_valid + k[1].n_valid + k[2].n_valid + k[3].n_valid, k[0].delta, 0});
  }
}
}  // namespace

void PoolIndex::build_work(Plan* p, const Tiling& t) {
  const int32_t ps = page_size_;
  p->bm_cross = t.bm_cross;
  for (size_t qi = 0; qi < p->query_spans.size(); ++qi) {
    const auto& ids = p->query_spans[qi];
    SpanPlan& prefix = p->spans[ids[0]];
    SpanPlan& cross = p->spans[ids.back()];
    const int32_t P = prefix.n_tok;
    prefix.canon0 = 0;
    prefix.final0 = 0;
    int32_t at = P;
    for (size_t c = 1; c + 1 < ids.size(); ++c) {
      SpanPlan& f = p->spans[ids[c]];
      f.canon0 = P;
      f.final0 = at;
      at += f.n_tok;
    }
    cross.canon0 = at;
    cross.final0 = at;
    p->max_pos = std::max(p->max_pos, at + cross.n_tok);
  }
  // ---- prefill: new pages and row tiles of every span that computes pages
  std::vector<int32_t> tile_span;  // per prefill tile: the span it belongs to
  {
    // room for every list (each padded by at most 3 pages per span)
    size_t kv_n = 0, new_n = 0, tile_n = 0;
    for (const auto& ids : p->query_spans) {
      const size_t pre = p->spans[ids[0]].pages.size() + 3;
      size_t all = 0;
      for (size_t c = 0; c < ids.size(); ++c) {
        const SpanPlan& s = p->spans[ids[c]];
        all += s.pages.size() + 3;
        if (c + 1 == ids.size() || s.n_hit >= static_cast<int32_t>(s.pages.size())) continue;
        kv_n += s.pages.size() + 3 + (s.kind == 1 ? pre : 0);
        new_n += s.pages.size() - s.n_hit;
        tile_n += (static_cast<size_t>(s.n_tok - s.n_hit * ps) + t.bm_prefill - 1) / t.bm_prefill;
      }
      kv_n += all;
    }
    p->kv.reserve(kv_n);
    p->k3_prefill.reserve(new_n);
    p->t_prefill.reserve(tile_n);
    p->rows_prefill.reserve(tile_n);
    tile_span.reserve(tile_n);
  }
  for (size_t qi = 0; qi < p->query_spans.size(); ++qi) {
    const auto& ids = p->query_spans[qi];
    const SpanPlan& prefix = p->spans[ids[0]];
    for (size_t c = 0; c + 1 < ids.size(); ++c) {
      const SpanPlan& s = p->spans[ids[c]];
      const int32_t np = static_cast<int32_t>(s.pages.size());
      if (s.n_hit >= np) continue;
      for (int32_t pg = s.n_hit; pg < np; ++pg)
        p->k3_prefill.push_back(NewPage{s.pages[pg], std::min(ps, s.n_tok - pg * ps),
                                        static_cast<int32_t>(s.row + pg * ps), s.canon0 + pg * ps});
      const int32_t kv0 = static_cast<int32_t>(p->kv.size());
      if (s.kind == 1) append_span(p->kv, prefix.pages, prefix.n_tok, ps, 0, 0, t.pad4);
      append_span(p->kv, s.pages, s.n_tok, ps, s.canon0, 0, t.pad4);
      const int32_t kv1 = static_cast<int32_t>(p->kv.size());
      const int32_t pre = (s.kind == 1) ? prefix.n_tok : 0;
      for (int32_t j0 = s.n_hit * ps; j0 < s.n_tok; j0 += t.bm_prefill) {
        int32_t n = std::min(t.bm_prefill, s.n_tok - j0);
        int32_t end = list_end(p->kv, kv0, kv1, s.canon0 + j0 + n - 1, t.pad4);
        p->t_prefill.push_back(WorkTile{static_cast<int32_t>(s.row + j0), n, s.canon0 + j0, kv0, end, -1, 0, 0});
        tile_span.push_back(ids[c]);
        p->rows_prefill.push_back(Plan::RowRun{s.row + j0, n});
        // rows j0..j0+n-1 see pre + j + 1 keys each
        p->prefill_pairs += static_cast<int64_t>(n) * (pre + 1) + static_cast<int64_t>(n) * (2 * j0 + n - 1) / 2;
      }
    }
  }
  order_prefill(p->t_prefill, tile_span, t, &p->prefill_chunks);
  // ---- cross: pages, key list in query order, split-KV row tiles
  std::vector<CrossTile> ct;
  int32_t max_pages = 0;
  for (size_t qi = 0; qi < p->query_spans.size(); ++qi) {
    const auto& ids = p->query_spans[qi];
    const SpanPlan& cross = p->spans[ids.back()];
    if (cross.n_tok == 0) continue;
    const int32_t wk3 = static_cast<int32_t>(p->k3_cross.size());
    for (size_t pg = 0; pg < cross.pages.size(); ++pg)
      p->k3_cross.push_back(NewPage{cross.pages[pg], std::min<int32_t>(ps, cross.n_tok - static_cast<int32_t>(pg) * ps),
                                    static_cast<int32_t>(cross.row + pg * ps), cross.final0 + static_cast<int32_t>(pg) * ps});
    const int32_t kv0 = static_cast<int32_t>(p->kv.size());
    const int32_t wkv0 = append_query_keys(*p, ids, ps, t.pad4, p->kv);
    const int32_t kv1 = static_cast<int32_t>(p->kv.size());
    p->cross_kv_pages += kv1 - kv0;
    for (int32_t j0 = 0; j0 < cross.n_tok; j0 += t.bm_cross) {
      int32_t n = std::min(t.bm_cross, cross.n_tok - j0);
      int32_t end = list_end(p->kv, kv0, kv1, cross.final0 + j0 + n - 1, t.pad4);
      ct.push_back(CrossTile{static_cast<int32_t>(cross.row + j0), n, cross.final0 + j0, kv0, end, wkv0, wk3,
                             static_cast<int32_t>(cross.pages.size())});
      max_pages = std::max(max_pages, end - kv0);
      p->rows_cross.push_back(Plan::RowRun{cross.row + j0, n});
      p->cross_pairs += static_cast<int64_t>(n) * (cross.final0 + 1) + static_cast<int64_t>(n) * (2 * j0 + n - 1) / 2;
    }
  }
  tile_cross(ct, max_pages, t, &p->t_cross, &p->combine, &p->n_parts, &p->n_cross_few, &p->kv_splits);
  tile_records(p->kv, t.pad4, &p->kv_tiles);
}

int PoolIndex::decode(Plan* p, const std::vector<int32_t>& n_new, const std::vector<int64_t>& rows,
                      const Tiling& t, std::string* msg) {
  const int32_t ps = page_size_;
  const size_t nq = p->query_spans.size();
  if (n_new.size() != nq || rows.size() != nq) {
    *msg = "decode: one token count and one row per query";
    return SPAN_EINVAL;
  }
  int64_t need = 0, total = 0;
  for (size_t q = 0; q < nq; ++q) {
    const SpanPlan& cross = p->spans[p->query_spans[q].back()];
    const int64_t n = n_new[q];
    if (n < 0 || (n > 0 && (rows[q] < 0 || rows[q] + n > std::numeric_limits<int32_t>::max())) ||
        static_cast<int64_t>(cross.final0) + cross.n_tok + n >= std::numeric_limits<int32_t>::max() / 2) {
      *msg = "decode: bad token count or row";
      return SPAN_EINVAL;
    }
    need += (cross.n_tok + n + ps - 1) / ps - (cross.n_tok + ps - 1) / ps;
    total += n;
  }
  if (need > free_count() + n_evictable_) {
    *msg = "pool exhausted: decode needs " + std::to_string(need) + " pages, " + std::to_string(free_count()) +
           " free, " + std::to_string(n_evictable_) + " evictable";
    return SPAN_ENOMEM;
  }
  Plan::DecodeStep& d = p->dec;
  d = Plan::DecodeStep{};
  std::vector<CrossTile> ct;
  int32_t max_pages = 0;
  for (size_t q = 0; q < nq; ++q) {
    const int32_t n = n_new[q];
    if (n == 0) continue;
    const auto& ids = p->query_spans[q];
    SpanPlan& cross = p->spans[ids.back()];
    const int32_t cur = cross.n_tok;
    while (static_cast<int64_t>(cross.pages.size()) * ps < static_cast<int64_t>(cur) + n) {
      if (free_count() == 0) evict_one(p);
      const int32_t pid = pop_free();
      PageRec& r = pages_[pid];
      r = PageRec{};
      r.last_use = p->tick;
      r.pins = 1;
      r.used = true;
      p->new_pages.push_back(pid);
      p->cross_pages.push_back(pid);
      cross.pages.push_back(pid);
      ++d.pages_new;
    }
    const int32_t pos_first = cross.final0 + cur;
    for (int32_t i = 0; i < n;) {
      const int32_t pg = (cur + i) / ps, s0 = (cur + i) % ps, m = std::min(ps - s0, n - i);
      d.writes.push_back(SlotWrite{cross.pages[pg], s0, m, static_cast<int32_t>(rows[q] + i), pos_first + i, {0, 0, 0}});
      i += m;
    }
    cross.n_tok = cur + n;
    p->max_pos = std::max(p->max_pos, cross.final0 + cross.n_tok);
    const int32_t kv0 = static_cast<int32_t>(d.kv.size());
    append_query_keys(*p, ids, ps, t.pad4, d.kv);
    const int32_t kv1 = static_cast<int32_t>(d.kv.size());
    for (int32_t j0 = 0; j0 < n; j0 += t.bm_cross) {
      const int32_t nn = std::min(t.bm_cross, n - j0);
      const int32_t end = list_end(d.kv, kv0, kv1, pos_first + j0 + nn - 1, t.pad4);
      ct.push_back(CrossTile{static_cast<int32_t>(rows[q] + j0), nn, pos_first + j0, kv0, end});
      max_pages = std::max(max_pages, end - kv0);
      d.rows.push_back(Plan::RowRun{rows[q] + j0, nn});
      d.pairs += static_cast<int64_t>(nn) * (pos_first + j0 + 1) + static_cast<int64_t>(nn) * (nn - 1) / 2;
    }
  }
  tile_cross(ct, max_pages, t, &d.tiles, &d.combine, &d.n_parts, &d.n_few, &d.kv_splits);
  tile_records(d.kv, t.pad4, &d.kv_tiles);
  d.tokens = total;
  p->decode_steps += 1;
  p->decode_tokens += total;
  p->decode_pages += d.pages_new;
  return SPAN_OK;
}

void PoolIndex::commit(Plan* p) {
  for (int32_t pid : p->new_pages) {
    PageRec& r = pages_[pid];
    if (!r.cacheable || !index_.try_emplace(r.hash, pid).second) continue;
    r.published = true;
  }
  for (int32_t pid : p->new_pages) {
    PageRec& r = pages_[pid];
    r.pins -= 1;
    if (!r.published) {
      push_free(pid);
    } else if (r.pins == 0) {
      make_evictable(pid);
    }
  }
  for (int32_t pid : p->hits) {
    PageRec& r = pages_[pid];
    r.pins -= 1;
    if (r.published && r.pins == 0) make_evictable(pid);
  }
  p->committed = true;
  --live_plans;
}

void PoolIndex::release(Plan* p) {
  if (p->committed) return;
  for (int32_t pid : p->new_pages) push_free(pid);
  for (int32_t pid : p->hits) {
    PageRec& r = pages_[pid];
    r.pins -= 1;
    if (r.published && r.pins == 0) make_evictable(pid);
  }
  p->committed = true;
  --live_plans;
}

}  // namespace spanq
