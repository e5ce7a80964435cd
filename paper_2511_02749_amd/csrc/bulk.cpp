// Bulk scheduling: an execution order for a bulk of span queries that clusters the
// reuse of fragments in time (section 5.8: a greedy heuristic clusters the requests
// of a bulk so that reused fragments are close together, which matters once the
// bulk's working set is larger than the cache).
//
// The heuristic simulates the pool at span granularity.  A span (the prefix or one
// fragment of a query, keyed by its page-hash chain) is resident or not; a span the
// pool already holds in full starts resident.  Each step picks the remaining query
// with the most pages in resident spans (ties: the lowest index), then applies it:
// its spans are touched, missing ones inserted, and least recently used spans
// evicted while the simulated pages exceed the pool's capacity.  O(n^2 k) for n
// queries of k spans.
#include <algorithm>
#include <cstdint>
#include <unordered_map>
#include <vector>

#include "../../include/spanq.h"
#include "capi_internal.h"
#include "planner.h"

using namespace spanq;

namespace {

struct SpanKey {
  uint64_t last;   // hash of the span's last page (identifies the whole chain)
  int64_t pages;
};

// The chain of one span, and how many of its leading pages the pool holds.
SpanKey span_key(const PoolIndex* index, uint64_t seed, const span_tokens& s, int32_t ps, bool* resident) {
  uint64_t h = seed;
  int64_t pages = 0, held = 0;
  bool run = true;
  for (int32_t p = 0; p * ps < s.n; ++p) {
    const int32_t n = std::min(ps, s.n - p * ps);
    h = page_hash(h, s.tokens + static_cast<int64_t>(p) * ps, n, p);
    ++pages;
    if (run && index->lookup(h) >= 0) {
      ++held;
    } else {
      run = false;
    }
  }
  *resident = pages > 0 && held == pages;
  return SpanKey{h, pages};
}

}  // namespace

extern "C" int span_bulk_order(const span_pool* pool, const span_query* qs, int32_t nq, int32_t* order) {
  if (!pool || nq < 0 || (nq > 0 && (!qs || !order))) return report(SPAN_EINVAL, "span_bulk_order: bad argument");
  const PoolIndex* index = pool_index(pool);
  const int32_t ps = index->page_size();
  const int64_t capacity = index->num_pages();
  // spans of every query, as indices into `keys`
  std::vector<SpanKey> keys;
  std::unordered_map<uint64_t, int32_t> by_hash;
  std::vector<std::vector<int32_t>> spans(static_cast<size_t>(nq));
  std::vector<char> resident;
  std::vector<int64_t> last_use;
  int64_t held_pages = 0;
  for (int32_t q = 0; q < nq; ++q) {
    const span_query& sq = qs[q];
    if (sq.n_frags < 0 || (sq.n_frags > 0 && !sq.frags) || sq.prefix.n < 0 || (sq.prefix.n > 0 && !sq.prefix.tokens))
      return report(SPAN_EINVAL, "span_bulk_order: bad query");
    auto add = [&](uint64_t seed, const span_tokens& s) -> uint64_t {
      bool res = false;
      SpanKey k = span_key(index, seed, s, ps, &res);
      if (k.pages == 0) return k.last;
      auto it = by_hash.find(k.last);
      if (it == by_hash.end()) {
        it = by_hash.emplace(k.last, static_cast<int32_t>(keys.size())).first;
        keys.push_back(k);
        resident.push_back(res ? 1 : 0);
        last_use.push_back(0);
        held_pages += res ? k.pages : 0;
      }
      spans[q].push_back(it->second);
      return k.last;
    };
    const uint64_t plast = add(SPAN_HASH_ROOT, sq.prefix);
    const uint64_t fseed = fragment_seed(sq.prefix.n > 0 ? plast : SPAN_HASH_ROOT);
    for (int32_t f = 0; f < sq.n_frags; ++f) {
      if (sq.frags[f].n < 0 || (sq.frags[f].n > 0 && !sq.frags[f].tokens))
        return report(SPAN_EINVAL, "span_bulk_order: bad fragment");
      add(fseed, sq.frags[f]);
    }
  }
  std::vector<char> done(static_cast<size_t>(nq), 0);
  for (int32_t step = 0; step < nq; ++step) {
    int32_t best = -1;
    int64_t best_score = -1;
    for (int32_t q = 0; q < nq; ++q) {
      if (done[q]) continue;
      int64_t score = 0;
      for (int32_t k : spans[q]) score += resident[k] ? keys[k].pages : 0;
      if (score > best_score) {
        best = q;
        best_score = score;
      }
    }
    order[step] = best;
    done[best] = 1;
    const int64_t t = step + 1;
    for (int32_t k : spans[best]) {
      if (!resident[k]) {
        resident[k] = 1;
        held_pages += keys[k].pages;
      }
      last_use[k] = t;
    }
    // evict least recently used spans (never the ones just used) down to capacity
    while (held_pages > capacity) {
      int32_t victim = -1;
      for (int32_t k = 0; k < static_cast<int32_t>(keys.size()); ++k)
        if (resident[k] && last_use[k] < t && (victim < 0 || last_use[k] < last_use[victim])) victim = k;
      if (victim < 0) break;
      resident[victim] = 0;
      held_pages -= keys[victim].pages;
    }
  }
  return SPAN_OK;
}
