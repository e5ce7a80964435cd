// Host-side checks of the planner, the serialized-query parser and bulk ordering.
// tests/test_host_sanitize.py builds this with g++ under AddressSanitizer and
// UndefinedBehaviorSanitizer, once with full 64-bit page hashes and once with
// SPANQ_TEST_HASH_BITS (page hashes cut to a few bits, so that unrelated pages
// collide all the time), and runs random streams through it.
//
// Planner: every plan (random queries over a small fragment set, random tilings of
// both kernels, with and without materialised repositioning, commit or release) is
// checked for
// - content: a page served as a hit holds exactly the tokens, page index and length
//   the query asks for (a hash collision must end as a miss, never as a wrong hit);
// - bounds of every page id and key-list range the GPU kernels would read;
// - the prefill tiles being a permutation of the row runs, the per-XCD chunking and
//   its balance, the repositioned copies.
// Parser: random and mutated token streams never read out of bounds and either
// fail cleanly or return ranges inside the stream.  Bulk order: a permutation.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
#include <string>
#include <vector>

#include "capi_internal.h"
#include "planner.h"
#include "spanq.h"

struct span_pool {
  spanq::PoolIndex* index;
};

namespace spanq {
int report(int code, const char*) { return code; }
const PoolIndex* pool_index(const span_pool* p) { return p->index; }
}  // namespace spanq

using namespace spanq;

static int g_fail = 0;
#define CHECK(cond, ...)                                                   \
  do {                                                                     \
    if (!(cond)) {                                                         \
      std::fprintf(stderr, "FAIL line %d (%s): ", __LINE__, #cond);        \
      std::fprintf(stderr, __VA_ARGS__);                                   \
      std::fprintf(stderr, "\n");                                          \
      if (++g_fail > 20) std::exit(1);                                     \
    }                                                                      \
  } while (0)

namespace {

using Tokens = std::vector<int32_t>;

struct PageContent {
  int32_t idx = -1;  // -1: a page no lookup may serve (cross page, copy)
  Tokens tok;
};

Tokens page_tokens(const Tokens& span, int32_t pg, int32_t ps) {
  const int32_t b = pg * ps;
  const int32_t e = std::min<int32_t>(static_cast<int32_t>(span.size()), b + ps);
  return Tokens(span.begin() + b, span.begin() + e);
}

int64_t work(const WorkTile& w) { return w.kv_end - w.kv_begin; }

void check_plan(const Plan& P, const std::vector<std::vector<const Tokens*>>& qspans, const Tiling& t,
                int64_t num_pages, int32_t ps, std::map<int32_t, PageContent>& shadow, int64_t* hits_checked) {
  for (size_t qi = 0; qi < P.query_spans.size(); ++qi) {
    const auto& ids = P.query_spans[qi];
    for (size_t c = 0; c < ids.size(); ++c) {
      const SpanPlan& sp = P.spans[ids[c]];
      const Tokens& tok = *qspans[qi][c];
      for (size_t pg = sp.kind == 2 ? 0 : sp.n_hit; pg < sp.pages.size(); ++pg) {
        PageContent pc;
        pc.idx = sp.kind == 2 ? -1 : static_cast<int32_t>(pg);
        pc.tok = page_tokens(tok, static_cast<int32_t>(pg), ps);
        shadow[sp.pages[pg]] = pc;
      }
    }
  }
  // content of hits (pages this plan writes first: a span may hit a page that an
  // earlier span of the same plan computes)
  std::set<int32_t> span_pages;
  for (size_t qi = 0; qi < P.query_spans.size(); ++qi) {
    const auto& ids = P.query_spans[qi];
    CHECK(ids.size() == qspans[qi].size(), "query %zu: %zu spans planned, %zu given", qi, ids.size(),
          qspans[qi].size());
    for (size_t c = 0; c < ids.size(); ++c) {
      const SpanPlan& sp = P.spans[ids[c]];
      const Tokens& tok = *qspans[qi][c];
      CHECK(static_cast<size_t>(sp.n_tok) == tok.size(), "span length");
      CHECK(static_cast<int64_t>(sp.pages.size()) == (sp.n_tok + ps - 1) / ps, "pages of a span");
      for (size_t pg = 0; pg < sp.pages.size(); ++pg) {
        const int32_t pid = sp.pages[pg];
        CHECK(pid >= 0 && pid < num_pages, "page id %d out of [0, %lld)", pid, static_cast<long long>(num_pages));
        span_pages.insert(pid);
        const Tokens want = page_tokens(tok, static_cast<int32_t>(pg), ps);
        if (sp.kind != 2 && static_cast<int32_t>(pg) < sp.n_hit) {
          auto it = shadow.find(pid);
          const bool ok = it != shadow.end() && it->second.idx == static_cast<int32_t>(pg) && it->second.tok == want;
          CHECK(ok, "query %zu span %zu page %zu: hit on page %d holding other content", qi, c, pg, pid);
          ++*hits_checked;
        }
      }
    }
  }
  // repositioned copies
  std::set<int32_t> dst;
  for (const MovePage& m : P.moves) {
    CHECK(m.src_page >= 0 && m.src_page < num_pages && m.dst_page >= 0 && m.dst_page < num_pages, "move bounds");
    CHECK(span_pages.count(m.src_page) == 1, "move source %d not in a block table", m.src_page);
    CHECK(span_pages.count(m.dst_page) == 0, "move copy %d is also in a block table", m.dst_page);
    CHECK(dst.insert(m.dst_page).second, "copy page %d used twice", m.dst_page);
    CHECK(m.delta > 0 && m.delta < P.max_pos, "move delta %d", m.delta);
    CHECK(m.n_valid >= 1 && m.n_valid <= ps, "move slots");
    shadow[m.dst_page] = PageContent{};
  }
  if (!t.materialize) CHECK(P.moves.empty(), "moves without materialisation");
  // key lists and work tiles
  for (const KvPage& k : P.kv) {
    CHECK(k.page_id >= 0 && k.page_id < num_pages, "key page %d", k.page_id);
    CHECK(k.n_valid >= 0 && k.n_valid <= ps, "key slots");
    CHECK(k.pos0 >= 0 && k.pos0 + ps <= P.max_pos + ps, "key position");
    if (t.materialize) CHECK(k.delta == 0 || dst.count(k.page_id) == 0, "copies are read at delta 0");
  }
  if (t.pad4) {
    CHECK(P.kv.size() % 4 == 0 && P.kv_tiles.size() * 4 == P.kv.size(), "tiled key list");
    for (const TileRec& r : P.kv_tiles)
      for (int i = 0; i < 4; ++i) CHECK(r.page_id[i] >= 0 && r.page_id[i] < num_pages, "tile page");
  }
  const int32_t nkv = static_cast<int32_t>(P.kv.size());
  auto check_tiles = [&](const std::vector<WorkTile>& ts, const char* what) {
    for (const WorkTile& w : ts) {
      CHECK(0 <= w.kv_begin && w.kv_begin < w.kv_end && w.kv_end <= nkv, "%s key range", what);
      if (t.pad4) CHECK(w.kv_begin % 4 == 0 && w.kv_end % 4 == 0, "%s tile alignment", what);
      CHECK(w.n_rows >= 1 && w.n_rows <= std::max(t.bm_prefill, t.bm_cross), "%s rows", what);
      CHECK(w.part < P.n_parts, "%s partial slot", what);
    }
  };
  check_tiles(P.t_prefill, "prefill");
  check_tiles(P.t_cross, "cross");
  for (const CombineTile& c : P.combine) CHECK(c.part0 >= 0 && c.part0 + c.n_parts <= P.n_parts, "combine slots");
  // prefill tiles: a permutation of the row runs
  std::multiset<std::pair<int64_t, int32_t>> runs, tiles;
  for (const auto& r : P.rows_prefill) runs.insert({r.row0, r.n});
  for (const WorkTile& w : P.t_prefill) tiles.insert({w.q_row0, w.n_rows});
  CHECK(runs == tiles, "prefill tiles are not the row runs");
  // per-XCD chunks
  const int hkv = t.kv_heads;
  const bool xcd = t.pad4 && (hkv == 1 || hkv == 2 || hkv == 4 || hkv == 8) && !P.t_prefill.empty();
  if (!xcd) {
    CHECK(P.prefill_chunks.empty(), "chunks without per-XCD queues");
    for (size_t i = 1; i < P.t_prefill.size(); ++i)
      CHECK(work(P.t_prefill[i - 1]) >= work(P.t_prefill[i]), "generic order is longest first");
  } else {
    const int R = 8 / hkv;
    CHECK(static_cast<int>(P.prefill_chunks.size()) == R + 1, "%zu chunk offsets for %d chunks",
          P.prefill_chunks.size(), R);
    if (static_cast<int>(P.prefill_chunks.size()) == R + 1) {
      CHECK(P.prefill_chunks[0] == 0 && P.prefill_chunks[R] == static_cast<int32_t>(P.t_prefill.size()),
            "chunk ends");
      int64_t total = 0, wmax = 0;
      for (const WorkTile& w : P.t_prefill) {
        total += work(w);
        wmax = std::max(wmax, work(w));
      }
      for (int c = 0; c < R; ++c) {
        CHECK(P.prefill_chunks[c] <= P.prefill_chunks[c + 1], "chunk offsets ascend");
        int64_t wc = 0;
        for (int32_t i = P.prefill_chunks[c]; i < P.prefill_chunks[c + 1]; ++i) wc += work(P.t_prefill[i]);
        // the long tiles are cut at equal shares of their work, the short ones dealt
        // to the lightest chunk: a chunk is within two tiles of the mean
        CHECK(wc * R <= total + 2 * R * wmax && wc * R >= total - 2 * R * wmax,
              "chunk %d holds %lld of %lld (max tile %lld)", c, static_cast<long long>(wc),
              static_cast<long long>(total), static_cast<long long>(wmax));
      }
    }
  }
}

struct Stream {
  std::mt19937_64 rng;
  std::vector<Tokens> frags, prefixes, crosses;
  explicit Stream(uint64_t seed) : rng(seed) {
    const int lens[] = {0, 1, 5, 15, 16, 17, 31, 32, 33, 47, 64, 80, 100};
    for (int i = 0; i < 14; ++i) {
      Tokens t(lens[rng() % 13]);
      for (auto& x : t) x = static_cast<int32_t>(rng() % 50);  // a small vocabulary: shared pages
      frags.push_back(t);
    }
    const int plens[] = {0, 5, 16, 33};
    for (int l : plens) {
      Tokens t(l);
      for (auto& x : t) x = static_cast<int32_t>(rng() % 50);
      prefixes.push_back(t);
    }
    for (int l : {0, 1, 9, 16, 40}) {
      Tokens t(l);
      for (auto& x : t) x = static_cast<int32_t>(1000 + rng() % 50);
      crosses.push_back(t);
    }
  }
  uint64_t pick(uint64_t n) { return rng() % n; }
};

void run_planner(uint64_t seed, int steps) {
  Stream st(seed);
  const int32_t ps = 16;
  const int64_t num_pages = 24 + static_cast<int64_t>(st.pick(120));  // small pools evict often
  PoolIndex index(num_pages, ps, SPAN_HASH_SPAN);
  std::map<int32_t, PageContent> shadow;
  int64_t hits = 0, plans = 0, full = 0;
  for (int s = 0; s < steps; ++s) {
    const int nq = 1 + static_cast<int>(st.pick(4));
    std::vector<QueryIn> qs(nq);
    std::vector<std::vector<const Tokens*>> qspans(nq);
    int64_t row = 0;
    for (int q = 0; q < nq; ++q) {
      const Tokens& pre = st.prefixes[st.pick(st.prefixes.size())];
      qs[q].prefix = SpanIn{pre.data(), static_cast<int32_t>(pre.size()), row};
      row += static_cast<int64_t>(pre.size());
      qspans[q].push_back(&pre);
      const int nf = static_cast<int>(st.pick(5));
      for (int f = 0; f < nf; ++f) {
        const Tokens& fr = st.frags[st.pick(st.frags.size())];
        qs[q].frags.push_back(SpanIn{fr.data(), static_cast<int32_t>(fr.size()), row});
        row += static_cast<int64_t>(fr.size());
        qspans[q].push_back(&fr);
      }
      const Tokens& cr = st.crosses[st.pick(st.crosses.size())];
      qs[q].cross = SpanIn{cr.data(), static_cast<int32_t>(cr.size()), row};
      row += static_cast<int64_t>(cr.size());
      qspans[q].push_back(&cr);
    }
    const int hkvs[] = {1, 2, 3, 4, 8};
    const int gs[] = {1, 2, 4, 8};
    const int hkv = hkvs[st.pick(5)], g = gs[st.pick(4)];
    const bool mfma = st.pick(2) == 0;
    Tiling t = tiling_for(mfma, mfma ? 256 / g : 64, g * hkv, hkv);
    t.materialize = st.pick(3) == 0;
    Plan P;
    std::string msg;
    const int64_t free_before = index.free_count(), cached_before = index.cached_count();
    const int rc = index.plan(qs, true, t, &P, &msg);
    if (rc == SPAN_ENOMEM) {
      CHECK(index.free_count() == free_before && index.cached_count() == cached_before, "ENOMEM changed the pool");
      ++full;
      continue;
    }
    CHECK(rc == 0, "plan failed: %s", msg.c_str());
    if (rc) continue;
    ++plans;
    check_plan(P, qspans, t, num_pages, ps, shadow, &hits);
    if (st.pick(4) != 0) {
      index.commit(&P);
    } else {
      index.release(&P);
    }
    CHECK(index.pinned_count() == 0, "pages still pinned after the plan ended");
    if (st.pick(50) == 0) {
      index.reset();
      shadow.clear();
    }
  }
  std::printf("planner seed %llu (%lld pages): %lld plans, %lld pool-full refusals, %lld evictions, %lld hit pages "
              "checked\n",
              static_cast<unsigned long long>(seed), static_cast<long long>(num_pages), static_cast<long long>(plans),
              static_cast<long long>(full), static_cast<long long>(index.total_evictions()),
              static_cast<long long>(hits));
  CHECK(hits > 0, "no hits at all");
}

void run_parser(uint64_t seed, int steps) {
  std::mt19937_64 rng(seed);
  const int32_t special[4] = {900, 901, 902, 903};  // PAD OPEN SEP CLOSE
  int64_t ok = 0, rejected = 0;
  for (int s = 0; s < steps; ++s) {
    const int32_t block = 1 + static_cast<int32_t>(rng() % 8);
    // a well-formed stream, then random mutations
    std::vector<int32_t> t;
    const int pre = static_cast<int>(rng() % 20);
    for (int i = 0; i < pre; ++i) t.push_back(static_cast<int32_t>(rng() % 100));
    auto align = [&]() {
      while (t.size() % block) t.push_back(special[0]);
    };
    const int nf = static_cast<int>(rng() % 4);
    int64_t open_at = -1;
    if (nf > 0) {
      align();
      open_at = static_cast<int64_t>(t.size());
      t.push_back(special[1]);
      for (int f = 0; f < nf; ++f) {
        if (f > 0) {
          align();
          t.push_back(special[2]);
        }
        const int n = static_cast<int>(rng() % 20);
        for (int i = 0; i < n; ++i) t.push_back(static_cast<int32_t>(rng() % 100));
      }
      align();
      t.push_back(special[3]);
      t.push_back(static_cast<int32_t>(open_at));
      const int cr = static_cast<int>(rng() % 10);
      for (int i = 0; i < cr; ++i) t.push_back(static_cast<int32_t>(rng() % 100));
    }
    const int muts = static_cast<int>(rng() % 3);
    for (int m = 0; m < muts && !t.empty(); ++m) {
      const size_t at = rng() % t.size();
      switch (rng() % 4) {
        case 0: t[at] = special[rng() % 4]; break;
        case 1: t.erase(t.begin() + static_cast<int64_t>(at)); break;
        case 2: t[at] = static_cast<int32_t>(rng() % 2000) - 500; break;  // also negative and large
        default: t.resize(at); break;
      }
    }
    const int32_t cap = static_cast<int32_t>(rng() % 4);
    std::vector<span_range> frags(static_cast<size_t>(std::max(cap, 1)));
    span_range prefix{}, cross{};
    int32_t n_frags = -1;
    const int rc = span_parse_serialized(t.empty() ? nullptr : t.data(), static_cast<int64_t>(t.size()), block,
                                         special, frags.data(), cap, &n_frags, &prefix, &cross);
    if (rc == SPAN_OK) {
      ++ok;
      const int64_t n = static_cast<int64_t>(t.size());
      CHECK(prefix.begin >= 0 && prefix.n >= 0 && prefix.begin + prefix.n <= n, "prefix range");
      CHECK(cross.begin >= 0 && cross.n >= 0 && cross.begin + cross.n <= n, "cross range");
      CHECK(n_frags >= 0, "fragment count");
      for (int32_t f = 0; f < std::min(n_frags, cap); ++f)
        CHECK(frags[f].begin >= 0 && frags[f].n >= 0 && frags[f].begin + frags[f].n <= n, "fragment range");
      if (muts == 0) CHECK(n_frags == nf, "fragments of a well-formed stream");
    } else {
      CHECK(rc == SPAN_EINVAL, "parser status %d", rc);
      CHECK(muts > 0, "a well-formed stream was rejected");
      ++rejected;
    }
  }
  std::printf("parser seed %llu: %lld parsed, %lld rejected\n", static_cast<unsigned long long>(seed),
              static_cast<long long>(ok), static_cast<long long>(rejected));
}

void run_bulk(uint64_t seed, int steps) {
  Stream st(seed);
  PoolIndex index(64, 16, SPAN_HASH_SPAN);
  span_pool pool{&index};
  for (int s = 0; s < steps; ++s) {
    const int nq = static_cast<int>(st.pick(12));
    std::vector<std::vector<span_tokens>> fr(nq);
    std::vector<span_query> qs(nq);
    for (int q = 0; q < nq; ++q) {
      const Tokens& pre = st.prefixes[st.pick(st.prefixes.size())];
      const int nf = static_cast<int>(st.pick(5));
      for (int f = 0; f < nf; ++f) {
        const Tokens& t = st.frags[st.pick(st.frags.size())];
        fr[q].push_back(span_tokens{t.data(), static_cast<int32_t>(t.size()), 0, 0});
      }
      qs[q].prefix = span_tokens{pre.data(), static_cast<int32_t>(pre.size()), 0, 0};
      qs[q].frags = fr[q].data();
      qs[q].n_frags = nf;
      qs[q].cross = span_tokens{nullptr, 0, 0, 0};
    }
    std::vector<int32_t> order(static_cast<size_t>(std::max(nq, 1)), -1);
    const int rc = span_bulk_order(&pool, qs.data(), nq, order.data());
    CHECK(rc == SPAN_OK, "bulk order status %d", rc);
    std::vector<int32_t> sorted(order.begin(), order.begin() + nq);
    std::sort(sorted.begin(), sorted.end());
    for (int q = 0; q < nq; ++q) CHECK(sorted[q] == q, "bulk order is not a permutation");
  }
}

}  // namespace

int main(int argc, char** argv) {
  const uint64_t seed = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
  const int steps = argc > 2 ? std::atoi(argv[2]) : 400;
  run_planner(seed, steps);
  run_parser(seed, steps * 5);
  run_bulk(seed, steps / 4);
  if (g_fail) {
    std::fprintf(stderr, "%d check(s) failed\n", g_fail);
    return 1;
  }
  std::printf("all checks passed\n");
  return 0;
}
