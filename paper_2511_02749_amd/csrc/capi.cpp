// C-ABI of the span-query prefill library: pools, plans, attention entry points.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdint>
#include <cstring>
#include <limits>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "../../include/spanq.h"
#include "capi_internal.h"
#include "kernels.h"
#include "planner.h"

using namespace spanq;

namespace {
thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SPAN_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t elem_size(int32_t dtype) { return dtype == SPAN_BF16 ? 2 : 4; }

}  // namespace

struct span_pool {
  span_pool_config cfg{};
  PoolIndex* index = nullptr;
  void* dev = nullptr;
  bool owns_dev = false;
  bool use_mfma = false;
  std::set<span_plan_t*> plans;
  std::vector<hipEvent_t> event_cache;  // reusable timing events
  std::vector<hipEvent_t> order_cache;  // reusable ordering events (no timing)
  float2* rope_tab = nullptr;           // (cos, sin) per [position][head_dim / 2]
  int64_t rope_n = 0;                   // positions in rope_tab
  // Tables replaced by a larger one.  A live plan may still launch kernels that read
  // the table it was planned with, so replaced tables (and the host copies their
  // uploads read from) stay allocated until the pool is destroyed; the table doubles
  // each time, so they add at most its current size.
  std::vector<float2*> rope_retired;
  std::vector<std::vector<float2>> rope_host;
};

namespace {
int max_parts(const std::vector<CombineTile>& c) {
  int m = 0;
  for (const CombineTile& t : c) m = std::max(m, static_cast<int>(t.n_parts));
  return m;
}

// The (m, l) half of a split-KV partial buffer, after its part_o_elems O elements.
float* part_ml_of(const span_pool* p, float* part, size_t part_o_elems) {
  if (!part) return nullptr;
  return reinterpret_cast<float*>(reinterpret_cast<unsigned char*>(part) +
                                  part_o_elems * part_elem_bytes(p->cfg.dtype == SPAN_BF16));
}

// Make the rotary table cover positions [0, need).  Computed on the host in double
// precision (angle reduced to [-pi, pi] before cos/sin), rounded once to float, and
// copied on `stream`: kernels of this plan on that stream follow the copy, and
// launches on other streams wait for the plan's ready event.  The table it replaces
// is retired, not freed, since plans made before may still read it.
int ensure_rope_table(span_pool* p, int64_t need, hipStream_t stream) {
  if (need <= p->rope_n) return SPAN_OK;
  int64_t n = 4096;
  while (n < need) n *= 2;
  const int half = p->cfg.head_dim / 2;
  std::vector<float2> tab(static_cast<size_t>(n) * half);
  const double two_pi = 6.283185307179586476925;
  for (int i = 0; i < half; ++i) {
    const double f = std::pow(static_cast<double>(p->cfg.rope_theta), -2.0 * i / p->cfg.head_dim);
    for (int64_t pos = 0; pos < n; ++pos) {
      double a = static_cast<double>(pos) * f;
      a -= two_pi * std::nearbyint(a / two_pi);
      tab[static_cast<size_t>(pos) * half + i] = float2{static_cast<float>(std::cos(a)), static_cast<float>(std::sin(a))};
    }
  }
  float2* dev = nullptr;
  hipError_t e = hipMalloc(&dev, tab.size() * sizeof(float2));
  if (e == hipSuccess) e = hipMemcpyAsync(dev, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) {
    if (dev) (void)hipFree(dev);
    return hip_fail(e, "rotary table");
  }
  if (p->rope_tab) p->rope_retired.push_back(p->rope_tab);
  p->rope_host.push_back(std::move(tab));
  p->rope_tab = dev;
  p->rope_n = n;
  return SPAN_OK;
}

hipEvent_t take_order_event(span_pool* p) {
  if (!p->order_cache.empty()) {
    hipEvent_t e = p->order_cache.back();
    p->order_cache.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

struct span_plan_t {
  span_pool* pool = nullptr;
  Plan plan;
  hipStream_t stream = nullptr;
  std::vector<unsigned char> host_meta;
  unsigned char* dev_meta = nullptr;
  float* part = nullptr;  // partial O (fp16 O / l for bf16 pools, fp32 O otherwise) then partial (m, l)
  size_t part_o_elems = 0;
  // device views
  const KvPage* kv = nullptr;
  const TileRec* kt = nullptr;
  const NewPage* k3p = nullptr;
  const NewPage* k3c = nullptr;
  const WorkTile* tp = nullptr;
  const WorkTile* tc = nullptr;
  const CombineTile* cb = nullptr;
  const MovePage* mv = nullptr;
  const float2* rope = nullptr;
  // item counters of the span-prefill kernel: kSchedSlots groups of kSchedWords
  // words, zeroed at upload and left zeroed by each launch; launches take them in
  // turn, so up to kSchedSlots launches of one plan may overlap (on different streams)
  static constexpr int kSchedSlots = 64;
  unsigned* sched = nullptr;
  const int32_t* xch = nullptr;  // per-XCD chunk offsets of the prefill tiles
  int prefill_queues = 0;         // queues of the last MFMA prefill launch (8: per XCD)
  unsigned sched_next = 0;
  int bm = kGenericBM;
  bool mfma = false;
  bool committed = false;
  double host_plan_us = 0.0;    // hashing, lookup, allocation, work lists
  double host_upload_us = 0.0;  // device metadata allocation and copy enqueue
  // timing: groups of events recorded around each launch (SPAN_FLAG_TIMING)
  std::vector<std::vector<hipEvent_t>> ev_prefill, ev_cross;
  // Stream ordering.  The metadata (and a grown rotary table) are copied on the
  // plan's stream.  The first launch on another stream records `ready` on the plan's
  // stream and makes that stream wait for it; destroy makes the plan's stream wait
  // for every such stream before the metadata is freed there.
  hipEvent_t ready = nullptr;
  std::vector<hipStream_t> foreign;
  // Device data in a caller-side region (span_plan_static) instead of stream-ordered
  // allocations: nothing to free at destroy, and the region is released for the
  // next such plan on the device.
  bool in_scratch = false;
  // Nested generation (span_plan_decode, span_decode_attend).  The last decode
  // step's device data (metadata and split-KV partials, allocated on the decode
  // stream), its host copy (kept until that copy is known to be done), and the
  // events of decode attention calls made on other streams: the next step and
  // destroy make the decode stream wait for them before the data are freed.
  struct DecodeDev {
    unsigned char* meta = nullptr;
    float* part = nullptr;
    size_t part_o_elems = 0;
    const SlotWrite* writes = nullptr;
    const KvPage* kv = nullptr;
    const TileRec* kt = nullptr;
    const WorkTile* tiles = nullptr;
    const CombineTile* cb = nullptr;
    const float2* rope = nullptr;
  } dec;
  std::vector<unsigned char> dec_host;
  hipEvent_t dec_copied = nullptr;  // recorded after the upload of dec_host
  hipStream_t dec_stream = nullptr;
  hipEvent_t dec_ready = nullptr;   // recorded on dec_stream after the upload
  std::vector<hipEvent_t> dec_pending;
  bool decoding = false;            // decode steps planned: prefill and cross calls are over
  std::vector<std::vector<hipEvent_t>> ev_decode;
};

namespace {
// The plan whose device data occupy each device's scratch region (span_plan_static).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
span_plan_t* g_scratch_owner[kMaxDevices] = {};
}  // namespace

int spanq::pool_device(const span_pool* pool) { return pool ? pool->cfg.device : -1; }

int spanq::report(int code, const char* msg) { return fail(code, msg); }

span_pool* spanq::plan_pool(const span_plan_t* plan) { return plan ? plan->pool : nullptr; }

const PoolIndex* spanq::pool_index(const span_pool* pool) { return pool->index; }

void spanq::pool_shape(const span_pool* pool, int32_t out[5]) {
  const span_pool_config& c = pool->cfg;
  out[0] = c.num_layers;
  out[1] = c.num_q_heads;
  out[2] = c.num_kv_heads;
  out[3] = c.head_dim;
  out[4] = c.dtype;
}

void spanq::plan_last_cross_rows(const span_plan_t* plan, std::vector<int64_t>* rows) {
  rows->clear();
  for (const auto& ids : plan->plan.query_spans) {
    const SpanPlan& c = plan->plan.spans[ids.back()];
    rows->push_back(c.n_tok > 0 ? c.row + c.n_tok - 1 : -1);
  }
}

namespace {
// Records n+1 events around n launches; returns an empty vector if timing is off.
struct Timer {
  std::vector<hipEvent_t> ev;
  hipStream_t s;
  Timer(bool on, int n, hipStream_t st, std::vector<hipEvent_t>& cache) : s(st) {
    if (!on) return;
    ev.resize(n + 1, nullptr);
    for (auto& e : ev) {
      if (!cache.empty()) {
        e = cache.back();
        cache.pop_back();
      } else if (hipEventCreate(&e) != hipSuccess) {
        e = nullptr;
      }
    }
  }
  void mark(int i) {
    if (!ev.empty() && ev[i]) (void)hipEventRecord(ev[i], s);
  }
};
void release_events(std::vector<std::vector<hipEvent_t>>& groups, std::vector<hipEvent_t>& cache) {
  for (auto& g : groups)
    for (auto e : g)
      if (e) cache.push_back(e);
  groups.clear();
}
}  // namespace

static int check_span(const span_tokens& s, const char* what) {
  if (s.n < 0 || (s.n > 0 && !s.tokens)) return fail(SPAN_EINVAL, std::string("span_plan: bad ") + what);
  if (s.n > 0 && (s.row < 0 || s.row + s.n > std::numeric_limits<int32_t>::max()))
    return fail(SPAN_EINVAL, std::string("span_plan: ") + what + " rows must lie in [0, 2^31)");
  return SPAN_OK;
}

template <typename T>
static size_t put(std::vector<unsigned char>& buf, const std::vector<T>& v) {
  size_t at = (buf.size() + 255) & ~static_cast<size_t>(255);
  buf.resize(at + v.size() * sizeof(T));
  if (!v.empty()) std::memcpy(buf.data() + at, v.data(), v.size() * sizeof(T));
  return at;
}

int spanq::plan_impl(span_pool* pool, const span_query* qs, int32_t nq, void* stream, span_plan_t** out,
                     unsigned char* region, size_t region_bytes, const char* who) {
  if (!pool || !out || nq < 0 || (nq > 0 && !qs)) return fail(SPAN_EINVAL, std::string(who) + ": bad argument");
  *out = nullptr;
  std::vector<QueryIn> in(static_cast<size_t>(nq));
  for (int32_t i = 0; i < nq; ++i) {
    const span_query& q = qs[i];
    int rc = check_span(q.prefix, "prefix");
    if (!rc) rc = check_span(q.cross, "cross");
    if (rc) return rc;
    if (q.n_frags < 0 || (q.n_frags > 0 && !q.frags)) return fail(SPAN_EINVAL, "span_plan: bad fragment list");
    if (pool->cfg.hash_mode == SPAN_HASH_STOCK && (q.n_frags != 0 || q.cross.n != 0))
      return fail(SPAN_EINVAL, "span_plan: stock hashing takes prefix-only queries");
    in[i].prefix = SpanIn{q.prefix.tokens, q.prefix.n, q.prefix.row};
    in[i].cross = SpanIn{q.cross.tokens, q.cross.n, q.cross.row};
    for (int32_t f = 0; f < q.n_frags; ++f) {
      rc = check_span(q.frags[f], "fragment");
      if (rc) return rc;
      in[i].frags.push_back(SpanIn{q.frags[f].tokens, q.frags[f].n, q.frags[f].row});
    }
  }
  span_plan_t* pl = new (std::nothrow) span_plan_t();
  if (!pl) return fail(SPAN_ENOMEM, "span_plan: host allocation");
  pl->pool = pool;
  pl->stream = static_cast<hipStream_t>(stream);
  const bool device = pool->cfg.device >= 0;
  pl->mfma = device && pool->use_mfma;
  pl->bm = pl->mfma ? mfma_bm(pool->cfg.num_q_heads / pool->cfg.num_kv_heads) : kGenericBM;
  Tiling t = tiling_for(pl->mfma, pl->bm, pool->cfg.num_q_heads, pool->cfg.num_kv_heads);
  t.materialize = (pool->cfg.flags & SPAN_FLAG_MATERIALIZE) != 0;
  std::string msg;
  const auto t_plan0 = std::chrono::steady_clock::now();
  int rc = pool->index->plan(in, true, t, &pl->plan, &msg);
  const auto t_plan1 = std::chrono::steady_clock::now();
  pl->host_plan_us = std::chrono::duration<double, std::micro>(t_plan1 - t_plan0).count();
  if (rc) {
    delete pl;
    return fail(rc, msg);
  }
  pool->plans.insert(pl);
  if (device) {
    Plan& P = pl->plan;
    const int d = pool->cfg.head_dim;
    hipError_t e = hipSetDevice(pool->cfg.device);
    if (e != hipSuccess) {
      span_plan_destroy(pl);
      return hip_fail(e, (std::string(who) + ": hipSetDevice").c_str());
    }
    if (region) {
      // no allocation: the rotary table must already cover the plan's positions
      if (P.max_pos + 1 > pool->rope_n) {
        span_plan_destroy(pl);
        return fail(SPAN_EINVAL, std::string(who) + ": the pool's rotary table covers " + std::to_string(pool->rope_n) +
                                     " positions, the plan needs " + std::to_string(P.max_pos + 1) +
                                     " (one span_plan of that length grows it)");
      }
    } else {
      rc = ensure_rope_table(pool, P.max_pos + 1, pl->stream);
      if (rc) {
        span_plan_destroy(pl);
        return rc;
      }
    }
    pl->rope = pool->rope_tab;
    auto& hb = pl->host_meta;
    size_t o_kv = put(hb, P.kv), o_kt = put(hb, P.kv_tiles), o_k3p = put(hb, P.k3_prefill),
           o_k3c = put(hb, P.k3_cross);
    size_t o_tp = put(hb, P.t_prefill), o_tc = put(hb, P.t_cross), o_cb = put(hb, P.combine),
           o_mv = put(hb, P.moves);
    size_t o_sc = put(hb, std::vector<unsigned>(kSchedWords * span_plan_t::kSchedSlots, 0u));
    size_t o_xc = put(hb, P.prefill_chunks);
    pl->part_o_elems = static_cast<size_t>(P.n_parts) * pool->cfg.num_q_heads * pl->bm * d;
    const size_t part_bytes = pl->part_o_elems * part_elem_bytes(pool->cfg.dtype == SPAN_BF16) +
                              static_cast<size_t>(P.n_parts) * pool->cfg.num_q_heads * pl->bm * 2 * sizeof(float);
    if (region) {
      const size_t meta_bytes = (hb.size() + 255) & ~static_cast<size_t>(255);
      if (meta_bytes + part_bytes > region_bytes) {
        span_plan_destroy(pl);
        return fail(SPAN_EINVAL, std::string(who) + ": the plan needs " + std::to_string(meta_bytes + part_bytes) +
                                     " bytes of device scratch, the limit is " + std::to_string(region_bytes));
      }
      {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        const int dv = pool->cfg.device;
        if (dv >= kMaxDevices) {
          span_plan_destroy(pl);
          return fail(SPAN_EINVAL, std::string(who) + ": device ordinal too large");
        }
        if (g_scratch_owner[dv]) {
          span_plan_destroy(pl);
          return fail(SPAN_ESTATE, std::string(who) + ": another plan of this kind is alive on the device");
        }
        g_scratch_owner[dv] = pl;
      }
      pl->in_scratch = true;
      pl->dev_meta = region;
      if (P.n_parts > 0) pl->part = reinterpret_cast<float*>(region + meta_bytes);
      e = hipMemcpyAsync(pl->dev_meta, hb.data(), hb.size(), hipMemcpyHostToDevice, pl->stream);
    } else {
      e = hipMallocAsync(reinterpret_cast<void**>(&pl->dev_meta), hb.size(), pl->stream);
      if (e == hipSuccess) e = hipMemcpyAsync(pl->dev_meta, hb.data(), hb.size(), hipMemcpyHostToDevice, pl->stream);
      if (e == hipSuccess && P.n_parts > 0)
        e = hipMallocAsync(reinterpret_cast<void**>(&pl->part), part_bytes, pl->stream);
    }
    if (e != hipSuccess) {
      span_plan_destroy(pl);
      return hip_fail(e, (std::string(who) + ": device metadata").c_str());
    }
    pl->host_upload_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t_plan1).count();
    pl->kv = reinterpret_cast<const KvPage*>(pl->dev_meta + o_kv);
    pl->kt = reinterpret_cast<const TileRec*>(pl->dev_meta + o_kt);
    pl->k3p = reinterpret_cast<const NewPage*>(pl->dev_meta + o_k3p);
    pl->k3c = reinterpret_cast<const NewPage*>(pl->dev_meta + o_k3c);
    pl->tp = reinterpret_cast<const WorkTile*>(pl->dev_meta + o_tp);
    pl->tc = reinterpret_cast<const WorkTile*>(pl->dev_meta + o_tc);
    pl->cb = reinterpret_cast<const CombineTile*>(pl->dev_meta + o_cb);
    pl->mv = reinterpret_cast<const MovePage*>(pl->dev_meta + o_mv);
    pl->sched = reinterpret_cast<unsigned*>(pl->dev_meta + o_sc);
    pl->xch = reinterpret_cast<const int32_t*>(pl->dev_meta + o_xc);
  }
  *out = pl;
  return SPAN_OK;
}

extern "C" {

const char* span_last_error(void) { return g_last_error.c_str(); }

uint64_t span_hash_mix(uint64_t x) { return mix64(x); }

int span_pool_bytes(const span_pool_config* c, size_t* bytes) {
  if (!c || !bytes) return fail(SPAN_EINVAL, "span_pool_bytes: null argument");
  if (c->num_layers < 1 || c->num_pages < 1 || c->num_kv_heads < 1 || c->head_dim < 1 || c->page_size < 1)
    return fail(SPAN_EINVAL, "span_pool_bytes: sizes must be positive");
  *bytes = static_cast<size_t>(c->num_layers) * static_cast<size_t>(c->num_pages) * 2 *
           static_cast<size_t>(c->num_kv_heads) * static_cast<size_t>(c->page_size) *
           static_cast<size_t>(c->head_dim) * elem_size(c->dtype);
  return SPAN_OK;
}

int span_pool_create(const span_pool_config* c, span_pool** out) {
  if (!c || !out) return fail(SPAN_EINVAL, "span_pool_create: null argument");
  *out = nullptr;
  if (c->dtype != SPAN_F32 && c->dtype != SPAN_BF16) return fail(SPAN_EINVAL, "span_pool_create: dtype");
  if (c->num_layers < 1 || c->num_pages < 1 || c->num_pages > std::numeric_limits<int32_t>::max())
    return fail(SPAN_EINVAL, "span_pool_create: num_layers >= 1 and 1 <= num_pages < 2^31 required");
  if (c->num_q_heads < 1 || c->num_kv_heads < 1 || c->num_q_heads % c->num_kv_heads != 0)
    return fail(SPAN_EINVAL, "span_pool_create: num_q_heads must be a positive multiple of num_kv_heads");
  if (c->hash_mode != SPAN_HASH_SPAN && c->hash_mode != SPAN_HASH_STOCK)
    return fail(SPAN_EINVAL, "span_pool_create: hash_mode");
  if (c->page_size < 1) return fail(SPAN_EINVAL, "span_pool_create: page_size");
  if (c->device >= 0) {
    if (c->page_size != kPage) return fail(SPAN_EINVAL, "span_pool_create: device pools use 16-token pages");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(SPAN_EINVAL, "span_pool_create: head_dim 64 or 128");
    if (c->hash_mode != SPAN_HASH_SPAN) return fail(SPAN_EINVAL, "span_pool_create: stock hashing is host-only");
    if (!(c->rope_theta > 0.f)) return fail(SPAN_EINVAL, "span_pool_create: rope_theta must be positive");
    if (c->kernel == SPAN_KERNEL_MFMA && !mfma_supported(c->num_q_heads, c->num_kv_heads, c->head_dim, c->dtype))
      return fail(SPAN_EINVAL, "span_pool_create: the MFMA kernel does not support this dtype/shape");
  }
  if (c->kernel < SPAN_KERNEL_AUTO || c->kernel > SPAN_KERNEL_MFMA) return fail(SPAN_EINVAL, "span_pool_create: kernel");
  span_pool* p = new (std::nothrow) span_pool();
  if (!p) return fail(SPAN_ENOMEM, "span_pool_create: host allocation");
  p->cfg = *c;
  if (c->device >= 0) {
    size_t need = 0;
    span_pool_bytes(c, &need);
    hipError_t e = hipSetDevice(c->device);
    if (e != hipSuccess) {
      delete p;
      return hip_fail(e, "span_pool_create: hipSetDevice");
    }
    if (c->device_buf) {
      if (c->device_bytes < need) {
        delete p;
        return fail(SPAN_EINVAL, "span_pool_create: device_buf smaller than span_pool_bytes()");
      }
      p->dev = c->device_buf;
    } else {
      e = hipMalloc(&p->dev, need);
      if (e != hipSuccess) {
        delete p;
        return hip_fail(e, "span_pool_create: hipMalloc of page memory");
      }
      p->owns_dev = true;
    }
    // Plans take their metadata and split-KV partials from the device's stream-ordered
    // pool; keep freed blocks cached there instead of returning them at each sync.
    hipMemPool_t mp = nullptr;
    if (hipDeviceGetDefaultMemPool(&mp, c->device) == hipSuccess && mp) {
      uint64_t keep = UINT64_MAX;
      (void)hipMemPoolSetAttribute(mp, hipMemPoolAttrReleaseThreshold, &keep);
    }
    p->use_mfma = c->kernel == SPAN_KERNEL_MFMA ||
                  (c->kernel == SPAN_KERNEL_AUTO && mfma_supported(c->num_q_heads, c->num_kv_heads, c->head_dim, c->dtype));
    // the first 4096 positions of the rotary table, ready before any plan
    int rc = ensure_rope_table(p, 1, nullptr);
    if (rc == SPAN_OK && hipDeviceSynchronize() != hipSuccess) rc = fail(SPAN_EHIP, "span_pool_create: rotary table copy");
    if (rc != SPAN_OK) {
      if (p->rope_tab) (void)hipFree(p->rope_tab);
      if (p->owns_dev) (void)hipFree(p->dev);
      delete p;
      return rc;
    }
  }
  p->index = new (std::nothrow) PoolIndex(c->num_pages, c->page_size, c->hash_mode);
  if (!p->index) {
    if (p->owns_dev) (void)hipFree(p->dev);
    delete p;
    return fail(SPAN_ENOMEM, "span_pool_create: host allocation");
  }
  *out = p;
  return SPAN_OK;
}

int span_plan_destroy(span_plan_t* plan);

int span_pool_destroy(span_pool* p) {
  if (!p) return fail(SPAN_EINVAL, "span_pool_destroy: null pool");
  std::vector<span_plan_t*> live(p->plans.begin(), p->plans.end());
  for (span_plan_t* pl : live) span_plan_destroy(pl);
  if (p->cfg.device >= 0) (void)hipDeviceSynchronize();
  for (hipEvent_t e : p->event_cache) (void)hipEventDestroy(e);
  for (hipEvent_t e : p->order_cache) (void)hipEventDestroy(e);
  if (p->rope_tab) (void)hipFree(p->rope_tab);
  for (float2* t : p->rope_retired) (void)hipFree(t);
  if (p->owns_dev && p->dev) (void)hipFree(p->dev);
  delete p->index;
  delete p;
  return SPAN_OK;
}

int span_pool_reset(span_pool* p) {
  if (!p) return fail(SPAN_EINVAL, "span_pool_reset: null pool");
  for (const span_plan_t* pl : p->plans)
    if (!pl->committed) return fail(SPAN_ESTATE, "span_pool_reset: an uncommitted plan is alive");
  p->index->reset();
  return SPAN_OK;
}

int span_pool_get_info(const span_pool* p, span_pool_info* info) {
  if (!p || !info) return fail(SPAN_EINVAL, "span_pool_get_info: null argument");
  info->num_pages = p->index->num_pages();
  info->free_pages = p->index->free_count();
  info->cached_pages = p->index->cached_count();
  info->pinned_pages = p->index->pinned_count();
  info->tick = p->index->tick();
  info->total_evictions = p->index->total_evictions();
  return SPAN_OK;
}

int span_pool_page_address(const span_pool* p, int32_t layer, int32_t page_id, void** base, int64_t* off) {
  if (!p || !base || !off) return fail(SPAN_EINVAL, "span_pool_page_address: null argument");
  if (p->cfg.device < 0) return fail(SPAN_ESTATE, "span_pool_page_address: host-only pool");
  if (layer < 0 || layer >= p->cfg.num_layers || page_id < 0 || page_id >= p->cfg.num_pages)
    return fail(SPAN_EINVAL, "span_pool_page_address: layer or page out of range");
  const int64_t page_elems = 2ll * p->cfg.num_kv_heads * p->cfg.page_size * p->cfg.head_dim;
  *base = p->dev;
  *off = (static_cast<int64_t>(layer) * p->cfg.num_pages + page_id) * page_elems;
  return SPAN_OK;
}

int span_pool_read_page(const span_pool* p, int32_t layer, int32_t page_id, void* host_dst, size_t bytes) {
  void* base = nullptr;
  int64_t off = 0;
  int rc = span_pool_page_address(p, layer, page_id, &base, &off);
  if (rc) return rc;
  const size_t es = elem_size(p->cfg.dtype);
  const size_t page_bytes = 2ull * p->cfg.num_kv_heads * p->cfg.page_size * p->cfg.head_dim * es;
  if (!host_dst || bytes < page_bytes) return fail(SPAN_EINVAL, "span_pool_read_page: destination too small");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "span_pool_read_page: hipDeviceSynchronize");
  e = hipMemcpy(host_dst, static_cast<unsigned char*>(base) + off * es, page_bytes, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "span_pool_read_page: hipMemcpy");
  return SPAN_OK;
}

int span_hash_pages(uint64_t seed, const int32_t* tok, int32_t n, int32_t page_size, int32_t include_partial,
                    uint64_t* out, int32_t* n_pages) {
  if ((!tok && n > 0) || n < 0 || page_size < 1 || !n_pages || (!out && n > 0))
    return fail(SPAN_EINVAL, "span_hash_pages: bad argument");
  uint64_t h = seed;
  int32_t w = 0;
  for (int32_t p = 0; p * page_size < n; ++p) {
    int32_t cnt = std::min(page_size, n - p * page_size);
    if (cnt < page_size && !include_partial) break;
    h = page_hash(h, tok + static_cast<int64_t>(p) * page_size, cnt, p);
    out[w++] = h;
  }
  *n_pages = w;
  return SPAN_OK;
}

int kv_lookup(const span_pool* p, const uint64_t* hashes, int32_t n, int32_t* page_ids, int32_t* n_leading) {
  if (!p || n < 0 || (n > 0 && (!hashes || !page_ids)) || !n_leading)
    return fail(SPAN_EINVAL, "kv_lookup: bad argument");
  int32_t lead = 0;
  bool run = true;
  for (int32_t i = 0; i < n; ++i) {
    page_ids[i] = static_cast<int32_t>(p->index->lookup(hashes[i]));
    if (run && page_ids[i] >= 0) {
      ++lead;
    } else {
      run = false;
    }
  }
  *n_leading = lead;
  return SPAN_OK;
}

int span_plan(span_pool* pool, const span_query* qs, int32_t nq, void* stream, span_plan_t** out) {
  return spanq::plan_impl(pool, qs, nq, stream, out, nullptr, 0, "span_plan");
}

int span_plan_stats(const span_plan_t* pl, span_stats* s) {
  if (!pl || !s) return fail(SPAN_EINVAL, "span_plan_stats: null argument");
  const Plan& P = pl->plan;
  s->pages_hit = P.pages_hit;
  s->pages_new = P.pages_new;
  s->pages_cross = static_cast<int64_t>(P.cross_pages.size());
  s->pages_evicted = static_cast<int64_t>(P.evicted.size());
  s->tokens_hit = P.tokens_hit;
  s->tokens_new = P.tokens_new;
  s->tokens_cross = P.tokens_cross;
  s->prefill_pairs = P.prefill_pairs;
  s->cross_pairs = P.cross_pairs;
  s->prefill_tiles = static_cast<int64_t>(P.t_prefill.size());
  s->cross_tiles = static_cast<int64_t>(P.t_cross.size());
  s->kv_splits = P.kv_splits;
  s->cross_kv_pages = P.cross_kv_pages;
  s->host_plan_us = pl->host_plan_us;
  s->host_upload_us = pl->host_upload_us;
  s->pages_moved = static_cast<int64_t>(P.moves.size());
  int64_t moved_tok = 0;
  for (const MovePage& m : P.moves) moved_tok += m.n_valid;
  s->tokens_moved = moved_tok;
  s->prefill_queues = pl->prefill_queues;
  s->decode_steps = P.decode_steps;
  s->decode_tokens = P.decode_tokens;
  s->decode_pages = P.decode_pages;
  s->decode_pairs = P.dec.pairs;
  return SPAN_OK;
}

int span_plan_moves(const span_plan_t* pl, int32_t* rec, int32_t cap, int32_t* n) {
  if (!pl || !n || cap < 0 || (cap > 0 && !rec)) return fail(SPAN_EINVAL, "span_plan_moves: bad argument");
  const auto& mv = pl->plan.moves;
  *n = static_cast<int32_t>(mv.size());
  for (int32_t i = 0; i < *n && i < cap; ++i) {
    rec[4 * i] = mv[i].src_page;
    rec[4 * i + 1] = mv[i].dst_page;
    rec[4 * i + 2] = mv[i].delta;
    rec[4 * i + 3] = mv[i].n_valid;
  }
  return SPAN_OK;
}

int span_plan_block_table(const span_plan_t* pl, int32_t query, int32_t span, int32_t* ids, int32_t cap, int32_t* n,
                          int32_t* n_hit) {
  if (!pl || !n || !n_hit || cap < 0 || (cap > 0 && !ids)) return fail(SPAN_EINVAL, "span_plan_block_table: bad argument");
  const Plan& P = pl->plan;
  if (query < 0 || query >= static_cast<int32_t>(P.query_spans.size()))
    return fail(SPAN_EINVAL, "span_plan_block_table: query out of range");
  const auto& sp = P.query_spans[query];
  const int32_t nfr = static_cast<int32_t>(sp.size()) - 2;
  if (span < -1 || span > nfr) return fail(SPAN_EINVAL, "span_plan_block_table: span out of range");
  const SpanPlan& s = P.spans[sp[span + 1]];
  *n = static_cast<int32_t>(s.pages.size());
  *n_hit = s.n_hit;
  for (int32_t i = 0; i < std::min(cap, *n); ++i) ids[i] = s.pages[i];
  return SPAN_OK;
}

int span_plan_evicted(const span_plan_t* pl, int32_t* ids, int32_t cap, int32_t* n) {
  if (!pl || !n || cap < 0 || (cap > 0 && !ids)) return fail(SPAN_EINVAL, "span_plan_evicted: bad argument");
  const auto& ev = pl->plan.evicted;
  *n = static_cast<int32_t>(ev.size());
  for (int32_t i = 0; i < std::min(cap, *n); ++i) ids[i] = ev[i];
  return SPAN_OK;
}

int span_plan_rows(const span_plan_t* pl, int64_t* rows, int64_t cap, int64_t* n_prefill, int64_t* n_cross) {
  if (!pl || !n_prefill || !n_cross || cap < 0 || (cap > 0 && !rows)) return fail(SPAN_EINVAL, "span_plan_rows: bad argument");
  const Plan& P = pl->plan;
  *n_prefill = 0;
  *n_cross = 0;
  for (const auto& rr : P.rows_prefill) *n_prefill += rr.n;
  for (const auto& rr : P.rows_cross) *n_cross += rr.n;
  int64_t w = 0;
  for (const auto* runs : {&P.rows_prefill, &P.rows_cross})
    for (const auto& rr : *runs)
      for (int32_t j = 0; j < rr.n && w < cap; ++j) rows[w++] = rr.row0 + j;
  return SPAN_OK;
}

// Launches on a stream other than the plan's wait for the plan's uploads.
static int order_after_upload(span_plan_t* pl, hipStream_t s, const char* who) {
  if (s == pl->stream) return SPAN_OK;
  if (std::find(pl->foreign.begin(), pl->foreign.end(), s) == pl->foreign.end()) {
    if (!pl->ready) {
      pl->ready = take_order_event(pl->pool);
      if (!pl->ready) return fail(SPAN_EHIP, std::string(who) + ": event creation");
      hipError_t e = hipEventRecord(pl->ready, pl->stream);
      if (e != hipSuccess) return hip_fail(e, who);
    }
    pl->foreign.push_back(s);
  }
  hipError_t e = hipStreamWaitEvent(s, pl->ready, 0);
  if (e != hipSuccess) return hip_fail(e, who);
  return SPAN_OK;
}

static int attention_common(span_plan_t* pl, int32_t layer, const char* who) {
  if (!pl) return fail(SPAN_EINVAL, std::string(who) + ": null plan");
  if (pl->pool->cfg.device < 0) return fail(SPAN_ESTATE, std::string(who) + ": host-only pool");
  if (pl->committed) return fail(SPAN_ESTATE, std::string(who) + ": plan already committed");
  if (layer < 0 || layer >= pl->pool->cfg.num_layers) return fail(SPAN_EINVAL, std::string(who) + ": layer out of range");
  return SPAN_OK;
}

static PoolGeom geom(const span_plan_t* pl, int32_t layer) {
  const span_pool_config& c = pl->pool->cfg;
  const int64_t page_elems = 2ll * c.num_kv_heads * c.page_size * c.head_dim;
  return PoolGeom{pl->pool->dev, static_cast<int64_t>(layer) * c.num_pages * page_elems, c.num_q_heads,
                  c.num_kv_heads, c.head_dim, c.dtype};
}

int span_prefill_fragments(span_plan_t* pl, int32_t layer, const void* q, const void* k, const void* v, void* out,
                           void* stream) {
  int rc = attention_common(pl, layer, "span_prefill_fragments");
  if (rc) return rc;
  if (pl->decoding) return fail(SPAN_ESTATE, "span_prefill_fragments: the plan has decode steps");
  const Plan& P = pl->plan;
  if (P.k3_prefill.empty() && P.t_prefill.empty()) return SPAN_OK;
  if (!q || !k || !v || !out) return fail(SPAN_EINVAL, "span_prefill_fragments: null activation pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  rc = order_after_upload(pl, s, "span_prefill_fragments");
  if (rc) return rc;
  PoolGeom g = geom(pl, layer);
  Timer tm((pl->pool->cfg.flags & SPAN_FLAG_TIMING) != 0, 2, s, pl->pool->event_cache);
  tm.mark(0);
  hipError_t e = launch_rope_write(g, pl->k3p, static_cast<int>(P.k3_prefill.size()), k, v, pl->rope, s);
  if (e != hipSuccess) return hip_fail(e, "span_prefill_fragments: page write");
  tm.mark(1);
  const int nt = static_cast<int>(P.t_prefill.size());
  unsigned* sched = pl->sched + kSchedWords * (pl->sched_next++ % span_plan_t::kSchedSlots);
  const int nch = P.prefill_chunks.empty() ? 0 : static_cast<int>(P.prefill_chunks.size()) - 1;
  e = pl->mfma ? launch_prefill_mfma(g, pl->tp, nt, pl->kt, q, out, pl->rope, sched, P.prefill_chunks.data(),
                                     pl->xch, nch, &pl->prefill_queues, s)
               : launch_attn_generic(g, pl->tp, nt, pl->kv, q, out, nullptr, nullptr, pl->rope, s);
  if (e != hipSuccess) return hip_fail(e, "span_prefill_fragments: attention");
  tm.mark(2);
  if (!tm.ev.empty()) pl->ev_prefill.push_back(tm.ev);
  return SPAN_OK;
}

int span_cross_attend(span_plan_t* pl, int32_t layer, const void* q, const void* k, const void* v, void* out,
                      void* stream) {
  int rc = attention_common(pl, layer, "span_cross_attend");
  if (rc) return rc;
  if (pl->decoding) return fail(SPAN_ESTATE, "span_cross_attend: the plan has decode steps");
  const Plan& P = pl->plan;
  if (P.t_cross.empty()) return SPAN_OK;
  if (!q || !k || !v || !out) return fail(SPAN_EINVAL, "span_cross_attend: null activation pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  rc = order_after_upload(pl, s, "span_cross_attend");
  if (rc) return rc;
  PoolGeom g = geom(pl, layer);
  Timer tm((pl->pool->cfg.flags & SPAN_FLAG_TIMING) != 0, 4, s, pl->pool->event_cache);
  tm.mark(0);
  // The MFMA cross kernel writes the cross-segment pages itself when every cross tile
  // is its own (none on the 16-row kernel); otherwise they are written first.
  const bool fused = pl->mfma && P.n_cross_few == 0 && !P.k3_cross.empty();
  hipError_t e =
      fused ? hipSuccess : launch_rope_write(g, pl->k3c, static_cast<int>(P.k3_cross.size()), k, v, pl->rope, s);
  if (e != hipSuccess) return hip_fail(e, "span_cross_attend: page write");
  tm.mark(1);
  // materialised repositioning: this layer's copies of shifted pages, keys rotated
  // to the final positions (the cross key lists name the copies, delta 0)
  e = launch_move_pages(g, pl->mv, static_cast<int>(P.moves.size()), pl->rope, s);
  if (e != hipSuccess) return hip_fail(e, "span_cross_attend: page moves");
  tm.mark(2);
  void* po = pl->part;
  float* pml = part_ml_of(pl->pool, pl->part, pl->part_o_elems);
  const int nt = static_cast<int>(P.t_cross.size());
  if (pl->mfma) {
    // the last n_cross_few tiles (few rows, two key groups) on the 16-row kernel
    const int nf = P.n_cross_few;
    CrossWrites w;
    if (fused) w = CrossWrites{pl->k3c, k, v};
    e = launch_attn_mfma(g, pl->tc, nt - nf, pl->kt, q, out, po, pml, pl->rope, w, s);
    if (e == hipSuccess && nf > 0) e = launch_few_mfma(g, pl->tc + (nt - nf), nf, pl->kt, q, po, pml, pl->rope, s);
  } else {
    e = launch_attn_generic(g, pl->tc, nt, pl->kv, q, out, po, pml, pl->rope, s);
  }
  if (e != hipSuccess) return hip_fail(e, "span_cross_attend: attention");
  tm.mark(3);
  e = launch_combine(g, pl->cb, static_cast<int>(P.combine.size()), po, pml, pl->bm, max_parts(P.combine), out, s);
  if (e != hipSuccess) return hip_fail(e, "span_cross_attend: combine");
  tm.mark(4);
  if (!tm.ev.empty()) pl->ev_cross.push_back(tm.ev);
  return SPAN_OK;
}

// Make stream s wait for the decode data's last readers: attention calls on other
// streams (their events) and the previous decode stream.
static int decode_drain(span_plan_t* pl, hipStream_t s, const char* who) {
  for (hipEvent_t ev : pl->dec_pending) {
    hipError_t e = hipStreamWaitEvent(s, ev, 0);
    pl->pool->order_cache.push_back(ev);
    if (e != hipSuccess) {
      pl->dec_pending.clear();
      return hip_fail(e, who);
    }
  }
  pl->dec_pending.clear();
  if (pl->dec_stream && pl->dec_stream != s) {
    hipEvent_t ev = take_order_event(pl->pool);
    if (!ev) return fail(SPAN_EHIP, std::string(who) + ": event creation");
    hipError_t e = hipEventRecord(ev, pl->dec_stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, ev, 0);
    pl->pool->order_cache.push_back(ev);
    if (e != hipSuccess) return hip_fail(e, who);
  }
  return SPAN_OK;
}

int span_plan_decode(span_plan_t* pl, const int32_t* n_new, const int64_t* rows, void* stream) {
  if (!pl) return fail(SPAN_EINVAL, "span_plan_decode: null plan");
  if (pl->committed) return fail(SPAN_ESTATE, "span_plan_decode: plan already committed");
  if (pl->in_scratch) return fail(SPAN_EINVAL, "span_plan_decode: decode steps allocate; not for span_plan_static plans");
  Plan& P = pl->plan;
  const size_t nq = P.query_spans.size();
  if (nq > 0 && (!n_new || !rows)) return fail(SPAN_EINVAL, "span_plan_decode: null argument");
  std::vector<int32_t> n(n_new, n_new + nq);
  std::vector<int64_t> r(rows, rows + nq);
  span_pool* pool = pl->pool;
  Tiling t = tiling_for(pl->mfma, pl->bm, pool->cfg.num_q_heads, pool->cfg.num_kv_heads);
  t.materialize = (pool->cfg.flags & SPAN_FLAG_MATERIALIZE) != 0;
  std::string msg;
  int rc = pool->index->decode(&P, n, r, t, &msg);
  if (rc) return fail(rc, "span_plan_decode: " + msg);
  pl->decoding = true;
  if (pool->cfg.device < 0) return SPAN_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSetDevice(pool->cfg.device);
  if (e != hipSuccess) return hip_fail(e, "span_plan_decode: hipSetDevice");
  // the previous step's device data are freed once their readers are done
  rc = decode_drain(pl, s, "span_plan_decode");
  if (rc) return rc;
  if (pl->dec.meta) (void)hipFreeAsync(pl->dec.meta, s);
  if (pl->dec.part) (void)hipFreeAsync(pl->dec.part, s);
  pl->dec = span_plan_t::DecodeDev{};
  rc = ensure_rope_table(pool, P.max_pos + 1, s);
  if (rc) return rc;
  // the host copy of the previous upload is reused once that upload is done
  if (pl->dec_copied && hipEventSynchronize(pl->dec_copied) != hipSuccess)
    return fail(SPAN_EHIP, "span_plan_decode: wait for the previous upload");
  const Plan::DecodeStep& d = P.dec;
  auto& hb = pl->dec_host;
  hb.clear();
  const size_t o_w = put(hb, d.writes), o_kv = put(hb, d.kv), o_kt = put(hb, d.kv_tiles), o_t = put(hb, d.tiles),
               o_cb = put(hb, d.combine);
  hb.resize((hb.size() + 255) & ~static_cast<size_t>(255));
  e = hipMallocAsync(reinterpret_cast<void**>(&pl->dec.meta), hb.size(), s);
  if (e == hipSuccess) e = hipMemcpyAsync(pl->dec.meta, hb.data(), hb.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !pl->dec_copied) e = hipEventCreateWithFlags(&pl->dec_copied, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(pl->dec_copied, s);
  pl->dec.part_o_elems = static_cast<size_t>(d.n_parts) * pool->cfg.num_q_heads * pl->bm * pool->cfg.head_dim;
  const size_t part_bytes = pl->dec.part_o_elems * part_elem_bytes(pool->cfg.dtype == SPAN_BF16) +
                            static_cast<size_t>(d.n_parts) * pool->cfg.num_q_heads * pl->bm * 2 * sizeof(float);
  if (e == hipSuccess && d.n_parts > 0) e = hipMallocAsync(reinterpret_cast<void**>(&pl->dec.part), part_bytes, s);
  if (e == hipSuccess && !pl->dec_ready) {
    pl->dec_ready = take_order_event(pool);
    if (!pl->dec_ready) e = hipErrorOutOfMemory;
  }
  if (e == hipSuccess) e = hipEventRecord(pl->dec_ready, s);
  if (e != hipSuccess) return hip_fail(e, "span_plan_decode: device metadata");
  pl->dec_stream = s;
  pl->dec.writes = reinterpret_cast<const SlotWrite*>(pl->dec.meta + o_w);
  pl->dec.kv = reinterpret_cast<const KvPage*>(pl->dec.meta + o_kv);
  pl->dec.kt = reinterpret_cast<const TileRec*>(pl->dec.meta + o_kt);
  pl->dec.tiles = reinterpret_cast<const WorkTile*>(pl->dec.meta + o_t);
  pl->dec.cb = reinterpret_cast<const CombineTile*>(pl->dec.meta + o_cb);
  pl->dec.rope = pool->rope_tab;
  return SPAN_OK;
}

int span_decode_attend(span_plan_t* pl, int32_t layer, const void* q, const void* k, const void* v, void* out,
                       void* stream) {
  int rc = attention_common(pl, layer, "span_decode_attend");
  if (rc) return rc;
  if (!pl->dec.meta) return fail(SPAN_ESTATE, "span_decode_attend: no decode step planned");
  const Plan::DecodeStep& d = pl->plan.dec;
  if (d.tokens == 0) return SPAN_OK;
  if (!q || !k || !v || !out) return fail(SPAN_EINVAL, "span_decode_attend: null activation pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool foreign = s != pl->dec_stream;
  if (foreign) {
    hipError_t e = hipStreamWaitEvent(s, pl->dec_ready, 0);
    if (e != hipSuccess) return hip_fail(e, "span_decode_attend: stream order");
  }
  PoolGeom g = geom(pl, layer);
  Timer tm((pl->pool->cfg.flags & SPAN_FLAG_TIMING) != 0, 1, s, pl->pool->event_cache);
  tm.mark(0);
  hipError_t e = launch_append_kv(g, pl->dec.writes, static_cast<int>(d.writes.size()), k, v, pl->dec.rope, s);
  if (e != hipSuccess) return hip_fail(e, "span_decode_attend: page write");
  void* po = pl->dec.part;
  float* pml = part_ml_of(pl->pool, pl->dec.part, pl->dec.part_o_elems);
  const int nt = static_cast<int>(d.tiles.size());
  if (pl->mfma) {
    const int nf = d.n_few;
    e = launch_attn_mfma(g, pl->dec.tiles, nt - nf, pl->dec.kt, q, out, po, pml, pl->dec.rope, CrossWrites{}, s);
    if (e == hipSuccess && nf > 0)
      e = launch_few_mfma(g, pl->dec.tiles + (nt - nf), nf, pl->dec.kt, q, po, pml, pl->dec.rope, s);
  } else {
    e = launch_attn_generic(g, pl->dec.tiles, nt, pl->dec.kv, q, out, po, pml, pl->dec.rope, s);
  }
  if (e != hipSuccess) return hip_fail(e, "span_decode_attend: attention");
  e = launch_combine(g, pl->dec.cb, static_cast<int>(d.combine.size()), po, pml, pl->bm, max_parts(d.combine), out, s);
  if (e != hipSuccess) return hip_fail(e, "span_decode_attend: combine");
  tm.mark(1);
  if (!tm.ev.empty()) pl->ev_decode.push_back(tm.ev);
  if (foreign) {
    hipEvent_t ev = take_order_event(pl->pool);
    if (!ev) return fail(SPAN_EHIP, "span_decode_attend: event creation");
    e = hipEventRecord(ev, s);
    pl->dec_pending.push_back(ev);
    if (e != hipSuccess) return hip_fail(e, "span_decode_attend: stream order");
  }
  return SPAN_OK;
}

static float elapsed(hipEvent_t a, hipEvent_t b) {
  float ms = 0.f;
  if (!a || !b || hipEventSynchronize(b) != hipSuccess || hipEventElapsedTime(&ms, a, b) != hipSuccess) return 0.f;
  return ms;
}

int span_plan_kernel_times(const span_plan_t* pl, span_kernel_times* t) {
  if (!pl || !t) return fail(SPAN_EINVAL, "span_plan_kernel_times: null argument");
  std::memset(t, 0, sizeof(*t));
  for (const auto& ev : pl->ev_prefill) {
    t->page_write_prefill_ms += elapsed(ev[0], ev[1]);
    t->prefill_attention_ms += elapsed(ev[1], ev[2]);
    t->prefill_calls += 1;
  }
  for (const auto& ev : pl->ev_cross) {
    t->page_write_cross_ms += elapsed(ev[0], ev[1]);
    t->page_move_ms += elapsed(ev[1], ev[2]);
    t->cross_attention_ms += elapsed(ev[2], ev[3]);
    t->combine_ms += elapsed(ev[3], ev[4]);
    t->cross_calls += 1;
  }
  for (const auto& ev : pl->ev_decode) {
    t->decode_ms += elapsed(ev[0], ev[1]);
    t->decode_calls += 1;
  }
  return SPAN_OK;
}

int span_plan_commit(span_plan_t* pl) {
  if (!pl) return fail(SPAN_EINVAL, "span_plan_commit: null plan");
  if (pl->committed) return fail(SPAN_ESTATE, "span_plan_commit: already committed");
  pl->pool->index->commit(&pl->plan);
  pl->committed = true;
  return SPAN_OK;
}

int span_plan_destroy(span_plan_t* pl) {
  if (!pl) return fail(SPAN_EINVAL, "span_plan_destroy: null plan");
  if (!pl->committed) pl->pool->index->release(&pl->plan);
  release_events(pl->ev_prefill, pl->pool->event_cache);
  release_events(pl->ev_cross, pl->pool->event_cache);
  release_events(pl->ev_decode, pl->pool->event_cache);
  // decode data: wait for their readers on the plan's stream, then free there
  if (pl->dec.meta || !pl->dec_pending.empty()) (void)decode_drain(pl, pl->stream, "span_plan_destroy");
  if (pl->dec.meta) (void)hipFreeAsync(pl->dec.meta, pl->stream);
  if (pl->dec.part) (void)hipFreeAsync(pl->dec.part, pl->stream);
  if (pl->dec_ready) pl->pool->order_cache.push_back(pl->dec_ready);
  if (pl->dec_copied) {
    (void)hipEventSynchronize(pl->dec_copied);
    (void)hipEventDestroy(pl->dec_copied);
  }
  // work enqueued on other streams must end before the plan's memory is released
  for (hipStream_t s : pl->foreign) {
    hipEvent_t ev = take_order_event(pl->pool);
    if (ev && hipEventRecord(ev, s) == hipSuccess) (void)hipStreamWaitEvent(pl->stream, ev, 0);
    if (ev) pl->pool->order_cache.push_back(ev);
  }
  if (pl->ready) pl->pool->order_cache.push_back(pl->ready);
  if (pl->in_scratch) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    g_scratch_owner[pl->pool->cfg.device] = nullptr;
  } else {
    if (pl->dev_meta) (void)hipFreeAsync(pl->dev_meta, pl->stream);
    if (pl->part) (void)hipFreeAsync(pl->part, pl->stream);
  }
  pl->pool->plans.erase(pl);
  delete pl;
  return SPAN_OK;
}

}  // extern "C"

namespace {
// One untimed launch, then reps launches between two events on stream s; the
// elapsed time in seconds.
template <class Launch>
int time_launches(Launch launch, int reps, hipStream_t s, const char* what, double* sec) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = launch();
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  for (int i = 0; e == hipSuccess && i < reps; ++i) e = launch();
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (e != hipSuccess) return hip_fail(e, what);
  *sec = 1e-3 * ms;
  return SPAN_OK;
}
}  // namespace

extern "C" {

int span_probe_mfma_peak(int32_t iters, int32_t reps, void* stream, double* tflops) {
  if (iters < 1 || reps < 1 || !tflops) return fail(SPAN_EINVAL, "span_probe_mfma_peak: bad argument");
  int n_cu = 0;
  hipError_t e = cu_count(&n_cu);
  if (e != hipSuccess) return hip_fail(e, "span_probe_mfma_peak: device attributes");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  double sec = 0.0;
  const int rc = time_launches([&] { return launch_probe_mfma(iters, n_cu, s); }, reps, s,
                               "span_probe_mfma_peak", &sec);
  if (rc != SPAN_OK) return rc;
  *tflops = probe_mfma_flops(iters, n_cu) * reps / sec * 1e-12;
  return SPAN_OK;
}

int span_probe_read_peak(const void* buf, size_t bytes, int32_t reps, void* stream, double* gbs) {
  if (!buf || reinterpret_cast<uintptr_t>(buf) % 16 != 0 || bytes == 0 || bytes % 16 != 0 || reps < 1 || !gbs)
    return fail(SPAN_EINVAL, "span_probe_read_peak: bad argument");
  int n_cu = 0;
  hipError_t e = cu_count(&n_cu);
  if (e != hipSuccess) return hip_fail(e, "span_probe_read_peak: device attributes");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  double sec = 0.0;
  const int rc = time_launches([&] { return launch_probe_read(buf, static_cast<int64_t>(bytes), n_cu, s); }, reps,
                               s, "span_probe_read_peak", &sec);
  if (rc != SPAN_OK) return rc;
  *gbs = static_cast<double>(bytes) * reps / sec * 1e-9;
  return SPAN_OK;
}

}  // extern "C"
