// Decoder stack around span attention: the model the span query's prefill runs
// through (the harness of the attention path).  Per layer, over the rows a plan
// computes (new prefix/fragment tokens, then cross tokens):
//
//   n = RMSNorm(x) g_attn; qkv = n W_qkv            hipBLASLt GEMM, bf16 out
//   q, k, v -> caller rows; span_prefill_fragments and span_cross_attend
//   x = x + o W_o                                    GEMM with the residual as C (beta 1)
//   n = RMSNorm(x) g_ffn; gu = n W_gate_up           GEMM
//   x = x + (silu(gate) * up) W_down                 SwiGLU kernel, GEMM with residual
//
// then the final RMSNorm of each query's last cross row, the LM head and the
// argmax (the first generated token).  GEMMs of at most 8 rows (decode steps) run
// on GEMV kernels of our own (HBM-bound: each weight read once), long reductions
// (the down projection) of 129..256 rows (a cache-hit query's question) on an MFMA
// kernel of our own that streams a transposed copy of the weights once with K split
// over the chip, the rest on hipBLASLt.  Rows that hit the cache are never
// computed: their keys and values are already in the pool's pages, which is the
// point of the method (section 5.6).
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <map>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "../../include/spanq.h"
#include "capi_internal.h"
#include "stack_kernels.h"

using namespace spanq;

namespace {

int hip_err(hipError_t e, const std::string& what) {
  return report(SPAN_EHIP, (what + ": " + hipGetErrorString(e)).c_str());
}

int lt_err(hipblasStatus_t st, const std::string& what) {
  return report(SPAN_EHIP, (what + ": hipBLASLt status " + std::to_string(static_cast<int>(st))).c_str());
}

// A device buffer that only grows (callers synchronise before it is replaced).
struct Buf {
  void* p = nullptr;
  size_t cap = 0;
  hipError_t ensure(size_t bytes) {
    if (bytes <= cap) return hipSuccess;
    if (p) {
      hipError_t e = hipFree(p);
      if (e != hipSuccess) return e;
      p = nullptr;
      cap = 0;
    }
    hipError_t e = hipMalloc(&p, bytes);
    if (e == hipSuccess) cap = bytes;
    return e;
  }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    cap = 0;
  }
  template <class T>
  T* as() const { return static_cast<T*>(p); }
};

// Row-major Y[M][N] = X[M][K] W[K][N] (+ Y when residual), bf16 in and out, fp32
// accumulation.  In hipBLASLt's column-major terms this is Y^T = W^T X^T: its A is W
// seen as an N x K matrix, its B is X seen as K x M, and its D is Y seen as N x M.
// Each (M, N, K) takes the heuristic's first choice.  That choice, and even one
// algorithm's split of the K loop, depend on M, so a row's result may change in its
// last bits with the number of rows computed together.
struct Gemm {
  hipblasLtHandle_t h = nullptr;
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  Buf ws;
  size_t ws_bytes = size_t{64} << 20;
  struct Plan {
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    hipblasLtMatmulAlgo_t algo{};
    size_t ws = 0;
  };
  std::map<std::tuple<int64_t, int64_t, int64_t, bool>, Plan> plans;
  // Up to 8 rows (decode steps) go to the GEMV kernels instead, with this fp32
  // scratch for their partial sums (sized by the caller before the launches); the
  // shapes skinny_gemm_fits takes to the skinny MFMA kernel when the weight has a
  // transposed copy, with sk_part for its K-slice partials.
  Buf gemv_part, sk_part;

  int init() {
    hipblasStatus_t st = hipblasLtCreate(&h);
    if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtCreate");
    st = hipblasLtMatmulDescCreate(&desc, HIPBLAS_COMPUTE_32F, HIP_R_32F);
    if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtMatmulDescCreate");
    st = hipblasLtMatmulPreferenceCreate(&pref);
    if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtMatmulPreferenceCreate");
    uint64_t wsb = ws_bytes;
    st = hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof(wsb));
    if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtMatmulPreferenceSetAttribute");
    hipError_t e = ws.ensure(ws_bytes);
    if (e != hipSuccess) return hip_err(e, "GEMM workspace");
    return SPAN_OK;
  }

  void destroy() {
    for (auto& kv : plans) {
      hipblasLtMatrixLayoutDestroy(kv.second.a);
      hipblasLtMatrixLayoutDestroy(kv.second.b);
      hipblasLtMatrixLayoutDestroy(kv.second.c);
    }
    plans.clear();
    gemv_part.release();
    sk_part.release();
    if (pref) hipblasLtMatmulPreferenceDestroy(pref);
    if (desc) hipblasLtMatmulDescDestroy(desc);
    if (h) hipblasLtDestroy(h);
    ws.release();
  }

  // wt: W^T [N][K], or null when the weight has no transposed copy
  // every GEMV of a layer of M rows fits the scratch (decode-sized M)
  bool gemv_layer(int64_t M, int64_t qkv_w, int64_t H, int64_t F, int64_t attn_w) const {
    if (M < 1 || M > 8) return false;
    const int m = static_cast<int>(M);
    return qkv_w % 8 == 0 && H % 8 == 0 && F % 8 == 0 &&
           gemv_part_bytes(m, static_cast<int>(qkv_w), static_cast<int>(H)) <= gemv_part.cap &&
           gemv_part_bytes(m, static_cast<int>(H), static_cast<int>(attn_w)) <= gemv_part.cap &&
           gemv_part_bytes(m, static_cast<int>(2 * F), static_cast<int>(H)) <= gemv_part.cap &&
           gemv_part_bytes(m, static_cast<int>(H), static_cast<int>(F)) <= gemv_part.cap;
  }

  // y += x W, then nout = RMSNorm(y) * gain in the same second pass when the skinny
  // kernel takes the shape with K split (bit for bit run + launch_rmsnorm); *fused
  // tells whether it did (otherwise only y += x W was done).
  int run_norm(const void* x, const void* w, const void* wt, void* y, int64_t M, int64_t N, int64_t K,
               const void* gain, void* nout, float eps, bool* fused, hipStream_t s) {
    *fused = false;
    if (wt && skinny_gemm_fits(M, N, K) && skinny_gemm_slices(static_cast<int>(M), static_cast<int>(N),
                                                              static_cast<int>(K)) > 1 &&
        skinny_gemm_part_bytes(static_cast<int>(M), static_cast<int>(N), static_cast<int>(K)) <= sk_part.cap) {
      hipError_t e = launch_skinny_gemm_norm(x, wt, y, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K),
                                             gain, nout, eps, sk_part.as<float>(), sk_part.cap, s);
      if (e != hipSuccess) return hip_err(e, "skinny GEMM with norm");
      *fused = true;
      return SPAN_OK;
    }
    return run(x, w, wt, y, M, N, K, true, s);
  }

  int run(const void* x, const void* w, const void* wt, void* y, int64_t M, int64_t N, int64_t K, bool residual,
          hipStream_t s) {
    if (M == 0) return SPAN_OK;
    if (wt && skinny_gemm_fits(M, N, K) &&
        skinny_gemm_part_bytes(static_cast<int>(M), static_cast<int>(N), static_cast<int>(K)) <= sk_part.cap) {
      hipError_t e = launch_skinny_gemm(x, wt, y, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K),
                                        residual, sk_part.as<float>(), sk_part.cap, s);
      if (e != hipSuccess) return hip_err(e, "skinny GEMM");
      return SPAN_OK;
    }
    if (M <= 8 && N % 8 == 0 && gemv_part_bytes(static_cast<int>(M), static_cast<int>(N), static_cast<int>(K)) <=
                                    gemv_part.cap) {
      hipError_t e = launch_gemv(x, w, y, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K), residual,
                                 gemv_part.as<float>(), gemv_part.cap, s);
      if (e != hipSuccess) return hip_err(e, "GEMV");
      return SPAN_OK;
    }
    auto key = std::make_tuple(M, N, K, residual);
    auto it = plans.find(key);
    if (it == plans.end()) {
      Plan p;
      hipblasStatus_t st = hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, N, K, N);
      if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, K, M, K);
      if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatrixLayoutCreate(&p.c, HIP_R_16BF, N, M, N);
      if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtMatrixLayoutCreate");
      hipblasLtMatmulHeuristicResult_t res[1];
      int n = 0;
      st = hipblasLtMatmulAlgoGetHeuristic(h, desc, p.a, p.b, p.c, p.c, pref, 1, res, &n);
      if (st != HIPBLAS_STATUS_SUCCESS || n < 1 || res[0].workspaceSize > ws_bytes) {
        hipblasLtMatrixLayoutDestroy(p.a);
        hipblasLtMatrixLayoutDestroy(p.b);
        hipblasLtMatrixLayoutDestroy(p.c);
        return report(SPAN_EHIP, ("hipBLASLt: no algorithm for M=" + std::to_string(M) + " N=" + std::to_string(N) +
                                  " K=" + std::to_string(K)).c_str());
      }
      p.algo = res[0].algo;
      p.ws = res[0].workspaceSize;
      it = plans.emplace(key, p).first;
    }
    const float alpha = 1.f, beta = residual ? 1.f : 0.f;
    const Plan& p = it->second;
    hipblasStatus_t st = hipblasLtMatmul(h, desc, &alpha, w, p.a, x, p.b, &beta, y, p.c, y, p.c, &p.algo, ws.p,
                                         p.ws ? ws_bytes : 0, s);
    if (st != HIPBLAS_STATUS_SUCCESS) return lt_err(st, "hipblasLtMatmul");
    return SPAN_OK;
  }
};

}  // namespace

struct span_model {
  span_pool* pool = nullptr;
  int device = 0;
  span_model_config cfg{};
  std::vector<const void*> attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down;
  // transposed copies (W^T [N][K]) for the skinny GEMM, all in wt_buf; null where a
  // matrix's shape does not suit that kernel
  std::vector<const void*> wt_qkv, wt_o, wt_gate_up, wt_down;
  Buf wt_buf;
  Gemm gemm;
  // compact activations over the computed rows
  Buf x, n, qkv, oc, gu, act;
  // caller-row activations the attention entry points read and write
  Buf q, k, v, o;
  // row lists, LM head
  Buf rows, toks, last, nf, part, logits, tok_out, best;
  int32_t* host_stage = nullptr;  // pinned staging of the row lists
  size_t host_stage_cap = 0;
  hipEvent_t staged = nullptr;     // the last upload from host_stage
};

namespace {

int check_config(span_pool* pool, const span_model_config* c) {
  if (!pool || !c) return report(SPAN_EINVAL, "span_model_create: null argument");
  int32_t sh[5];
  pool_shape(pool, sh);
  if (pool_device(pool) < 0) return report(SPAN_EINVAL, "span_model_create: the pool must be a device pool");
  if (sh[4] != SPAN_BF16) return report(SPAN_EINVAL, "span_model_create: the pool must hold bf16 pages");
  if (c->num_layers != sh[0] || c->num_q_heads != sh[1] || c->num_kv_heads != sh[2] || c->head_dim != sh[3])
    return report(SPAN_EINVAL, "span_model_create: layers, heads and head_dim must equal the pool's");
  if (c->hidden < 8 || c->hidden % 8 != 0 || c->hidden > 8192)
    return report(SPAN_EINVAL, "span_model_create: hidden must be a multiple of 8 in [8, 8192]");
  if (c->ffn < 8 || c->ffn % 8 != 0) return report(SPAN_EINVAL, "span_model_create: ffn must be a positive multiple of 8");
  if (c->vocab < 8 || c->vocab % 8 != 0) return report(SPAN_EINVAL, "span_model_create: vocab must be a positive multiple of 8");
  if (!(c->rms_eps > 0.f)) return report(SPAN_EINVAL, "span_model_create: rms_eps must be positive");
  if (!c->embed || !c->final_norm || !c->lm_head || !c->attn_norm || !c->w_qkv || !c->w_o || !c->ffn_norm ||
      !c->w_gate_up || !c->w_down)
    return report(SPAN_EINVAL, "span_model_create: null weight pointer");
  for (int l = 0; l < c->num_layers; ++l)
    if (!c->attn_norm[l] || !c->w_qkv[l] || !c->w_o[l] || !c->ffn_norm[l] || !c->w_gate_up[l] || !c->w_down[l])
      return report(SPAN_EINVAL, "span_model_create: null weight pointer in a layer table");
  return SPAN_OK;
}

// The pinned staging area for a call's row lists, at least n words, once the
// previous call's upload from it is done.
int stage_area(span_model* m, size_t n, int32_t** out, const char* who) {
  hipError_t e = hipEventSynchronize(m->staged);  // the previous upload has left the staging area
  if (e == hipSuccess && n > m->host_stage_cap) {
    if (m->host_stage) e = hipHostFree(m->host_stage);
    m->host_stage = nullptr;
    m->host_stage_cap = 0;
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&m->host_stage), n * sizeof(int32_t), 0);
    if (e == hipSuccess) m->host_stage_cap = n;
  }
  if (e != hipSuccess) return hip_err(e, std::string(who) + ": pinned staging");
  *out = m->host_stage;
  return SPAN_OK;
}

// Scratch of the GEMV path for T <= 8 rows: the largest of the four GEMMs' partials.
size_t gemv_scratch(const span_model_config& c, int T) {
  const int qkv_w = (c.num_q_heads + 2 * c.num_kv_heads) * c.head_dim;
  size_t b = gemv_part_bytes(T, qkv_w, c.hidden);
  b = std::max(b, gemv_part_bytes(T, c.hidden, c.num_q_heads * c.head_dim));
  b = std::max(b, gemv_part_bytes(T, 2 * c.ffn, c.hidden));
  return std::max(b, gemv_part_bytes(T, c.hidden, c.ffn));
}

// Scratch of the skinny GEMM for T rows: the largest of the four GEMMs' K-slice partials.
size_t skinny_scratch(const span_model_config& c, int64_t T) {
  const int64_t shapes[4][2] = {{(c.num_q_heads + 2 * c.num_kv_heads) * c.head_dim, c.hidden},
                                {c.hidden, c.num_q_heads * c.head_dim},
                                {2 * c.ffn, c.hidden},
                                {c.hidden, c.ffn}};
  size_t b = 0;
  for (const auto& nk : shapes)
    if (skinny_gemm_fits(T, nk[0], nk[1]))
      b = std::max(b, skinny_gemm_part_bytes(static_cast<int>(T), static_cast<int>(nk[0]), static_cast<int>(nk[1])));
  return b;
}

// Buffers for T compact rows whose attention rows lie in [0, R), then the upload of
// the row list (compact row i -> attention row), the tokens and the LM-head rows.
// Buffers grow with the stream drained, so no launch still reads the old ones.
int prepare(span_model* m, int64_t T, int64_t R, const int32_t* h_rows, const int32_t* h_toks, const int32_t* h_last,
            int nh, hipStream_t s, const char* who) {
  const span_model_config& c = m->cfg;
  const int H = c.hidden, hq = c.num_q_heads, hkv = c.num_kv_heads, d = c.head_dim, F = c.ffn, V = c.vocab;
  const int64_t qkv_w = static_cast<int64_t>(hq + 2 * hkv) * d;
  const size_t bf = 2;
  const size_t Tz = static_cast<size_t>(T), Rz = static_cast<size_t>(R);
  struct Need {
    Buf* b;
    size_t bytes;
  } needs[] = {
      {&m->x, Tz * H * bf}, {&m->n, Tz * H * bf}, {&m->qkv, Tz * qkv_w * bf}, {&m->oc, Tz * hq * d * bf},
      {&m->gu, Tz * 2 * F * bf}, {&m->act, Tz * F * bf}, {&m->q, Rz * hq * d * bf}, {&m->k, Rz * hkv * d * bf},
      {&m->v, Rz * hkv * d * bf}, {&m->o, Rz * hq * d * bf}, {&m->rows, Tz * 4 + 4}, {&m->toks, Tz * 4 + 4},
      {&m->last, static_cast<size_t>(nh) * 4 + 32}, {&m->nf, static_cast<size_t>(8) * H * bf},
      {&m->part, static_cast<size_t>(lm_head_chunks(H)) * 8 * V * 4}, {&m->logits, static_cast<size_t>(8) * V * 4},
      {&m->tok_out, 8 * 4}, {&m->best, argmax_scratch_bytes(8, V)},
      {&m->gemm.gemv_part, T <= 8 ? gemv_scratch(c, static_cast<int>(T)) : 0},
      {&m->gemm.sk_part, skinny_scratch(c, T)}};
  bool grow = false;
  for (const Need& nd : needs) grow |= nd.bytes > nd.b->cap;
  hipError_t e = hipSuccess;
  if (grow) {
    e = hipStreamSynchronize(s);
    for (const Need& nd : needs)
      if (e == hipSuccess) e = nd.b->ensure(nd.bytes);
    if (e != hipSuccess) return hip_err(e, std::string(who) + ": activation buffers");
  }
  e = T > 0 ? hipMemcpyAsync(m->rows.p, h_rows, Tz * 4, hipMemcpyHostToDevice, s) : hipSuccess;
  if (e == hipSuccess && T > 0) e = hipMemcpyAsync(m->toks.p, h_toks, Tz * 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && nh > 0) e = hipMemcpyAsync(m->last.p, h_last, static_cast<size_t>(nh) * 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipEventRecord(m->staged, s);
  if (e != hipSuccess) return hip_err(e, std::string(who) + ": row lists");
  return SPAN_OK;
}

// Embeddings of the T compact rows, then n_layers decoder layers; attn(l) runs the
// span attention of layer l on the q/k/v/o buffers.  base >= 0: compact row i is
// attention row base + i for every i, so the output projection reads the attention
// output in place instead of through a gather.
template <class Attn>
int run_layers(span_model* m, int64_t T, int n_layers, int64_t base, hipStream_t s, const char* who, Attn attn) {
  const span_model_config& c = m->cfg;
  const int H = c.hidden, hq = c.num_q_heads, hkv = c.num_kv_heads, d = c.head_dim, F = c.ffn;
  const int64_t qkv_w = static_cast<int64_t>(hq + 2 * hkv) * d;
  const int32_t* rows = m->rows.as<int32_t>();
  const std::string w(who);
  hipError_t e = launch_copy_rows(m->x.p, c.embed, m->toks.as<int32_t>(), T, H * 2, false, s);
  if (e != hipSuccess) return hip_err(e, w + ": embedding");
  // Up to 8 rows: every GEMM is a GEMV whose second pass also does the step after it
  // (q/k/v split, SwiGLU, the next RMSNorm), bit for bit the separate kernels' result.
  const bool gv = m->gemm.gemv_layer(T, qkv_w, H, F, static_cast<int64_t>(hq) * d);
  float* gp = m->gemm.gemv_part.as<float>();
  const size_t gcap = m->gemm.gemv_part.cap;
  const int Ti = static_cast<int>(T);
  if (gv && n_layers > 0) {
    e = launch_rmsnorm(m->x.p, nullptr, m->attn_norm[0], m->n.p, T, H, c.rms_eps, s);
    if (e != hipSuccess) return hip_err(e, w + ": attention norm");
  }
  bool normed = false;  // m->n already holds the attention norm of layer l
  for (int l = 0; l < n_layers; ++l) {
    int rc;
    if (gv) {
      e = launch_gemv_qkv(m->n.p, m->w_qkv[l], Ti, H, rows, hq * d, hkv * d, m->q.p, m->k.p, m->v.p, gp, gcap, s);
      if (e != hipSuccess) return hip_err(e, w + ": q/k/v GEMV");
    } else {
      if (!normed) {
        e = launch_rmsnorm(m->x.p, nullptr, m->attn_norm[l], m->n.p, T, H, c.rms_eps, s);
        if (e != hipSuccess) return hip_err(e, w + ": attention norm");
      }
      rc = m->gemm.run(m->n.p, m->w_qkv[l], m->wt_qkv[l], m->qkv.p, T, qkv_w, H, false, s);
      if (rc) return rc;
      e = launch_scatter_qkv(m->qkv.p, rows, T, hq * d, hkv * d, m->q.p, m->k.p, m->v.p, s);
      if (e != hipSuccess) return hip_err(e, w + ": q/k/v scatter");
    }
    rc = attn(l);
    if (rc) return rc;
    const void* oc = m->oc.p;
    if (base >= 0) {
      oc = static_cast<const char*>(m->o.p) + base * hq * d * 2;
    } else {
      e = launch_copy_rows(m->oc.p, m->o.p, rows, T, hq * d * 2, false, s);
      if (e != hipSuccess) return hip_err(e, w + ": attention output gather");
    }
    if (gv) {
      e = launch_gemv_residual_norm(oc, m->w_o[l], m->x.p, Ti, H, hq * d, m->ffn_norm[l], m->n.p, c.rms_eps, gp, gcap,
                                    s);
      if (e != hipSuccess) return hip_err(e, w + ": output GEMV");
      e = launch_gemv_swiglu(m->n.p, m->w_gate_up[l], m->act.p, Ti, F, H, gp, gcap, s);
      if (e != hipSuccess) return hip_err(e, w + ": gate/up GEMV");
      if (l + 1 < n_layers) {
        e = launch_gemv_residual_norm(m->act.p, m->w_down[l], m->x.p, Ti, H, F, m->attn_norm[l + 1], m->n.p,
                                      c.rms_eps, gp, gcap, s);
        if (e != hipSuccess) return hip_err(e, w + ": down GEMV");
      } else {
        rc = m->gemm.run(m->act.p, m->w_down[l], m->wt_down[l], m->x.p, T, H, F, true, s);
        if (rc) return rc;
      }
      continue;
    }
    rc = m->gemm.run(oc, m->w_o[l], m->wt_o[l], m->x.p, T, H, static_cast<int64_t>(hq) * d, true, s);
    if (rc) return rc;
    e = launch_rmsnorm(m->x.p, nullptr, m->ffn_norm[l], m->n.p, T, H, c.rms_eps, s);
    if (e != hipSuccess) return hip_err(e, w + ": ffn norm");
    rc = m->gemm.run(m->n.p, m->w_gate_up[l], m->wt_gate_up[l], m->gu.p, T, 2 * static_cast<int64_t>(F), H, false, s);
    if (rc) return rc;
    e = launch_swiglu(m->gu.p, m->act.p, T, F, s);
    if (e != hipSuccess) return hip_err(e, w + ": swiglu");
    if (l + 1 < n_layers) {
      rc = m->gemm.run_norm(m->act.p, m->w_down[l], m->wt_down[l], m->x.p, T, H, F, m->attn_norm[l + 1], m->n.p,
                            c.rms_eps, &normed, s);
    } else {
      rc = m->gemm.run(m->act.p, m->w_down[l], m->wt_down[l], m->x.p, T, H, F, true, s);
    }
    if (rc) return rc;
  }
  return SPAN_OK;
}

// Final RMSNorm, LM head and argmax of the nh compact rows listed in m->last, in
// groups of up to 8 (a group padded to 1, 2, 4 or 8 rows repeats its last row).
// Logits to logits_out [nh][vocab] if given; tokens to *toks if given (waits).
int lm_head(span_model* m, int nh, float* logits_out, std::vector<int32_t>* toks, hipStream_t s, const char* who) {
  const span_model_config& c = m->cfg;
  const int H = c.hidden, V = c.vocab;
  const size_t bf = 2;
  if (toks) toks->assign(static_cast<size_t>(nh), -1);
  hipError_t e = hipSuccess;
  for (int g0 = 0; g0 < nh; g0 += 8) {
    const int ng = std::min(8, nh - g0);
    const int np = ng <= 1 ? 1 : ng <= 2 ? 2 : ng <= 4 ? 4 : 8;
    e = launch_rmsnorm(m->x.p, m->last.as<int32_t>() + g0, c.final_norm, m->nf.p, ng, H, c.rms_eps, s);
    for (int r = ng; e == hipSuccess && r < np; ++r)
      e = hipMemcpyAsync(static_cast<char*>(m->nf.p) + static_cast<size_t>(r) * H * bf,
                         static_cast<char*>(m->nf.p) + static_cast<size_t>(ng - 1) * H * bf, H * bf,
                         hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = launch_lm_head(m->nf.p, c.lm_head, m->part.as<float>(), np, H, V, s);
    float* lg = logits_out ? logits_out + static_cast<size_t>(g0) * V : nullptr;
    if (e == hipSuccess) e = launch_argmax(m->part.as<float>(), np, ng, H, V, lg, m->tok_out.as<int32_t>(), m->best.p, s);
    if (e == hipSuccess && toks)
      e = hipMemcpyAsync(toks->data() + g0, m->tok_out.p, static_cast<size_t>(ng) * 4, hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_err(e, std::string(who) + ": LM head");
  }
  if (toks) {
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_err(e, std::string(who) + ": tokens");
  }
  return SPAN_OK;
}

// W^T copies of every layer matrix whose shape the skinny GEMM takes (at 256 rows; the
// row range does not change which shapes fit), in one allocation, made once.
int make_transposed(span_model* m) {
  const span_model_config& c = m->cfg;
  const int L = c.num_layers;
  const int64_t dims[4][2] = {{c.hidden, (c.num_q_heads + 2 * c.num_kv_heads) * c.head_dim},
                              {c.num_q_heads * c.head_dim, c.hidden},
                              {c.hidden, 2 * c.ffn},
                              {c.ffn, c.hidden}};  // K x N of W
  std::vector<const void*>* src[4] = {&m->w_qkv, &m->w_o, &m->w_gate_up, &m->w_down};
  // the weights may have been written on any stream of the device: wait for all of them
  hipError_t e0 = hipDeviceSynchronize();
  if (e0 != hipSuccess) return hip_err(e0, "span_model_create: waiting for the weights");
  std::vector<const void*>* dst[4] = {&m->wt_qkv, &m->wt_o, &m->wt_gate_up, &m->wt_down};
  size_t total = 0;
  for (int i = 0; i < 4; ++i)
    if (skinny_gemm_fits(256, dims[i][1], dims[i][0])) total += static_cast<size_t>(L) * dims[i][0] * dims[i][1] * 2;
  for (int i = 0; i < 4; ++i) dst[i]->assign(static_cast<size_t>(L), nullptr);
  if (total == 0) return SPAN_OK;
  hipError_t e = m->wt_buf.ensure(total);
  if (e != hipSuccess) return hip_err(e, "span_model_create: transposed weights");
  char* at = m->wt_buf.as<char>();
  for (int i = 0; i < 4 && e == hipSuccess; ++i) {
    if (!skinny_gemm_fits(256, dims[i][1], dims[i][0])) continue;
    for (int l = 0; l < L && e == hipSuccess; ++l) {
      e = launch_transpose_bf16((*src[i])[l], at, dims[i][0], dims[i][1], nullptr);
      (*dst[i])[l] = at;
      at += static_cast<size_t>(dims[i][0]) * dims[i][1] * 2;
    }
  }
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) return hip_err(e, "span_model_create: transposing the weights");
  return SPAN_OK;
}

}  // namespace

extern "C" {

int span_model_create(span_pool* pool, const span_model_config* cfg, span_model** out) {
  if (!out) return report(SPAN_EINVAL, "span_model_create: null argument");
  *out = nullptr;
  int rc = check_config(pool, cfg);
  if (rc) return rc;
  span_model* m = new (std::nothrow) span_model();
  if (!m) return report(SPAN_ENOMEM, "span_model_create: host allocation");
  m->pool = pool;
  m->device = pool_device(pool);
  m->cfg = *cfg;
  const int L = cfg->num_layers;
  m->attn_norm.assign(cfg->attn_norm, cfg->attn_norm + L);
  m->w_qkv.assign(cfg->w_qkv, cfg->w_qkv + L);
  m->w_o.assign(cfg->w_o, cfg->w_o + L);
  m->ffn_norm.assign(cfg->ffn_norm, cfg->ffn_norm + L);
  m->w_gate_up.assign(cfg->w_gate_up, cfg->w_gate_up + L);
  m->w_down.assign(cfg->w_down, cfg->w_down + L);
  m->cfg.attn_norm = m->cfg.w_qkv = m->cfg.w_o = m->cfg.ffn_norm = m->cfg.w_gate_up = m->cfg.w_down = nullptr;
  hipError_t e = hipSetDevice(m->device);
  if (e != hipSuccess) {
    delete m;
    return hip_err(e, "span_model_create: hipSetDevice");
  }
  rc = m->gemm.init();
  if (rc == SPAN_OK) {
    e = hipEventCreateWithFlags(&m->staged, hipEventDisableTiming);
    if (e != hipSuccess) rc = hip_err(e, "span_model_create: event");
  }
  if (rc == SPAN_OK) rc = make_transposed(m);
  if (rc) {
    m->gemm.destroy();
    m->wt_buf.release();
    if (m->staged) (void)hipEventDestroy(m->staged);
    delete m;
    return rc;
  }
  *out = m;
  return SPAN_OK;
}

int span_model_destroy(span_model* m) {
  if (!m) return report(SPAN_EINVAL, "span_model_destroy: null model");
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  m->gemm.destroy();
  m->wt_buf.release();
  for (Buf* b : {&m->x, &m->n, &m->qkv, &m->oc, &m->gu, &m->act, &m->q, &m->k, &m->v, &m->o, &m->rows, &m->toks,
                 &m->last, &m->nf, &m->part, &m->logits, &m->tok_out, &m->best})
    b->release();
  if (m->host_stage) (void)hipHostFree(m->host_stage);
  if (m->staged) (void)hipEventDestroy(m->staged);
  delete m;
  return SPAN_OK;
}

int span_model_forward(span_model* m, span_plan_t* plan, const int32_t* row_tokens, int64_t n_rows, int32_t n_layers,
                       void* hidden_out, float* logits_out, int32_t* first_tokens, void* stream) {
  if (!m || !plan || (!row_tokens && n_rows > 0) || n_rows < 0)
    return report(SPAN_EINVAL, "span_model_forward: bad argument");
  if (plan_pool(plan) != m->pool) return report(SPAN_EINVAL, "span_model_forward: the plan belongs to another pool");
  const span_model_config& c = m->cfg;
  if (n_layers < 0 || n_layers > c.num_layers)
    return report(SPAN_EINVAL, "span_model_forward: n_layers must lie in [0, num_layers]");
  if ((first_tokens || logits_out) && n_layers != c.num_layers)
    return report(SPAN_EINVAL, "span_model_forward: the LM head needs every layer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSetDevice(m->device);
  if (e != hipSuccess) return hip_err(e, "span_model_forward: hipSetDevice");

  // ---- the rows the plan computes, their tokens, each query's last cross row
  int64_t n_pre = 0, n_cross = 0;
  int rc = span_plan_rows(plan, nullptr, 0, &n_pre, &n_cross);
  if (rc) return rc;
  const int64_t T = n_pre + n_cross;
  std::vector<int64_t> rows64(static_cast<size_t>(T));
  rc = span_plan_rows(plan, rows64.data(), T, &n_pre, &n_cross);
  if (rc) return rc;
  std::vector<int64_t> last_rows;
  plan_last_cross_rows(plan, &last_rows);
  const int nq = static_cast<int>(last_rows.size());
  std::unordered_map<int64_t, int32_t> last_at;
  for (int64_t r : last_rows)
    if (r >= 0) last_at.emplace(r, -1);
  int32_t* h_rows = nullptr;
  rc = stage_area(m, 2 * static_cast<size_t>(T) + static_cast<size_t>(nq) + 8, &h_rows, "span_model_forward");
  if (rc) return rc;
  int32_t* h_toks = h_rows + T;
  int32_t* h_last = h_toks + T;
  for (int64_t i = 0; i < T; ++i) {
    const int64_t r = rows64[static_cast<size_t>(i)];
    if (r < 0 || r >= n_rows) return report(SPAN_EINVAL, "span_model_forward: a planned row lies outside row_tokens");
    const int32_t t = row_tokens[r];
    if (t < 0 || t >= c.vocab) return report(SPAN_EINVAL, "span_model_forward: token id outside the vocabulary");
    h_rows[i] = static_cast<int32_t>(r);
    h_toks[i] = t;
    auto it = last_at.find(r);
    if (it != last_at.end()) it->second = static_cast<int32_t>(i);
  }
  std::vector<int> q_of;  // queries with a cross row, in order
  for (int qi = 0; qi < nq; ++qi)
    if (last_rows[qi] >= 0) {
      const int32_t at = last_at[last_rows[qi]];
      if (at < 0) return report(SPAN_EINVAL, "span_model_forward: a query's last cross row is not computed by the plan");
      h_last[q_of.size()] = at;
      q_of.push_back(qi);
    }
  const int nh = static_cast<int>(q_of.size());
  int64_t base = T > 0 ? h_rows[0] : -1;
  for (int64_t i = 1; i < T && base >= 0; ++i)
    if (h_rows[i] != base + i) base = -1;
  rc = prepare(m, T, n_rows, h_rows, h_toks, h_last, nh, s, "span_model_forward");
  if (rc) return rc;
  rc = run_layers(m, T, n_layers, base, s, "span_model_forward", [&](int l) {
    int r = span_prefill_fragments(plan, l, m->q.p, m->k.p, m->v.p, m->o.p, s);
    if (!r) r = span_cross_attend(plan, l, m->q.p, m->k.p, m->v.p, m->o.p, s);
    return r;
  });
  if (rc) return rc;
  if (hidden_out) {
    e = launch_copy_rows(hidden_out, m->x.p, m->rows.as<int32_t>(), T, c.hidden * 2, true, s);
    if (e != hipSuccess) return hip_err(e, "span_model_forward: hidden state scatter");
  }
  if (first_tokens)
    for (int qi = 0; qi < nq; ++qi) first_tokens[qi] = -1;
  if ((first_tokens || logits_out) && nh > 0) {
    std::vector<int32_t> toks;
    rc = lm_head(m, nh, logits_out, first_tokens ? &toks : nullptr, s, "span_model_forward");
    if (rc) return rc;
    if (first_tokens)
      for (int i = 0; i < nh; ++i) first_tokens[q_of[i]] = toks[i];
  }
  return SPAN_OK;
}

int span_model_decode(span_model* m, span_plan_t* plan, const int32_t* tokens, float* logits_out, int32_t* next_tokens,
                      void* stream) {
  if (!m || !plan) return report(SPAN_EINVAL, "span_model_decode: null argument");
  if (plan_pool(plan) != m->pool) return report(SPAN_EINVAL, "span_model_decode: the plan belongs to another pool");
  const span_model_config& c = m->cfg;
  std::vector<int64_t> last_rows;
  plan_last_cross_rows(plan, &last_rows);
  const int nq = static_cast<int>(last_rows.size());
  if (nq > 0 && !tokens) return report(SPAN_EINVAL, "span_model_decode: null token list");
  std::vector<int> q_of;  // decoding queries, in order
  std::vector<int32_t> n_new(static_cast<size_t>(nq), 0);
  std::vector<int64_t> rows(static_cast<size_t>(nq), 0);
  for (int qi = 0; qi < nq; ++qi) {
    if (tokens[qi] < 0) continue;
    if (tokens[qi] >= c.vocab) return report(SPAN_EINVAL, "span_model_decode: token id outside the vocabulary");
    n_new[qi] = 1;
    rows[qi] = static_cast<int64_t>(q_of.size());
    q_of.push_back(qi);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSetDevice(m->device);
  if (e != hipSuccess) return hip_err(e, "span_model_decode: hipSetDevice");
  if (next_tokens)
    for (int qi = 0; qi < nq; ++qi) next_tokens[qi] = -1;
  const int nd = static_cast<int>(q_of.size());
  if (nd == 0) return SPAN_OK;
  int rc = span_plan_decode(plan, n_new.data(), rows.data(), s);
  if (rc) return rc;
  // one compact row per decoding query; its attention row is the same index
  int32_t* h_rows = nullptr;
  rc = stage_area(m, 3 * static_cast<size_t>(nd) + 8, &h_rows, "span_model_decode");
  if (rc) return rc;
  int32_t* h_toks = h_rows + nd;
  int32_t* h_last = h_toks + nd;
  for (int i = 0; i < nd; ++i) {
    h_rows[i] = i;
    h_toks[i] = tokens[q_of[i]];
    h_last[i] = i;
  }
  rc = prepare(m, nd, nd, h_rows, h_toks, h_last, nd, s, "span_model_decode");
  if (rc) return rc;
  rc = run_layers(m, nd, c.num_layers, 0, s, "span_model_decode",
                  [&](int l) { return span_decode_attend(plan, l, m->q.p, m->k.p, m->v.p, m->o.p, s); });
  if (rc) return rc;
  if (!next_tokens && !logits_out) return SPAN_OK;
  std::vector<int32_t> toks;
  rc = lm_head(m, nd, logits_out, next_tokens ? &toks : nullptr, s, "span_model_decode");
  if (rc) return rc;
  if (next_tokens)
    for (int i = 0; i < nd; ++i) next_tokens[q_of[i]] = toks[i];
  return SPAN_OK;
}

int span_probe_gemm(const void* x, const void* w, void* y, int64_t M, int64_t N, int64_t K, int32_t residual,
                    int32_t reps, void* stream, int32_t* kernel, double* sec_per_call) {
  if (!x || !w || !y || M < 1 || N < 8 || N % 8 != 0 || K < 8 || K % 8 != 0 || reps < 0 || M > (int64_t{1} << 24) ||
      N > (int64_t{1} << 24) || K > (int64_t{1} << 24))
    return report(SPAN_EINVAL, "span_probe_gemm: bad argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Gemm g;
  Buf wt, y2;
  auto done = [&](int rc) {
    (void)hipStreamSynchronize(s);
    g.destroy();
    wt.release();
    y2.release();
    return rc;
  };
  int rc = g.init();
  if (rc) return done(rc);
  const int Mi = static_cast<int>(M), Ni = static_cast<int>(N), Ki = static_cast<int>(K);
  const bool skinny = skinny_gemm_fits(M, N, K);
  hipError_t e = hipSuccess;
  if (skinny) {
    e = wt.ensure(static_cast<size_t>(N) * K * 2);
    if (e == hipSuccess) e = launch_transpose_bf16(w, wt.p, K, N, s);
    if (e == hipSuccess) e = g.sk_part.ensure(std::max<size_t>(16, skinny_gemm_part_bytes(Mi, Ni, Ki)));
  } else if (M <= 8) {
    e = g.gemv_part.ensure(gemv_part_bytes(Mi, Ni, Ki));
  }
  if (e != hipSuccess) return done(hip_err(e, "span_probe_gemm: set-up"));
  rc = g.run(x, w, skinny ? wt.p : nullptr, y, M, N, K, residual != 0, s);
  if (rc) return done(rc);
  if (kernel) *kernel = skinny ? 2 : (M <= 8 ? 1 : 0);
  if (sec_per_call && reps > 0) {
    e = y2.ensure(static_cast<size_t>(M) * N * 2);
    if (e == hipSuccess) e = hipMemcpyAsync(y2.p, y, static_cast<size_t>(M) * N * 2, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return done(hip_err(e, "span_probe_gemm: timing buffer"));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    e = hipEventCreate(&e0);
    if (e == hipSuccess) e = hipEventCreate(&e1);
    if (e == hipSuccess) e = hipEventRecord(e0, s);
    for (int i = 0; e == hipSuccess && rc == SPAN_OK && i < reps; ++i)
      rc = g.run(x, w, skinny ? wt.p : nullptr, y2.p, M, N, K, residual != 0, s);
    if (e == hipSuccess && rc == SPAN_OK) e = hipEventRecord(e1, s);
    if (e == hipSuccess && rc == SPAN_OK) e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess && rc == SPAN_OK) e = hipEventElapsedTime(&ms, e0, e1);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (rc) return done(rc);
    if (e != hipSuccess) return done(hip_err(e, "span_probe_gemm: timing"));
    *sec_per_call = 1e-3 * ms / reps;
  }
  return done(SPAN_OK);
}

}  // extern "C"
