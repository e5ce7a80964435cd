/*
 * spanq.h - span-query prefill attention over a paged KV cache (MI355X, gfx950).
 *
 * A span query (Castro et al., "Using Span Queries to Optimize for Cache and
 * Attention Locality", Def. 2-3) of the RAG / judge form
 *     G( cross-join( prefix, plus(F_1, ..., F_n), cross ) )
 * presents a shared prefix, n commuting fragments (the children of the
 * commutative join, section 4.3) in some order, and a non-commuting cross
 * segment (question, judge prompt).  This library executes its prefill:
 *
 *   span_plan              hash every page of every span, look each span up in
 *                          the page cache (stop at the first miss), deduplicate
 *                          fragments across the batch, allocate or evict pages,
 *                          and build the device work lists (sections 2, 5.4).
 *   span_prefill_fragments rotate and write the keys/values of every new prefix
 *                          and fragment token into its page, then run span-prefill
 *                          attention: a fragment token attends to the whole prefix
 *                          and causally to its own fragment, at canonical
 *                          positions (section 5.6; section 5.1 footnote).
 *   span_cross_attend      write the cross tokens' pages, then run cross
 *                          attention: a cross token attends to the prefix, to all
 *                          fragments in this query's order, and causally to the
 *                          cross segment, with every cached page repositioned to
 *                          its place in this query (section 5.5).
 *   kv_lookup              the longest cached run of a chain of page hashes
 *                          (section 2).
 *
 * Conventions
 * - Every function returns an int status: SPAN_OK (0) or a negative SPAN_E*
 *   code; none throws or aborts.  span_last_error() gives a thread-local message
 *   for the most recent failure on the calling thread.
 * - Tokens are int32.  A page holds 16 tokens (page_size, device pools); every
 *   span starts on a fresh page and its last page may be partial.
 * - Activations are row-major arrays in the caller's row numbering:
 *       q, out: [rows][num_q_heads][head_dim]     k, v: [rows][num_kv_heads][head_dim]
 *   element type = the pool dtype (SPAN_F32: float, SPAN_BF16: bfloat16 bits).
 *   Token j of a span lives in row span.row + j.  q and k are BEFORE rotary
 *   encoding.  Only rows of tokens the plan computes (new prefix/fragment tokens
 *   and all cross tokens) are read or written.
 * - Query head h reads kv head floor(h * num_kv_heads / num_q_heads).
 * - Rotary encoding: rotate-half pairs (i, i + d/2), inverse frequency
 *   rope_theta^(-2i/d).
 * - Device work is enqueued asynchronously on the caller's HIP stream (void* =
 *   hipStream_t; NULL = the null stream).  Caller buffers must stay alive until that
 *   work completes.  A plan's device metadata (and a grown rotary table) are copied
 *   on the stream given to span_plan; an attention call on any other stream first
 *   makes that stream wait (hipStreamWaitEvent) for those copies, and
 *   span_plan_destroy releases the plan's device memory on the plan's stream only
 *   after the work already enqueued on every stream the plan was launched on.
 * - A pool is not thread-safe; use one thread per pool.
 */
#ifndef SPANQ_H
#define SPANQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPAN_OK 0
#define SPAN_EINVAL (-1)  /* bad argument or unsupported shape */
#define SPAN_ENOMEM (-2)  /* pool exhausted: more pages needed than free or evictable */
#define SPAN_EHIP (-3)    /* a HIP runtime call failed */
#define SPAN_ESTATE (-4)  /* call-order violation (e.g. attention after commit) */

#define SPAN_F32 0
#define SPAN_BF16 1

#define SPAN_HASH_SPAN 0  /* per-span chains: fragments hit in any order (section 5.4) */
#define SPAN_HASH_STOCK 1 /* one chain over the whole prompt, partial tail page never
                             cached (section 2); prefix-only queries, host-only pools */

#define SPAN_KERNEL_AUTO 0    /* bf16 MFMA kernel where the shape allows, else generic */
#define SPAN_KERNEL_GENERIC 1 /* vector-ALU kernel, any supported shape / dtype */
#define SPAN_KERNEL_MFMA 2    /* bf16 MFMA kernel: bf16 pools, head_dim 64 or 128, num_q_heads /
                                 num_kv_heads in {1, 2, 4, 8} (SPAN_EINVAL otherwise) */

#define SPAN_FLAG_TIMING 1    /* bracket every kernel launch with HIP events (span_plan_kernel_times) */
#define SPAN_FLAG_MATERIALIZE 2 /* materialised repositioning (the re-rotation of cached blocks of
                                   section 5.5, CIDRA): plans copy every page that cross rows read at a shifted
                                   position into a transient page whose keys sit at the final positions;
                                   see span_plan.  Default (flag clear): cross attention rotates at read
                                   time and nothing is copied. */

typedef struct span_pool span_pool;
typedef struct span_plan_t span_plan_t;

typedef struct {
  int32_t num_layers;   /* >= 1; each layer has its own page slab */
  int32_t num_q_heads;  /* multiple of num_kv_heads */
  int32_t num_kv_heads;
  int32_t head_dim;     /* 64 or 128 */
  int32_t page_size;    /* 16 for device pools; any >= 1 for host-only pools */
  int32_t dtype;        /* SPAN_F32 or SPAN_BF16 */
  int32_t hash_mode;    /* SPAN_HASH_SPAN or SPAN_HASH_STOCK */
  int32_t kernel;       /* SPAN_KERNEL_* */
  int32_t device;       /* HIP device ordinal, or -1 for a host-only pool (no device
                           memory: planning and lookup only) */
  int32_t flags;        /* SPAN_FLAG_* */
  float rope_theta;
  int64_t num_pages;    /* pages per layer */
  void* device_buf;     /* optional caller-owned device buffer of span_pool_bytes();
                           NULL = the library allocates (and frees) it */
  size_t device_bytes;
} span_pool_config;

/* Bytes of device memory a pool with this config needs:
 *   num_layers * num_pages * 2 * num_kv_heads * page_size * head_dim * elem_size.
 * Page layout (one layer): K as [kv_head][slot][head_dim], then V as
 * [kv_head][head_dim][v_pos(slot)] (transposed so the P.V contraction reads it
 * directly), where v_pos swaps bits 2 and 3 of the slot (device pools, 16 slots). */
int span_pool_bytes(const span_pool_config* cfg, size_t* bytes);

/* Create a pool.  With device >= 0 the page memory is device memory (allocated
 * here unless device_buf is given).  *out receives the handle. */
int span_pool_create(const span_pool_config* cfg, span_pool** out);

/* Destroy a pool and every plan still attached to it.  Frees library-owned memory. */
int span_pool_destroy(span_pool* pool);

/* Forget every cached page (all pages free, LRU clock unchanged).  SPAN_ESTATE if
 * an uncommitted plan is alive (committed plans hold no pages). */
int span_pool_reset(span_pool* pool);

typedef struct {
  int64_t num_pages;
  int64_t free_pages;
  int64_t cached_pages;    /* published pages */
  int64_t pinned_pages;    /* pages held by live plans */
  int64_t tick;            /* LRU clock: number of successful span_plan calls */
  int64_t total_evictions;
} span_pool_info;
int span_pool_get_info(const span_pool* pool, span_pool_info* info);

/* Base device address of the page memory and the element offset of (layer, page):
 * K of kv head h, slot s, dim i at base + off + (h*page_size + s)*head_dim + i;
 * V at base + off + num_kv_heads*page_size*head_dim + (h*head_dim + i)*page_size + v_pos(s),
 * v_pos(s) = (s & 3) | ((s & 4) << 1) | ((s & 8) >> 1). */
int span_pool_page_address(const span_pool* pool, int32_t layer, int32_t page_id,
                           void** base, int64_t* elem_offset);

/* ---------------------------------------------------------------- hashing */

/* Chain seeds of the page hash (section 5.4: a fragment's chain starts from the
 * prefix, never from its left siblings).
 *   prefix chain seed      = SPAN_HASH_ROOT
 *   fragment chain seed    = mix(last prefix page hash, or SPAN_HASH_ROOT if the
 *                                prefix is empty, XOR SPAN_HASH_FRAG_TAG)
 * mix = SplitMix64 (Steele, Lea, Flood 2014): x + 0x9E3779B97F4A7C15, then
 * xor-shift 30 / multiply 0xBF58476D1CE4E5B9 / xor-shift 27 / multiply
 * 0x94D049BB133111EB / xor-shift 31.
 * Page i of a chain: h = previous page's hash (or the seed); h = mix(h ^ t) for
 * each token t (as uint32); page hash = mix(h ^ (n << 32) ^ i), n = tokens in page. */
#define SPAN_HASH_ROOT 0x243F6A8885A308D3ull
#define SPAN_HASH_FRAG_TAG 0x13198A2E03707344ull
uint64_t span_hash_mix(uint64_t x);

/* Hashes of the pages of one chain.  out must hold ceil(n / page_size) values;
 * with include_partial == 0 a trailing partial page is not hashed.  *n_pages
 * receives the number written. */
int span_hash_pages(uint64_t seed, const int32_t* tokens, int32_t n, int32_t page_size,
                    int32_t include_partial, uint64_t* out, int32_t* n_pages);

/* Section 2 lookup: page_ids[i] = cached page holding hash i or -1; *n_leading_hits
 * = number of leading hits (lookup stops at the first miss).  Pure: no LRU touch,
 * no content check (span_plan also compares the stored tokens). */
int kv_lookup(const span_pool* pool, const uint64_t* hashes, int32_t n, int32_t* page_ids,
              int32_t* n_leading_hits);

/* ---------------------------------------------------------------- planning */

typedef struct {
  const int32_t* tokens;  /* host memory, n tokens */
  int32_t n;              /* >= 0 */
  int32_t reserved;
  int64_t row;            /* caller row of token 0 in q/k/v/out */
} span_tokens;

typedef struct {
  span_tokens prefix;       /* shared prefix (may be empty) */
  const span_tokens* frags; /* n_frags commuting children, in this query's order */
  int32_t n_frags;
  int32_t reserved;
  span_tokens cross;        /* trailing non-commuting segment (may be empty) */
} span_query;

/* Plan a batch of queries (sections 2 and 5.4).  Pages of the prefix and of each
 * fragment are hashed per span and looked up, stopping at each span's first miss;
 * a span already scheduled earlier in the batch is a hit for later ones.  Missing
 * pages and the cross pages are allocated (lowest free id first; with no free page
 * the least recently used unpinned cached page is evicted, a span's tail pages
 * first).  All pages the plan uses are pinned until commit (cache pages) or destroy
 * (cross pages).  The device work lists are copied once, on `stream`.
 * SPAN_ENOMEM (pool unchanged) if the batch needs more pages than are free or
 * evictable.  Host-only pools plan but cannot run attention.
 * With SPAN_FLAG_MATERIALIZE the plan also allocates, after all other pages, one
 * transient page per distinct (page, shift) that a query with a cross segment
 * reads at a shifted position (a fragment page with final != canonical position;
 * a page read at two shifts gets two copies, one read at the same shift by several
 * queries one); they count in the capacity check and are freed like cross pages. */
int span_plan(span_pool* pool, const span_query* queries, int32_t n_queries, void* stream,
              span_plan_t** out);

typedef struct {
  int64_t pages_hit;        /* prefix/fragment pages served from cache (incl. batch dedup) */
  int64_t pages_new;        /* prefix/fragment pages to compute */
  int64_t pages_cross;      /* transient cross pages */
  int64_t pages_evicted;
  int64_t tokens_hit;
  int64_t tokens_new;       /* prefix/fragment tokens to compute */
  int64_t tokens_cross;
  int64_t prefill_pairs;    /* (query, key) pairs the span mask allows, prefill rows */
  int64_t cross_pairs;      /* same, cross rows */
  int64_t prefill_tiles;
  int64_t cross_tiles;      /* work items including KV splits */
  int64_t kv_splits;        /* KV splits per cross row tile */
  int64_t cross_kv_pages;   /* page reads of the cross pass per kv head */
  double host_plan_us;      /* host time of hashing, lookup, allocation and work lists */
  double host_upload_us;    /* host time of device metadata allocation + copy enqueue */
  int64_t pages_moved;      /* SPAN_FLAG_MATERIALIZE: transient repositioned copies */
  int64_t tokens_moved;     /* filled slots of those copies */
  int64_t prefill_queues;   /* work queues of the last bf16 MFMA prefill launch: 8 (one per XCD,
                               each reading one kv head of a group of spans), 1, or 0 (none yet) */
  int64_t decode_steps;     /* span_plan_decode calls so far */
  int64_t decode_tokens;    /* tokens they appended */
  int64_t decode_pages;     /* transient pages they allocated */
  int64_t decode_pairs;     /* (query, key) pairs of the last decode step's rows */
} span_stats;
int span_plan_stats(const span_plan_t* plan, span_stats* stats);

/* Block table of one span: span = -1 prefix, 0..n_frags-1 fragment children,
 * n_frags cross.  Writes up to cap page ids; *n = pages of the span, *n_hit =
 * leading pages that were hits. */
int span_plan_block_table(const span_plan_t* plan, int32_t query, int32_t span, int32_t* page_ids,
                          int32_t cap, int32_t* n, int32_t* n_hit);

/* Repositioned copies of a SPAN_FLAG_MATERIALIZE plan (none otherwise): record i
 * is rec[4i..4i+3] = (source page, copy page, shift in positions, filled slots),
 * for i < cap; *n = number of copies. */
int span_plan_moves(const span_plan_t* plan, int32_t* rec, int32_t cap, int32_t* n);

/* Page ids evicted by this plan, in eviction order. */
int span_plan_evicted(const span_plan_t* plan, int32_t* page_ids, int32_t cap, int32_t* n);

/* Caller rows the plan reads (q, k, v) and writes (out): the new prefix/fragment
 * token rows (prefill) then the cross rows, in work order. */
int span_plan_rows(const span_plan_t* plan, int64_t* rows, int64_t cap, int64_t* n_prefill,
                   int64_t* n_cross);

/* Device scratch reserved per GPU for span_plan_static (64 MiB). */
#define SPAN_STATIC_SCRATCH_BYTES (64u << 20)

/* span_plan for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same planning,
 * same arguments, same kernels; the plan's device data (work lists, scheduling
 * counters, split-KV partials) go to a device array of SPAN_STATIC_SCRATCH_BYTES
 * that the library holds on each GPU until the process ends, instead of the
 * stream-ordered allocations span_plan makes.  No hipMalloc, hipFree or other
 * device allocation is made by this call or by the attention calls and destroy of
 * its plan.
 * - SPAN_EINVAL if the plan's device data exceed SPAN_STATIC_SCRATCH_BYTES, or if
 *   the pool's rotary table does not cover the plan's positions (a pool covers 4096
 *   positions from creation; one span_plan of a longer query grows it).  The plan
 *   is then released as by span_plan_destroy without commit: pages it evicted stay
 *   evicted.
 * - SPAN_ESTATE while another span_plan_static plan on the same GPU is alive
 *   (created and not yet destroyed): every such plan on a GPU shares its array.
 * - The array keeps the last plan's contents; what must start at zero (the
 *   scheduling counters) is part of the copy each call makes on `stream`.  A plan
 *   made after an earlier one was destroyed overwrites the array on its own
 *   stream: the caller must order it after the earlier plan's kernels (one stream,
 *   or a synchronisation); calls that overlap on one GPU race. */
int span_plan_static(span_pool* pool, const span_query* queries, int32_t n_queries, void* stream,
                     span_plan_t** out);

/* ---------------------------------------------------------------- attention */

/* Prefill of the new prefix and fragment tokens for one layer (sections 5.1, 5.6):
 * rotate each new key at its canonical position (prefix token t at t, fragment
 * token j at P + j), write keys and values into their pages, then write out[row] =
 * softmax over the span mask of q.k / sqrt(d) times V, with the query also at its
 * canonical position.  No-op when every page hit.  Calls on one plan may run
 * concurrently on different streams, up to 64 of them in flight at once (the
 * bf16 kernel schedules its work items through per-launch counters the plan owns);
 * the ordering after the plan's uploads is enforced as described above. */
int span_prefill_fragments(span_plan_t* plan, int32_t layer, const void* q, const void* k,
                           const void* v, void* out, void* stream);

/* Cross attention for one layer (sections 5.5, 5.6): write the cross tokens' keys
 * and values into the plan's transient pages, then for every cross row attend to the
 * prefix, to every fragment in this query's order and causally to the cross segment,
 * all at final positions (index in prefix | F_s1 | ... | F_sn | cross).  Cached
 * fragment keys are rotated by (final - canonical) position as they are read; pages
 * are never rewritten.  On a SPAN_FLAG_MATERIALIZE pool the layer's repositioned
 * copies are written first (keys rotated by the shift, values copied) and the cross
 * rows read those, unrotated.  Must follow span_prefill_fragments for the same layer. */
int span_cross_attend(span_plan_t* plan, int32_t layer, const void* q, const void* k, const void* v,
                      void* out, void* stream);

/* Publish the plan's new prefix/fragment pages in the cache index, unpin its pages
 * and free its cross pages.  Call after the last layer's kernels are enqueued; pages
 * released here may be reused by the next plan's kernels, so a next plan on another
 * stream must be ordered after this plan's work by the caller. */
int span_plan_commit(span_plan_t* plan);

/* Free the plan.  Without a prior commit its new pages are freed unpublished and its
 * hits unpinned.  Device metadata is released on the plan's stream, ordered after
 * the work enqueued so far on every stream the plan's attention calls used; the
 * call itself does not wait for the device. */
int span_plan_destroy(span_plan_t* plan);

/* ---------------------------------------------------------------- nested generation */

/* Decode steps after the first token (section 5.7: a generate G over a cross
 * segment; section 6: the judge steps of a tree reduction).  A step appends
 * n_new[q] tokens (caller rows rows[q] .. rows[q] + n_new[q] - 1; 0 for a query
 * that is not decoding) to the end of each query's cross segment: they take the
 * positions after it, their keys and values go into the cross segment's pages
 * (new transient pages as the last one fills, allocated and evicted for like
 * span_plan's, freed at commit or destroy), and each new row attends to the
 * prefix, every fragment at its final position and causally to the whole cross
 * segment, as a cross row would.  The step's work lists are copied on `stream`.
 * Call after the plan's span_prefill_fragments / span_cross_attend calls for
 * every layer: once a step is planned those two return SPAN_ESTATE.
 * SPAN_ENOMEM (plan and pool unchanged) if the pages do not fit; SPAN_ESTATE after
 * commit; SPAN_EINVAL for plans of span_plan_static (a step allocates).  Host-only
 * pools plan the step (pages, positions) without device work. */
int span_plan_decode(span_plan_t* plan, const int32_t* n_new, const int64_t* rows, void* stream);

/* The last decode step for one layer: write the new tokens' keys (rotated at their
 * positions) and values into their pages, then out[row] = attention of each new
 * row as span_plan_decode describes.  q, k, v, out as for span_cross_attend (rows
 * are caller rows).  Calls on a stream other than the step's wait for its upload;
 * the next step and destroy wait for them. */
int span_decode_attend(span_plan_t* plan, int32_t layer, const void* q, const void* k, const void* v, void* out,
                       void* stream);

/* ---------------------------------------------------------------- bulk scheduling */

/* An execution order for a bulk of n_queries queries that clusters fragment reuse in
 * time (section 5.8).  Greedy: the pool is simulated at span granularity (a prefix
 * or fragment, keyed by its page-hash chain, is resident or not; spans the pool
 * holds in full start resident; capacity = the pool's pages); each step takes the
 * remaining query with the most pages in resident spans (ties: the lowest index),
 * marks its spans used and evicts least recently used spans down to the capacity.
 * order[0 .. n_queries) receives a permutation of 0 .. n_queries - 1.  The pool is
 * only read.  O(n_queries^2 x spans per query). */
int span_bulk_order(const span_pool* pool, const span_query* queries, int32_t n_queries, int32_t* order);

/* ---------------------------------------------------------------- serialized queries */

typedef struct {
  int64_t begin;  /* first token of the span in the serialized stream */
  int64_t n;      /* tokens (special and pad tokens excluded) */
} span_range;

/* Parse a serialized span query (sections 5.2 and 5.3, Def. 4): the token stream of
 * G(Cross(prefix, Plus(F_1, ..., F_n), cross)) as
 *     prefix  OPEN F_1  SEP F_2 ... SEP F_n  CLOSE pos  cross
 * where every special token starts a block of `block` tokens, PAD tokens fill the
 * end of the block before it, and the token after CLOSE is the position of the OPEN
 * (so no parsing stack is needed).  special = {PAD, OPEN, SEP, CLOSE} token ids.
 * Writes the prefix and cross ranges and up to cap fragment ranges (in order);
 * *n_frags = the number of fragments.  A stream with no OPEN is all cross segment.
 * SPAN_EINVAL (with the offending position in span_last_error) for a special token
 * off a block start, inside a span or after the join, a nested join, a missing CLOSE,
 * or a CLOSE pointing elsewhere than its OPEN. */
int span_parse_serialized(const int32_t* tokens, int64_t n, int32_t block, const int32_t special[4],
                          span_range* frags, int32_t cap, int32_t* n_frags, span_range* prefix, span_range* cross);

/* ---------------------------------------------------------------- decoder stack */

/* A decoder stack that a span query's prefill runs through (the paper's latency
 * results are whole-model time to first token, sections 5.6 and 5.7; it names no
 * architecture for them).  The layer is the pre-norm Llama block:
 *     n = RMSNorm(x) g_attn;  q | k | v = n W_qkv;  o = span attention (the calls above)
 *     h = x + o W_o;  n2 = RMSNorm(h) g_ffn;  x' = h + (silu(n2 W_gate) * (n2 W_up)) W_down
 * with RMSNorm(x) = x / sqrt(mean(x^2) + eps) and silu(z) = z / (1 + e^-z); then a
 * final RMSNorm and the LM head on each query's last cross token, and the argmax of
 * its logits (lowest id on ties) as the first generated token.
 * Weights are caller-owned device memory, bf16, row-major, x @ W convention
 * (W is [in][out]); the per-layer tables are host arrays of num_layers pointers.
 * The model copies the tables; the weights must outlive it.  At creation it also
 * makes a transposed copy of each layer matrix that its few-row GEMM kernel takes (a
 * reduction K at least 4 times the output width N, N a multiple of 64, K of 256:
 * the down projection of usual FFNs), read by forward calls of 129..256 rows, so
 * weights changed after span_model_create are not seen by those calls. */
typedef struct span_model span_model;


typedef struct {
  int32_t num_layers;    /* == the pool's */
  int32_t hidden;        /* multiple of 8, at most 8192 */
  int32_t num_q_heads;   /* == the pool's */
  int32_t num_kv_heads;  /* == the pool's */
  int32_t head_dim;      /* == the pool's */
  int32_t ffn;           /* SwiGLU width, multiple of 8 */
  int32_t vocab;         /* multiple of 8 */
  float rms_eps;         /* > 0 */
  int32_t reserved;      /* 0 */
  const void* embed;                /* [vocab][hidden] */
  const void* const* attn_norm;     /* per layer [hidden] */
  const void* const* w_qkv;         /* per layer [hidden][(num_q_heads + 2 num_kv_heads) head_dim]: q | k | v */
  const void* const* w_o;           /* per layer [num_q_heads head_dim][hidden] */
  const void* const* ffn_norm;      /* per layer [hidden] */
  const void* const* w_gate_up;     /* per layer [hidden][2 ffn]: gate | up */
  const void* const* w_down;        /* per layer [ffn][hidden] */
  const void* final_norm;           /* [hidden] */
  const void* lm_head;              /* [hidden][vocab] */
} span_model_config;

/* Bind a model to a bf16 device pool of the same layers and heads.  Allocates a
 * GEMM workspace and the transposed weight copies (waits for the device, so that
 * weights written on any stream are complete, then for the transposition);
 * activation buffers are allocated by the first forward call and
 * grown when a later one needs more.  SPAN_EINVAL on a shape mismatch. */
int span_model_create(span_pool* pool, const span_model_config* cfg, span_model** out);
int span_model_destroy(span_model* model);

/* Run the rows a plan computes (span_plan_rows: new prefix/fragment tokens, then
 * cross tokens) through the first n_layers layers, calling span_prefill_fragments
 * and span_cross_attend of `plan` per layer; cached rows are not computed, their
 * keys and values are read from the pool's pages.
 * - row_tokens: host int32 [n_rows], the token id at each caller row (the rows of
 *   the plan's spans must lie below n_rows).
 * - hidden_out: optional device bf16 [n_rows][hidden]; receives the residual stream
 *   after n_layers layers at the computed rows (other rows untouched).
 * - logits_out: optional device float [m][vocab], m = number of the plan's queries
 *   with a cross segment, in query order: the LM head logits of each one's last
 *   cross token.  Needs n_layers == num_layers.
 * - first_tokens: optional host int32 [n_queries]: the argmax of those logits, -1
 *   for a query without a cross segment.  Needs n_layers == num_layers; the call
 *   then waits for the stream.
 * Work is enqueued on `stream`.  The model's buffers are reused by the next call:
 * calls on one model are ordered by the caller (one stream). */
int span_model_forward(span_model* model, span_plan_t* plan, const int32_t* row_tokens, int64_t n_rows,
                       int32_t n_layers, void* hidden_out, float* logits_out, int32_t* first_tokens, void* stream);

/* One greedy decode step of nested generation (sections 5.7 and 6), after
 * span_model_forward on the same plan: every query q with tokens[q] >= 0 feeds that
 * token (typically the one it generated last) as the next token of its cross
 * segment; it runs through every layer, attending as span_plan_decode describes
 * (which this calls, one token per decoding query), and the final norm, LM head and
 * argmax give next_tokens[q] (-1 for queries with tokens[q] < 0).  logits_out, if
 * not NULL, receives [decoding queries][vocab] float32, in query order.  The
 * model's own buffers hold the step's activations. */
int span_model_decode(span_model* model, span_plan_t* plan, const int32_t* tokens, float* logits_out,
                      int32_t* next_tokens, void* stream);

/* ---------------------------------------------------------------- debug */

/* Kernel durations of a plan's launches on a pool created with SPAN_FLAG_TIMING,
 * measured with HIP events recorded on the launch stream, summed over every layer
 * call so far; launches counts the attention calls timed.  Waits for the events. */
typedef struct {
  float page_write_prefill_ms;  /* K3 over new prefix/fragment pages */
  float prefill_attention_ms;   /* span-prefill attention */
  float page_write_cross_ms;    /* K3 over cross pages */
  float cross_attention_ms;     /* cross attention (all KV splits) */
  float combine_ms;             /* KV-split merge */
  float page_move_ms;           /* SPAN_FLAG_MATERIALIZE: repositioned copies */
  float decode_ms;              /* decode steps: page writes, attention and merge */
  int32_t prefill_calls;
  int32_t cross_calls;
  int32_t decode_calls;
} span_kernel_times;
int span_plan_kernel_times(const span_plan_t* plan, span_kernel_times* times);

const char* span_last_error(void);

/* Copy one page (K then V, page layout above) of one layer to host memory; synchronous. */
int span_pool_read_page(const span_pool* pool, int32_t layer, int32_t page_id, void* host_dst,
                        size_t bytes);

/* ---------------------------------------------------------------- machine peaks */

/* Not part of the method: these measure what this GPU attains for the two resources
 * the attention kernels are bound by, to read the kernels' rates against beside the
 * published peaks.  Each launches its kernel once untimed, then `reps` times between
 * two HIP events on `stream` (0 = the null stream), and waits for them.
 * SPAN_EINVAL on a bad argument, SPAN_EHIP on a HIP error. */

/* bf16 MFMA rate: two waves on every SIMD of every compute unit each run `iters`
 * rounds of four independent v_mfma_f32_32x32x16_bf16 chains with register operands
 * and nothing else.  Stores dense TFLOP/s (2 * 32 * 32 * 16 flop per MFMA) in *tflops. */
int span_probe_mfma_peak(int32_t iters, int32_t reps, void* stream, double* tflops);

/* HBM read rate: a grid-stride kernel reads `bytes` (a positive multiple of 16) of
 * device memory at `buf` (caller-owned, 16-byte aligned) with 16-byte non-temporal
 * loads, four in flight per lane.  A buffer well past the 256 MiB last-level cache
 * (1 GiB or more) measures HBM.  Stores GB/s (10^9 bytes per second) in *gbs.
 * SPAN_EINVAL also for a buffer that is not 16-byte aligned. */
int span_probe_read_peak(const void* buf, size_t bytes, int32_t reps, void* stream, double* gbs);

/* The model stack's GEMM on caller buffers: Y[M][N] = X[M][K] W[K][N] (+ Y when
 * residual != 0), bf16 row-major device memory (16-byte aligned), fp32 accumulation,
 * through the same dispatch span_model_forward uses for M rows: the GEMV kernels for
 * M <= 8, the skinny MFMA kernel for 129..256 rows when K >= 4 N, N is a multiple of
 * 64 and K of 256 (from a transposed copy of W this call makes), hipBLASLt otherwise.  N and K
 * multiples of 8.  *kernel (if given) receives 1 (GEMV), 2 (skinny) or 0 (hipBLASLt).
 * With reps > 0 and sec_per_call given, reps more calls into a scratch copy of Y are
 * timed between two events and the mean seconds per call stored.  Waits for `stream`
 * before returning.  Allocates its scratch; SPAN_EINVAL on a bad argument, SPAN_EHIP
 * on a HIP or hipBLASLt error. */
int span_probe_gemm(const void* x, const void* w, void* y, int64_t M, int64_t N, int64_t K, int32_t residual,
                    int32_t reps, void* stream, int32_t* kernel, double* sec_per_call);

#ifdef __cplusplus
}
#endif
#endif /* SPANQ_H */
