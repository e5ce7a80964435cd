// Internal entries shared by the C-ABI sources (not part of the public ABI).
#pragma once
#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/spanq.h"

namespace spanq {

// span_plan's work.  With region == nullptr the plan's device data (work lists,
// scheduling counters, split-KV partials) come from the device's stream-ordered
// allocator and the rotary table grows as needed.  With a region, they are placed
// in region[0, region_bytes) (256-byte aligned device memory of the pool's device)
// and nothing is allocated: SPAN_EINVAL if they do not fit or the table is too
// short, SPAN_ESTATE while another plan holds the device's region.  `who` names
// the entry point in error messages.
int plan_impl(span_pool* pool, const span_query* qs, int32_t nq, void* stream, span_plan_t** out,
              unsigned char* region, size_t region_bytes, const char* who);

// Device ordinal of a pool; -1 for a null or host-only pool.
int pool_device(const span_pool* pool);

// Record a failure for span_last_error and return its status.
int report(int code, const char* msg);

// The page index of a pool (host side).
const class PoolIndex* pool_index(const span_pool* pool);

// The pool a plan was made on.
span_pool* plan_pool(const span_plan_t* plan);

// Pool shape: {num_layers, num_q_heads, num_kv_heads, head_dim, dtype}.
void pool_shape(const span_pool* pool, int32_t out[5]);

// Caller row of each query's last cross token, -1 for a query without one.
void plan_last_cross_rows(const span_plan_t* plan, std::vector<int64_t>* rows);

}  // namespace spanq
