// span_plan_static: span_plan for callers that cannot allocate device memory.
//
// The plan's device data live in `scratch`, a file-scope device array of
// SPAN_STATIC_SCRATCH_BYTES per GPU, held until the process ends.  Host code never
// passes the array's name to a kernel or a copy (on the host it is only a stand-in
// for the symbol): the device address is taken once per device with
// hipGetSymbolAddress, with that device current, and kept in g_scratch_ptr.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/spanq.h"
#include "capi_internal.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[SPAN_STATIC_SCRATCH_BYTES];

std::mutex g_mu;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device`; the first call per device looks it up.
hipError_t scratch_on(int device, unsigned char** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[device]) {
    int prev = 0;
    hipError_t e = hipGetDevice(&prev);
    if (e == hipSuccess && prev != device) e = hipSetDevice(device);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev != device) (void)hipSetDevice(prev);
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace

extern "C" int span_plan_static(span_pool* pool, const span_query* queries, int32_t n_queries, void* stream,
                                span_plan_t** out) {
  if (!pool || !out) return spanq::report(SPAN_EINVAL, "span_plan_static: null argument");
  *out = nullptr;
  const int device = spanq::pool_device(pool);
  if (device < 0) return spanq::report(SPAN_EINVAL, "span_plan_static: needs a device pool");
  if (device >= kMaxDevices) return spanq::report(SPAN_EINVAL, "span_plan_static: device ordinal too large");
  unsigned char* region = nullptr;
  const hipError_t e = scratch_on(device, &region);
  if (e != hipSuccess)
    return spanq::report(SPAN_EHIP, (std::string("span_plan_static: hipGetSymbolAddress: ") + hipGetErrorString(e)).c_str());
  return spanq::plan_impl(pool, queries, n_queries, stream, out, region, SPAN_STATIC_SCRATCH_BYTES, "span_plan_static");
}
