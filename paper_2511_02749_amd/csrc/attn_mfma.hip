// bf16 MFMA span attention (gfx950).
#include <hip/hip_runtime.h>

#include "../../include/spanq.h"
#include "kernels.h"

namespace spanq {

bool mfma_supported(int hq, int hkv, int d, int dtype) {
  (void)hq; (void)hkv; (void)d; (void)dtype;
  return false;
}

hipError_t launch_attn_mfma(const PoolGeom&, const WorkTile*, int, const KvPage*, const void*, void*, float*, float*,
                            const double*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace spanq
