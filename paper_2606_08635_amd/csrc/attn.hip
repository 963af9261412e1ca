// Attention-mode score (Sec. 3, Sec. 4.3): placeholder until the MFMA kernel lands.
#include "skv_internal.h"

namespace skv {

uint64_t attn_scratch_bytes(const Geometry&, int32_t, int32_t) { return 0; }

hipError_t launch_score_attn(const Geometry&, int32_t, int32_t, const uint16_t*, const uint16_t*,
                             const double*, void*, double*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace skv
