// DMS-masked chunked prefill attention (placeholder until the MFMA kernel lands).
#include "dms_common.h"

namespace dms {

hipError_t launch_prefill_attention(const dms_config&, const Layout&, void*, void*, void*, int,
                                    int, const int32_t*, const int32_t*, int, int, const void*,
                                    const void*, const void*, const uint8_t*, float*,
                                    hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace dms
