// bf16 MFMA forward for the main shapes (placeholder until the MFMA kernel lands).
#include "common.h"

namespace hsa {

bool forward_mfma_supported(const Dims&, bool) { return false; }

hipError_t launch_forward_mfma(const Dims&, const void*, const void*, const void*,
                               const int32_t*, const float*, void*, void*, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace hsa
