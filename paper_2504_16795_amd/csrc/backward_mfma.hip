// bf16 MFMA backward for the main shapes (placeholder until the MFMA kernels land).
#include "common.h"

namespace hsa {

bool backward_mfma_supported(const Dims&, bool) { return false; }
size_t backward_mfma_workspace(const Dims&) { return 0; }

hipError_t launch_backward_mfma(const Dims&, const void*, const void*, const void*,
                                const float*, const int32_t*, const float*, const void*, void*,
                                void*, void*, void*, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace hsa
