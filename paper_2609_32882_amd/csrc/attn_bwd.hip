// Block-sparse attention backward (placeholder until the kernels land).
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

hipError_t launch_attn_bwd(int, int, const void*, const void*, const void*, const void*, const float*,
                           const void*, const int32_t*, const int32_t*, const int32_t*, const int32_t*,
                           int64_t, void*, void*, void*, float*, int, int, int, int, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace vsa2
