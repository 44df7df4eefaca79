// Routing forward kernels for d_head = 128, bf16 X.
#include "route_kernel.hpp"

namespace mhl {
namespace route_detail {
template hipError_t launch_dh_dtype<128, false>(
    const void*, const float*, const float*, int64_t, int, int, int, int32_t*,
    float*, int32_t*, uint32_t*, hipStream_t);
}  // namespace route_detail
}  // namespace mhl
