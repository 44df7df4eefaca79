// Routing forward dispatch over d_head and the X dtype; the kernels live in
// route_kernel.hpp and are instantiated in route_<dh>_<dtype>.hip.

#include "launch.hpp"

namespace mhl {
namespace route_detail {
template <int DH, bool XF32>
hipError_t launch_dh_dtype(const void* X, const float* W, const float* bias,
                           int64_t T, int Nh, int Ne, int k, int32_t* idx,
                           float* gate, int32_t* partial, uint32_t* ticket,
                           hipStream_t s);
}  // namespace route_detail

using route_detail::launch_dh_dtype;

hipError_t launch_route_fwd(const void* X, const float* W_router,
                            const float* bias, int64_t T, int Nh, int dh,
                            int Ne, int k, bool x_f32, int32_t* idx,
                            float* gate, int32_t* partial, uint32_t* ticket,
                            hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dh == 128)
    return x_f32 ? launch_dh_dtype<128, true>(X, W_router, bias, T, Nh, Ne, k, idx, gate, partial, ticket, s)
                 : launch_dh_dtype<128, false>(X, W_router, bias, T, Nh, Ne, k, idx, gate, partial, ticket, s);
  if (dh == 64)
    return x_f32 ? launch_dh_dtype<64, true>(X, W_router, bias, T, Nh, Ne, k, idx, gate, partial, ticket, s)
                 : launch_dh_dtype<64, false>(X, W_router, bias, T, Nh, Ne, k, idx, gate, partial, ticket, s);
  return hipErrorInvalidValue;
}

}  // namespace mhl
