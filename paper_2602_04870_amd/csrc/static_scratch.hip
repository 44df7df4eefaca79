// The static scratch of the allocation-free entry point (mhlmoe_route_static):
// device memory for callers that cannot allocate (code under graph capture,
// serving loops).  The array's name is a host-side stand-in, not a device
// address: host code uses only the address hipGetSymbolAddress gives, once
// per device (each device holds its own copy, at its own address).
#include <mutex>

#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace
}  // namespace mhl

static __device__ __align__(256) uint8_t scratch[mhl::kStaticScratchBytes];

namespace mhl {

hipError_t static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace mhl
