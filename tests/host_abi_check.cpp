// Host-side driver of the libmhlmoe C ABI for the sanitizer tier: compiled
// with the ABI's own source (argument validation and workspace layout) and
// with -fsanitize=address,undefined, it sizes every entry point's workspace
// over a table of shapes (valid, boundary and invalid) and walks the argument
// errors of every entry point.  Nothing here reaches a kernel: the kernel
// launchers are replaced by stubs that abort.  Output: one line per
// workspace query ("ws op T Nh dh Ne k dff dtype status bytes") and
// "FAIL ..." lines for argument checks that return an unexpected status.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "mhlmoe.h"

namespace {

struct S {
  int64_t T;
  int Nh, dh, Ne, k, dff;
};

const S kShapes[] = {
    // the five workloads and the GELU ones
    {256, 4, 64, 16, 2, 128},        {4096, 8, 128, 64, 8, 256},
    {16384, 16, 128, 128, 8, 256},   {16384, 16, 128, 256, 16, 128},
    {65536, 8, 128, 1024, 32, 128},  {8192, 8, 128, 384, 4, 256},
    {8192, 8, 128, 768, 8, 128},
    // edge shapes of the GPU tests
    {1, 2, 64, 8, 2, 64},            {37, 3, 128, 40, 5, 96},
    {129, 2, 128, 33, 3, 128},       {255, 2, 64, 16, 16, 64},
    {300, 2, 128, 64, 1, 32},        {200, 2, 128, 100, 32, 128},
    {77, 1, 64, 1, 1, 64},           {513, 2, 128, 1024, 8, 64},
    {70, 2, 128, 48, 4, 512},        {45, 2, 128, 20, 3, 480},
    {16, 1024, 64, 4, 2, 32},        {0, 2, 64, 8, 2, 64},
    // boundaries: the largest supported extents, T * k just below 2^31
    {(int64_t(1) << 31) / 32 - 1, 1, 128, 1024, 32, 512},
    {(int64_t(1) << 26), 1024, 128, 1024, 32, 512},
    {1, 1024, 128, 1024, 32, 32},
    // invalid or unsupported
    {-1, 2, 64, 8, 2, 64},           {16, 0, 64, 8, 2, 64},
    {16, 1025, 64, 8, 2, 64},        {16, 2, 96, 8, 2, 64},
    {16, 2, 64, 8, 9, 64},           {16, 2, 64, 8, 0, 64},
    {16, 2, 64, 40, 33, 64},         {16, 2, 64, 1025, 2, 64},
    {16, 2, 64, 8, 2, 0},            {16, 2, 64, 8, 2, 544},
    {16, 2, 64, 8, 2, 48},           {int64_t(1) << 31, 2, 64, 8, 2, 64},
    {int64_t(1) << 62, 2, 64, 8, 2, 64},
};

int g_fail = 0;

void expect(const char* what, mhlmoe_status got, mhlmoe_status want) {
  if (got != want) {
    std::printf("FAIL %s: status %d, expected %d (%s)\n", what, (int)got, (int)want,
                mhlmoe_last_error());
    ++g_fail;
  }
}

}  // namespace

int main() {
  for (const S& s : kShapes)
    for (int op = 0; op <= 7; ++op)
      for (int dt = 0; dt <= 1; ++dt) {
        size_t bytes = 0;
        const mhlmoe_status st = mhlmoe_workspace_size((mhlmoe_op)op, s.T, s.Nh, s.dh, s.Ne, s.k,
                                                       s.dff, (mhlmoe_dtype)dt, &bytes);
        std::printf("ws %d %lld %d %d %d %d %d %d %d %zu\n", op, (long long)s.T, s.Nh, s.dh, s.Ne,
                    s.k, s.dff, dt, (int)st, st == MHLMOE_OK ? bytes : size_t(0));
      }
  size_t b = 0;
  expect("workspace_size NULL bytes",
         mhlmoe_workspace_size(MHLMOE_OP_LAYER, 16, 2, 64, 8, 2, 64, MHLMOE_BF16, nullptr),
         MHLMOE_EINVAL);
  expect("workspace_size unknown op",
         mhlmoe_workspace_size((mhlmoe_op)99, 16, 2, 64, 8, 2, 64, MHLMOE_BF16, &b),
         MHLMOE_EINVAL);
  expect("workspace_size unknown dtype",
         mhlmoe_workspace_size(MHLMOE_OP_ROUTE, 16, 2, 64, 8, 2, 64, (mhlmoe_dtype)5, &b),
         MHLMOE_EINVAL);

  // Argument errors: A stands for any 16-byte aligned non-NULL device
  // pointer (never dereferenced: every call below fails its checks first).
  void* A = reinterpret_cast<void*>(uintptr_t(0x10000));
  void* M = reinterpret_cast<void*>(uintptr_t(0x10004));  // misaligned
  float* Af = static_cast<float*>(A);
  int32_t* Ai = static_cast<int32_t*>(A);
  const size_t ws = size_t(1) << 30;
  const mhlmoe_dtype bf = MHLMOE_BF16;
  expect("route NULL X", mhlmoe_route(nullptr, Af, nullptr, 16, 2, 64, 8, 2, bf, Ai, Af, Ai, A, ws, nullptr), MHLMOE_EINVAL);
  expect("route misaligned gate", mhlmoe_route(A, Af, nullptr, 16, 2, 64, 8, 2, bf, Ai, (float*)M, Ai, A, ws, nullptr), MHLMOE_EINVAL);
  expect("route small workspace", mhlmoe_route(A, Af, nullptr, 16, 2, 64, 8, 2, bf, Ai, Af, Ai, A, 8, nullptr), MHLMOE_EWORKSPACE);
  expect("route k > Ne", mhlmoe_route(A, Af, nullptr, 16, 2, 64, 8, 9, bf, Ai, Af, Ai, A, ws, nullptr), MHLMOE_EINVAL);
  expect("route_static too large", mhlmoe_route_static(A, Af, nullptr, int64_t(1) << 22, 8, 128, 1024, 8, bf, Ai, Af, Ai, nullptr), MHLMOE_EWORKSPACE);
  expect("route_static NULL counts", mhlmoe_route_static(A, Af, nullptr, 16, 2, 64, 8, 2, bf, Ai, Af, nullptr, nullptr), MHLMOE_EINVAL);
  expect("route_backward NULL dgate", mhlmoe_route_backward(A, Af, Ai, Af, nullptr, 16, 2, 64, 8, 2, bf, A, Af, A, ws, nullptr), MHLMOE_EINVAL);
  expect("bucket NULL offsets", mhlmoe_bucket(Ai, 16, 2, 8, 2, Ai, nullptr, Ai, A, ws, nullptr), MHLMOE_EINVAL);
  expect("bucket k > Ne", mhlmoe_bucket(Ai, 16, 2, 8, 9, Ai, Ai, Ai, A, ws, nullptr), MHLMOE_EINVAL);
  expect("experts NULL W3", mhlmoe_experts(A, Ai, Af, A, nullptr, A, 16, 2, 64, 8, 2, 64, bf, A, A, ws, nullptr), MHLMOE_EINVAL);
  expect("experts d_ff 48", mhlmoe_experts(A, Ai, Af, A, A, A, 16, 2, 64, 8, 2, 48, bf, A, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("experts workspace misaligned", mhlmoe_experts(A, Ai, Af, A, A, A, 16, 2, 64, 8, 2, 64, bf, A, M, ws, nullptr), MHLMOE_EINVAL);
  expect("layer NULL W_router", mhlmoe_layer(A, nullptr, nullptr, A, A, A, 16, 2, 64, 8, 2, 64, bf, A, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EINVAL);
  expect("layer d_head 96", mhlmoe_layer(A, Af, nullptr, A, A, A, 16, 2, 96, 8, 2, 64, bf, A, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("experts_gelu d_ff 80", mhlmoe_experts_gelu(A, Ai, Af, A, A, 16, 2, 128, 8, 2, 80, MHLMOE_F32, A, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("layer_gelu d_head 96", mhlmoe_layer_gelu(A, Af, nullptr, A, A, 16, 2, 96, 8, 2, 96, bf, A, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("layer_backward fp32", mhlmoe_layer_backward(A, Af, A, A, A, Ai, Af, A, 16, 2, 64, 8, 2, 64, MHLMOE_F32, A, Af, Af, Af, Af, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("layer_backward NULL dW2", mhlmoe_layer_backward(A, Af, A, A, A, Ai, Af, A, 16, 2, 64, 8, 2, 64, bf, A, Af, Af, Af, nullptr, A, ws, nullptr), MHLMOE_EINVAL);
  expect("layer_gelu_backward small workspace", mhlmoe_layer_gelu_backward(A, Af, A, A, Ai, Af, A, 16, 2, 64, 8, 2, 64, bf, A, Af, Af, Af, A, 16, nullptr), MHLMOE_EWORKSPACE);
  expect("layer_routed NULL R", mhlmoe_layer_routed(A, nullptr, Af, nullptr, A, A, A, 16, 2, 64, 8, 2, 64, bf, A, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EINVAL);
  expect("backward_routed dR == dX", mhlmoe_layer_backward_routed(A, A, Af, A, A, A, Ai, Af, A, 16, 2, 64, 8, 2, 64, bf, A, A, Af, Af, Af, Af, A, ws, nullptr), MHLMOE_EINVAL);
  expect("latent d_model 0", mhlmoe_latent_layer(A, A, Af, nullptr, A, A, A, A, 16, 0, 2, 64, 8, 2, 64, 0, bf, A, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EUNSUPPORTED);
  expect("latent routing_tokens 2", mhlmoe_latent_layer(A, A, Af, nullptr, A, A, A, A, 16, 64, 2, 64, 8, 2, 64, 2, bf, A, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, A, ws, nullptr), MHLMOE_EINVAL);
  expect("latent_backward NULL dout", mhlmoe_latent_layer_backward(A, A, Af, A, A, A, A, A, nullptr, A, Ai, Af, nullptr, 16, 64, 2, 64, 8, 2, 64, 0, bf, A, Af, Af, Af, Af, Af, Af, A, ws, nullptr), MHLMOE_EINVAL);
  expect("bias_update negative rate", mhlmoe_bias_update(Ai, Af, 2, 8, -1.0f, nullptr), MHLMOE_EINVAL);
  expect("bias_update 1025 experts", mhlmoe_bias_update(Ai, Af, 2, 1025, 1.0f, nullptr), MHLMOE_EINVAL);
  expect("timing_query NULL", mhlmoe_timing_query(nullptr, nullptr, nullptr), MHLMOE_EINVAL);
  std::printf("done %d failures\n", g_fail);
  return g_fail == 0 ? 0 : 1;
}
