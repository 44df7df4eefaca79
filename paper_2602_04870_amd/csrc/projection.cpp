// Dense projections around the per-head MoEs (Eq. (5)-(6)): row-major GEMMs
// through hipBLASLt, the library GEMM of ROCm (these are plain dense
// contractions with no per-expert structure, so a tuned library kernel is the
// right tool).  Plans (descriptors, layouts and the heuristic's algorithm)
// are cached per device and shape, at most kMaxPlans of them (a caller whose
// batch size keeps changing would otherwise grow the cache without bound; it
// is emptied when full); a hipBLASLt handle is created once per device on
// first use.

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <map>
#include <mutex>
#include <tuple>

#include "launch.hpp"

namespace mhl {
namespace {

struct Plan {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  hipblasLtMatmulAlgo_t algo{};
  size_t ws = 0;
};

// (device, M, N, K, transA, transB, input type, output type, accumulate)
using PlanKey = std::tuple<int, int64_t, int64_t, int64_t, bool, bool, int, int, bool>;

constexpr size_t kMaxPlans = 256;

std::mutex g_mu;
std::map<int, hipblasLtHandle_t> g_handles;
std::map<PlanKey, Plan> g_plans;

void destroy_plan(Plan& p) {
  if (p.a) hipblasLtMatrixLayoutDestroy(p.a);
  if (p.b) hipblasLtMatrixLayoutDestroy(p.b);
  if (p.c) hipblasLtMatrixLayoutDestroy(p.c);
  if (p.desc) hipblasLtMatmulDescDestroy(p.desc);
  p = Plan{};
}

hipError_t to_hip(hipblasStatus_t st) {
  switch (st) {
    case HIPBLAS_STATUS_SUCCESS: return hipSuccess;
    case HIPBLAS_STATUS_ALLOC_FAILED: return hipErrorOutOfMemory;
    case HIPBLAS_STATUS_INVALID_VALUE: return hipErrorInvalidValue;
    case HIPBLAS_STATUS_NOT_SUPPORTED: return hipErrorNotSupported;
    default: return hipErrorUnknown;
  }
}

#define MHL_BLAS(expr)                                   \
  do {                                                   \
    const hipblasStatus_t st_ = (expr);                  \
    if (st_ != HIPBLAS_STATUS_SUCCESS) return to_hip(st_); \
  } while (0)

// Zero fill (used for an empty contraction, K == 0, where the product is 0).
__global__ __launch_bounds__(256) void zero_kernel(uint16_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = 0u;
}

hipError_t handle_for(int dev, hipblasLtHandle_t* h) {
  auto it = g_handles.find(dev);
  if (it != g_handles.end()) {
    *h = it->second;
    return hipSuccess;
  }
  MHL_BLAS(hipblasLtCreate(h));
  g_handles[dev] = *h;
  return hipSuccess;
}

// Column-major view of the row-major product C[M][N] = op(A) op(B): hipBLASLt
// computes C^T = op(B)^T op(A)^T, i.e. an (N x M) column-major result whose
// first operand is B and second is A.  A row-major [r][c] array is the
// column-major (c x r) matrix with leading dimension c.
hipError_t make_plan(hipblasLtHandle_t h, int64_t M, int64_t N, int64_t K, bool ta, bool tb,
                     hipDataType tin, hipDataType tout, size_t ws_limit, Plan* p) {
  const hipblasOperation_t opB = tb ? HIPBLAS_OP_T : HIPBLAS_OP_N;
  const hipblasOperation_t opA = ta ? HIPBLAS_OP_T : HIPBLAS_OP_N;
  MHL_BLAS(hipblasLtMatmulDescCreate(&p->desc, HIPBLAS_COMPUTE_32F, HIP_R_32F));
  MHL_BLAS(hipblasLtMatmulDescSetAttribute(p->desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opB, sizeof(opB)));
  MHL_BLAS(hipblasLtMatmulDescSetAttribute(p->desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opA, sizeof(opA)));
  // B stored [K][N] (tb false) is column-major N x K; stored [N][K], K x N.
  MHL_BLAS(tb ? hipblasLtMatrixLayoutCreate(&p->b, tin, K, N, K)
              : hipblasLtMatrixLayoutCreate(&p->b, tin, N, K, N));
  // A stored [M][K] (ta false) is column-major K x M; stored [K][M], M x K.
  MHL_BLAS(ta ? hipblasLtMatrixLayoutCreate(&p->a, tin, M, K, M)
              : hipblasLtMatrixLayoutCreate(&p->a, tin, K, M, K));
  MHL_BLAS(hipblasLtMatrixLayoutCreate(&p->c, tout, N, M, N));
  hipblasLtMatmulPreference_t pref = nullptr;
  MHL_BLAS(hipblasLtMatmulPreferenceCreate(&pref));
  const uint64_t lim = ws_limit;
  hipblasStatus_t st = hipblasLtMatmulPreferenceSetAttribute(
      pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &lim, sizeof(lim));
  hipblasLtMatmulHeuristicResult_t res[1];
  int n = 0;
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatmulAlgoGetHeuristic(h, p->desc, p->b, p->a, p->c, p->c, pref, 1, res, &n);
  hipblasLtMatmulPreferenceDestroy(pref);
  if (st != HIPBLAS_STATUS_SUCCESS) return to_hip(st);
  if (n < 1 || res[0].state != HIPBLAS_STATUS_SUCCESS) return hipErrorNotSupported;
  p->algo = res[0].algo;
  p->ws = res[0].workspaceSize;
  return hipSuccess;
}

}  // namespace

hipError_t gemm_rowmajor(int64_t M, int64_t N, int64_t K, const void* A, bool ta, const void* B,
                         bool tb, bool bf16_in, bool f32_out, bool accumulate, void* C,
                         void* blas_ws, size_t blas_ws_bytes, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  if (K == 0) {
    if (accumulate) return hipSuccess;
    // M * N elements of 4 bytes (fp32) or 2 (bf16), cleared as 2-byte units.
    const int64_t units = (f32_out || !bf16_in ? 2 : 1) * M * N;
    const int64_t blocks = ceil_div(units, 256) < 1024 ? ceil_div(units, 256) : 1024;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint16_t*)C, units);
    return hipGetLastError();
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const hipDataType tin = bf16_in ? HIP_R_16BF : HIP_R_32F;
  const hipDataType tout = f32_out ? HIP_R_32F : tin;
  // The lock is held through the enqueue, so no other thread can empty the
  // cache (destroying this plan's descriptors) while they are in use.
  std::lock_guard<std::mutex> lk(g_mu);
  hipblasLtHandle_t h = nullptr;
  e = handle_for(dev, &h);
  if (e != hipSuccess) return e;
  const PlanKey key{dev, M, N, K, ta, tb, (int)tin, (int)tout, accumulate};
  auto it = g_plans.find(key);
  if (it == g_plans.end()) {
    Plan p;
    e = make_plan(h, M, N, K, ta, tb, tin, tout, blas_ws_bytes, &p);
    if (e != hipSuccess) {
      destroy_plan(p);
      return e;
    }
    // Emptied when full (matmuls already enqueued do not refer to the
    // host-side descriptors any more).
    if (g_plans.size() >= kMaxPlans) {
      for (auto& kv : g_plans) destroy_plan(kv.second);
      g_plans.clear();
    }
    it = g_plans.emplace(key, p).first;
  }
  const Plan& plan = it->second;
  if (plan.ws > blas_ws_bytes) return hipErrorInvalidValue;
  const float alpha = 1.0f, beta = accumulate ? 1.0f : 0.0f;
  MHL_BLAS(hipblasLtMatmul(h, plan.desc, &alpha, B, plan.b, A, plan.a, &beta, C, plan.c, C,
                           plan.c, &plan.algo, blas_ws, blas_ws_bytes, s));
  return hipGetLastError();
}

}  // namespace mhl
