// The libmhlmoe C ABI: argument validation, workspace layout and the launch
// sequence of every entry point.  No allocation, no host synchronisation
// (unless MHLMOE_DEBUG=1 is set, which synchronises and checks after every
// launch).

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mhlmoe.h"
#include "launch.hpp"

namespace {

thread_local std::string g_error;

mhlmoe_status fail(mhlmoe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

bool debug_sync() {
  static const bool on = [] {
    const char* v = std::getenv("MHLMOE_DEBUG");
    return v != nullptr && v[0] == '1';
  }();
  return on;
}

struct Shape {
  int64_t T;
  int Nh, dh, Ne, k, dff;
  mhlmoe_dtype dtype;
  int64_t slots() const { return T * k; }  // per head
  size_t esize() const { return dtype == MHLMOE_F32 ? 4 : 2; }
};

mhlmoe_status check_route_shape(const Shape& s) {
  if (s.T < 0) return fail(MHLMOE_EINVAL, "T must be >= 0 (got %lld)", (long long)s.T);
  if (s.Nh < 1) return fail(MHLMOE_EINVAL, "n_heads must be >= 1 (got %d)", s.Nh);
  if (s.Nh > mhl::kMaxHeadsSupported)
    return fail(MHLMOE_EUNSUPPORTED, "n_heads must be <= %d", mhl::kMaxHeadsSupported);
  if (s.k < 1) return fail(MHLMOE_EINVAL, "top_k must be >= 1 (got %d)", s.k);
  if (s.Ne < 1) return fail(MHLMOE_EINVAL, "n_experts must be >= 1 (got %d)", s.Ne);
  if (s.k > s.Ne) return fail(MHLMOE_EINVAL, "top_k (%d) > n_experts (%d)", s.k, s.Ne);
  if (s.k > 32) return fail(MHLMOE_EUNSUPPORTED, "top_k %d > 32", s.k);
  if (s.Ne > 1024) return fail(MHLMOE_EUNSUPPORTED, "n_experts %d > 1024", s.Ne);
  // T * top_k < 2^31, tested without forming the product (T may be huge)
  if (s.T > ((int64_t(1) << 31) - 1) / s.k)
    return fail(MHLMOE_EUNSUPPORTED, "T * top_k must be < 2^31");
  if (s.dtype != MHLMOE_F32 && s.dtype != MHLMOE_BF16)
    return fail(MHLMOE_EINVAL, "unknown dtype %d", (int)s.dtype);
  return MHLMOE_OK;
}

mhlmoe_status check_dh(const Shape& s) {
  if (s.dh != 64 && s.dh != 128)
    return fail(MHLMOE_EUNSUPPORTED, "d_head %d not in {64, 128}", s.dh);
  return MHLMOE_OK;
}

mhlmoe_status check_backward_dtype(const Shape& s) {
  if (s.dtype != MHLMOE_BF16) return fail(MHLMOE_EUNSUPPORTED, "layer backward supports bf16 only");
  return MHLMOE_OK;
}

mhlmoe_status check_ffn_shape(const Shape& s) {
  if (s.dff < 32 || s.dff > 512 || s.dff % 32 != 0)
    return fail(MHLMOE_EUNSUPPORTED, "d_ff %d must be a multiple of 32 in [32, 512]", s.dff);
  return MHLMOE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

mhlmoe_status need(const void* p, const char* name) {
  if (p == nullptr) return fail(MHLMOE_EINVAL, "%s is NULL", name);
  if (!aligned16(p)) return fail(MHLMOE_EINVAL, "%s is not 16-byte aligned", name);
  return MHLMOE_OK;
}

// Tensors with a T-sized dimension may be NULL when T == 0.
mhlmoe_status need_rows(const void* p, const char* name, int64_t T) {
  return T == 0 ? (p != nullptr && !aligned16(p)
                       ? fail(MHLMOE_EINVAL, "%s is not 16-byte aligned", name)
                       : MHLMOE_OK)
                : need(p, name);
}

mhlmoe_status maybe(const void* p, const char* name) {
  if (p != nullptr && !aligned16(p)) return fail(MHLMOE_EINVAL, "%s is not 16-byte aligned", name);
  return MHLMOE_OK;
}

#define MHL_TRY(expr)                       \
  do {                                      \
    const mhlmoe_status st_ = (expr);       \
    if (st_ != MHLMOE_OK) return st_;       \
  } while (0)

// Workspace: a list of 256-byte aligned regions.
struct Layout {
  size_t ticket = 0, counts = 0, partial = 0, base = 0, offsets = 0, tile_start = 0,
         tile_info = 0, head_base = 0, perm = 0, yslot = 0, idx = 0, gate = 0, dg = 0, ds = 0,
         dw_order = 0, rdw_base = 0, rdw_part = 0, lat_x = 0, lat_r = 0, lat_y = 0, lat_dy = 0, lat_dx = 0, lat_dr = 0,
         blas = 0, total = 0;
};

size_t bump(size_t& cur, size_t bytes) {
  const size_t at = cur;
  cur += (bytes + 255) & ~size_t(255);
  return at;
}

Layout make_layout(mhlmoe_op op, const Shape& s) {
  if (op == MHLMOE_OP_LATENT_LAYER || op == MHLMOE_OP_LATENT_BACKWARD) {
    // The inner layer's (or layer backward's) workspace first, then the
    // latent activations the caller did not keep and hipBLASLt's workspace.
    const bool fwd = op == MHLMOE_OP_LATENT_LAYER;
    Layout L = make_layout(fwd ? MHLMOE_OP_LAYER : MHLMOE_OP_LAYER_BACKWARD, s);
    size_t cur = L.total;
    const size_t lat = s.esize() * (size_t)s.T * s.Nh * s.dh;
    if (fwd) {
      L.lat_x = bump(cur, lat);
      L.lat_r = bump(cur, lat);
      L.lat_y = bump(cur, lat);
    } else {
      L.lat_dy = bump(cur, lat);
      L.lat_dx = bump(cur, lat);
      L.lat_dr = bump(cur, lat);
    }
    L.blas = bump(cur, mhl::kBlasWorkspace);
    L.total = cur;
    return L;
  }
  Layout L;
  size_t cur = 0;
  const int64_t nblk = mhl::num_token_blocks(s.T);
  const size_t hist_bytes = sizeof(int32_t) * (size_t)s.Nh * nblk * s.Ne;
  L.ticket = bump(cur, sizeof(uint32_t));
  L.counts = bump(cur, sizeof(int32_t) * (size_t)s.Nh * s.Ne);
  L.partial = bump(cur, hist_bytes);
  if (op == MHLMOE_OP_ROUTE) {
    L.total = cur;
    return L;
  }
  L.base = bump(cur, hist_bytes);
  if (op == MHLMOE_OP_BUCKET) {
    L.total = cur;
    return L;
  }
  if (op == MHLMOE_OP_ROUTE_BACKWARD) {  // clustering (no tile list), dS, dW_router sums
    L.offsets = bump(cur, sizeof(int32_t) * (size_t)s.Nh * (s.Ne + 1));
    L.perm = bump(cur, sizeof(int32_t) * (size_t)s.Nh * s.slots());
    L.ds = bump(cur, sizeof(float) * (size_t)s.T * s.Nh * s.k);
    L.rdw_base = bump(cur, sizeof(int32_t) * ((size_t)s.Nh * s.Ne + 1));
    L.rdw_part = bump(cur, sizeof(float) * (size_t)mhl::rdw_max_segments(s.T, s.Nh, s.Ne, s.k) *
                               s.dh);
    L.total = cur;
    return L;
  }
  const int64_t mt = mhl::max_tiles_per_head(s.T, s.k, s.Ne);
  L.offsets = bump(cur, sizeof(int32_t) * (size_t)s.Nh * (s.Ne + 1));
  L.tile_start = bump(cur, sizeof(int32_t) * (size_t)s.Nh * (s.Ne + 1));
  L.tile_info = bump(cur, sizeof(mhl::TileInfo) * (size_t)s.Nh * mt);
  L.head_base = bump(cur, sizeof(int32_t) * (size_t)(s.Nh + 1));
  L.perm = bump(cur, sizeof(int32_t) * (size_t)s.Nh * s.slots());
  L.yslot = bump(cur, s.esize() * (size_t)s.T * s.Nh * s.k * s.dh);
  if (op == MHLMOE_OP_LAYER) {
    L.idx = bump(cur, sizeof(int32_t) * (size_t)s.T * s.Nh * s.k);
    L.gate = bump(cur, sizeof(float) * (size_t)s.T * s.Nh * s.k);
  }
  if (op == MHLMOE_OP_LAYER_BACKWARD) {  // yslot holds the per-slot dX_expert
    L.dg = bump(cur, sizeof(float) * (size_t)s.T * s.Nh * s.k);
    L.ds = bump(cur, sizeof(float) * (size_t)s.T * s.Nh * s.k);
    L.dw_order = bump(cur, sizeof(int32_t) * (size_t)s.Nh * s.Ne);
    L.rdw_base = bump(cur, sizeof(int32_t) * ((size_t)s.Nh * s.Ne + 1));
    L.rdw_part = bump(cur, sizeof(float) * (size_t)mhl::rdw_max_segments(s.T, s.Nh, s.Ne, s.k) *
                               s.dh);
  }
  L.total = cur;
  return L;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(reinterpret_cast<uint8_t*>(ws) + off);
}

mhlmoe_status check_ws(mhlmoe_op op, const Shape& s, void* ws, size_t ws_bytes, Layout& L) {
  L = make_layout(op, s);
  if (L.total > 0) {
    if (ws == nullptr) return fail(MHLMOE_EWORKSPACE, "workspace is NULL (need %zu bytes)", L.total);
    if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
      return fail(MHLMOE_EINVAL, "workspace is not 256-byte aligned");
    if (ws_bytes < L.total)
      return fail(MHLMOE_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, L.total);
  }
  return MHLMOE_OK;
}

mhlmoe_status launched(hipError_t e, const char* what, hipStream_t stream) {
  if (e == hipSuccess && debug_sync()) {
    e = hipStreamSynchronize(stream);
    if (e == hipSuccess) e = hipGetLastError();
  }
  if (e != hipSuccess) return fail(MHLMOE_EHIP, "%s: %s", what, hipGetErrorString(e));
  return MHLMOE_OK;
}

// Optional per-kernel timing: each launch bracketed by two events on its own
// stream.  Events are pooled and reused; nothing is recorded when off.
struct TimingRecord {
  const char* name;  // string literal
  hipEvent_t start, stop;
};
std::atomic<bool> g_timing{false};
std::mutex g_timing_mu;
std::vector<TimingRecord> g_records;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launch one kernel (the callable returns the launch's hipError_t).
template <class F>
mhlmoe_status run_kernel(const char* name, hipStream_t stream, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  const bool timing = g_timing.load(std::memory_order_relaxed);
  if (timing) {
    std::lock_guard<std::mutex> lk(g_timing_mu);
    a = take_event();
    b = take_event();
    if (a) hipEventRecord(a, stream);
  }
  const hipError_t e = launch();
  if (timing && a && b) {
    hipEventRecord(b, stream);
    std::lock_guard<std::mutex> lk(g_timing_mu);
    g_records.push_back(TimingRecord{name, a, b});
  }
  return launched(e, name, stream);
}

// Clustering from the per-block histograms in the workspace: counts,
// offsets, (tile_rows > 0) the FFN tile list, and perm.
mhlmoe_status run_cluster(const Shape& s, const int32_t* idx, int32_t* counts, int32_t* offsets,
                          int32_t* perm, int tile_rows, const Layout& L, void* ws,
                          hipStream_t stream) {
  const int64_t mt = mhl::max_tiles_per_head(s.T, s.k, s.Ne);
  int32_t* partial = at<int32_t>(ws, L.partial);
  int32_t* base = at<int32_t>(ws, L.base);
  int32_t* tile_start = tile_rows > 0 ? at<int32_t>(ws, L.tile_start) : nullptr;
  mhl::TileInfo* tiles = tile_rows > 0 ? at<mhl::TileInfo>(ws, L.tile_info) : nullptr;
  int32_t* head_base = tile_rows > 0 ? at<int32_t>(ws, L.head_base) : nullptr;
  uint32_t* ticket = at<uint32_t>(ws, L.ticket);
  MHL_TRY(run_kernel("count_scan", stream, [&] {
    return mhl::launch_count_scan(partial, s.T, s.Nh, s.Ne, tile_rows, counts, base, offsets,
                                  tile_start, ticket, stream);
  }));
  MHL_TRY(run_kernel("scatter", stream, [&] {
    return mhl::launch_scatter(idx, base, offsets, tile_start, head_base, s.T, s.Nh, s.Ne, s.k,
                               tile_rows, mt, perm, tiles, stream);
  }));
  return MHLMOE_OK;
}

// Clustering, grouped FFN and combine, given idx/gate and the per-block
// histograms in the workspace (counts: caller's array or NULL).  W3 == NULL
// selects the two-matrix GELU expert (W1 = W_in, W2 = W_out).
mhlmoe_status run_experts(const Shape& s, const void* X, const int32_t* idx, const float* gate,
                          int32_t* counts, const void* W1, const void* W3, const void* W2,
                          void* Y, const Layout& L, void* ws, hipStream_t stream) {
  const bool f32 = s.dtype == MHLMOE_F32;
  int32_t* perm = at<int32_t>(ws, L.perm);
  const mhl::TileInfo* tiles = at<mhl::TileInfo>(ws, L.tile_info);
  const int32_t* head_base = at<int32_t>(ws, L.head_base);
  void* yslot = at<void>(ws, L.yslot);
  if (counts == nullptr) counts = at<int32_t>(ws, L.counts);
  MHL_TRY(run_cluster(s, idx, counts, at<int32_t>(ws, L.offsets), perm,
                      mhl::ffn_tile_rows(s.T, s.Nh, s.dh, s.Ne, s.k, s.dff, f32), L, ws,
                      stream));
  MHL_TRY(run_kernel("ffn", stream, [&] {
    if (W3 == nullptr)
      return mhl::launch_ffn_gelu(X, gate, perm, tiles, head_base, W1, W2, s.T, s.Nh, s.dh, s.Ne,
                                  s.k, s.dff, f32, yslot, stream);
    return mhl::launch_ffn(X, gate, perm, tiles, head_base, W1, W3, W2, s.T, s.Nh, s.dh, s.Ne, s.k,
                           s.dff, f32, yslot, stream);
  }));
  // The bf16 d_h-128 kernels (SwiGLU and GELU) leave the gate to the
  // combine.
  const bool gated = mhl::ffn_slots_gated(s.T, s.Nh, s.dh, s.dff, f32);
  MHL_TRY(run_kernel("combine", stream, [&] {
    return mhl::launch_combine(yslot, gated ? nullptr : gate, s.T, s.Nh, s.dh, s.k, f32, Y,
                               stream);
  }));
  return MHLMOE_OK;
}

// The forward layer: routing from R (X itself, or the separate routing
// sub-tokens of Sec. 4.4), then the experts on X.  W3 == NULL selects the
// two-matrix GELU expert.
mhlmoe_status layer_impl(const Shape& s, const void* X, const void* R, const float* W_router,
                         const float* bias, const void* W1, const void* W3, const void* W2,
                         void* Y, int32_t* idx, float* gate, int32_t* counts, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need_rows(R, "R", s.T));
  MHL_TRY(need(W_router, "W_router"));
  MHL_TRY(maybe(bias, "bias"));
  MHL_TRY(need(W1, W3 == nullptr ? "W_in" : "W1"));
  MHL_TRY(need(W2, W3 == nullptr ? "W_out" : "W2"));
  MHL_TRY(need_rows(Y, "Y", s.T));
  MHL_TRY(maybe(idx, "idx"));
  MHL_TRY(maybe(gate, "gate"));
  MHL_TRY(maybe(counts, "counts"));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_LAYER, s, workspace, workspace_bytes, L));
  if (idx == nullptr) idx = at<int32_t>(workspace, L.idx);
  if (gate == nullptr) gate = at<float>(workspace, L.gate);
  int32_t* partial = at<int32_t>(workspace, L.partial);
  if (s.T == 0) {
    if (counts == nullptr) return MHLMOE_OK;
    return run_kernel("count_scan", stream, [&] {
      return mhl::launch_count_scan(partial, s.T, s.Nh, s.Ne, 0, counts, nullptr, nullptr,
                                    nullptr, nullptr, stream);
    });
  }
  MHL_TRY(run_kernel("route_fwd", stream, [&] {
    return mhl::launch_route_fwd(R, W_router, bias, s.T, s.Nh, s.dh, s.Ne, s.k,
                                 s.dtype == MHLMOE_F32, idx, gate, partial,
                                 at<uint32_t>(workspace, L.ticket), stream);
  }));
  return run_experts(s, X, idx, gate, counts, W1, W3, W2, Y, L, workspace, stream);
}

// The layer backward.  dR == NULL: the router read X, and its input
// gradient is added into dX.  Otherwise the router read R: its input
// gradient goes to dR and dW_router is taken against R.  W3 == NULL selects
// the two-matrix GELU expert (W1 = W_in, W2 = W_out; dW3 is not written).
mhlmoe_status backward_impl(const Shape& s, const void* X, const void* R, const float* W_router,
                            const void* W1, const void* W3, const void* W2, const int32_t* idx,
                            const float* gate, const void* dY, void* dX, void* dR,
                            float* dW_router, float* dW1, float* dW3, float* dW2,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(check_backward_dtype(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need_rows(R, "R", s.T));
  MHL_TRY(need(W_router, "W_router"));
  const bool gelu = W3 == nullptr;
  MHL_TRY(need(W1, gelu ? "W_in" : "W1"));
  MHL_TRY(need(W2, gelu ? "W_out" : "W2"));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(need_rows(gate, "gate", s.T));
  MHL_TRY(need_rows(dY, "dY", s.T));
  MHL_TRY(need_rows(dX, "dX", s.T));
  MHL_TRY(need(dW_router, "dW_router"));
  MHL_TRY(need(dW1, gelu ? "dW_in" : "dW1"));
  if (!gelu) MHL_TRY(need(dW3, "dW3"));
  MHL_TRY(need(dW2, gelu ? "dW_out" : "dW2"));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_LAYER_BACKWARD, s, workspace, workspace_bytes, L));
  void* ws = workspace;
  int32_t* perm = at<int32_t>(ws, L.perm);
  int32_t* offsets = at<int32_t>(ws, L.offsets);
  int32_t* order = at<int32_t>(ws, L.dw_order);
  const mhl::TileInfo* tiles = at<mhl::TileInfo>(ws, L.tile_info);
  const int32_t* head_base = at<int32_t>(ws, L.head_base);
  void* dxslot = at<void>(ws, L.yslot);
  float* dg = at<float>(ws, L.dg);
  float* dS = at<float>(ws, L.ds);
  // Clustering of the forward's idx (with T == 0 it still yields all-zero
  // offsets, so the weight-gradient kernels write zeros everywhere).
  MHL_TRY(run_kernel("hist", stream, [&] {
    return mhl::launch_hist(idx, s.T, s.Nh, s.Ne, s.k, at<int32_t>(ws, L.partial),
                            at<uint32_t>(ws, L.ticket), stream);
  }));
  MHL_TRY(run_cluster(s, idx, at<int32_t>(ws, L.counts), offsets, perm, mhl::kTileRows, L, ws,
                      stream));
  MHL_TRY(run_kernel("bwd_dx", stream, [&] {
    return mhl::launch_bwd_dx(X, dY, gate, perm, tiles, head_base, W1, W3, W2, s.T, s.Nh, s.dh,
                              s.Ne, s.k, s.dff, dxslot, dg, stream);
  }));
  MHL_TRY(run_kernel("bwd_combine", stream, [&] {
    return mhl::launch_bwd_combine(idx, gate, dg, dxslot, W_router, s.T, s.Nh, s.dh, s.Ne, s.k,
                                   dX, dR, dS, stream);
  }));
  // dW_router from the router's input (X, or R with separate routing
  // sub-tokens) by the segment-parallel kernels.
  MHL_TRY(run_kernel("bwd_dw", stream, [&] {
    return mhl::launch_bwd_dw(X, dY, gate, perm, offsets, order, W1, W3, W2, s.T, s.Nh, s.dh,
                              s.Ne, s.k, s.dff, dW1, gelu ? nullptr : dW3, dW2, stream);
  }));
  return run_kernel("router_dw", stream, [&] {
    return mhl::launch_router_dw(R, false, dS, perm, offsets, s.T, s.Nh, s.dh, s.Ne, s.k,
                                 at<int32_t>(ws, L.rdw_base), at<float>(ws, L.rdw_part),
                                 dW_router, stream);
  });
}

mhlmoe_status check_latent(int64_t T, int d_model, int routing_tokens) {
  if (d_model < 1 || d_model > 65536)
    return fail(MHLMOE_EUNSUPPORTED, "d_model must be in [1, 65536] (got %d)", d_model);
  if (routing_tokens != 0 && routing_tokens != 1)
    return fail(MHLMOE_EINVAL, "routing_tokens must be 0 or 1 (got %d)", routing_tokens);
  if (T * (int64_t)d_model >= (int64_t(1) << 40))
    return fail(MHLMOE_EUNSUPPORTED, "T * d_model too large");
  return MHLMOE_OK;
}

// One projection GEMM (see mhl::gemm_rowmajor) with the workspace's
// hipBLASLt region.
mhlmoe_status project(const char* name, int64_t M, int64_t N, int64_t K, const void* A, bool ta,
                      const void* B, bool tb, bool bf16, bool f32_out, bool accumulate, void* C,
                      const Layout& L, void* ws, hipStream_t stream) {
  return run_kernel(name, stream, [&] {
    return mhl::gemm_rowmajor(M, N, K, A, ta, B, tb, bf16, f32_out, accumulate, C,
                              at<void>(ws, L.blas), mhl::kBlasWorkspace, stream);
  });
}

// Argument checks of the routing forward.
mhlmoe_status check_route_args(const Shape& s, const void* X, const float* W_router,
                               const float* bias, const int32_t* idx, const float* gate,
                               const int32_t* counts) {
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need(W_router, "W_router"));
  MHL_TRY(maybe(bias, "bias"));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(need_rows(gate, "gate", s.T));
  MHL_TRY(need(counts, "counts"));
  return MHLMOE_OK;
}

// The routing forward on a checked workspace (ws laid out as L): route_fwd
// writes every per-block histogram row it covers, and count_scan reads only
// those, so nothing in ws needs to start at zero.
mhlmoe_status route_impl(const Shape& s, const void* X, const float* W_router, const float* bias,
                         int32_t* idx, float* gate, int32_t* counts, const Layout& L, void* ws,
                         hipStream_t stream) {
  int32_t* partial = at<int32_t>(ws, L.partial);
  MHL_TRY(run_kernel("route_fwd", stream, [&] {
    return mhl::launch_route_fwd(X, W_router, bias, s.T, s.Nh, s.dh, s.Ne, s.k,
                                 s.dtype == MHLMOE_F32, idx, gate, partial, nullptr, stream);
  }));
  return run_kernel("count_scan", stream, [&] {
    return mhl::launch_count_scan(partial, s.T, s.Nh, s.Ne, 0, counts, nullptr, nullptr, nullptr,
                                  nullptr, stream);
  });
}

}  // namespace

extern "C" {

int mhlmoe_version(void) { return 100; }

const char* mhlmoe_last_error(void) { return g_error.c_str(); }

mhlmoe_status mhlmoe_workspace_size(mhlmoe_op op, int64_t T, int n_heads, int d_head,
                                    int n_experts, int top_k, int d_ff, mhlmoe_dtype dtype,
                                    size_t* bytes) {
  g_error.clear();
  if (bytes == nullptr) return fail(MHLMOE_EINVAL, "bytes is NULL");
  const Shape s{T, n_heads, d_head, n_experts, top_k, d_ff, dtype};
  MHL_TRY(check_route_shape(s));
  switch (op) {
    case MHLMOE_OP_ROUTE:
      MHL_TRY(check_dh(s));
      break;
    case MHLMOE_OP_BUCKET:
      break;
    case MHLMOE_OP_EXPERTS:
    case MHLMOE_OP_LAYER:
      MHL_TRY(check_dh(s));
      MHL_TRY(check_ffn_shape(s));
      break;
    case MHLMOE_OP_LAYER_BACKWARD:
    case MHLMOE_OP_LATENT_BACKWARD:
      MHL_TRY(check_dh(s));
      MHL_TRY(check_ffn_shape(s));
      MHL_TRY(check_backward_dtype(s));
      break;
    case MHLMOE_OP_LATENT_LAYER:
      MHL_TRY(check_dh(s));
      MHL_TRY(check_ffn_shape(s));
      break;
    case MHLMOE_OP_ROUTE_BACKWARD:
      MHL_TRY(check_dh(s));
      break;
    default:
      return fail(MHLMOE_EINVAL, "unknown op %d", (int)op);
  }
  *bytes = make_layout(op, s).total;
  return MHLMOE_OK;
}

mhlmoe_status mhlmoe_route(const void* X, const float* W_router, const float* bias, int64_t T,
                           int n_heads, int d_head, int n_experts, int top_k, mhlmoe_dtype dtype,
                           int32_t* idx, float* gate, int32_t* counts, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, 0, dtype};
  MHL_TRY(check_route_args(s, X, W_router, bias, idx, gate, counts));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_ROUTE, s, workspace, workspace_bytes, L));
  return route_impl(s, X, W_router, bias, idx, gate, counts, L, workspace, stream);
}

mhlmoe_status mhlmoe_route_static(const void* X, const float* W_router, const float* bias,
                                  int64_t T, int n_heads, int d_head, int n_experts, int top_k,
                                  mhlmoe_dtype dtype, int32_t* idx, float* gate, int32_t* counts,
                                  hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, 0, dtype};
  MHL_TRY(check_route_args(s, X, W_router, bias, idx, gate, counts));
  const Layout L = make_layout(MHLMOE_OP_ROUTE, s);
  if (L.total > mhl::kStaticScratchBytes)
    return fail(MHLMOE_EWORKSPACE,
                "mhlmoe_route_static needs %zu bytes of scratch for this shape; its static "
                "scratch holds %zu (use mhlmoe_route with a workspace)",
                L.total, mhl::kStaticScratchBytes);
  void* ws = nullptr;
  const hipError_t e = mhl::static_scratch(&ws);
  if (e != hipSuccess) return fail(MHLMOE_EHIP, "static scratch: %s", hipGetErrorString(e));
  return route_impl(s, X, W_router, bias, idx, gate, counts, L, ws, stream);
}

mhlmoe_status mhlmoe_route_backward(const void* X, const float* W_router, const int32_t* idx,
                                    const float* gate, const float* dgate, int64_t T, int n_heads,
                                    int d_head, int n_experts, int top_k, mhlmoe_dtype dtype,
                                    void* dX, float* dW_router, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, 0, dtype};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need(W_router, "W_router"));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(need_rows(gate, "gate", s.T));
  MHL_TRY(need_rows(dgate, "dgate", s.T));
  MHL_TRY(need_rows(dX, "dX", s.T));
  MHL_TRY(need(dW_router, "dW_router"));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_ROUTE_BACKWARD, s, workspace, workspace_bytes, L));
  void* ws = workspace;
  int32_t* offsets = at<int32_t>(ws, L.offsets);
  int32_t* perm = at<int32_t>(ws, L.perm);
  float* dS = at<float>(ws, L.ds);
  const bool f32 = dtype == MHLMOE_F32;
  // Clustering of idx (with T == 0: all-zero offsets, so dW_router is zeros).
  MHL_TRY(run_kernel("hist", stream, [&] {
    return mhl::launch_hist(idx, s.T, s.Nh, s.Ne, s.k, at<int32_t>(ws, L.partial),
                            at<uint32_t>(ws, L.ticket), stream);
  }));
  MHL_TRY(run_cluster(s, idx, at<int32_t>(ws, L.counts), offsets, perm, 0, L, ws, stream));
  MHL_TRY(run_kernel("route_bwd", stream, [&] {
    return mhl::launch_route_bwd(idx, gate, dgate, W_router, s.T, s.Nh, s.dh, s.Ne, s.k, f32, dX,
                                 dS, stream);
  }));
  return run_kernel("router_dw", stream, [&] {
    return mhl::launch_router_dw(X, f32, dS, perm, offsets, s.T, s.Nh, s.dh, s.Ne, s.k,
                                 at<int32_t>(ws, L.rdw_base), at<float>(ws, L.rdw_part),
                                 dW_router, stream);
  });
}

mhlmoe_status mhlmoe_bucket(const int32_t* idx, int64_t T, int n_heads, int n_experts, int top_k,
                            int32_t* counts, int32_t* offsets, int32_t* perm, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, 64, n_experts, top_k, 0, MHLMOE_BF16};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(maybe(counts, "counts"));
  MHL_TRY(need(offsets, "offsets"));
  MHL_TRY(need_rows(perm, "perm", s.T));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_BUCKET, s, workspace, workspace_bytes, L));
  MHL_TRY(run_kernel("hist", stream, [&] {
    return mhl::launch_hist(idx, s.T, s.Nh, s.Ne, s.k, at<int32_t>(workspace, L.partial),
                            at<uint32_t>(workspace, L.ticket), stream);
  }));
  if (counts == nullptr) counts = at<int32_t>(workspace, L.counts);
  return run_cluster(s, idx, counts, offsets, perm, 0, L, workspace, stream);
}

mhlmoe_status mhlmoe_experts(const void* X, const int32_t* idx, const float* gate, const void* W1,
                             const void* W3, const void* W2, int64_t T, int n_heads, int d_head,
                             int n_experts, int top_k, int d_ff, mhlmoe_dtype dtype, void* Y,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, d_ff, dtype};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(need_rows(gate, "gate", s.T));
  MHL_TRY(need(W1, "W1"));
  MHL_TRY(need(W3, "W3"));
  MHL_TRY(need(W2, "W2"));
  MHL_TRY(need_rows(Y, "Y", s.T));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_EXPERTS, s, workspace, workspace_bytes, L));
  if (s.T == 0) return MHLMOE_OK;
  MHL_TRY(run_kernel("hist", stream, [&] {
    return mhl::launch_hist(idx, s.T, s.Nh, s.Ne, s.k, at<int32_t>(workspace, L.partial),
                            at<uint32_t>(workspace, L.ticket), stream);
  }));
  return run_experts(s, X, idx, gate, nullptr, W1, W3, W2, Y, L, workspace, stream);
}

mhlmoe_status mhlmoe_layer(const void* X, const float* W_router, const float* bias, const void* W1,
                           const void* W3, const void* W2, int64_t T, int n_heads, int d_head,
                           int n_experts, int top_k, int d_ff, mhlmoe_dtype dtype, void* Y,
                           int32_t* idx, float* gate, int32_t* counts, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  MHL_TRY(need(W3, "W3"));
  return layer_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, X, W_router,
                    bias, W1, W3, W2, Y, idx, gate, counts, workspace, workspace_bytes, stream);
}

mhlmoe_status mhlmoe_layer_routed(const void* X, const void* R, const float* W_router,
                                  const float* bias, const void* W1, const void* W3,
                                  const void* W2, int64_t T, int n_heads, int d_head,
                                  int n_experts, int top_k, int d_ff, mhlmoe_dtype dtype, void* Y,
                                  int32_t* idx, float* gate, int32_t* counts, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  return layer_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, R, W_router,
                    bias, W1, W3, W2, Y, idx, gate, counts, workspace, workspace_bytes, stream);
}

mhlmoe_status mhlmoe_experts_gelu(const void* X, const int32_t* idx, const float* gate,
                                  const void* W_in, const void* W_out, int64_t T, int n_heads,
                                  int d_head, int n_experts, int top_k, int d_ff,
                                  mhlmoe_dtype dtype, void* Y, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, d_ff, dtype};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(need_rows(X, "X", s.T));
  MHL_TRY(need_rows(idx, "idx", s.T));
  MHL_TRY(need_rows(gate, "gate", s.T));
  MHL_TRY(need(W_in, "W_in"));
  MHL_TRY(need(W_out, "W_out"));
  MHL_TRY(need_rows(Y, "Y", s.T));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_EXPERTS, s, workspace, workspace_bytes, L));
  if (s.T == 0) return MHLMOE_OK;
  MHL_TRY(run_kernel("hist", stream, [&] {
    return mhl::launch_hist(idx, s.T, s.Nh, s.Ne, s.k, at<int32_t>(workspace, L.partial),
                            at<uint32_t>(workspace, L.ticket), stream);
  }));
  return run_experts(s, X, idx, gate, nullptr, W_in, nullptr, W_out, Y, L, workspace, stream);
}

mhlmoe_status mhlmoe_layer_gelu(const void* X, const float* W_router, const float* bias,
                                const void* W_in, const void* W_out, int64_t T, int n_heads,
                                int d_head, int n_experts, int top_k, int d_ff,
                                mhlmoe_dtype dtype, void* Y, int32_t* idx, float* gate,
                                int32_t* counts, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  g_error.clear();
  return layer_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, X, W_router,
                    bias, W_in, nullptr, W_out, Y, idx, gate, counts, workspace, workspace_bytes,
                    stream);
}

mhlmoe_status mhlmoe_layer_backward(const void* X, const float* W_router, const void* W1,
                                    const void* W3, const void* W2, const int32_t* idx,
                                    const float* gate, const void* dY, int64_t T, int n_heads,
                                    int d_head, int n_experts, int top_k, int d_ff,
                                    mhlmoe_dtype dtype, void* dX, float* dW_router, float* dW1,
                                    float* dW3, float* dW2, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  MHL_TRY(need(W3, "W3"));
  return backward_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, X, W_router,
                       W1, W3, W2, idx, gate, dY, dX, nullptr, dW_router, dW1, dW3, dW2,
                       workspace, workspace_bytes, stream);
}

mhlmoe_status mhlmoe_layer_gelu_backward(const void* X, const float* W_router, const void* W_in,
                                         const void* W_out, const int32_t* idx, const float* gate,
                                         const void* dY, int64_t T, int n_heads, int d_head,
                                         int n_experts, int top_k, int d_ff, mhlmoe_dtype dtype,
                                         void* dX, float* dW_router, float* dW_in, float* dW_out,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream) {
  g_error.clear();
  return backward_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, X, W_router,
                       W_in, nullptr, W_out, idx, gate, dY, dX, nullptr, dW_router, dW_in,
                       nullptr, dW_out, workspace, workspace_bytes, stream);
}

mhlmoe_status mhlmoe_layer_backward_routed(const void* X, const void* R, const float* W_router,
                                           const void* W1, const void* W3, const void* W2,
                                           const int32_t* idx, const float* gate, const void* dY,
                                           int64_t T, int n_heads, int d_head, int n_experts,
                                           int top_k, int d_ff, mhlmoe_dtype dtype, void* dX,
                                           void* dR, float* dW_router, float* dW1, float* dW3,
                                           float* dW2, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
  g_error.clear();
  if (T > 0 && dR == nullptr) return fail(MHLMOE_EINVAL, "dR is NULL");
  MHL_TRY(maybe(dR, "dR"));
  if (T > 0 && dR == dX) return fail(MHLMOE_EINVAL, "dR and dX must be distinct buffers");
  // With T == 0 (dR may then be NULL) either path writes zero weight
  // gradients.
  return backward_impl(Shape{T, n_heads, d_head, n_experts, top_k, d_ff, dtype}, X, R, W_router,
                       W1, W3, W2, idx, gate, dY, dX, dR, dW_router, dW1, dW3, dW2, workspace,
                       workspace_bytes, stream);
}

mhlmoe_status mhlmoe_latent_layer(const void* x, const void* W_in, const float* W_router,
                                  const float* bias, const void* W1, const void* W3,
                                  const void* W2, const void* W_out, int64_t T, int d_model,
                                  int n_heads, int d_head, int n_experts, int top_k, int d_ff,
                                  int routing_tokens, mhlmoe_dtype dtype, void* out, void* X_lat,
                                  void* R_lat, void* Y_lat, int32_t* idx, float* gate,
                                  int32_t* counts, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, d_ff, dtype};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(check_latent(T, d_model, routing_tokens));
  MHL_TRY(need_rows(x, "x", s.T));
  MHL_TRY(need(W_in, "W_in"));
  MHL_TRY(need(W_out, "W_out"));
  MHL_TRY(need_rows(out, "out", s.T));
  MHL_TRY(maybe(X_lat, "X_lat"));
  MHL_TRY(maybe(R_lat, "R_lat"));
  MHL_TRY(maybe(Y_lat, "Y_lat"));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_LATENT_LAYER, s, workspace, workspace_bytes, L));
  const bool bf16 = dtype == MHLMOE_BF16;
  const int64_t N = (int64_t)s.Nh * s.dh;
  if (X_lat == nullptr) X_lat = at<void>(workspace, L.lat_x);
  if (R_lat == nullptr) R_lat = at<void>(workspace, L.lat_r);
  if (Y_lat == nullptr) Y_lat = at<void>(workspace, L.lat_y);
  if (!routing_tokens) R_lat = X_lat;
  // Eq. (5) (Eq. (9) with routing sub-tokens): the latent sub-tokens, whose
  // split into heads is the [T][n_heads][d_head] view of each row.
  MHL_TRY(project("proj_in", s.T, N, d_model, x, false, W_in, true, bf16, false, false, X_lat, L,
                  workspace, stream));
  if (routing_tokens) {
    const void* W_in_r = static_cast<const uint8_t*>(W_in) + s.esize() * (size_t)N * d_model;
    MHL_TRY(project("proj_in", s.T, N, d_model, x, false, W_in_r, true, bf16, false, false, R_lat,
                    L, workspace, stream));
  }
  MHL_TRY(layer_impl(s, X_lat, R_lat, W_router, bias, W1, W3, W2, Y_lat, idx, gate, counts,
                     workspace, workspace_bytes, stream));
  // Eq. (6): the output projection of the concatenated head outputs.
  return project("proj_out", s.T, d_model, N, Y_lat, false, W_out, true, bf16, false, false, out,
                 L, workspace, stream);
}

mhlmoe_status mhlmoe_latent_layer_backward(
    const void* x, const void* W_in, const float* W_router, const void* W1, const void* W3,
    const void* W2, const void* W_out, const void* X_lat, const void* R_lat, const void* Y_lat,
    const int32_t* idx, const float* gate, const void* dout, int64_t T, int d_model, int n_heads,
    int d_head, int n_experts, int top_k, int d_ff, int routing_tokens, mhlmoe_dtype dtype,
    void* dx, float* dW_in, float* dW_router, float* dW1, float* dW3, float* dW2, float* dW_out,
    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_error.clear();
  const Shape s{T, n_heads, d_head, n_experts, top_k, d_ff, dtype};
  MHL_TRY(check_route_shape(s));
  MHL_TRY(check_dh(s));
  MHL_TRY(check_ffn_shape(s));
  MHL_TRY(check_backward_dtype(s));
  MHL_TRY(check_latent(T, d_model, routing_tokens));
  MHL_TRY(need_rows(x, "x", s.T));
  MHL_TRY(need(W_in, "W_in"));
  MHL_TRY(need(W_out, "W_out"));
  MHL_TRY(need_rows(X_lat, "X_lat", s.T));
  if (routing_tokens) MHL_TRY(need_rows(R_lat, "R_lat", s.T));
  MHL_TRY(need_rows(Y_lat, "Y_lat", s.T));
  MHL_TRY(need_rows(dout, "dout", s.T));
  MHL_TRY(need_rows(dx, "dx", s.T));
  MHL_TRY(need(dW_in, "dW_in"));
  MHL_TRY(need(dW_out, "dW_out"));
  Layout L;
  MHL_TRY(check_ws(MHLMOE_OP_LATENT_BACKWARD, s, workspace, workspace_bytes, L));
  const int64_t N = (int64_t)s.Nh * s.dh;
  void* dY = at<void>(workspace, L.lat_dy);
  void* dXl = at<void>(workspace, L.lat_dx);
  void* dRl = routing_tokens ? at<void>(workspace, L.lat_dr) : nullptr;
  // Through the output projection: dY_lat = dout W_out, dW_out = dout^T Y_lat.
  MHL_TRY(project("proj_bwd", s.T, N, d_model, dout, false, W_out, false, true, false, false, dY,
                  L, workspace, stream));
  MHL_TRY(project("proj_bwd", d_model, N, s.T, dout, true, Y_lat, false, true, true, false, dW_out,
                  L, workspace, stream));
  // The heads (Algorithm 2 and the expert backward).
  MHL_TRY(backward_impl(s, X_lat, routing_tokens ? R_lat : X_lat, W_router, W1, W3, W2, idx,
                        gate, dY, dXl, dRl, dW_router, dW1, dW3, dW2, workspace,
                        workspace_bytes, stream));
  // Through the input projection: dW_in = [dX_lat; dR_lat]^T x and
  // dx = dX_lat W_in_x (+ dR_lat W_in_r).
  MHL_TRY(project("proj_bwd", N, d_model, s.T, dXl, true, x, false, true, true, false, dW_in, L,
                  workspace, stream));
  MHL_TRY(project("proj_bwd", s.T, d_model, N, dXl, false, W_in, false, true, false, false, dx, L,
                  workspace, stream));
  if (routing_tokens) {
    const void* W_in_r = static_cast<const uint8_t*>(W_in) + s.esize() * (size_t)N * d_model;
    MHL_TRY(project("proj_bwd", N, d_model, s.T, dRl, true, x, false, true, true, false,
                    dW_in + N * d_model, L, workspace, stream));
    MHL_TRY(project("proj_bwd", s.T, d_model, N, dRl, false, W_in_r, false, true, false, true, dx,
                    L, workspace, stream));
  }
  return MHLMOE_OK;
}

mhlmoe_status mhlmoe_bias_update(const int32_t* counts, float* bias, int n_heads, int n_experts,
                                 float rate, hipStream_t stream) {
  g_error.clear();
  if (n_heads < 1 || n_heads > mhl::kMaxHeadsSupported)
    return fail(MHLMOE_EINVAL, "n_heads must be in [1, %d] (got %d)", mhl::kMaxHeadsSupported,
                n_heads);
  if (n_experts < 1 || n_experts > 1024)
    return fail(MHLMOE_EINVAL, "n_experts must be in [1, 1024] (got %d)", n_experts);
  if (!std::isfinite(rate) || rate < 0.0f)
    return fail(MHLMOE_EINVAL, "rate must be finite and >= 0");
  MHL_TRY(need(counts, "counts"));
  MHL_TRY(need(bias, "bias"));
  return run_kernel("bias_update", stream, [&] {
    return mhl::launch_bias_update(counts, n_heads, n_experts, rate, bias, stream);
  });
}

mhlmoe_status mhlmoe_timing_enable(int on) {
  g_error.clear();
  g_timing.store(on != 0);
  return MHLMOE_OK;
}

mhlmoe_status mhlmoe_timing_query(const char* kernel, double* total_ms, int64_t* launches) {
  g_error.clear();
  if (kernel == nullptr || total_ms == nullptr || launches == nullptr)
    return fail(MHLMOE_EINVAL, "kernel, total_ms and launches must be non-NULL");
  std::lock_guard<std::mutex> lk(g_timing_mu);
  double sum = 0.0;
  int64_t n = 0;
  for (const TimingRecord& r : g_records) {
    if (std::strcmp(r.name, kernel) != 0) continue;
    hipError_t e = hipEventSynchronize(r.stop);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return fail(MHLMOE_EHIP, "timing %s: %s", kernel, hipGetErrorString(e));
    sum += ms;
    ++n;
  }
  *total_ms = sum;
  *launches = n;
  return MHLMOE_OK;
}

mhlmoe_status mhlmoe_timing_reset(void) {
  g_error.clear();
  std::lock_guard<std::mutex> lk(g_timing_mu);
  for (const TimingRecord& r : g_records) {
    hipEventSynchronize(r.stop);
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_records.clear();
  return MHLMOE_OK;
}

}  // extern "C"
