// IO-aware routing forward (Algorithm 1, Sec. 3.3) for gfx950 — kernel
// templates.  Each (d_head, X dtype) pair is instantiated in its own
// translation unit (route_<dh>_<dtype>.hip) so they compile in parallel.
//
// One workgroup = 4 wavefronts = 128 tokens of one head.  The head's router
// weights stream through LDS in blocks of 32 experts (double buffered); each
// wavefront computes the 32-expert x 32-token score tile S^T = W_blk X_blk^T
// with 32x32 MFMAs, so every lane ends up holding 16 scores of ONE token.
// Each lane keeps a sorted top-k list of (score + bias, expert) in registers
// and inserts only candidates that beat its current k-th key; the two lanes
// that share a token merge their lists through a cross-lane shuffle at the
// end.  The bias is then removed (Algorithm 1), the gate softmax over the k
// unbiased scores is taken (Eq. (2)-(3)) and idx / gate are written.  The
// T x N_e score matrix never leaves the chip.  A per-block expert histogram
// is accumulated in LDS and written for the clustering step.
//
// FP32 router (Sec. 2.2): for bf16 X the fp32 router weights are split on the
// fly into hi = bf16(w) and lo = bf16(w - hi); X*hi + X*lo (two bf16 MFMAs,
// exact products, fp32 accumulation) is accurate to ~2^-17 relative, the
// level of an fp32 dot product.  fp32 X uses the fp32 MFMA directly.
//
// The register list holds the best KC >= k candidates (KC a power of two);
// the first k of it are the result.  Ties: each lane visits its experts in
// ascending index order and inserts on strictly greater keys, so an equal
// later key never displaces an earlier one; the final cross-lane merge is a
// bitonic merge under the (key descending, index ascending) total order.

#include <math.h>

#pragma once

#include "device_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace route_detail {

constexpr int kRouteWaves = 4;
constexpr int kRouteThreads = kRouteWaves * kWave;
constexpr int kExpertBlock = 32;
constexpr int kMaxExperts = 1024;
static_assert(kRouteWaves * 32 == kTokensPerBlock, "token block mismatch");

template <int DH, bool XF32>
struct RouteSmem;

template <int DH>
struct RouteSmem<DH, false> {
  static constexpr int kStride = DH + 8;  // bf16 per row: 16-byte pad
  uint16_t w[2][2][kExpertBlock * kStride];  // [buffer][hi, lo]
  float b[2][kExpertBlock];
  int hist[kMaxExperts];
};

template <int DH>
struct RouteSmem<DH, true> {
  static constexpr int kStride = DH + 4;  // floats per row: 16-byte pad
  float w[2][kExpertBlock * kStride];
  float b[2][kExpertBlock];
  int hist[kMaxExperts];
};

// Branch-free sorted (descending) insertion of candidate (c, ci): every slot
// the candidate beats shifts down by one and the candidate lands in the
// first of them; a candidate not above the last key changes nothing.  Only
// strictly greater keys move, so an equal later key stays behind.
template <int KC>
__device__ __forceinline__ void topk_insert(float (&lk)[KC], int (&li)[KC],
                                            float c, int ci) {
  bool here = c > lk[KC - 1];
#pragma unroll
  for (int p = KC - 1; p >= 1; --p) {
    const bool above = c > lk[p - 1];
    const float kk = here ? c : lk[p];
    const int ii = here ? ci : li[p];
    lk[p] = above ? lk[p - 1] : kk;
    li[p] = above ? li[p - 1] : ii;
    here = above;
  }
  lk[0] = here ? c : lk[0];
  li[0] = here ? ci : li[0];
}

// Insert a block of candidates; for long lists the block is skipped when no
// lane of the wavefront has a candidate above its current last key.
template <int KC>
__device__ __forceinline__ void topk_insert_block(float (&lk)[KC], int (&li)[KC],
                                                  const f32x16& acc, int e0, int lane,
                                                  int Ne, bool ragged) {
  float c[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int e = e0 + mfma32_row(v, lane);
    c[v] = (ragged && e >= Ne) ? -INFINITY : acc[v];
  }
  if (KC >= 16) {
    float m = c[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) m = fmaxf(m, c[v]);
    if (!__any(m > lk[KC - 1])) return;
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) topk_insert<KC>(lk, li, c[v], e0 + mfma32_row(v, lane));
}

__device__ __forceinline__ bool key_before(float a, int ai, float b, int bi) {
  return a > b || (a == b && ai < bi);
}

// Merge this lane's sorted list with the partner lane's (lane ^ 32): the
// element-wise best of A[i] and B[KC-1-i] is the top-KC of the union in
// bitonic order, which log2(KC) half-cleaner stages then sort.
template <int KC>
__device__ __forceinline__ void topk_merge_partner(float (&lk)[KC], int (&li)[KC]) {
  float pk[KC];
  int pi[KC];
#pragma unroll
  for (int q = 0; q < KC; ++q) {
    pk[q] = __shfl_xor(lk[q], 32, kWave);
    pi[q] = __shfl_xor(li[q], 32, kWave);
  }
#pragma unroll
  for (int i = 0; i < KC; ++i) {
    const bool mine = key_before(lk[i], li[i], pk[KC - 1 - i], pi[KC - 1 - i]);
    lk[i] = mine ? lk[i] : pk[KC - 1 - i];
    li[i] = mine ? li[i] : pi[KC - 1 - i];
  }
#pragma unroll
  for (int d = KC / 2; d >= 1; d >>= 1) {
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      if ((i & d) == 0) {
        const bool swap = key_before(lk[i + d], li[i + d], lk[i], li[i]);
        const float a = lk[i], b = lk[i + d];
        const int ai = li[i], bi = li[i + d];
        lk[i] = swap ? b : a;
        lk[i + d] = swap ? a : b;
        li[i] = swap ? bi : ai;
        li[i + d] = swap ? ai : bi;
      }
    }
  }
}

template <int DH>
struct WBlockRegs {
  static constexpr int kN = DH / 32;  // float4 per thread per 32 x DH block
  f32x4 v[kN];
  float bias;
};

template <int DH>
__device__ __forceinline__ void load_w_block(const float* __restrict__ Wh,
                                             const float* __restrict__ bh,
                                             int e0, int Ne,
                                             WBlockRegs<DH>& r) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = tid + kRouteThreads * i;
    const int row = (4 * q) / DH;
    const int col = (4 * q) % DH;
    const int e = e0 + row;
    if (e < Ne) {
      r.v[i] = *reinterpret_cast<const f32x4*>(Wh + (int64_t)e * DH + col);
    } else {
      r.v[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  r.bias = 0.f;
  if (bh != nullptr && tid < kExpertBlock && e0 + tid < Ne) r.bias = bh[e0 + tid];
}

template <int DH>
__device__ __forceinline__ void store_w_block(RouteSmem<DH, false>& sm, int buf,
                                              const WBlockRegs<DH>& r) {
  constexpr int S = RouteSmem<DH, false>::kStride;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = tid + kRouteThreads * i;
    const int row = (4 * q) / DH;
    const int col = (4 * q) % DH;
    u32x2 hi, lo;
    hi[0] = pack_bf16x2(r.v[i][0], r.v[i][1]);
    hi[1] = pack_bf16x2(r.v[i][2], r.v[i][3]);
    // w - bf16(w) is exact in fp32
    lo[0] = pack_bf16x2(r.v[i][0] - bf16_bits_to_f32(hi[0] & 0xFFFFu),
                        r.v[i][1] - bf16_bits_to_f32(hi[0] >> 16));
    lo[1] = pack_bf16x2(r.v[i][2] - bf16_bits_to_f32(hi[1] & 0xFFFFu),
                        r.v[i][3] - bf16_bits_to_f32(hi[1] >> 16));
    *reinterpret_cast<u32x2*>(&sm.w[buf][0][row * S + col]) = hi;
    *reinterpret_cast<u32x2*>(&sm.w[buf][1][row * S + col]) = lo;
  }
  if (tid < kExpertBlock) sm.b[buf][tid] = r.bias;
}

template <int DH>
__device__ __forceinline__ void store_w_block(RouteSmem<DH, true>& sm, int buf,
                                              const WBlockRegs<DH>& r) {
  constexpr int S = RouteSmem<DH, true>::kStride;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = tid + kRouteThreads * i;
    const int row = (4 * q) / DH;
    const int col = (4 * q) % DH;
    *reinterpret_cast<f32x4*>(&sm.w[buf][row * S + col]) = r.v[i];
  }
  if (tid < kExpertBlock) sm.b[buf][tid] = r.bias;
}

// X fragments of one lane: token (lane % 32), d_h elements 16 s + 8 g + [0, 8)
// for every 16-wide k-step s, g = lane / 32.
template <int DH, bool XF32>
struct XFrag;

template <int DH>
struct XFrag<DH, false> {
  u32x4 x[DH / 16];
  __device__ __forceinline__ void load(const void* X, int64_t row, bool ok, int g) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(X) + row * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s)
      x[s] = ok ? *reinterpret_cast<const u32x4*>(p + 16 * s) : u32x4{0u, 0u, 0u, 0u};
  }
};

template <int DH>
struct XFrag<DH, true> {
  f32x4 x[DH / 16][2];
  __device__ __forceinline__ void load(const void* X, int64_t row, bool ok, int g) {
    const float* p = reinterpret_cast<const float*>(X) + row * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      x[s][0] = ok ? *reinterpret_cast<const f32x4*>(p + 16 * s) : f32x4{0.f, 0.f, 0.f, 0.f};
      x[s][1] = ok ? *reinterpret_cast<const f32x4*>(p + 16 * s + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

// Score tile for 32 experts x the lane's token, accumulator initialised with
// the bias so the result is the biased key s + b.
template <int DH>
__device__ __forceinline__ f32x16 score_tile(const RouteSmem<DH, false>& sm, int buf,
                                             const XFrag<DH, false>& xf, int lane) {
  constexpr int S = RouteSmem<DH, false>::kStride;
  const int g = lane >> 5, c = lane & 31;
  f32x16 acc;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 b4 = *reinterpret_cast<const f32x4*>(&sm.b[buf][8 * q + 4 * g]);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[4 * q + i] = b4[i];
  }
  const uint16_t* wh = &sm.w[buf][0][c * S + 8 * g];
  const uint16_t* wl = &sm.w[buf][1][c * S + 8 * g];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const bf16x8 xb = as_bf16x8(xf.x[s]);
    acc = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(wh + 16 * s)), xb, acc);
    acc = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(wl + 16 * s)), xb, acc);
  }
  return acc;
}

template <int DH>
__device__ __forceinline__ f32x16 score_tile(const RouteSmem<DH, true>& sm, int buf,
                                             const XFrag<DH, true>& xf, int lane) {
  constexpr int S = RouteSmem<DH, true>::kStride;
  const int g = lane >> 5, c = lane & 31;
  f32x16 acc;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 b4 = *reinterpret_cast<const f32x4*>(&sm.b[buf][8 * q + 4 * g]);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[4 * q + i] = b4[i];
  }
  const float* w = &sm.w[buf][c * S + 8 * g];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const f32x4 w0 = *reinterpret_cast<const f32x4*>(w + 16 * s);
    const f32x4 w1 = *reinterpret_cast<const f32x4*>(w + 16 * s + 4);
#pragma unroll
    for (int p = 0; p < 4; ++p) acc = mfma32_f32(w0[p], xf.x[s][0][p], acc);
#pragma unroll
    for (int p = 0; p < 4; ++p) acc = mfma32_f32(w1[p], xf.x[s][1][p], acc);
  }
  return acc;
}

template <int DH, bool XF32, int KC>
__global__ __launch_bounds__(kRouteThreads) void route_fwd_kernel(
    const void* __restrict__ X, const float* __restrict__ W_router,
    const float* __restrict__ bias, int64_t T, int Nh, int Ne, int k,
    int32_t* __restrict__ idx, float* __restrict__ gate,
    int32_t* __restrict__ partial, uint32_t* __restrict__ ticket) {
  __shared__ RouteSmem<DH, XF32> sm;
  // Reset the clustering step's completion counter for the next kernel.
  if (ticket != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *ticket = 0u;

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int nblk = gridDim.x;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid & (kWave - 1);
  const int g = lane >> 5;
  const int64_t t = (int64_t)blk * kTokensPerBlock + wave * 32 + (lane & 31);
  const bool tok_ok = t < T;

  const float* Wh = W_router + (int64_t)h * Ne * DH;
  const float* bh = bias ? bias + (int64_t)h * Ne : nullptr;

  for (int e = tid; e < Ne; e += kRouteThreads) sm.hist[e] = 0;

  XFrag<DH, XF32> xf;
  xf.load(X, t * Nh + h, tok_ok, g);

  // Sorted list of the best KC candidates seen by this lane (empty slots are
  // (-inf, INT_MAX) and lose to every real candidate).
  float lk[KC];
  int li[KC];
#pragma unroll
  for (int p = 0; p < KC; ++p) {
    lk[p] = -INFINITY;
    li[p] = 0x7fffffff;
  }

  const int nb = (Ne + kExpertBlock - 1) / kExpertBlock;
  WBlockRegs<DH> wr;
  load_w_block<DH>(Wh, bh, 0, Ne, wr);
  store_w_block<DH>(sm, 0, wr);
  __syncthreads();

  for (int b = 0; b < nb; ++b) {
    const int buf = b & 1;
    const int e0 = b * kExpertBlock;
    if (b + 1 < nb) load_w_block<DH>(Wh, bh, e0 + kExpertBlock, Ne, wr);

    const f32x16 acc = score_tile<DH>(sm, buf, xf, lane);
    topk_insert_block<KC>(lk, li, acc, e0, lane, Ne, e0 + kExpertBlock > Ne);

    if (b + 1 < nb) store_w_block<DH>(sm, buf ^ 1, wr);
    __syncthreads();
  }

  // Merge with the partner lane holding the other 16 experts of each tile.
  topk_merge_partner<KC>(lk, li);

  if (g == 0 && tok_ok) {
    // Slots left empty by non-finite scores get expert 0 so that nothing below
    // indexes out of range (the result is unspecified for such inputs).
#pragma unroll
    for (int p = 0; p < KC; ++p) li[p] = (unsigned)li[p] < (unsigned)Ne ? li[p] : 0;
    // Remove the bias (Algorithm 1) and take the softmax over the k scores.
    float s[KC];
    float m = -INFINITY;
#pragma unroll
    for (int p = 0; p < KC; ++p) {
      if (p < k) {
        s[p] = bh ? lk[p] - bh[li[p]] : lk[p];
        m = fmaxf(m, s[p]);
      }
    }
    float z = 0.f;
#pragma unroll
    for (int p = 0; p < KC; ++p) {
      if (p < k) {
        s[p] = expf(s[p] - m);
        z += s[p];
      }
    }
    const float inv = 1.0f / z;
    const int64_t o = (t * Nh + h) * k;
#pragma unroll
    for (int p = 0; p < KC; ++p) {
      if (p < k) {
        idx[o + p] = li[p];
        gate[o + p] = s[p] * inv;
        atomicAdd(&sm.hist[li[p]], 1);
      }
    }
  }
  __syncthreads();
  int32_t* out = partial + ((int64_t)h * nblk + blk) * Ne;
  for (int e = tid; e < Ne; e += kRouteThreads) out[e] = sm.hist[e];
}

template <int DH, bool XF32>
hipError_t launch_dh_dtype(const void* X, const float* W, const float* bias,
                           int64_t T, int Nh, int Ne, int k, int32_t* idx,
                           float* gate, int32_t* partial, uint32_t* ticket,
                           hipStream_t s) {
  const dim3 grid((unsigned)num_token_blocks(T), (unsigned)Nh);
  const dim3 block(kRouteThreads);
#define MHL_ROUTE_CASE(KC)                                                        \
  if (k <= KC) {                                                                  \
    hipLaunchKernelGGL((route_fwd_kernel<DH, XF32, KC>), grid, block, 0, s, X, W, \
                       bias, T, Nh, Ne, k, idx, gate, partial, ticket);           \
    return hipGetLastError();                                                     \
  }
  MHL_ROUTE_CASE(2)
  MHL_ROUTE_CASE(4)
  MHL_ROUTE_CASE(8)
  MHL_ROUTE_CASE(16)
  MHL_ROUTE_CASE(32)
#undef MHL_ROUTE_CASE
  return hipErrorInvalidValue;
}

}  // namespace route_detail
}  // namespace mhl
