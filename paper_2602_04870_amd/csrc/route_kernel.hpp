// IO-aware routing forward (Algorithm 1, Sec. 3.3) for gfx950 — kernel
// templates.  Each (d_head, X dtype) pair is instantiated in its own
// translation unit (route_<dh>_<dtype>.hip) so they compile in parallel.
//
// One workgroup = 8 wavefronts = 128 tokens of one head: 4 token groups of
// 32 tokens times 2 expert halves (the even and the odd 32-expert blocks).
// The head's router weights stream through LDS in blocks of 32 experts
// (double buffered per half); each wavefront computes 32-expert x 32-token
// score tiles S^T = W_blk X_blk^T with 32x32 MFMAs, so every lane holds 16
// scores of ONE token per tile.  Splitting the experts over two wavefronts
// gives two wavefronts per token group, which hides the latency of the
// selection network when there are few tokens.
//
// Selection keys pack the order-preserving image of the fp32 biased score
// s + b with the complement of the expert index, so one unsigned compare
// orders by score descending and, among equal scores, by index ascending
// (the tie-break).  With N_e > 128 (> 256 at d_h = 128) the key is wide:
// the whole image and the index side by side (the packing of Algorithm 1)
// in the mantissa of a double in [1, 2), compared by v_max_f64 / v_min_f64.
// With fewer experts it is 32 bits: the image with its low
// b = ceil(log2 N_e) bits replaced by the index, so a compare-exchange is
// one v_max_u32 and one v_min_u32.  Scores whose images agree above those b bits
// (a relative difference below 2^(b-23), at the level of the router score's
// own rounding) are then ordered by index; every other comparison is exact.
// The b dropped bits of each candidate stay in registers (one byte each) and
// are written to LDS after the score loop, so the selected scores, and from
// them the gates, are the exact fp32 values.
// Each lane keeps the best KC >= k keys of its candidates sorted in
// registers.  A tile's 16 new candidates are merged in with compare-exchange
// networks (the block sorted by Batcher's odd-even merge sort, an
// elementwise maximum against the reversed list tail, a bitonic merge, and
// at KC = 32 an odd-even merge of the list's two sorted halves), which costs
// fewer operations per candidate than inserting them one by one once
// KC >= 8; for KC <= 4 candidates are inserted.  The two lanes holding a token's two 16-expert halves, then the
// two expert halves, merge their lists the same way.  The bias is then
// removed (Algorithm 1), the gate softmax over the k unbiased scores is
// taken (Eq. (2)-(3)) and idx / gate are written.  The T x N_e score matrix
// never leaves the chip.  A per-block expert histogram is accumulated in
// LDS and written for the clustering step.
//
// FP32 router (Sec. 2.2): for bf16 X the fp32 router weights are split on the
// fly into hi = bf16(w) and lo = bf16(w - hi); X*hi + X*lo (two bf16 MFMAs,
// exact products, fp32 accumulation) is accurate to ~2^-17 relative, the
// level of an fp32 dot product.  fp32 X uses the fp32 MFMA directly.

#include <math.h>

#include <type_traits>

#pragma once

#include "device_common.hpp"
#include "launch.hpp"
#include "sort_networks.hpp"

namespace mhl {
namespace route_detail {

constexpr int kRouteGroups = 4;   // 32-token groups per workgroup
constexpr int kRouteHalves = 2;   // expert halves (even / odd blocks)
constexpr int kRouteWaves = kRouteGroups * kRouteHalves;
constexpr int kRouteThreads = kRouteWaves * kWave;
constexpr int kHalfThreads = kRouteGroups * kWave;  // threads staging one half's block
constexpr int kExpertBlock = 32;
constexpr int kMaxExperts = 1024;
static_assert(kRouteGroups * 32 == kTokensPerBlock, "token block mismatch");

template <int DH, bool XF32>
struct RouteSmem;

template <int DH>
struct RouteSmem<DH, false> {
  static constexpr int kStride = DH + 8;  // bf16 per row: 16-byte pad
  uint16_t w[kRouteHalves][2][2][kExpertBlock * kStride];  // [half][buffer][hi, lo]
  float b[kRouteHalves][2][kExpertBlock];
  int hist[kMaxExperts];
};

template <int DH>
struct RouteSmem<DH, true> {
  static constexpr int kStride = DH + 4;  // floats per row: 16-byte pad
  float w[kRouteHalves][2][kExpertBlock * kStride];
  float b[kRouteHalves][2][kExpertBlock];
  int hist[kMaxExperts];
};

// ---------------------------------------------------------------------------
// Packed selection keys and compare-exchange networks (descending order).
// ---------------------------------------------------------------------------
// Order-preserving image of an fp32 value (-0 taken as +0): unsigned order
// of the images is the numeric order of the values.
__device__ __forceinline__ uint32_t orderable(float v) {
  const uint32_t b = __float_as_uint(v + 0.0f);
  return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}
__device__ __forceinline__ float from_orderable(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o ^ 0x80000000u) : ~o);
}

// Key of expert e with image o.  Wide keys (exact): the 52-bit integer
// image * 2^20 + (2^20 - 1 - e) placed in the mantissa of a double of
// exponent 0 (a value in [1, 2)), so that the order of the doubles is the
// order of the integers and a compare-exchange is one v_max_f64 and one
// v_min_f64 (a 64-bit integer one takes a 64-bit compare and four selects);
// the empty key is +0, below every real key.  32 bits (e <= mask = 2^b - 1):
// the image with its low b bits replaced by mask - e.
constexpr int kWideIndexBits = 20;  // experts per head < 2^20
template <typename K>
__device__ __forceinline__ K make_key(uint32_t o, int e, uint32_t mask) {
  if constexpr (sizeof(K) == 8)
    return __builtin_bit_cast(double, (0x3FFull << 52) | ((uint64_t)o << kWideIndexBits) |
                                          (uint64_t)(((1u << kWideIndexBits) - 1) & ~(uint32_t)e));
  else return (o & ~mask) | (mask & ~(uint32_t)e);
}
__device__ __forceinline__ int key_expert(double p, uint32_t) {
  return (int)(((1u << kWideIndexBits) - 1) & ~(uint32_t)__builtin_bit_cast(uint64_t, p));
}
__device__ __forceinline__ uint32_t key_image(double p, uint32_t) {
  return (uint32_t)(__builtin_bit_cast(uint64_t, p) >> kWideIndexBits);
}
__device__ __forceinline__ int key_expert(uint32_t p, uint32_t mask) { return (int)(~p & mask); }
// The image with its dropped low bits still to be restored.
__device__ __forceinline__ uint32_t key_image(uint32_t p, uint32_t mask) { return p & ~mask; }

// a <- max(a, b), b <- min(a, b)
// The wide keys are finite doubles in [1, 2) or +0, never NaN; through
// fmax / fmin the compiler would still quiet every operand it cannot prove
// quiet (one more v_max_f64 per operand coming through a loop phi), so the
// two instructions are written out (6% of the route at 1024 experts).
__device__ __forceinline__ double dmax(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ double dmin(double a, double b) {
  double r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ void cex(double& a, double& b) {
  const double hi = dmax(a, b), lo = dmin(a, b);
  a = hi;
  b = lo;
}
__device__ __forceinline__ void cex(uint32_t& a, uint32_t& b) {
  const uint32_t hi = a > b ? a : b, lo = a > b ? b : a;
  a = hi;
  b = lo;
}
__device__ __forceinline__ double kmax(double a, double b) { return dmax(a, b); }
__device__ __forceinline__ uint32_t kmax(uint32_t a, uint32_t b) { return b > a ? b : a; }
// cex as the compare-exchange of the odd-even networks
struct Cex {
  template <typename K>
  __device__ __forceinline__ void operator()(K& a, K& b) const { cex(a, b); }
};

// The value of lane l ^ 32, valid in lanes 0-31 (v_permlane32_swap).
__device__ __forceinline__ uint32_t upper_half(uint32_t v) { return permlane32_swap(v, v)[1]; }
__device__ __forceinline__ double upper_half(double d) {
  const uint64_t v = __builtin_bit_cast(uint64_t, d);
  return __builtin_bit_cast(double,
                            ((uint64_t)upper_half((uint32_t)(v >> 32)) << 32) | upper_half((uint32_t)v));
}

// Sort a bitonic sequence of N keys descending (half-cleaner stages).
template <int N, typename K>
__device__ __forceinline__ void bitonic_merge(K* v) {
#pragma unroll
  for (int j = N >> 1; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int l = i ^ j;
      if (l > i) cex(v[i], v[l]);
    }
}

// L (KC sorted) <- the best KC of L and the 16 candidates c (unsorted; c is
// clobbered).
template <int KC, typename K>
__device__ __forceinline__ void merge_block(K (&L)[KC], K (&c)[16]) {
  if constexpr (KC <= 4) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      K x = c[v];
#pragma unroll
      for (int p = 0; p < KC; ++p) cex(L[p], x);
    }
  } else if constexpr (KC == 8) {
    // top 8 of the block: sort both halves, keep the larger of each
    // mirrored pair (a bitonic sequence), sort it
    oe_sort<0, 7>(c, Cex{});
    oe_sort<8, 15>(c, Cex{});
    K t[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = kmax(c[i], c[15 - i]);
    bitonic_merge<8>(t);
#pragma unroll
    for (int i = 0; i < 8; ++i) L[i] = kmax(L[i], t[7 - i]);
    bitonic_merge<8>(L);
  } else {
    static_assert(KC == 16 || KC == 32, "list length");
    oe_sort<0, 15>(c, Cex{});
    // the best 16 of the list tail and the block
    K* tail = L + (KC - 16);
#pragma unroll
    for (int i = 0; i < 16; ++i) tail[i] = kmax(tail[i], c[15 - i]);
    bitonic_merge<16>(tail);
    // the head and the new tail are sorted runs: merge them
    if constexpr (KC == 32) oe_merge<0, 31, 1>(L, Cex{});
  }
}

// L (32 sorted) <- the best 32 of L and two tiles' candidates a, b
// (unsorted, clobbered): the 32 candidates sorted (Batcher, 191
// compare-exchanges), an elementwise maximum against L reversed (a bitonic
// sequence holding the best 32), a bitonic merge (80): 271 per two tiles
// against 320 for two merge_block calls.
template <typename K>
__device__ __forceinline__ void merge_pair32(K (&L)[32], K (&a)[16], K (&b)[16]) {
  K c[32];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    c[i] = a[i];
    c[16 + i] = b[i];
  }
  oe_sort<0, 31>(c, Cex{});
#pragma unroll
  for (int i = 0; i < 32; ++i) L[i] = kmax(L[i], c[31 - i]);
  bitonic_merge<32>(L);
}

// L <- the best KC of L and another sorted list P.
template <int KC, typename K>
__device__ __forceinline__ void merge_lists(K (&L)[KC], const K (&P)[KC]) {
#pragma unroll
  for (int i = 0; i < KC; ++i) L[i] = kmax(L[i], P[KC - 1 - i]);
  bitonic_merge<KC>(L);
}

// ---------------------------------------------------------------------------
// Router weight blocks: fp32 from global memory, split into bf16 hi/lo (bf16
// X) or kept fp32, staged in LDS.
// ---------------------------------------------------------------------------
template <int DH>
struct WBlockRegs {
  static constexpr int kN = DH * kExpertBlock / 4 / kHalfThreads;  // float4 per thread
  f32x4 v[kN];
  float bias;
};

// Thread ht (0 .. kHalfThreads-1) of a half loads its share of the block of
// experts e0 .. e0+31 (rows past Ne read as zero).
template <int DH>
__device__ __forceinline__ void load_w_block(const float* __restrict__ Wh,
                                             const float* __restrict__ bh, int e0, int Ne,
                                             int ht, WBlockRegs<DH>& r) {
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = ht + kHalfThreads * i;
    const int row = (4 * q) / DH;
    const int col = (4 * q) % DH;
    const int e = e0 + row;
    r.v[i] = e < Ne ? *reinterpret_cast<const f32x4*>(Wh + (int64_t)e * DH + col)
                    : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  r.bias = 0.f;
  if (bh != nullptr && ht < kExpertBlock && e0 + ht < Ne) r.bias = bh[e0 + ht];
}

template <int DH>
__device__ __forceinline__ void store_w_block(RouteSmem<DH, false>& sm, int half, int buf,
                                              int ht, const WBlockRegs<DH>& r) {
  constexpr int S = RouteSmem<DH, false>::kStride;
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = ht + kHalfThreads * i;
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
    *reinterpret_cast<u32x2*>(&sm.w[half][buf][0][row * S + col]) = hi;
    *reinterpret_cast<u32x2*>(&sm.w[half][buf][1][row * S + col]) = lo;
  }
  if (ht < kExpertBlock) sm.b[half][buf][ht] = r.bias;
}

template <int DH>
__device__ __forceinline__ void store_w_block(RouteSmem<DH, true>& sm, int half, int buf,
                                              int ht, const WBlockRegs<DH>& r) {
  constexpr int S = RouteSmem<DH, true>::kStride;
#pragma unroll
  for (int i = 0; i < WBlockRegs<DH>::kN; ++i) {
    const int q = ht + kHalfThreads * i;
    const int row = (4 * q) / DH;
    const int col = (4 * q) % DH;
    *reinterpret_cast<f32x4*>(&sm.w[half][buf][row * S + col]) = r.v[i];
  }
  if (ht < kExpertBlock) sm.b[half][buf][ht] = r.bias;
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
// the bias so the result is the biased key s + b.  CH accumulation chains
// (1 or 2) are summed at the end: two halve the dependent MFMA sequence but
// take 16 more registers.
template <int DH, int CH>
__device__ __forceinline__ f32x16 score_tile(const RouteSmem<DH, false>& sm, int half, int buf,
                                             const XFrag<DH, false>& xf, int lane) {
  constexpr int S = RouteSmem<DH, false>::kStride;
  const int g = lane >> 5, c = lane & 31;
  f32x16 acc;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 b4 = *reinterpret_cast<const f32x4*>(&sm.b[half][buf][8 * q + 4 * g]);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[4 * q + i] = b4[i];
  }
  const uint16_t* wh = &sm.w[half][buf][0][c * S + 8 * g];
  const uint16_t* wl = &sm.w[half][buf][1][c * S + 8 * g];
  // two chains: hi products in one, lo products in the other
  f32x16 acc2 = zero16();
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const bf16x8 xb = as_bf16x8(xf.x[s]);
    acc = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(wh + 16 * s)), xb, acc);
    if constexpr (CH == 2)
      acc2 = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(wl + 16 * s)), xb, acc2);
    else
      acc = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(wl + 16 * s)), xb, acc);
  }
  if constexpr (CH == 2) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] += acc2[v];
  }
  return acc;
}

template <int DH, int CH>
__device__ __forceinline__ f32x16 score_tile(const RouteSmem<DH, true>& sm, int half, int buf,
                                             const XFrag<DH, true>& xf, int lane) {
  constexpr int S = RouteSmem<DH, true>::kStride;
  const int g = lane >> 5, c = lane & 31;
  f32x16 acc;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 b4 = *reinterpret_cast<const f32x4*>(&sm.b[half][buf][8 * q + 4 * g]);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[4 * q + i] = b4[i];
  }
  const float* w = &sm.w[half][buf][c * S + 8 * g];
  // two chains: even k in one, odd k in the other
  f32x16 acc2 = zero16();
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const f32x4 w0 = *reinterpret_cast<const f32x4*>(w + 16 * s);
    const f32x4 w1 = *reinterpret_cast<const f32x4*>(w + 16 * s + 4);
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const float a = p < 4 ? w0[p] : w1[p - 4];
      const float b = xf.x[s][p >> 2][p & 3];
      if (CH == 2 && (p & 1)) acc2 = mfma32_f32(a, b, acc2);
      else acc = mfma32_f32(a, b, acc);
    }
  }
  if constexpr (CH == 2) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] += acc2[v];
  }
  return acc;
}

// 32-bit keys serve N_e up to 256 (one byte of dropped bits per candidate):
// a lane's candidates of at most MI iterations (2 for N_e <= 128, 4 for
// N_e <= 256) keep their dropped bits in registers (MI = 0: 64-bit keys).
// N_e <= 256 needs the byte table of d_h = 128's larger weight buffers.
constexpr int kK32Experts = 128;
constexpr int kK32WideExperts = 256;
template <int DH>
constexpr int k32_max_iters(int Ne) {
  return Ne <= kK32Experts ? 2 : (DH == 128 && Ne <= kK32WideExperts) ? 4 : 0;
}

// Four wavefronts per SIMD, i.e. two workgroups per CU (at most 128
// registers per lane), where the kernel fits: 32-bit keys (with at most 16
// keys per list for N_e > 128), or 64-bit keys with lists of up to 8; the
// rest, and fp32 X at d_h = 128 (64 registers of X fragments), get two
// wavefronts per SIMD.
template <int DH, bool XF32, int KC, int MI>
constexpr int route_waves_per_simd() {
  if (XF32 && DH == 128) return 2;
  return (MI == 2 || (MI == 4 && KC <= 16) || (MI == 0 && KC <= 8)) ? 4 : 2;
}

// MI > 0: 32-bit keys; MI = 0: 64-bit keys.
template <int DH, bool XF32, int KC, int MI>
__global__ __launch_bounds__(kRouteThreads, (route_waves_per_simd<DH, XF32, KC, MI>())) void route_fwd_kernel(
    const void* __restrict__ X, const float* __restrict__ W_router,
    const float* __restrict__ bias, int64_t T, int Nh, int Ne, int k,
    int32_t* __restrict__ idx, float* __restrict__ gate,
    int32_t* __restrict__ partial, uint32_t* __restrict__ ticket) {
  constexpr bool K32 = MI > 0;
  using K = std::conditional_t<K32, uint32_t, double>;
  __shared__ RouteSmem<DH, XF32> sm;
  // Reset the clustering step's completion counter for the next kernel.
  if (ticket != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *ticket = 0u;

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int nblk = gridDim.x;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int tg = wave % kRouteGroups;    // token group
  const int half = wave / kRouteGroups;  // expert half: blocks half, half + 2, ...
  const int ht = tid % kHalfThreads;     // thread index within the half
  const int lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int64_t t = (int64_t)blk * kTokensPerBlock + tg * 32 + c;
  const bool tok_ok = t < T;
  // 32-bit keys: index bits b with 2^b >= N_e
  uint32_t mask = 0;
  if constexpr (K32) {
    while (mask + 1 < (uint32_t)Ne) mask = 2 * mask + 1;
  }

  const float* Wh = W_router + (int64_t)h * Ne * DH;
  const float* bh = bias ? bias + (int64_t)h * Ne : nullptr;

  for (int e = tid; e < Ne; e += kRouteThreads) sm.hist[e] = 0;

  XFrag<DH, XF32> xf;
  xf.load(X, t * Nh + h, tok_ok, g);

  // Best KC keys of this lane's candidates, sorted descending (0 = empty:
  // below every real key).
  K L[KC];
#pragma unroll
  for (int p = 0; p < KC; ++p) L[p] = 0;
  // 32-bit keys: the dropped image bits of the lane's 16 candidates of
  // iteration i, one byte each (candidate v in byte v % 4 of word v / 4).
  uint32_t low[K32 ? MI : 1][4];

  const int nb = (Ne + kExpertBlock - 1) / kExpertBlock;
  const int niter = (nb + kRouteHalves - 1) / kRouteHalves;
  WBlockRegs<DH> wr;
  load_w_block<DH>(Wh, bh, half * kExpertBlock, Ne, ht, wr);
  store_w_block<DH>(sm, half, 0, ht, wr);
  __syncthreads();

  // 32-key lists with wide keys: the candidates of every other tile wait in
  // pend and two tiles are merged at once (merge_pair32).
  constexpr bool PAIR = !K32 && KC == 32;
  K pend[PAIR ? 16 : 1];
  bool have_pend = false;
  auto iteration = [&](int it, uint32_t (&lw)[4]) {
    const int buf = it & 1;
    const int b = kRouteHalves * it + half;  // this half's block
    if (it + 1 < niter) load_w_block<DH>(Wh, bh, (b + kRouteHalves) * kExpertBlock, Ne, ht, wr);
    if (b < nb) {
      const int e0 = b * kExpertBlock;
      const f32x16 acc = score_tile<DH, (MI == 2 || (MI == 0 && KC <= 8)) ? 2 : 1>(sm, half, buf, xf, lane);
      K cand[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int e = e0 + mfma32_row(v, lane);
        const uint32_t o = orderable(acc[v]);
        cand[v] = e < Ne ? make_key<K>(o, e, mask) : K(0);
        if constexpr (K32) {
          if ((v & 3) == 0) lw[v >> 2] = 0;
          lw[v >> 2] |= (o & mask) << (8 * (v & 3));
        }
      }
      if constexpr (PAIR) {
        if (have_pend) {
          merge_pair32(L, pend, cand);
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) pend[v] = cand[v];
        }
        have_pend = !have_pend;
      } else {
        merge_block<KC>(L, cand);
      }
    }
    if (it + 1 < niter) store_w_block<DH>(sm, half, buf ^ 1, ht, wr);
    __syncthreads();
  };
  if constexpr (K32) {
    // (the host picks MI with niter <= MI)
#pragma unroll
    for (int it = 0; it < MI; ++it)
      if (it < niter) iteration(it, low[it]);
  } else {
    for (int it = 0; it < niter; ++it) iteration(it, low[0]);
    if constexpr (PAIR) {
      if (have_pend) merge_block<KC>(L, pend);
    }
  }

  // After the score loop the weight buffers hold, in order: (32-bit keys)
  // the dropped image bits as bytes [token][expert], then the lists that
  // the second expert half hands to the first.
  const int tstride = nb * kExpertBlock + 4;  // bytes per token row (skewed)
  uint8_t* tab = reinterpret_cast<uint8_t*>(&sm.w);
  const int tab_bytes = K32 ? (kTokensPerBlock * tstride + 15) & ~15 : 0;
  K* xch = reinterpret_cast<K*>(tab + tab_bytes);
  static_assert(kTokensPerBlock * (MI * kRouteHalves * kExpertBlock + 4) +
                        sizeof(uint32_t) * kTokensPerBlock * 32 <= sizeof(sm.w),
                "byte table and exchange lists fit");
  static_assert(sizeof(K) * kTokensPerBlock * KC <= sizeof(sm.w), "exchange lists fit");
  if constexpr (K32) {
#pragma unroll
    for (int it = 0; it < MI; ++it) {
      const int b = kRouteHalves * it + half;
      if (it < niter && b < nb) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<uint32_t*>(tab + (tg * 32 + c) * tstride + b * kExpertBlock + 8 * q +
                                       4 * g) = low[it][q];
      }
    }
  }

  // Merge with the partner lane holding the other 16 experts of each tile;
  // from here on only lanes 0-31 carry the token's list.
  {
    K P[KC];
#pragma unroll
    for (int p = 0; p < KC; ++p) P[p] = upper_half(L[p]);
    merge_lists<KC>(L, P);
  }
  // Merge the two expert halves through LDS.
  if (half == 1 && g == 0) {
#pragma unroll
    for (int p = 0; p < KC; ++p) xch[(tg * 32 + c) * KC + p] = L[p];
  }
  __syncthreads();
  if (half == 0 && g == 0) {
    K P[KC];
#pragma unroll
    for (int p = 0; p < KC; ++p) P[p] = xch[(tg * 32 + c) * KC + p];
    merge_lists<KC>(L, P);
  }

  if (half == 0 && g == 0 && tok_ok) {
    int li[KC];
    float s[KC];
    // Slots left empty by non-finite scores get expert 0 so that nothing
    // below indexes out of range (the result is unspecified for such inputs).
#pragma unroll
    for (int p = 0; p < KC; ++p) {
      const int e = key_expert(L[p], mask);
      li[p] = (unsigned)e < (unsigned)Ne ? e : 0;
    }
    // Remove the bias (Algorithm 1) and take the softmax over the k scores.
    float m = -INFINITY;
#pragma unroll
    for (int p = 0; p < KC; ++p) {
      if (p < k) {
        uint32_t o = key_image(L[p], mask);
        if constexpr (K32) o |= tab[(tg * 32 + c) * tstride + li[p]];
        const float kv = from_orderable(o);
        s[p] = bh ? kv - bh[li[p]] : kv;
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
#pragma unroll
    for (int p = 0; p < KC; ++p)
      if (p < k) s[p] *= inv;
    const int64_t o = (t * Nh + h) * k;
    if ((k & 3) == 0) {
      // rows start 16-byte aligned (16-byte aligned tensors, k % 4 == 0)
#pragma unroll
      for (int p = 0; p < KC; p += 4) {
        if (p < k) {
          *reinterpret_cast<u32x4*>(idx + o + p) =
              u32x4{(uint32_t)li[p], (uint32_t)li[p + 1], (uint32_t)li[p + 2], (uint32_t)li[p + 3]};
          *reinterpret_cast<f32x4*>(gate + o + p) = f32x4{s[p], s[p + 1], s[p + 2], s[p + 3]};
        }
      }
    } else {
#pragma unroll
      for (int p = 0; p < KC; ++p) {
        if (p < k) {
          idx[o + p] = li[p];
          gate[o + p] = s[p];
        }
      }
    }
#pragma unroll
    for (int p = 0; p < KC; ++p)
      if (p < k) atomicAdd(&sm.hist[li[p]], 1);
  }
  // The histogram is complete once every LDS operation is; the idx / gate
  // stores may still be in flight.
  barrier_vm<63>();
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
  const int mi = k32_max_iters<DH>(Ne);
#define MHL_ROUTE_LAUNCH(KC, MI)                                                            \
  hipLaunchKernelGGL((route_fwd_kernel<DH, XF32, KC, MI>), grid, block, 0, s, X, W, bias, T, \
                     Nh, Ne, k, idx, gate, partial, ticket)
#define MHL_ROUTE_CASE(KC)                                 \
  if (k <= KC) {                                           \
    if (mi == 2) MHL_ROUTE_LAUNCH(KC, 2);                  \
    else if constexpr (DH == 128) {                        \
      if (mi == 4) MHL_ROUTE_LAUNCH(KC, 4);                \
      else MHL_ROUTE_LAUNCH(KC, 0);                        \
    } else MHL_ROUTE_LAUNCH(KC, 0);                        \
    return hipGetLastError();                              \
  }
  MHL_ROUTE_CASE(2)
  MHL_ROUTE_CASE(4)
  MHL_ROUTE_CASE(8)
  MHL_ROUTE_CASE(16)
  MHL_ROUTE_CASE(32)
#undef MHL_ROUTE_CASE
#undef MHL_ROUTE_LAUNCH
  return hipErrorInvalidValue;
}

}  // namespace route_detail
}  // namespace mhl
