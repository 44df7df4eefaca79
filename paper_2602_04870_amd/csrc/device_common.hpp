// Device helpers shared by the libmhlmoe kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace mhl {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kWave = 64;


typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// Two fp32 -> packed bf16 (element 0 in the low half), round to nearest even
// (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// silu(z) = z / (1 + e^-z) with the hardware exp2 and reciprocal.
__device__ __forceinline__ float silu_fast(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

// 32x32 output tile of a 32x32xK MFMA: lane l holds column (l % 32) and, for
// accumulator element v, row 8*(v/4) + 4*(l/32) + (v%4).
__device__ __forceinline__ int mfma32_row(int v, int lane) {
  return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

// floor(n / k) for 0 <= n < 2^31 and 1 <= k <= 32 as one multiply and a
// shift: with S = 31 + ceil(log2 k) and m = ceil(2^S / k) = 2^S / k + d
// (0 <= d < 1; m <= 2^32, so n m < 2^63), n m / 2^S = n / k + n d / 2^S,
// and n d / 2^S < 2^31 / 2^S = 2^-ceil(log2 k) <= 1/k, less than the gap
// from n / k up to the next integer whenever the floor could change.
struct DivMagic {
  uint64_t m;
  int shift;
};
__host__ __device__ __forceinline__ DivMagic div_magic(int k) {
  int c = 0;
  while ((1 << c) < k) ++c;
  const int S = 31 + c;
  return DivMagic{((uint64_t(1) << S) + (uint64_t)k - 1) / (uint64_t)k, S};
}
__device__ __forceinline__ int div_by_magic(int n, DivMagic d) {
  return (int)(((uint64_t)(uint32_t)n * d.m) >> d.shift);
}

__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Inclusive prefix sum over one wavefront.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    int o = __shfl_up(v, d, kWave);
    if (lane >= d) v += o;
  }
  return v;
}

// v_permlane32_swap: lanes 32-63 of a trade values with lanes 0-31 of b.
__device__ __forceinline__ u32x2 permlane32_swap(uint32_t a, uint32_t b) {
  const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
  return u32x2{r[0], r[1]};
}

// Wait until at most N vector-memory operations of this wavefront are
// outstanding and all its LDS operations are done, then barrier the
// workgroup.  Unlike __syncthreads() (which waits for every load), this
// keeps the N most recent loads, the prefetches, in flight.  The empty asm
// statements keep the compiler from moving memory operations across it.
template <int N>
__device__ __forceinline__ void barrier_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait until this wavefront's LDS operations are done (vector-memory
// operations, e.g. LDS DMA, may stay in flight), then barrier the workgroup.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt 63, expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// f(std::integral_constant<int, i>{}) for i = I, ..., N - 1, unrolled at
// compile time (so f can use i in constant expressions).
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// gelu(z) = z Phi(z) for the forward FFN, with the normal CDF written as a
// logistic function of an odd polynomial: Phi(z) ~ 1 / (1 + e^{-z P(z^2)}),
// P of degree 4 fitted by weighted minimax of logit Phi on [0, 6] (gelu_fit.py
// beside this file prints the constants; |Phi error| <= 1.6e-6 in fp32, far
// below the bf16 rounding of the intermediate).  The constants are P's
// coefficients times -log2(e), so the exponential is one exp2.  Large |z|:
// exp2 goes to 0 or +inf and the result to z or -0, as gelu does.
__device__ __forceinline__ float gelu_logistic(float z) {
  const float z2 = z * z;
  float p = fmaf(-4.087395155e-06f, z2, 1.055776665e-04f);
  p = fmaf(p, z2, 2.545143943e-04f);
  p = fmaf(p, z2, -1.050070599e-01f);
  p = fmaf(p, z2, -2.302165031e+00f);
  const float e = __builtin_amdgcn_exp2f(z * p);
  return z * __builtin_amdgcn_rcpf(1.0f + e);
}

// gelu(z) = z/2 (1 + erf(z / sqrt 2)) and gelu'(z) = Phi(z) + z phi(z)
// together, for the backward, with erf from Abramowitz & Stegun 7.1.26:
// erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) e^{-x^2},
// t = 1 / (1 + p x) for x >= 0 (|error| <= 1.5e-7), extended as an odd
// function.  With x = |z| / sqrt 2, e^{-x^2} = e^{-z^2/2} is both the factor
// of the erf formula and, divided by sqrt(2 pi), the normal density phi(z), so
// one exponential serves both.
__device__ __forceinline__ void gelu_and_grad(float z, float& g, float& dg) {
  const float x = fabsf(z) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  float p = fmaf(1.061405429f, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  const float e = __builtin_amdgcn_exp2f((-1.4426950408889634f * x) * x);
  const float erf_abs = fmaf(-(p * t), e, 1.0f);
  const float hz = 0.5f * z;
  g = fmaf(hz, copysignf(erf_abs, z), hz);
  const float phi_cdf = fmaf(0.5f, copysignf(erf_abs, z), 0.5f);  // Phi(z)
  dg = fmaf(z * 0.3989422804014327f, e, phi_cdf);                // Phi + z phi
}

}  // namespace mhl
