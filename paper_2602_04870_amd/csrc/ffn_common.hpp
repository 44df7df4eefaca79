// Device pieces shared by the expert forward and backward kernels: the
// XOR-swizzled LDS row layout, the W2 column regrouping, and the gathered
// slot-row operand fragments.
#pragma once

#include "device_common.hpp"

namespace mhl {

// LDS rows are stored as NJ 16-byte chunks with no padding; chunk j of row r
// sits at position j ^ f(r), chosen so that 16 consecutive rows reading the
// same logical chunk touch 16 distinct 16-byte bank groups (64 banks x 4 B).
template <int NJ>
__device__ __forceinline__ int swz(int j, int r) {
  constexpr int R = NJ >= 16 ? 1 : 16 / NJ;  // rows per 256-byte bank row
  constexpr int M = NJ >= 16 ? 16 : NJ;
  return j ^ ((r / R) % M);
}

// W2 columns of a chunk are regrouped in LDS so that the eight elements one
// lane feeds to a GEMM2 MFMA are contiguous: 4-element group G (logical
// columns 4G..4G+3) is stored at group position (G & ~3) | swap of bits 0, 1.
__device__ __forceinline__ int w2_group_pos(int G) {
  return (G & ~3) | ((G & 1) << 1) | ((G >> 1) & 1);
}

// The wavefront's 32 gathered slot rows as MFMA operand fragments: lane
// (g, c) holds row c, d_h elements 16 s + 8 g + [0, 8) for k-step s.
template <int DH, bool F32>
struct RowFrag;

template <int DH>
struct RowFrag<DH, false> {
  u32x4 x[DH / 16];
  __device__ __forceinline__ void load(const void* X, int64_t row, bool ok, int g) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(X) + row * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s)
      x[s] = ok ? *reinterpret_cast<const u32x4*>(p + 16 * s) : u32x4{0u, 0u, 0u, 0u};
  }
};

template <int DH>
struct RowFrag<DH, true> {
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

}  // namespace mhl
