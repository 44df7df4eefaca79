// IO-aware expert computation (Sec. 3.4) for gfx950: a dropless grouped
// SwiGLU FFN over the expert-clustered slot list, and the gate-weighted
// combine of Eq. (1).
//
// One workgroup = one tile = up to 128 clustered slots of one (head, expert);
// each of its 2 wavefronts owns 64 slots (two 32-slot MFMA column blocks).
// The wavefront gathers its slots' sub-token rows X[t, h, :] straight into
// MFMA operand registers, then walks d_ff in chunks of 32 rows:
//
//   GEMM1  A^T = W1_c X^T, B^T = W3_c X^T   (32 x 32 tiles, K = d_h)
//   H^T    = silu(A^T) * B^T                 (registers only)
//   GEMM2  Y^T += W2_c H^T                   (K = the 32-wide chunk)
//
// The accumulator layout of GEMM1 (lane = slot, 16 d_ff rows per lane) is
// reused directly as the operand of GEMM2 by permuting the K order of the W2
// fragment to match, so the d_ff-wide intermediate never leaves registers.
// The weight chunks (W1_c, W3_c: 32 x d_h; W2_c: d_h x 32) are staged in LDS,
// double buffered, and shared by both wavefronts.  Outputs are scaled by the
// slot's gate and written to a per-slot buffer yslot[T][Nh][k][d_h]; the
// combine kernel then sums each token's k slots in j order (deterministic,
// no atomics).

#include <math.h>

#include "device_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kFfnThreads = kFfnWaves * kWave;
constexpr int kChunk = 32;

template <int DH, bool F32>
struct FfnSmem;

template <int DH>
struct FfnSmem<DH, false> {
  static constexpr int kS1 = DH + 8;     // bf16 per W1/W3 chunk row
  static constexpr int kS2 = kChunk + 8; // bf16 per W2 chunk row
  uint16_t w1[2][kChunk * kS1];
  uint16_t w3[2][kChunk * kS1];
  uint16_t w2[2][DH * kS2];
};

template <int DH>
struct FfnSmem<DH, true> {
  static constexpr int kS1 = DH + 4;
  static constexpr int kS2 = kChunk + 4;
  float w1[2][kChunk * kS1];
  float w3[2][kChunk * kS1];
  float w2[2][DH * kS2];
};

// Cooperative 16-byte loads of one d_ff chunk of W1, W3 (32 contiguous rows of
// d_h) and W2 (d_h rows of 32 elements, row stride d_ff).
template <int DH, bool F32>
struct ChunkLoader {
  static constexpr int E = F32 ? 4 : 2;
  static constexpr int PER16 = 16 / E;                // elements per 16 bytes
  static constexpr int U1 = kChunk * DH / PER16;       // units of W1 (or W3)
  static constexpr int R2 = kChunk / PER16;            // units per W2 row
  static constexpr int U2 = DH * R2;
  static constexpr int U = 2 * U1 + U2;
  static constexpr int NPT = U / kFfnThreads;
  static_assert(U % kFfnThreads == 0, "chunk does not split evenly");
  u32x4 r[NPT];

  __device__ __forceinline__ void load(const uint8_t* w1, const uint8_t* w3,
                                       const uint8_t* w2, int dff, int f0) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int u = tid + kFfnThreads * i;
      const uint8_t* src;
      if (u < U1) {
        src = w1 + ((int64_t)f0 * DH) * E + (int64_t)u * 16;
      } else if (u < 2 * U1) {
        src = w3 + ((int64_t)f0 * DH) * E + (int64_t)(u - U1) * 16;
      } else {
        const int u2 = u - 2 * U1;
        const int n = u2 / R2, col = (u2 % R2) * PER16;
        src = w2 + ((int64_t)n * dff + f0 + col) * E;
      }
      r[i] = *reinterpret_cast<const u32x4*>(src);
    }
  }

  __device__ __forceinline__ void store(FfnSmem<DH, F32>& sm, int buf) const {
    using S = FfnSmem<DH, F32>;
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int u = tid + kFfnThreads * i;
      void* dst;
      if (u < 2 * U1) {
        const int uu = u < U1 ? u : u - U1;
        const int el = uu * PER16;
        const int row = el / DH, col = el % DH;
        dst = u < U1 ? (void*)&sm.w1[buf][row * S::kS1 + col]
                     : (void*)&sm.w3[buf][row * S::kS1 + col];
      } else {
        const int u2 = u - 2 * U1;
        const int n = u2 / R2, col = (u2 % R2) * PER16;
        dst = (void*)&sm.w2[buf][n * S::kS2 + col];
      }
      *reinterpret_cast<u32x4*>(dst) = r[i];
    }
  }
};

// Per-lane operand fragments of the wave's gathered slot rows.
template <int DH, bool F32>
struct RowFrag;

template <int DH>
struct RowFrag<DH, false> {
  u32x4 x[2][DH / 16];
  __device__ __forceinline__ void load(int tb, const void* X, int64_t row, bool ok, int g) {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(X) + row * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s)
      x[tb][s] = ok ? *reinterpret_cast<const u32x4*>(p + 16 * s) : u32x4{0u, 0u, 0u, 0u};
  }
};

template <int DH>
struct RowFrag<DH, true> {
  f32x4 x[2][DH / 16][2];
  __device__ __forceinline__ void load(int tb, const void* X, int64_t row, bool ok, int g) {
    const float* p = reinterpret_cast<const float*>(X) + row * DH + 8 * g;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      x[tb][s][0] = ok ? *reinterpret_cast<const f32x4*>(p + 16 * s) : f32x4{0.f, 0.f, 0.f, 0.f};
      x[tb][s][1] = ok ? *reinterpret_cast<const f32x4*>(p + 16 * s + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// One d_ff chunk: GEMM1 for both column blocks, SwiGLU, GEMM2 accumulate.
template <int DH>
__device__ __forceinline__ void chunk_compute(const FfnSmem<DH, false>& sm, int buf,
                                              const RowFrag<DH, false>& xf,
                                              f32x16 (&y)[2][DH / 32], int lane) {
  using S = FfnSmem<DH, false>;
  const int g = lane >> 5, c = lane & 31;
  f32x16 a[2], b[2];
  a[0] = a[1] = b[0] = b[1] = zero16();
  const uint16_t* w1 = &sm.w1[buf][c * S::kS1 + 8 * g];
  const uint16_t* w3 = &sm.w3[buf][c * S::kS1 + 8 * g];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const bf16x8 f1 = as_bf16x8(*reinterpret_cast<const u32x4*>(w1 + 16 * s));
    const bf16x8 f3 = as_bf16x8(*reinterpret_cast<const u32x4*>(w3 + 16 * s));
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const bf16x8 xb = as_bf16x8(xf.x[tb][s]);
      a[tb] = mfma32_bf16(f1, xb, a[tb]);
      b[tb] = mfma32_bf16(f3, xb, b[tb]);
    }
  }
  // H^T element v of this lane is d_ff row 8*(v/4) + 4*g + v%4 of the chunk.
  u32x4 hp[2][2];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = 8 * hh + 2 * i;
        hp[tb][hh][i] = pack_bf16x2(silu(a[tb][v]) * b[tb][v],
                                    silu(a[tb][v + 1]) * b[tb][v + 1]);
      }
  // GEMM2 K-step hh covers accumulator elements v in [8 hh, 8 hh + 8), i.e.
  // d_ff rows 16 hh + 8 (p/4) + 4 g + p%4 for operand element p; the W2
  // fragment is read in that same order.
#pragma unroll
  for (int nb = 0; nb < DH / 32; ++nb) {
    const uint16_t* w2 = &sm.w2[buf][(32 * nb + c) * S::kS2 + 4 * g];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const u32x2 lo = *reinterpret_cast<const u32x2*>(w2 + 16 * hh);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(w2 + 16 * hh + 8);
      const bf16x8 f2 = as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) y[tb][nb] = mfma32_bf16(f2, as_bf16x8(hp[tb][hh]), y[tb][nb]);
    }
  }
}

template <int DH>
__device__ __forceinline__ void chunk_compute(const FfnSmem<DH, true>& sm, int buf,
                                              const RowFrag<DH, true>& xf,
                                              f32x16 (&y)[2][DH / 32], int lane) {
  using S = FfnSmem<DH, true>;
  const int g = lane >> 5, c = lane & 31;
  f32x16 a[2], b[2];
  a[0] = a[1] = b[0] = b[1] = zero16();
  const float* w1 = &sm.w1[buf][c * S::kS1 + 8 * g];
  const float* w3 = &sm.w3[buf][c * S::kS1 + 8 * g];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const f32x4 f1 = *reinterpret_cast<const f32x4*>(w1 + 16 * s + 4 * half);
      const f32x4 f3 = *reinterpret_cast<const f32x4*>(w3 + 16 * s + 4 * half);
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int tb = 0; tb < 2; ++tb) {
          a[tb] = mfma32_f32(f1[p], xf.x[tb][s][half][p], a[tb]);
          b[tb] = mfma32_f32(f3[p], xf.x[tb][s][half][p], b[tb]);
        }
    }
  }
  float hv[2][16];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int v = 0; v < 16; ++v) hv[tb][v] = silu(a[tb][v]) * b[tb][v];
#pragma unroll
  for (int nb = 0; nb < DH / 32; ++nb) {
    const float* w2 = &sm.w2[buf][(32 * nb + c) * S::kS2 + 4 * g];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const f32x4 lo = *reinterpret_cast<const f32x4*>(w2 + 16 * hh);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(w2 + 16 * hh + 8);
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const float wv = p < 4 ? lo[p] : hi[p - 4];
#pragma unroll
        for (int tb = 0; tb < 2; ++tb) y[tb][nb] = mfma32_f32(wv, hv[tb][8 * hh + p], y[tb][nb]);
      }
    }
  }
}

template <int DH, bool F32>
__global__ __launch_bounds__(kFfnThreads) void ffn_kernel(
    const void* __restrict__ X, const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const TileInfo* __restrict__ tile_info,
    const int32_t* __restrict__ ntiles, const void* __restrict__ W1,
    const void* __restrict__ W3, const void* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, int dff, int64_t max_tiles, void* __restrict__ yslot) {
  __shared__ FfnSmem<DH, F32> sm;
  constexpr int E = F32 ? 4 : 2;

  const int h = blockIdx.y;
  const int tile = blockIdx.x;
  if (tile >= ntiles[h]) return;
  const TileInfo ti = tile_info[(int64_t)h * max_tiles + tile];
  const int e = ti.expert;

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int wrow0 = ti.row_begin + wave * kFfnRowsPerWave;
  const bool wave_active = wrow0 < ti.row_end;

  const int32_t* P = perm + (int64_t)h * T * k;
  RowFrag<DH, F32> xf;
  int64_t out_off[2];
  float gv[2];
  bool ok[2];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int r = wrow0 + 32 * tb + c;
    ok[tb] = r < ti.row_end;
    const int slot = ok[tb] ? P[r] : 0;
    const int64_t t = slot / k;
    const int j = slot - (int)t * k;
    const int64_t tok_head = t * Nh + h;
    xf.load(tb, X, tok_head, ok[tb], g);
    gv[tb] = ok[tb] ? gate[tok_head * k + j] : 0.f;
    out_off[tb] = (tok_head * k + j) * DH;
  }

  const int64_t he = (int64_t)h * Ne + e;
  const uint8_t* w1 = reinterpret_cast<const uint8_t*>(W1) + he * dff * DH * E;
  const uint8_t* w3 = reinterpret_cast<const uint8_t*>(W3) + he * dff * DH * E;
  const uint8_t* w2 = reinterpret_cast<const uint8_t*>(W2) + he * DH * dff * E;

  f32x16 y[2][DH / 32];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) y[tb][nb] = zero16();

  ChunkLoader<DH, F32> ld;
  const int nc = dff / kChunk;
  ld.load(w1, w3, w2, dff, 0);
  ld.store(sm, 0);
  __syncthreads();
  for (int ch = 0; ch < nc; ++ch) {
    const int buf = ch & 1;
    if (ch + 1 < nc) ld.load(w1, w3, w2, dff, (ch + 1) * kChunk);
    if (wave_active) chunk_compute<DH>(sm, buf, xf, y, lane);
    if (ch + 1 < nc) ld.store(sm, buf ^ 1);
    __syncthreads();
  }

  // Y^T tile: lane holds slot column c, d_h rows 32 nb + 8 q + 4 g + [0, 4).
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    if (!ok[tb]) continue;
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = 32 * nb + 8 * q + 4 * g;
        const float v0 = gv[tb] * y[tb][nb][4 * q + 0];
        const float v1 = gv[tb] * y[tb][nb][4 * q + 1];
        const float v2 = gv[tb] * y[tb][nb][4 * q + 2];
        const float v3 = gv[tb] * y[tb][nb][4 * q + 3];
        if (F32) {
          float* o = reinterpret_cast<float*>(yslot) + out_off[tb] + n;
          *reinterpret_cast<f32x4*>(o) = f32x4{v0, v1, v2, v3};
        } else {
          uint16_t* o = reinterpret_cast<uint16_t*>(yslot) + out_off[tb] + n;
          *reinterpret_cast<u32x2*>(o) = u32x2{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
        }
      }
  }
}

// Y[row] = sum_{j<k} yslot[row][j] in fixed j order; one thread per 8
// consecutive output elements.
template <int DH, bool F32>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ yslot,
                                                      int64_t rows, int k,
                                                      void* __restrict__ Y) {
  constexpr int TPR = DH / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / TPR;
  const int part = (int)(gid % TPR);
  if (row >= rows) return;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int j = 0; j < k; ++j) {
    const int64_t off = (row * k + j) * DH + part * 8;
    if (F32) {
      const float* p = reinterpret_cast<const float*>(yslot) + off;
      const f32x4 a = *reinterpret_cast<const f32x4*>(p);
      const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i] += a[i];
        acc[4 + i] += b[i];
      }
    } else {
      const u32x4 v = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(yslot) + off);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += bf16_bits_to_f32(v[i] & 0xFFFFu);
        acc[2 * i + 1] += bf16_bits_to_f32(v[i] >> 16);
      }
    }
  }
  const int64_t o = row * DH + part * 8;
  if (F32) {
    float* p = reinterpret_cast<float*>(Y) + o;
    *reinterpret_cast<f32x4*>(p) = f32x4{acc[0], acc[1], acc[2], acc[3]};
    *reinterpret_cast<f32x4*>(p + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
  } else {
    *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(Y) + o) =
        u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
              pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
  }
}

template <int DH, bool F32>
hipError_t ffn_dispatch(const void* X, const float* gate, const int32_t* perm,
                        const TileInfo* ti, const int32_t* ntiles, const void* W1,
                        const void* W3, const void* W2, int64_t T, int Nh, int Ne,
                        int k, int dff, int64_t max_tiles, void* yslot, hipStream_t s) {
  const dim3 grid((unsigned)max_tiles, (unsigned)Nh);
  hipLaunchKernelGGL((ffn_kernel<DH, F32>), grid, dim3(kFfnThreads), 0, s, X, gate,
                     perm, ti, ntiles, W1, W3, W2, T, Nh, Ne, k, dff, max_tiles, yslot);
  return hipGetLastError();
}

template <int DH, bool F32>
hipError_t combine_dispatch(const void* yslot, int64_t T, int Nh, int k, void* Y,
                            hipStream_t s) {
  const int64_t rows = T * Nh;
  const int64_t threads = rows * (DH / 8);
  const dim3 grid((unsigned)ceil_div(threads, 256));
  hipLaunchKernelGGL((combine_kernel<DH, F32>), grid, dim3(256), 0, s, yslot, rows, k, Y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ffn(const void* X, const float* gate, const int32_t* perm,
                      const TileInfo* tile_info, const int32_t* ntiles,
                      const void* W1, const void* W3, const void* W2,
                      int64_t T, int Nh, int dh, int Ne, int k, int dff,
                      bool f32, int64_t max_tiles, void* yslot, hipStream_t s) {
  if (T == 0) return hipSuccess;
#define MHL_FFN(DH, F)                                                           \
  return ffn_dispatch<DH, F>(X, gate, perm, tile_info, ntiles, W1, W3, W2, T, Nh, \
                             Ne, k, dff, max_tiles, yslot, s)
  if (dh == 128) {
    if (f32) MHL_FFN(128, true);
    MHL_FFN(128, false);
  }
  if (dh == 64) {
    if (f32) MHL_FFN(64, true);
    MHL_FFN(64, false);
  }
#undef MHL_FFN
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const void* yslot, int64_t T, int Nh, int dh, int k,
                          bool f32, void* Y, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dh == 128)
    return f32 ? combine_dispatch<128, true>(yslot, T, Nh, k, Y, s)
               : combine_dispatch<128, false>(yslot, T, Nh, k, Y, s);
  if (dh == 64)
    return f32 ? combine_dispatch<64, true>(yslot, T, Nh, k, Y, s)
               : combine_dispatch<64, false>(yslot, T, Nh, k, Y, s);
  return hipErrorInvalidValue;
}

}  // namespace mhl
