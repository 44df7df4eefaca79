// IO-aware expert computation (Sec. 3.4) for gfx950: a dropless grouped
// SwiGLU FFN over the expert-clustered slot list, and the gate-weighted
// combine of Eq. (1).
//
// One workgroup = one tile = up to 128 clustered slots of one (head, expert);
// each of its 4 wavefronts owns 32 slots (one 32-slot MFMA column block), so
// a wavefront needs under 256 registers and two fit on a SIMD (one's SwiGLU
// VALU work overlaps the other's MFMAs).  The wavefront gathers its slots'
// sub-token rows X[t, h, :] straight into MFMA operand registers, then walks
// d_ff in chunks of 32 rows:
//
//   GEMM1  A^T = W1_c X^T, B^T = W3_c X^T   (32 x 32 tiles, K = d_h)
//   H^T    = silu(A^T) * B^T                 (registers only)
//   GEMM2  Y^T += W2_c H^T                   (K = the 32-wide chunk)
//
// The accumulator layout of GEMM1 (lane = slot, 16 d_ff rows per lane) is
// reused directly as the operand of GEMM2 by permuting the K order of the W2
// fragment to match, so the d_ff-wide intermediate never leaves registers.
// The weight chunks (W1_c, W3_c: 32 x d_h; W2_c: d_h x 32) are staged in LDS,
// double buffered, XOR-swizzled against bank conflicts, and shared by the
// four wavefronts.  Outputs are scaled by the
// slot's gate and written to a per-slot buffer yslot[T][Nh][k][d_h]; the
// combine kernel then sums each token's k slots in j order (deterministic,
// no atomics).

#include <math.h>

#include "device_common.hpp"
#include "ffn_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kFfnThreads = kFfnWaves * kWave;
constexpr int kChunk = 32;  // d_ff rows per pipeline step
static_assert(kFfnRowsPerWave == 32, "one 32-slot MFMA column block per wavefront");

template <int DH, bool F32>
struct FfnLayout {
  static constexpr int E = F32 ? 4 : 2;
  static constexpr int NJ1 = DH * E / 16;      // 16-byte chunks per W1/W3 row
  static constexpr int NJ2 = kChunk * E / 16;  // 16-byte chunks per W2 row
  static constexpr int W13_BYTES = kChunk * NJ1 * 16;
  static constexpr int W2_BYTES = DH * NJ2 * 16;
  static constexpr int STAGE = 2 * W13_BYTES + W2_BYTES;
  static constexpr int U1 = kChunk * NJ1;  // 16-byte units of W1 (and of W3)
  static constexpr int U2 = DH * NJ2;      // 16-byte units of W2
  static constexpr int NPT = (2 * U1 + U2) / kFfnThreads;
  static_assert(U1 % kFfnThreads == 0 && U2 % kFfnThreads == 0, "uneven chunk split");
};

// Cooperative loads of one d_ff chunk (W1/W3 rows f0..f0+31, W2 columns
// f0..f0+31) into registers, then into one LDS stage.  Unit i of a thread is
// W1 for i < U1/T, W3 for the next U1/T, W2 after that (T = threads); the
// source and LDS offsets are recomputed per use to save registers.
template <int DH, bool F32>
struct ChunkLoader {
  using L = FfnLayout<DH, F32>;
  static constexpr int N1 = L::U1 / kFfnThreads;
  u32x4 r[L::NPT];

  __device__ __forceinline__ void load(const uint8_t* w1, const uint8_t* w3, const uint8_t* w2,
                                       int ch, int dff) {
    const int tid = threadIdx.x;
    const int64_t o13 = (int64_t)ch * kChunk * DH * L::E;
    const int64_t o2 = (int64_t)ch * kChunk * L::E;
#pragma unroll
    for (int i = 0; i < L::NPT; ++i) {
      const uint8_t* src;
      if (i < 2 * N1) {
        const int uu = tid + kFfnThreads * (i % N1);
        src = (i < N1 ? w1 : w3) + o13 + uu * 16;
      } else {
        const int uu = tid + kFfnThreads * (i - 2 * N1);
        src = w2 + o2 + (int64_t)(uu / L::NJ2) * dff * L::E + (uu % L::NJ2) * 16;
      }
      r[i] = *reinterpret_cast<const u32x4*>(src);
    }
  }

  __device__ __forceinline__ void store(uint8_t* stage) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < L::NPT; ++i) {
      if (i < 2 * N1) {
        const int uu = tid + kFfnThreads * (i % N1);
        const int row = uu / L::NJ1, j = uu % L::NJ1;
        const int o = (i < N1 ? 0 : L::W13_BYTES) + row * L::NJ1 * 16 + swz<L::NJ1>(j, row) * 16;
        *reinterpret_cast<u32x4*>(stage + o) = r[i];
      } else {
        const int uu = tid + kFfnThreads * (i - 2 * N1);
        const int n = uu / L::NJ2, m = uu % L::NJ2;
        uint8_t* rowp = stage + 2 * L::W13_BYTES + n * L::NJ2 * 16;
        if (F32) {
          *reinterpret_cast<u32x4*>(rowp + swz<L::NJ2>(w2_group_pos(m), n) * 16) = r[i];
        } else {
          const int p0 = w2_group_pos(2 * m), p1 = w2_group_pos(2 * m + 1);
          *reinterpret_cast<u32x2*>(rowp + swz<L::NJ2>(p0 >> 1, n) * 16 + (p0 & 1) * 8) =
              u32x2{r[i][0], r[i][1]};
          *reinterpret_cast<u32x2*>(rowp + swz<L::NJ2>(p1 >> 1, n) * 16 + (p1 & 1) * 8) =
              u32x2{r[i][2], r[i][3]};
        }
      }
    }
  }
};

// One d_ff chunk for the wavefront's 32 rows:
//   GEMM1  A^T = W1_c X^T, B^T = W3_c X^T  (lane: slot c, d_ff rows 8(v/4) + 4g + v%4)
//   H^T    = silu(A^T) * B^T               (registers)
//   GEMM2  Y^T += W2_c H^T                  (K order permuted to H's lane layout)
template <int DH>
__device__ __forceinline__ void chunk_compute(const uint8_t* stage, const RowFrag<DH, false>& xf,
                                              f32x16 (&y)[DH / 32], int lane) {
  using L = FfnLayout<DH, false>;
  const int g = lane >> 5, c = lane & 31;
  const uint8_t* r1 = stage + c * L::NJ1 * 16;
  const uint8_t* r3 = r1 + L::W13_BYTES;
  f32x16 a, b;
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const int o = swz<L::NJ1>(2 * s + g, c) * 16;
    const bf16x8 f1 = as_bf16x8(*reinterpret_cast<const u32x4*>(r1 + o));
    const bf16x8 f3 = as_bf16x8(*reinterpret_cast<const u32x4*>(r3 + o));
    const bf16x8 xb = as_bf16x8(xf.x[s]);
    a = mfma32_bf16(f1, xb, s == 0 ? zero16() : a);
    b = mfma32_bf16(f3, xb, s == 0 ? zero16() : b);
  }
  u32x4 hp[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = 8 * hh + 2 * i;
      hp[hh][i] = pack_bf16x2(silu_fast(a[v]) * b[v], silu_fast(a[v + 1]) * b[v + 1]);
    }
  const uint8_t* w2 = stage + 2 * L::W13_BYTES;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) {
      const int n = 32 * nb + c;
      const bf16x8 f2 = as_bf16x8(*reinterpret_cast<const u32x4*>(
          w2 + n * L::NJ2 * 16 + swz<L::NJ2>(2 * hh + g, n) * 16));
      y[nb] = mfma32_bf16(f2, as_bf16x8(hp[hh]), y[nb]);
    }
  }
}

template <int DH>
__device__ __forceinline__ void chunk_compute(const uint8_t* stage, const RowFrag<DH, true>& xf,
                                              f32x16 (&y)[DH / 32], int lane) {
  using L = FfnLayout<DH, true>;
  const int g = lane >> 5, c = lane & 31;
  const uint8_t* r1 = stage + c * L::NJ1 * 16;
  const uint8_t* r3 = r1 + L::W13_BYTES;
  f32x16 a = zero16(), b = zero16();
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int o = swz<L::NJ1>(4 * s + 2 * g + half, c) * 16;
      const f32x4 f1 = *reinterpret_cast<const f32x4*>(r1 + o);
      const f32x4 f3 = *reinterpret_cast<const f32x4*>(r3 + o);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        a = mfma32_f32(f1[p], xf.x[s][half][p], a);
        b = mfma32_f32(f3[p], xf.x[s][half][p], b);
      }
    }
  }
  float hv[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) hv[v] = silu_fast(a[v]) * b[v];
  const uint8_t* w2 = stage + 2 * L::W13_BYTES;
#pragma unroll
  for (int nb = 0; nb < DH / 32; ++nb) {
    const int n = 32 * nb + c;
    const uint8_t* rowp = w2 + n * L::NJ2 * 16;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const f32x4 lo = *reinterpret_cast<const f32x4*>(rowp + swz<L::NJ2>(4 * hh + 2 * g, n) * 16);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(rowp + swz<L::NJ2>(4 * hh + 2 * g + 1, n) * 16);
#pragma unroll
      for (int p = 0; p < 8; ++p) y[nb] = mfma32_f32(p < 4 ? lo[p] : hi[p - 4], hv[8 * hh + p], y[nb]);
    }
  }
}

// State of one tile as seen by one lane: its slot row, the gathered X
// fragments, the gate and where the output row goes.
template <int DH, bool F32>
struct TileRows {
  RowFrag<DH, F32> xf;
  float gv;
  int64_t out_off;
  int slot;
  bool ok;
};

// Persistent workgroups walk the compact tile list: XCD x (workgroups are
// dispatched round-robin over the XCDs) owns the contiguous tile range
// [x n / 8, (x + 1) n / 8), so one expert's adjacent tiles run on one XCD at
// about the same time and share its L2; within it the workgroups stride by
// their count.  While a tile computes, the next tile's descriptor, slot rows,
// X fragments, gate and first weight chunk are fetched, so a tile starts
// without a dependent round trip to memory.
template <int DH, bool F32>
__global__ __launch_bounds__(kFfnThreads, 2) void ffn_kernel(
    const void* __restrict__ X, const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const TileInfo* __restrict__ tiles,
    const int32_t* __restrict__ head_base, const void* __restrict__ W1,
    const void* __restrict__ W3, const void* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, int dff, void* __restrict__ yslot) {
  using L = FfnLayout<DH, F32>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * L::STAGE];

  const int ntot = head_base[Nh];
  const int xcd = (int)(blockIdx.x % kXcds);
  const int nper = (int)(gridDim.x / kXcds);
  const int t_hi = (int)((int64_t)ntot * (xcd + 1) / kXcds);
  int tcur = (int)((int64_t)ntot * xcd / kXcds) + (int)(blockIdx.x / kXcds);
  if (tcur >= t_hi) return;

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int64_t head_slots = T * k;
  const int nc = dff / kChunk;
  const int64_t wbytes = (int64_t)dff * DH * L::E;  // one expert's W1 (= W3 = W2) bytes

  auto expert_base = [&](const TileInfo& ti) {
    return ((int64_t)ti.head * Ne + ti.expert) * wbytes;
  };
  auto slot_of = [&](const TileInfo& ti, bool& ok) {
    const int r = ti.row_begin + wave * kFfnRowsPerWave + c;
    ok = r < ti.row_end;
    return ok ? perm[(int64_t)ti.head * head_slots + r] : 0;
  };
  auto gather = [&](const TileInfo& ti, TileRows<DH, F32>& tr) {
    const int64_t t = tr.slot / k;
    const int j = tr.slot - (int)t * k;
    const int64_t tok_head = t * Nh + ti.head;
    tr.xf.load(X, tok_head, tr.ok, g);
    tr.gv = tr.ok ? gate[tok_head * k + j] : 0.f;
    tr.out_off = (tok_head * k + j) * DH;
  };
  const uint8_t* w1b = reinterpret_cast<const uint8_t*>(W1);
  const uint8_t* w3b = reinterpret_cast<const uint8_t*>(W3);
  const uint8_t* w2b = reinterpret_cast<const uint8_t*>(W2);

  TileInfo ti = tiles[tcur];
  TileRows<DH, F32> cur;
  cur.slot = slot_of(ti, cur.ok);
  gather(ti, cur);

  ChunkLoader<DH, F32> ld;
  int64_t eb = expert_base(ti);
  ld.load(w1b + eb, w3b + eb, w2b + eb, 0, dff);
  ld.store(smem);
  __syncthreads();
  int stage = 0;

  while (true) {
    const int tnext = tcur + nper;
    const bool has_next = tnext < t_hi;
    TileInfo tn = ti;
    TileRows<DH, F32> nxt;
    nxt.ok = false;
    nxt.slot = 0;
    const bool wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;

    f32x16 y[DH / 32];
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) y[nb] = zero16();

    for (int ch = 0; ch < nc; ++ch) {
      if (has_next) {
        if (ch == 0) tn = tiles[tnext];
        if (ch == (nc > 1 ? 1 : 0)) nxt.slot = slot_of(tn, nxt.ok);
        if (ch == (nc > 2 ? 2 : nc - 1)) gather(tn, nxt);
      }
      if (ch + 1 < nc) {
        ld.load(w1b + eb, w3b + eb, w2b + eb, ch + 1, dff);
      } else if (has_next) {
        const int64_t en = expert_base(tn);
        ld.load(w1b + en, w3b + en, w2b + en, 0, dff);
      }
      if (wave_active) chunk_compute<DH>(smem + stage * L::STAGE, cur.xf, y, lane);
      if (ch + 1 < nc || has_next) ld.store(smem + (stage ^ 1) * L::STAGE);
      __syncthreads();
      stage ^= 1;
    }

    // Y^T tile: lane holds slot column c, d_h rows 32 nb + 8 q + 4 g + [0, 4).
    if (cur.ok) {
#pragma unroll
      for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const int n = 32 * nb + 8 * qq + 4 * g;
          const float v0 = cur.gv * y[nb][4 * qq + 0];
          const float v1 = cur.gv * y[nb][4 * qq + 1];
          const float v2 = cur.gv * y[nb][4 * qq + 2];
          const float v3 = cur.gv * y[nb][4 * qq + 3];
          if (F32) {
            float* o = reinterpret_cast<float*>(yslot) + cur.out_off + n;
            *reinterpret_cast<f32x4*>(o) = f32x4{v0, v1, v2, v3};
          } else {
            uint16_t* o = reinterpret_cast<uint16_t*>(yslot) + cur.out_off + n;
            *reinterpret_cast<u32x2*>(o) = u32x2{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
          }
        }
    }
    if (!has_next) break;
    ti = tn;
    cur = nxt;
    eb = expert_base(ti);
    tcur = tnext;
  }
}

// Y[row] = sum_{j<k} yslot[row][j] in fixed j order; one thread per 8
// consecutive output elements.  All k loads are issued before the sums.
template <int DH, bool F32>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ yslot,
                                                      int64_t rows, int k,
                                                      void* __restrict__ Y) {
  constexpr int TPR = DH / 8;
  constexpr int KU = 8;  // slots loaded per round
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / TPR;
  const int part = (int)(gid % TPR);
  if (row >= rows) return;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  const int64_t base = row * k * DH + part * 8;
  for (int j0 = 0; j0 < k; j0 += KU) {
    if (F32) {
      f32x4 a[KU], b[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
          const float* p = reinterpret_cast<const float*>(yslot) + base + (int64_t)(j0 + u) * DH;
          a[u] = *reinterpret_cast<const f32x4*>(p);
          b[u] = *reinterpret_cast<const f32x4*>(p + 4);
        }
      }
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[i] += a[u][i];
            acc[4 + i] += b[u][i];
          }
        }
      }
    } else {
      u32x4 v[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u)
        if (j0 + u < k)
          v[u] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(yslot) + base +
                                                 (int64_t)(j0 + u) * DH);
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[2 * i] += bf16_bits_to_f32(v[u][i] & 0xFFFFu);
            acc[2 * i + 1] += bf16_bits_to_f32(v[u][i] >> 16);
          }
        }
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
                        const TileInfo* ti, const int32_t* head_base, const void* W1,
                        const void* W3, const void* W2, int64_t T, int Nh, int Ne,
                        int k, int dff, void* yslot, hipStream_t s) {
  hipLaunchKernelGGL((ffn_kernel<DH, F32>), dim3(kFfnGrid), dim3(kFfnThreads), 0, s, X, gate,
                     perm, ti, head_base, W1, W3, W2, T, Nh, Ne, k, dff, yslot);
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
                      const TileInfo* tile_info, const int32_t* head_base,
                      const void* W1, const void* W3, const void* W2,
                      int64_t T, int Nh, int dh, int Ne, int k, int dff,
                      bool f32, void* yslot, hipStream_t s) {
  if (T == 0) return hipSuccess;
#define MHL_FFN(DH, F)                                                               \
  return ffn_dispatch<DH, F>(X, gate, perm, tile_info, head_base, W1, W3, W2, T, Nh, \
                             Ne, k, dff, yslot, s)
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
