// Backward of the Multi-Head LatentMoE layer for gfx950: routing backward
// (Algorithm 2, Sec. 3.3) and the gradient of Eq. (1)-(3) with the SwiGLU
// expert.  Nothing from the forward is stored except idx and gate; the expert
// intermediate is recomputed.
//
// Per slot (token t, head h, k-slot j, expert e, gate g):
//   a = W1 x, b = W3 x, u = silu(a) * b          (recomputed)
//   v = W2^T dy                                   (one GEMM gives both:)
//   dg = <dy, W2 u> = <v, u>,   du = g v
//   da = du * b * silu'(a),     db = du * silu(a)
//   dX_expert = W1^T da + W3^T db
//   dW1 += da x^T, dW3 += db x^T, dW2 += dy (g u)^T
// Per token: dS_j = g_j (dg_j - sum_j' g_j' dg_j')  (softmax backward)
//   dX = sum_j dS_j W_r[h, e_j] + dX_expert_j     (Algorithm 2's dX)
//   dW_r[h, e] += dS x over the slots of e        (Algorithm 2's dW_r)
//
// Kernels (all deterministic, no floating-point atomics):
//   bwd_dx_kernel     tiles of 32 slots of one expert (the forward's tile list):
//                     a, b, v, dg and the per-slot dX_expert, d_ff streamed
//                     through LDS in chunks of 32 as in the forward FFN;
//   bwd_combine_kernel per (t, h): dS and dX in fixed j order;
//   bwd_dw_kernel     one workgroup per (expert, 32-wide d_ff chunk) with the
//                     chunk's weights resident in LDS, looping over all of the
//                     expert's slots (the next 32 slots' rows fetched while the
//                     current ones are used); each wavefront accumulates
//                     dW1/dW3/dW2 in registers, then the four partial sums
//                     are added in a fixed order.  Experts are
//                     taken in decreasing order of slot count (dw_order_kernel)
//                     so the longest workgroups start first.  For the contraction over slots
//                     GEMM1 is taken with slots as rows, so a, b, v arrive with
//                     one d_ff index per lane and the slot axis in registers;
//   rdw_plan / router_dw_seg / router_dw_fix
//                     dW_r from the router's input rows, the expert's slots
//                     cut into segments spread over workgroups.

#include <math.h>

#include "device_common.hpp"
#include "ffn_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kBwdThreads = 256;  // 4 wavefronts
constexpr int kChunk = 32;

// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives
// element i % 4 of the 8-byte pieces addressed by lanes i / 4, 4 + i / 4,
// 8 + i / 4 and 12 + i / 4 (so four rows of 4 columns, one row per
// addressing lane quad, come back as one column per lane).
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 lds_read_tr16(const uint8_t* p) {
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(p));
  return __builtin_bit_cast(u32x2, r);
}

__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

// Row swizzle of the backward's LDS matrices: 16-byte unit j of row r sits
// at position swz_tr(j, r) = j ^ mask(r), a linear bijection of the row's
// place in 16 bank rows.  It keeps three read forms free of bank conflicts:
//  - 32 rows reading one logical unit with ds_read_b128 (the 32x32 operand
//    form: 16 lanes served together hold 16 distinct rows mod 16);
//  - 16 rows reading units u0 + lane / 16 (the 16x16x32 operand form): the
//    LDS serves a ds_read_b128 in four cycles, to the lanes of equal bit 5
//    and equal parity of bits 2-4, so for 256-byte rows the mask's images of
//    row bits 2 and 3 must stay independent of rows 0-1's after adding the
//    unit bit that lane bit 4 contributes;
//  - four consecutive rows r0..r0+3 (r0 a multiple of 4) each reading one
//    aligned 64-byte piece (ds_read_b64_tr_b16 fragments): their masks differ
//    in the two bits above the piece (256-byte rows) or, two rows to a bank
//    row, in the bit above it, so the 16 units land in 16 bank groups.
template <int NJ>
__device__ __forceinline__ int swz_tr(int j, int r) {
  static_assert(NJ == 8 || NJ == 16, "rows of 128 or 256 bytes");
  if constexpr (NJ == 16) {
    const int m = r & 15;
    return j ^ (((m & 3) << 2) | ((((m >> 2) ^ (m >> 3)) & 1) << 1) | ((m >> 3) & 1));
  } else {
    const int m = (r >> 1) & 7;
    return j ^ (((m & 1) << 2) | (m >> 1));
  }
}

// ---------------------------------------------------------------------------
// Weight-chunk layouts in LDS (bf16):
//   W1_c, W3_c  [32 f][DH n]   rows f, 16-byte units of n swizzled by swz_tr
//   W2_c        [DH n][32 f]   rows n, 16-byte units of f XOR-swizzled by n / 8
//   or W2_c^T   [32 f][DH n]   as W1_c (transposed on store, for a kernel
//                              that keeps the chunk for all its slots)
// Operands whose K runs down a column (W2^T for v from W2_c, W1^T / W3^T
// for dX) are read with ds_read_b64_tr_b16 (lds_read_tr16).
// ---------------------------------------------------------------------------
template <int DH>
struct BwdLayout {
  static constexpr int NJ1 = DH * 2 / 16;  // 16-byte chunks per W1_c / W3_c row
  static constexpr int NAT = kChunk * NJ1 * 16;  // bytes of one chunk matrix (any of the three)
  static constexpr int W2ROW = kChunk * 2;       // bytes per W2_c row (64)
};

template <int DH>
__device__ __forceinline__ int w13_byte(int f, int n) {
  using L = BwdLayout<DH>;
  return f * L::NJ1 * 16 + swz_tr<L::NJ1>(n >> 3, f) * 16 + (n & 7) * 2;
}

template <int DH>
__device__ __forceinline__ int w2_byte(int n, int f) {
  using L = BwdLayout<DH>;
  return n * L::W2ROW + (((f >> 3) ^ ((n >> 3) & 3)) << 4) + (f & 7) * 2;
}

// MFMA operand fragment (eight K of one M / N index per lane) from a matrix
// in LDS whose rows are K: lane l takes column col0 + l % 32 and, for
// elements 0-3 and 4-7, rows ra(g) .. ra(g) + 3 and rb(g) .. rb(g) + 3,
// g = l / 32.  Lane j of each 16-lane group addresses row r + j / 4,
// columns col + 4 (j % 4) .. + 3 (see lds_read_tr16).  addr(row, col) gives
// the byte offset of an 8-byte aligned piece of four columns.
template <typename Addr>
__device__ __forceinline__ bf16x8 tr_fragment(const uint8_t* base, const Addr& addr, int ra0,
                                              int ra1, int rb0, int rb1, int col0) {
  const int lane = lane_id();
  const int grp = lane >> 4, j = lane & 15;
  const int col = col0 + 16 * (grp & 1) + 4 * (j & 3);
  const int ra = (grp >> 1) ? ra1 : ra0, rb = (grp >> 1) ? rb1 : rb0;
  const u32x2 lo = lds_read_tr16(base + addr(ra + (j >> 2), col));
  const u32x2 hi = lds_read_tr16(base + addr(rb + (j >> 2), col));
  return as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
}

// Loads one d_ff chunk f0..f0+31 of one expert (W1/W3 rows and W2 rows, in
// 16-byte units), then stores it to a stage W1_c | W3_c | W2_c (W2_c^T when
// W2T).  GELU (the two-matrix expert): W1 is W_in, W2 is W_out, and the W3
// part is neither loaded nor stored.
template <int DH, bool W2T, bool GELU = false>
struct BwdChunkLoader {
  static constexpr int U13 = kChunk * DH / 8;  // 16-byte units of W1 (or W3) chunk
  static constexpr int U2 = DH * kChunk / 8;   // 16-byte units of the W2 chunk
  static constexpr int NPT = (2 * U13 + U2) / kBwdThreads;
  static constexpr int N13 = U13 / kBwdThreads;
  static_assert((2 * U13 + U2) % kBwdThreads == 0 && U13 % kBwdThreads == 0, "uneven split");
  u32x4 r[NPT];

  // tid: the thread's index among the kBwdThreads that share the chunk
  __device__ __forceinline__ void load(const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                                       int f0, int dff, int tid) {
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      if (GELU && i >= N13 && i < 2 * N13) continue;
      const uint16_t* src;
      if (i < 2 * N13) {
        const int uu = tid + kBwdThreads * (i % N13);
        const int f = uu / (DH / 8), n8 = uu % (DH / 8);
        src = (i < N13 ? w1 : w3) + (int64_t)(f0 + f) * DH + n8 * 8;
      } else {
        const int uu = tid + kBwdThreads * (i - 2 * N13);
        const int n = uu / (kChunk / 8), f8 = uu % (kChunk / 8);
        src = w2 + (int64_t)n * dff + f0 + f8 * 8;
      }
      r[i] = *reinterpret_cast<const u32x4*>(src);
    }
  }

  __device__ __forceinline__ void store(uint8_t* stage, int tid) const {
    using L = BwdLayout<DH>;
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      if (GELU && i >= N13 && i < 2 * N13) continue;
      if (i < 2 * N13) {
        const int uu = tid + kBwdThreads * (i % N13);
        const int f = uu / (DH / 8), n8 = uu % (DH / 8);
        *reinterpret_cast<u32x4*>(stage + (i < N13 ? 0 : L::NAT) + w13_byte<DH>(f, n8 * 8)) = r[i];
      } else {
        const int uu = tid + kBwdThreads * (i - 2 * N13);
        const int n = uu / (kChunk / 8), f8 = uu % (kChunk / 8);
        if (W2T) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const uint32_t word = r[i][q >> 1];
            *reinterpret_cast<uint16_t*>(stage + 2 * L::NAT + w13_byte<DH>(f8 * 8 + q, n)) =
                (uint16_t)((q & 1) ? (word >> 16) : (word & 0xFFFFu));
          }
        } else {
          *reinterpret_cast<u32x4*>(stage + 2 * L::NAT + w2_byte<DH>(n, f8 * 8)) = r[i];
        }
      }
    }
  }
};

// One d_ff chunk f0..f0+31 of one expert straight from global memory into a
// stage W1_c | W3_c | W2_c (the layouts of w13_byte and w2_byte) by LDS DMA.
// The stage is 3 NAT bytes, filled by 1 KiB instructions: instruction d of
// wavefront w fills piece kBwdWaves d + w, so the matrix it belongs to
// depends on d alone and is a compile-time constant.  Lane l's 16 bytes land
// at byte 16 l of the piece, a physical 16-byte unit whose logical unit the
// lane's source offset picks (the XOR swizzles are their own inverses).  The
// source offsets of chunk 0 are fixed per lane and computed once; chunk f0
// adds a wavefront-uniform offset (f0 rows of W1 / W3, f0 columns of W2)
// given as the buffer instruction's scalar offset, so issuing a chunk takes
// no vector instructions.  GELU skips the W3 part.  Completion is tracked by
// vmcnt; no register holds the chunk.
constexpr int kBwdWaves = kBwdThreads / kWave;

template <int DH, bool GELU>
struct BwdDma {
  using L = BwdLayout<DH>;
  static constexpr int IPM = L::NAT / 1024;       // 1 KiB pieces per matrix
  static constexpr int DPW = 3 * IPM / kBwdWaves;  // instructions per wavefront
  // of which issued (GELU skips the W3 part)
  static constexpr int ISSUED = GELU ? DPW - IPM / kBwdWaves : DPW;
  static_assert(L::NAT % 1024 == 0 && IPM % kBwdWaves == 0, "uniform DMA split");
  uint32_t voff[DPW];  // source byte offset of the lane's unit in its matrix, chunk 0

  __device__ __forceinline__ void init(int wave, int lane, int dff) {
#pragma unroll
    for (int d = 0; d < DPW; ++d) {
      const int m = kBwdWaves * d / IPM;  // 0: W1, 1: W3, 2: W2
      const int b = ((kBwdWaves * d + wave) % IPM) * 1024 + 16 * lane;
      if (m < 2) {
        const int f = b / (L::NJ1 * 16), p = (b / 16) % L::NJ1;
        voff[d] = (uint32_t)(f * DH + swz_tr<L::NJ1>(p, f) * 8) * 2;
      } else {
        const int n = b / L::W2ROW, p = (b / 16) % (L::W2ROW / 16);
        voff[d] = (uint32_t)(n * dff + (p ^ ((n >> 3) & 3)) * 8) * 2;
      }
    }
  }

  // r1, r3, r2: buffer resources over the expert's W1, W3, W2 (wave: the
  // wavefront's index, uniform).
  __device__ __forceinline__ void issue(uint8_t* stage, __amdgpu_buffer_rsrc_t r1,
                                        __amdgpu_buffer_rsrc_t r3, __amdgpu_buffer_rsrc_t r2,
                                        int wave, int f0) const {
#pragma unroll
    for (int d = 0; d < DPW; ++d) {
      const int m = kBwdWaves * d / IPM;
      if (GELU && m == 1) continue;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          m == 0 ? r1 : (m == 1 ? r3 : r2),
          (__attribute__((address_space(3))) void*)(stage + 1024 * (kBwdWaves * d + wave)), 16,
          voff[d], m < 2 ? f0 * DH * 2 : f0 * 2, 0, 0);
    }
  }
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t bwd_rsrc(const uint16_t* base, int num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, num_bytes, 0x00020000);
}

// ---------------------------------------------------------------------------
// dX_expert and dg per slot.
// ---------------------------------------------------------------------------
// GELU: the two-matrix expert (W1 = W_in, W2 = W_out; W3 unused):
// h = gelu(a), dg = <v, h>, da = g v gelu'(a), dX_expert = W_in^T da.
template <int DH, bool GELU>
// Two workgroups per CU (two wavefronts per SIMD) so one's loads overlap the
// other's matrix work; at d_h 128 this costs a few spilled registers.
__global__ __launch_bounds__(kBwdThreads, 2) void bwd_dx_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ dY,
    const float* __restrict__ gate, const int32_t* __restrict__ perm,
    const TileInfo* __restrict__ tiles, const int32_t* __restrict__ head_base,
    const uint16_t* __restrict__ W1, const uint16_t* __restrict__ W3,
    const uint16_t* __restrict__ W2, int64_t T, int Nh, int Ne, int k, int dff,
    uint16_t* __restrict__ dxslot, float* __restrict__ dgslot) {
  using L = BwdLayout<DH>;
  constexpr int STAGE = 3 * L::NAT;
  __shared__ __attribute__((aligned(16))) uint8_t smem[3 * STAGE];

  const int ntot = 2 * head_base[Nh];  // half-tile work items
  const int xcd = (int)(blockIdx.x % kXcds);
  const int nper = (int)(gridDim.x / kXcds);
  const int t_hi = (int)((int64_t)ntot * (xcd + 1) / kXcds);
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int nc = dff / kChunk;
  const int wbytes = dff * DH * 2;  // one expert's W1, W3 or W2
  BwdDma<DH, GELU> dma;
  dma.init(wave, lane, dff);
  auto rsrcs = [&](const TileInfo& t, __amdgpu_buffer_rsrc_t& r1, __amdgpu_buffer_rsrc_t& r3,
                   __amdgpu_buffer_rsrc_t& r2) {
    const int64_t eo = ((int64_t)t.head * Ne + t.expert) * dff * DH;
    r1 = bwd_rsrc(W1 + eo, wbytes);
    r3 = bwd_rsrc(W3 + eo, wbytes);
    r2 = bwd_rsrc(W2 + eo, wbytes);
  };

  // Chunk ch of a tile sits in stage (s0 + ch) % 3 of a three-stage ring:
  // step ch fetches chunk ch + 2, which has two steps to land.  A tile's
  // chunks 0 and 1 are fetched when the tile starts, beside its slot rows.
  // (Fetching them during the previous tile's last steps was measured slower
  // where most tiles hold a few slots of a cold expert: the rows then wait
  // behind them.)
  // The second half of an expert's last tile is empty when that tile has at
  // most 128 slots: such items are skipped (no weights fetched for them).
  auto next_item = [&](int i, TileInfo& t) {
    for (; i < t_hi; i += nper) {
      t = half_tile(tiles, i);
      if (t.row_begin < t.row_end) break;
    }
    return i;
  };
  int s0 = 0;
  TileInfo ti{};
  __amdgpu_buffer_rsrc_t r1, r3, r2;
  int tile = next_item((int)((int64_t)ntot * xcd / kXcds) + (int)(blockIdx.x / kXcds), ti);
  if (tile < t_hi) rsrcs(ti, r1, r3, r2);
  for (int tnext; tile < t_hi; tile = tnext) {
    const int r = ti.row_begin + wave * kFfnRowsPerWave + c;
    const bool ok = r < ti.row_end;
    const bool wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;
    const int slot = ok ? perm[(int64_t)ti.head * T * k + r] : 0;
    // stages s0 and s0 + 1 (mod 3) were last read three and two steps ago
    // (or never), each before a barrier
    dma.issue(smem + s0 * STAGE, r1, r3, r2, wave, 0);
    const int64_t t = slot / k;
    const int j = slot - (int)t * k;
    const int64_t th = t * Nh + ti.head;
    RowFrag<DH, false> xf, df;
    xf.load(X, th, ok, g);
    df.load(dY, th, ok, g);
    const float gs = ok ? gate[th * k + j] : 0.f;
    // the next tile's descriptor, read ahead
    TileInfo tn{};
    __amdgpu_buffer_rsrc_t n1, n3, n2;
    tnext = next_item(tile + nper, tn);
    if (tnext < t_hi) rsrcs(tn, n1, n3, n2);
    if (nc > 1) {
      dma.issue(smem + (s0 == 2 ? 0 : s0 + 1) * STAGE, r1, r3, r2, wave, kChunk);
      barrier_vm<BwdDma<DH, GELU>::ISSUED>();  // chunk 0 and the rows landed
    } else {
      barrier_vm<0>();
    }

    f32x16 dx[DH / 32];
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) dx[nb] = zero16();
    float dg = 0.f;

    for (int ch = 0, sc = s0; ch < nc; ++ch, sc = sc == 2 ? 0 : sc + 1) {
      const uint8_t* st = smem + sc * STAGE;
      // stage sc + 2 (mod 3) was last read in step ch - 1, before its barrier
      const bool ahead = ch + 2 < nc;
      if (ahead)
        dma.issue(smem + (sc == 0 ? 2 : sc - 1) * STAGE, r1, r3, r2, wave, (ch + 2) * kChunk);
      if (wave_active) {
        const uint8_t* r1 = st + c * L::NJ1 * 16;
        const uint8_t* r3 = r1 + L::NAT;
        const auto w2a = [](int n, int f) { return w2_byte<DH>(n, f); };
        f32x16 a, b, v;
#pragma unroll
        for (int s = 0; s < DH / 16; ++s) {
          const int o = swz_tr<L::NJ1>(2 * s + g, c) * 16;
          const bf16x8 xb = as_bf16x8(xf.x[s]);
          const bf16x8 db8 = as_bf16x8(df.x[s]);
          a = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(r1 + o)), xb, s == 0 ? zero16() : a);
          if (!GELU)
            b = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(r3 + o)), xb, s == 0 ? zero16() : b);
          // W2^T row f = c: column c of W2_c at n = 16 s + 8 g + [0, 8)
          const bf16x8 w2f = tr_fragment(st + 2 * L::NAT, w2a, 16 * s, 16 * s + 8, 16 * s + 4,
                                         16 * s + 12, 0);
          v = mfma32_bf16(w2f, db8, s == 0 ? zero16() : v);
        }
        // lane: slot c; element e: d_ff row 8(e/4) + 4g + e%4 of the chunk
        u32x4 pa[2], pb[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float da2[2], db2[2];
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const int e = 8 * hh + 2 * i + q;
              if (GELU) {
                float h, dh;
                gelu_and_grad(a[e], h, dh);
                dg += v[e] * h;
                da2[q] = gs * v[e] * dh;
                db2[q] = 0.f;
              } else {
                const float sg = sigmoid_fast(a[e]);
                const float sl = a[e] * sg;
                dg += v[e] * (sl * b[e]);
                const float du = gs * v[e];
                da2[q] = du * b[e] * (sg + sl * (1.0f - sg));
                db2[q] = du * sl;
              }
            }
            pa[hh][i] = pack_bf16x2(da2[0], da2[1]);
            pb[hh][i] = pack_bf16x2(db2[0], db2[1]);
          }
        // dX_expert^T (rows n, columns slots) += W1_c^T da + W3_c^T db: W1^T /
        // W3^T rows n = 32 nb + c are columns of W1_c / W3_c, taken at d_ff
        // rows 16 hh + 8 (p / 4) + 4 g + p % 4 to match pa / pb's order.
        const auto w13a = [](int f, int n) { return w13_byte<DH>(f, n); };
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int nb = 0; nb < DH / 32; ++nb) {
            const bf16x8 t1 = tr_fragment(st, w13a, 16 * hh, 16 * hh + 4, 16 * hh + 8,
                                          16 * hh + 12, 32 * nb);
            dx[nb] = mfma32_bf16(t1, as_bf16x8(pa[hh]), dx[nb]);
            if (!GELU) {
              const bf16x8 t3 = tr_fragment(st + L::NAT, w13a, 16 * hh, 16 * hh + 4, 16 * hh + 8,
                                            16 * hh + 12, 32 * nb);
              dx[nb] = mfma32_bf16(t3, as_bf16x8(pb[hh]), dx[nb]);
            }
          }
      }
      // chunk ch + 1 landed (chunk ch + 2's DMA may stay in flight)
      if (ahead) barrier_vm<BwdDma<DH, GELU>::ISSUED>();
      else barrier_vm<0>();
    }

    dg += __shfl_xor(dg, 32, kWave);
    if (ok) {
      if (g == 0) dgslot[th * k + j] = dg;
      uint16_t* o = dxslot + (th * k + j) * DH;
#pragma unroll
      for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const int n = 32 * nb + 8 * qq + 4 * g;
          *reinterpret_cast<u32x2*>(o + n) =
              u32x2{pack_bf16x2(dx[nb][4 * qq], dx[nb][4 * qq + 1]),
                    pack_bf16x2(dx[nb][4 * qq + 2], dx[nb][4 * qq + 3])};
        }
    }
    s0 = (s0 + nc) % 3;
    ti = tn;
    r1 = n1;
    r3 = n3;
    r2 = n2;
  }
}

// ---------------------------------------------------------------------------
// dS and dX per (t, h).  One thread per 8 consecutive dX elements.
// ---------------------------------------------------------------------------
// With SPLIT (separate routing sub-tokens, Sec. 4.4) the router term
// sum_j dS_j W_r[h, e_j] goes to dR and dX keeps the expert terms.
// U: slots whose loads are in flight together (16 where a row has at least
// 32 slots: fewer latency waits per row; 8 otherwise, where 16 would leave
// the slots of a short row to the one-at-a-time tail).
template <int DH, bool SPLIT, int U>
__global__ __launch_bounds__(256) void bwd_combine_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ gate,
    const float* __restrict__ dgslot, const uint16_t* __restrict__ dxslot,
    const float* __restrict__ W_router, int64_t rows, int Nh, int Ne, int k,
    uint16_t* __restrict__ dX, uint16_t* __restrict__ dR, float* __restrict__ dS) {
  constexpr int TPR = DH / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / TPR;  // t * Nh + h
  const int part = (int)(gid % TPR);
  if (row >= rows) return;
  const int h = (int)(row % Nh);
  const int64_t base = row * k;
  float sgd = 0.f;
#pragma unroll 8
  for (int j = 0; j < k; ++j) sgd += gate[base + j] * dgslot[base + j];
  float acc[8], accr[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = accr[i] = 0.f;
  float* ar = SPLIT ? accr : acc;
  // The slots are taken in j order, U at a time: their loads are issued
  // together so that U rows are in flight, then summed one j after another.
  // The per-slot input gradients are read once: non-temporal loads.
  auto add = [&](int j, float gj, float dg, const f32x4& w0, const f32x4& w1, const u32x4& xs) {
    const float ds = gj * (dg - sgd);
    if (part == 0) dS[base + j] = ds;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ar[i] += ds * w0[i];
      ar[4 + i] += ds * w1[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += bf16_bits_to_f32(xs[i] & 0xFFFFu);
      acc[2 * i + 1] += bf16_bits_to_f32(xs[i] >> 16);
    }
  };
  auto wrow = [&](int j) {
    int e = idx[base + j];
    e = (unsigned)e < (unsigned)Ne ? e : 0;
    return W_router + ((int64_t)h * Ne + e) * DH + part * 8;
  };
  int j = 0;
  for (; j + U <= k; j += U) {
    float gj[U], dg[U];
    f32x4 w0[U], w1[U];
    u32x4 xs[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      gj[u] = gate[base + j + u];
      dg[u] = dgslot[base + j + u];
      const float* wr = wrow(j + u);
      w0[u] = *reinterpret_cast<const f32x4*>(wr);
      w1[u] = *reinterpret_cast<const f32x4*>(wr + 4);
      xs[u] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4*>(dxslot + (base + j + u) * DH + part * 8));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) add(j + u, gj[u], dg[u], w0[u], w1[u], xs[u]);
  }
  for (; j < k; ++j) {
    const float* wr = wrow(j);
    add(j, gate[base + j], dgslot[base + j], *reinterpret_cast<const f32x4*>(wr),
        *reinterpret_cast<const f32x4*>(wr + 4),
        __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(dxslot + (base + j) * DH + part * 8)));
  }
  *reinterpret_cast<u32x4*>(dX + row * DH + part * 8) =
      u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
            pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
  if (SPLIT)
    *reinterpret_cast<u32x4*>(dR + row * DH + part * 8) =
        u32x4{pack_bf16x2(accr[0], accr[1]), pack_bf16x2(accr[2], accr[3]),
              pack_bf16x2(accr[4], accr[5]), pack_bf16x2(accr[6], accr[7])};
}

// ---------------------------------------------------------------------------
// Processing order of the (head, expert) pairs for the weight gradients:
// a stable counting sort by floor(log2(slots + 1)), largest first.  One
// workgroup; thread t takes the contiguous pairs [t n / 256, (t + 1) n / 256).
// ---------------------------------------------------------------------------
constexpr int kOrderThreads = 256;
constexpr int kOrderBuckets = 32;

__device__ __forceinline__ int order_bucket(int c) {
  return kOrderBuckets - 1 - (31 - __clz(c + 1));  // 0 for the largest counts
}

__global__ __launch_bounds__(kOrderThreads) void dw_order_kernel(const int32_t* __restrict__ offsets,
                                                                 int Nh, int Ne,
                                                                 int32_t* __restrict__ order) {
  __shared__ int cnt[kOrderBuckets][kOrderThreads];
  const int t = threadIdx.x;
  const int64_t n = (int64_t)Nh * Ne;
  const int64_t i0 = n * t / kOrderThreads, i1 = n * (t + 1) / kOrderThreads;
  auto count_of = [&](int64_t i) {
    const int64_t h = i / Ne, e = i - h * Ne;
    const int32_t* o = offsets + h * (Ne + 1) + e;
    return o[1] - o[0];
  };
  for (int b = 0; b < kOrderBuckets; ++b) cnt[b][t] = 0;
  for (int64_t i = i0; i < i1; ++i) ++cnt[order_bucket(count_of(i))][t];
  __syncthreads();
  if (t < kWave) {
    // exclusive prefix over (bucket, thread) in bucket-major order
    int run = 0;
    for (int b = 0; b < kOrderBuckets; ++b) {
      for (int q = 0; q < kOrderThreads; q += kWave) {
        const int v = cnt[b][q + t];
        const int inc = wave_inclusive_scan(v);
        cnt[b][q + t] = run + inc - v;
        run += __shfl(inc, kWave - 1, kWave);
      }
    }
  }
  __syncthreads();
  int pos[kOrderBuckets];
  for (int b = 0; b < kOrderBuckets; ++b) pos[b] = cnt[b][t];
  for (int64_t i = i0; i < i1; ++i) order[pos[order_bucket(count_of(i))]++] = (int32_t)i;
}

// ---------------------------------------------------------------------------
// Weight gradients of one (head, expert, d_ff chunk).
// ---------------------------------------------------------------------------
template <int DH>
struct DwSmem {
  static constexpr int W_BYTES = 3 * BwdLayout<DH>::NAT;  // W1_c | W3_c | W2_c^T
  static constexpr int ROWB = DH * 2 + 16;                // padded tile row (bytes)
  static constexpr int TILE = 32 * ROWB;                  // one 32-slot tile
  static constexpr int WAVE = 2 * TILE + 32 * 4;          // x, dy tiles + g
  static constexpr int RED = 3 * 32 * DH * 4;             // one wave's dW partial (fp32)
  // the tiles, or (after the slot loop) three waves' partials side by side
  static constexpr int TOTAL = W_BYTES + 4 * WAVE > 3 * RED ? W_BYTES + 4 * WAVE : 3 * RED;
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

// GELU: the two-matrix expert (W1 = W_in, W2 = W_out): dW_in += da x^T with
// da = g v gelu'(a), dW_out += dy (g gelu(a))^T; no dW3.
template <int DH, bool GELU>
__global__ __launch_bounds__(kBwdThreads) void bwd_dw_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ dY,
    const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ order, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W3,
    const uint16_t* __restrict__ W2, int64_t T, int Nh, int Ne, int k, int dff,
    float* __restrict__ dW1, float* __restrict__ dW3, float* __restrict__ dW2) {
  using L = BwdLayout<DH>;
  using S = DwSmem<DH>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[S::TOTAL];
  constexpr int NB = DH / 32;

  // workgroup (pair p of the order, chunk ch).  Workgroup i runs on XCD
  // i % 8; the nch chunks of one pair take consecutive places of one XCD's
  // sequence, so they run together and that XCD's L2 serves the slot rows
  // they all gather.  Places past the last pair (the grid rounds the pair
  // count up to a multiple of 8) have nothing to do.
  const int nch = dff / kChunk;
  const int xcd = (int)(blockIdx.x % kXcds), seq = (int)(blockIdx.x / kXcds);
  const int p = (seq / nch) * kXcds + xcd;
  if (p >= Nh * Ne) return;
  const int32_t pair = order[p];
  const int ch = seq % nch, h = pair / Ne, e = pair - h * Ne;
  const int f0 = ch * kChunk;
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int row0 = offsets[(int64_t)h * (Ne + 1) + e];
  const int row1 = offsets[(int64_t)h * (Ne + 1) + e + 1];
  const int64_t eoff = ((int64_t)h * Ne + e) * dff * DH;

  {
    BwdChunkLoader<DH, true, GELU> ld;
    ld.load(W1 + eoff, W3 + eoff, W2 + eoff, f0, dff, threadIdx.x);
    ld.store(smem, threadIdx.x);
  }
  uint8_t* wtile = smem + S::W_BYTES + wave * S::WAVE;
  uint8_t* xt = wtile;
  uint8_t* dyt = wtile + S::TILE;
  float* gsh = reinterpret_cast<float*>(wtile + 2 * S::TILE);
  __syncthreads();

  f32x16 acc1[NB], acc3[NB], acc2[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc1[nb] = acc3[nb] = acc2[nb] = zero16();

  const uint8_t* w1r = smem + c * L::NJ1 * 16;  // row f = c of W1_c
  const int64_t head_slots = T * k;
  const int32_t* perm_h = perm + (int64_t)h * head_slots;

  // The rows of the 32 slots at r0 (lane c: slot r0 + c): x and dy
  // fragments and gate.
  struct Rows {
    RowFrag<DH, false> xf, df;
    float gs;
  };
  auto fetch = [&](int r0, Rows& q) {
    const int r = r0 + c;
    const bool ok = r < row1;
    const int slot = ok ? perm_h[r] : 0;
    const int64_t t = slot / k;
    const int j = slot - (int)t * k;
    const int64_t th = t * Nh + h;
    q.xf.load(X, th, ok, g);
    q.df.load(dY, th, ok, g);
    q.gs = ok ? gate[th * k + j] : 0.f;
  };

  // One group of 32 slots: its rows (in q) go to the wavefront's LDS tiles,
  // then q takes the rows of the group at r_next (loads in flight while this
  // group is computed); the MFMAs read the rows from the tiles.
  auto body = [&](Rows& q, int r_next) {
    // tiles in LDS, [slot][DH] with a padded row stride
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      *reinterpret_cast<u32x4*>(xt + c * S::ROWB + (16 * s + 8 * g) * 2) = q.xf.x[s];
      *reinterpret_cast<u32x4*>(dyt + c * S::ROWB + (16 * s + 8 * g) * 2) = q.df.x[s];
    }
    if (g == 0) gsh[c] = q.gs;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (r_next < row1) fetch(r_next, q);

    // a, b, v with slots as rows: lane = d_ff index c of the chunk,
    // element e = slot 8(e/4) + 4g + e%4 of the tile.
    f32x16 a, b, v;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      const int o = swz_tr<L::NJ1>(2 * s + g, c) * 16;
      const bf16x8 f1 = as_bf16x8(*reinterpret_cast<const u32x4*>(w1r + o));
      const bf16x8 f3 = as_bf16x8(*reinterpret_cast<const u32x4*>(w1r + L::NAT + o));
      const bf16x8 f2 = as_bf16x8(*reinterpret_cast<const u32x4*>(w1r + 2 * L::NAT + o));
      const bf16x8 xs =
          as_bf16x8(*reinterpret_cast<const u32x4*>(xt + c * S::ROWB + (16 * s + 8 * g) * 2));
      const bf16x8 ys =
          as_bf16x8(*reinterpret_cast<const u32x4*>(dyt + c * S::ROWB + (16 * s + 8 * g) * 2));
      a = mfma32_bf16(xs, f1, s == 0 ? zero16() : a);
      if (!GELU) b = mfma32_bf16(xs, f3, s == 0 ? zero16() : b);
      v = mfma32_bf16(ys, f2, s == 0 ? zero16() : v);
    }
    float gsl[16];
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      const f32x4 g4 = *reinterpret_cast<const f32x4*>(gsh + 8 * qd + 4 * g);
#pragma unroll
      for (int i = 0; i < 4; ++i) gsl[4 * qd + i] = g4[i];
    }
    u32x4 pda[2], pdb[2], pgu[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float da2[2], db2[2], gu2[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int el = 8 * hh + 2 * i + q;
          if (GELU) {
            float h, dh;
            gelu_and_grad(a[el], h, dh);
            da2[q] = gsl[el] * v[el] * dh;
            db2[q] = 0.f;
            gu2[q] = gsl[el] * h;
          } else {
            const float sg = sigmoid_fast(a[el]);
            const float sl = a[el] * sg;
            const float du = gsl[el] * v[el];
            da2[q] = du * b[el] * (sg + sl * (1.0f - sg));
            db2[q] = du * sl;
            gu2[q] = gsl[el] * sl * b[el];
          }
        }
        pda[hh][i] = pack_bf16x2(da2[0], da2[1]);
        pdb[hh][i] = pack_bf16x2(db2[0], db2[1]);
        pgu[hh][i] = pack_bf16x2(gu2[0], gu2[1]);
      }
    // Contractions over the tile's slots.  K-step hh covers slots
    // 16 hh + 8 (p/4) + 4 g + p%4 for operand element p (as a, b, v above).
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        // x and dy columns n = 32 nb + c at those slots, from the row-major
        // tiles by transposing reads: lane j of each 16-lane group points at
        // slot row r0 + j / 4, columns n0 + 4 (j % 4) .. + 3, and lane i of the
        // group receives column n0 + i at rows r0 .. r0 + 3 (group 2 g + q:
        // n0 = 32 nb + 16 q; rows 16 hh + 4 g and 16 hh + 8 + 4 g for
        // elements 0-3 and 4-7).
        const int grp = lane >> 4, jj = lane & 15;
        const int trow = 16 * hh + 4 * (grp >> 1) + (jj >> 2);
        const int tcol = (32 * nb + 16 * (grp & 1) + 4 * (jj & 3)) * 2;
        const u32x2 x0 = lds_read_tr16(xt + trow * S::ROWB + tcol);
        const u32x2 x1 = lds_read_tr16(xt + (trow + 8) * S::ROWB + tcol);
        const u32x2 y0 = lds_read_tr16(dyt + trow * S::ROWB + tcol);
        const u32x2 y1 = lds_read_tr16(dyt + (trow + 8) * S::ROWB + tcol);
        const bf16x8 xb = as_bf16x8(u32x4{x0[0], x0[1], x1[0], x1[1]});
        const bf16x8 yb = as_bf16x8(u32x4{y0[0], y0[1], y1[0], y1[1]});
        // dW1_c[f][n] += sum_s da[s][f] x[s][n]   (rows f = lane, cols n)
        acc1[nb] = mfma32_bf16(as_bf16x8(pda[hh]), xb, acc1[nb]);
        if (!GELU) acc3[nb] = mfma32_bf16(as_bf16x8(pdb[hh]), xb, acc3[nb]);
        // dW2_c[n][f] += sum_s dy[s][n] (g u)[s][f]  (rows n, cols f = lane)
        acc2[nb] = mfma32_bf16(yb, as_bf16x8(pgu[hh]), acc2[nb]);
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // Each wavefront takes every fourth group of 32 slots; the next group's
  // rows are fetched while the current group is processed.
  {
    Rows q;
    int r0 = row0 + wave * 32;
    if (r0 < row1) fetch(r0, q);
    for (; r0 < row1; r0 += 4 * 32) body(q, r0 + 4 * 32);
  }

  // Fixed-order sum of the four wavefronts' partial gradients (wavefront 0's
  // plus 1's, then 2's, then 3's); wavefronts that received no group of
  // slots hold zeros and are left out (nact is the same for the whole
  // workgroup).  Waves 1-3 write their partials to separate LDS regions at
  // once, so one barrier serves the whole sum.
  __syncthreads();  // every wave is done with the weight and tile areas
  const int nact = row1 - row0 >= 4 * 32 ? 4 : (row1 - row0 + 31) / 32;
  if (wave >= 1 && wave < nact) {
    float* red = reinterpret_cast<float*>(smem + (wave - 1) * S::RED);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        red[((0 * NB + nb) * 16 + v) * kWave + lane] = acc1[nb][v];
        if (!GELU) red[((1 * NB + nb) * 16 + v) * kWave + lane] = acc3[nb][v];
        red[((2 * NB + nb) * 16 + v) * kWave + lane] = acc2[nb][v];
      }
  }
  __syncthreads();
  if (wave != 0) return;
  for (int w = 1; w < nact; ++w) {
    const float* red = reinterpret_cast<const float*>(smem + (w - 1) * S::RED);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        acc1[nb][v] += red[((0 * NB + nb) * 16 + v) * kWave + lane];
        if (!GELU) acc3[nb][v] += red[((1 * NB + nb) * 16 + v) * kWave + lane];
        acc2[nb][v] += red[((2 * NB + nb) * 16 + v) * kWave + lane];
      }
  }
  // acc1/acc3: row f = 8(v/4) + 4g + v%4 of the chunk, column n = 32 nb + c.
  // acc2: row n = 32 nb + 8(v/4) + 4g + v%4, column f = c.
  float* d1 = dW1 + eoff + (int64_t)f0 * DH;
  float* d3 = GELU ? nullptr : dW3 + eoff + (int64_t)f0 * DH;
  float* d2 = dW2 + eoff + f0;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int rr = 8 * (v >> 2) + 4 * g + (v & 3);
      d1[(int64_t)rr * DH + 32 * nb + c] = acc1[nb][v];
      if (!GELU) d3[(int64_t)rr * DH + 32 * nb + c] = acc3[nb][v];
      d2[(int64_t)(32 * nb + rr) * dff + c] = acc2[nb][v];
    }
}

// ---------------------------------------------------------------------------
// Weight gradients of one (head, expert, d_ff chunk) at d_h 128, split over
// d_h: wavefront w owns columns 32 w .. 32 w + 31 of dW1_c and dW3_c and the
// same rows of dW2_c, so no wavefront holds a partial of another's output
// and nothing is summed across wavefronts.  The expert's slots are taken 64
// at a time (two groups of 32):
//   A. wavefront w computes a, b, v = W1 x, W3 x, W2^T dy for group w / 2
//      and chunk rows 16 (w % 2) .. + 15 with 16x16x32 MFMAs (d_ff rows as
//      M, slots as N, d_h as K), then the SwiGLU backward of those
//      elements, and stores da, db and g u as [slot][d_ff row] bf16 in LDS
//      (each lane's four d_ff rows of one slot as one 8-byte piece);
//   B. every wavefront contracts its d_h block over the 64 slots: dW1_c +=
//      da^T x, dW3_c += db^T x, dW2_c += dy^T (g u) (32x32x16 MFMAs, every
//      operand a slot-contiguous column, read by ds_read_b64_tr_b16).
// With an even number of chunks a workgroup takes two (CPW = 2: 8
// wavefronts, 136 KiB of LDS, one workgroup per CU), so the gathered rows
// serve twice the work, and the next 64 slots' rows go by LDS DMA into the
// other of two row buffers during A and B; otherwise one chunk (68 KiB, two
// workgroups per CU) and the next rows are loaded into registers during A
// and B and stored to the single row buffer after B.  The slot numbers come
// from perm one iteration earlier still.  Either way two wavefronts per
// SIMD, at most 256 registers each.
// ---------------------------------------------------------------------------
constexpr int kDw2DRow = kChunk * 2;  // bytes of a [slot][f] row: 8 pieces of 8 bytes
template <int CPW>  // d_ff chunks per workgroup (4 wavefronts each)
struct Dw2Smem {
  static constexpr int DH = 128;
  static constexpr int SI = 64;                          // slots per iteration
  static constexpr int WCH = 3 * BwdLayout<DH>::NAT;     // one chunk: W1_c | W3_c | W2_c^T
  static constexpr int TROW = DH * 2;                    // tile row: 16 units, swz_tr
  static constexpr int TILE = SI * TROW;
  static constexpr int DMAT = SI * kDw2DRow;
  // Row tiles (X then dY) and gates: double buffered where the rows come by
  // LDS DMA (CPW = 2), single where they go through registers (CPW = 1).
  static constexpr int NBUF = CPW == 2 ? 2 : 1;
  static constexpr int RBUF = 2 * TILE;                  // one buffer: X | dY
  static constexpr int X_OFF = CPW * WCH;
  static constexpr int DY_OFF = X_OFF + TILE;
  static constexpr int D_OFF = X_OFF + NBUF * RBUF;      // per chunk: da | db | g u
  static constexpr int G_OFF = D_OFF + CPW * 3 * DMAT;   // gates of the 64 slots, per buffer
  static constexpr int TOTAL = G_OFF + NBUF * SI * 4;
  static_assert(CPW == 1 ? TOTAL <= 80 * 1024 : TOTAL <= 160 * 1024,
                "two workgroups per CU with one chunk, one with two");
};

// Byte of (slot s, d_ff row f) in a [slot][f] matrix: 8-byte pieces (four
// f) XOR-ed with bits 1-3 of s.  LDS writes go 128 bytes per cycle, so 16
// consecutive slots writing one piece with ds_write_b64 must hit 16 distinct
// 8-byte positions of a 128-byte bank row (two slots per row, eight pieces);
// the transposed reads (four consecutive slots, 32 bytes of f each, and the
// other 16-lane group the other 32 bytes) cover every bank of the four rows
// once, whatever the XOR.
__device__ __forceinline__ int dslot_byte(int s, int f) {
  return s * kDw2DRow + (((f >> 2) ^ ((s >> 1) & 7)) << 3) + (f & 3) * 2;
}

__device__ __forceinline__ f32x4 mfma16_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <bool GELU, int CPW>
__global__ __launch_bounds__(kBwdThreads * CPW, CPW == 1 ? 2 : 1) void bwd_dw2_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ dY,
    const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ order, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W3,
    const uint16_t* __restrict__ W2, int64_t T, int Nh, int Ne, int k, int dff,
    float* __restrict__ dW1, float* __restrict__ dW3, float* __restrict__ dW2) {
  constexpr int DH = 128;
  using L = BwdLayout<DH>;
  using S = Dw2Smem<CPW>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[S::TOTAL];

  // workgroup (pair p of the order, chunks CPW cg .. CPW cg + CPW - 1),
  // placed as in bwd_dw_kernel; wavefront w works on chunk CPW cg + w / 4
  const int ngrp = dff / kChunk / CPW;
  const int xcd = (int)(blockIdx.x % kXcds), seq = (int)(blockIdx.x / kXcds);
  const int pidx = (seq / ngrp) * kXcds + xcd;
  if (pidx >= Nh * Ne) return;
  const int32_t pair = order[pidx];
  const int h = pair / Ne, e = pair - h * Ne;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int cq = wave >> 2, wl = wave & 3;  // the wavefront's chunk of the group, its place there
  const int ch = (seq % ngrp) * CPW + cq;
  const int f0 = ch * kChunk;
  uint8_t* const wst = smem + cq * S::WCH;             // the chunk's weights
  const int doff = S::D_OFF + cq * 3 * S::DMAT;        // its da | db | g u
  const int row0 = offsets[(int64_t)h * (Ne + 1) + e];
  const int row1 = offsets[(int64_t)h * (Ne + 1) + e + 1];
  const int64_t eoff = ((int64_t)h * Ne + e) * dff * DH;
  const int32_t* perm_h = perm + (int64_t)h * T * k;
  float* gsh = reinterpret_cast<float*>(smem + S::G_OFF);

  // Row loading: lane l of wavefront w takes tile rows r = RPW w + 4 i +
  // l / 16 (i < NI), physical 16-byte unit l % 16 (its logical unit is the
  // XOR of that with the row's swz_tr mask).  A row past the expert's last
  // slot loads nothing (the expert may have no slot, the batch no token)
  // and holds zeros with gate 0, so its terms vanish.
  constexpr int RPW = S::SI / (4 * CPW), NI = RPW / 4;
  constexpr bool DMA = CPW == 2;  // rows by LDS DMA into two buffers
  const int pu = lane & 15, rq = lane >> 4;
  const DivMagic kmag = div_magic(k);  // slot / k without a division
  u32x4 px[DMA ? 1 : NI], pd[DMA ? 1 : NI];
  float pg[NI];
  int sn[NI];
  // A row past the expert's last slot: -1, or (DMA) -1 - the slot of the
  // expert's last row, whose row the DMA then re-reads (finite values; the
  // gate 0 makes its terms vanish).  Only called when the expert has a slot.
  auto slots_at = [&](int base, int* out) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = base + RPW * wave + 4 * i + rq;
      out[i] = r < row1 ? perm_h[r] : DMA ? -1 - perm_h[row1 - 1] : -1;
    }
  };
  // DMA form: rows of instruction i of wavefront w are tile rows RPW w + 4 i
  // + [0, 4), 1 KiB of LDS at a uniform base, lane l's 16 bytes at 16 l
  // (row l / 16, physical unit l % 16): the layout the register path stores.
  auto fetch_dma = [&](const int* sl4, int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = RPW * wave + 4 * i + rq;
      const bool ok = sl4[i] >= 0;
      const int sl = ok ? sl4[i] : -1 - sl4[i];
      const int64_t t = div_by_magic(sl, kmag);
      const int j = sl - (int)t * k;
      const int64_t th = t * Nh + h;
      const int u = swz_tr<L::NJ1>(pu, r);
      uint8_t* dst = smem + S::X_OFF + buf * S::RBUF + (RPW * wave + 4 * i) * S::TROW;
      __builtin_amdgcn_global_load_lds(X + th * DH + 8 * u,
                                        (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(dY + th * DH + 8 * u,
                                        (__attribute__((address_space(3))) void*)(dst + S::TILE),
                                        16, 0, 0);
      pg[i] = ok ? gate[th * k + j] : 0.f;
    }
  };
  auto stash_gates = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (pu == 0) gsh[buf * S::SI + RPW * wave + 4 * i + rq] = pg[i];
  };
  auto fetch = [&](const int* sl4) {
    if constexpr (!DMA)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = RPW * wave + 4 * i + rq;
      const bool ok = sl4[i] >= 0;
      const int sl = ok ? sl4[i] : 0;
      const int64_t t = div_by_magic(sl, kmag);
      const int j = sl - (int)t * k;
      const int64_t th = t * Nh + h;
      const int u = swz_tr<L::NJ1>(pu, r);
      const u32x4 zero = {0u, 0u, 0u, 0u};
      px[i] = ok ? *reinterpret_cast<const u32x4*>(X + th * DH + 8 * u) : zero;
      pd[i] = ok ? *reinterpret_cast<const u32x4*>(dY + th * DH + 8 * u) : zero;
      pg[i] = ok ? gate[th * k + j] : 0.f;
    }
  };
  auto stash = [&]() {
    if constexpr (!DMA)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = RPW * wave + 4 * i + rq;
      *reinterpret_cast<u32x4*>(smem + S::X_OFF + r * S::TROW + pu * 16) = px[i];
      *reinterpret_cast<u32x4*>(smem + S::DY_OFF + r * S::TROW + pu * 16) = pd[i];
      if (pu == 0) gsh[r] = pg[i];
    }
  };

  if constexpr (DMA) {
    // (no row is fetched for an expert without a slot: the batch may be
    // empty)
    if (row0 < row1) {
      int sc[NI];
      slots_at(row0, sc);
      fetch_dma(sc, 0);
      slots_at(row0 + S::SI, sn);
    }
    BwdChunkLoader<DH, true, GELU> ld;  // each chunk by its 4 wavefronts
    ld.load(W1 + eoff, W3 + eoff, W2 + eoff, f0, dff, tid & (kBwdThreads - 1));
    ld.store(wst, tid & (kBwdThreads - 1));
    if (row0 < row1) stash_gates(0);
    barrier_vm<0>();  // the rows landed; weights and gates stored
  } else {
    int sc[NI];
    slots_at(row0, sc);
    fetch(sc);
    slots_at(row0 + S::SI, sn);
    BwdChunkLoader<DH, true, GELU> ld;  // each chunk by its 4 wavefronts
    ld.load(W1 + eoff, W3 + eoff, W2 + eoff, f0, dff, tid & (kBwdThreads - 1));
    ld.store(wst, tid & (kBwdThreads - 1));
    stash();
    __syncthreads();
  }
  int cb = 0;  // the row buffer of the current 64 slots (DMA form)

  f32x16 acc1 = zero16(), acc3 = zero16(), acc2 = zero16();
  const int gq = wl >> 1, fh = wl & 1;  // phase A: slot group, half of the chunk rows
  const int nb = wl;                    // phase B: d_h block

  for (int base = row0; base < row1; base += S::SI) {
    const bool more = base + S::SI < row1;
    // the other buffer was last read in the previous iteration, before its
    // closing barrier
    if (more) {
      if constexpr (DMA) fetch_dma(sn, cb ^ 1);
      else fetch(sn);
      slots_at(base + 2 * S::SI, sn);
    }
    uint8_t* const xt = smem + S::X_OFF + (DMA ? cb * S::RBUF : 0);  // this iteration's rows
    const float* const gt = gsh + (DMA ? cb * S::SI : 0);

    // A. a, b, v for chunk rows 16 fh + [0, 16) (M) and slots 32 gq + 16 t +
    // [0, 16) (N), K = d_h in steps of 32: lane l holds chunk rows 16 fh +
    // 4 (l / 16) + [0, 4) of slot 32 gq + 16 t + l % 16.
    f32x4 a[2], b[2], v[2];
    {
      const int fr = 16 * fh + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks) {
        const int u = 4 * ks + (lane >> 4);
        const int ow = fr * L::NJ1 * 16 + swz_tr<L::NJ1>(u, fr) * 16;
        const bf16x8 w1f = as_bf16x8(*reinterpret_cast<const u32x4*>(wst + ow));
        const bf16x8 w3f =
            GELU ? w1f : as_bf16x8(*reinterpret_cast<const u32x4*>(wst + L::NAT + ow));
        const bf16x8 w2f = as_bf16x8(*reinterpret_cast<const u32x4*>(wst + 2 * L::NAT + ow));
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int sr = 32 * gq + 16 * t + (lane & 15);
          const int ot = sr * S::TROW + swz_tr<L::NJ1>(u, sr) * 16;
          const bf16x8 xs = as_bf16x8(*reinterpret_cast<const u32x4*>(xt + ot));
          const bf16x8 ys = as_bf16x8(*reinterpret_cast<const u32x4*>(xt + S::TILE + ot));
          const f32x4 z = {0.f, 0.f, 0.f, 0.f};
          a[t] = mfma16_bf16(w1f, xs, ks == 0 ? z : a[t]);
          if (!GELU) b[t] = mfma16_bf16(w3f, xs, ks == 0 ? z : b[t]);
          v[t] = mfma16_bf16(w2f, ys, ks == 0 ? z : v[t]);
        }
      }
      // Issue order: the fragment reads of K steps 0 and 1, then each
      // step's MFMAs followed by the reads of the step after next, so a
      // step's reads land while the previous step's MFMAs run (left alone,
      // the compiler waits for each step's reads with the MFMA pipe idle).
      {
        constexpr int NR = GELU ? 6 : 7, NM = GELU ? 4 : 6, NK = DH / 32;
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * NR, 0);
#pragma unroll
        for (int ks = 0; ks < NK; ++ks) {
          __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
          if (ks + 2 < NK) __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
        }
      }
      // SwiGLU (GELU) backward of the 8 elements, stored as [slot][f]
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int sl = 32 * gq + 16 * t + (lane & 15);
        const float gs = gt[sl];
        float da[4], db[4], gu[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (GELU) {
            float hv, dh;
            gelu_and_grad(a[t][i], hv, dh);
            da[i] = gs * v[t][i] * dh;
            db[i] = 0.f;
            gu[i] = gs * hv;
          } else {
            const float sg = sigmoid_fast(a[t][i]);
            const float si = a[t][i] * sg;
            const float du = gs * v[t][i];
            da[i] = du * b[t][i] * (sg + si * (1.0f - sg));
            db[i] = du * si;
            gu[i] = gs * si * b[t][i];
          }
        }
        const int od = doff + dslot_byte(sl, 16 * fh + 4 * (lane >> 4));
        *reinterpret_cast<u32x2*>(smem + od) = u32x2{pack_bf16x2(da[0], da[1]), pack_bf16x2(da[2], da[3])};
        if (!GELU)
          *reinterpret_cast<u32x2*>(smem + od + S::DMAT) =
              u32x2{pack_bf16x2(db[0], db[1]), pack_bf16x2(db[2], db[3])};
        *reinterpret_cast<u32x2*>(smem + od + 2 * S::DMAT) =
            u32x2{pack_bf16x2(gu[0], gu[1]), pack_bf16x2(gu[2], gu[3])};
      }
    }
    barrier_lds();

    // B. contraction over the 64 slots in K steps of 16 (slots sb + 8 (l /
    // 32) + [0, 8) per lane): dW1_c / dW3_c rows f = lane % 32 (A: da^T,
    // db^T) times x columns 32 nb + lane % 32 (B); dW2_c rows 32 nb + lane %
    // 32 (A: dy^T) times g u columns f (B).  Every operand runs down a
    // column of a [slot][...] matrix: ds_read_b64_tr_b16 of slots r0..r0+3
    // and r0+4..r0+7.
    {
      const int grp = lane >> 4, jj = lane & 15;
      const int tcol = (32 * nb + 16 * (grp & 1) + 4 * (jj & 3)) * 2;
      const int fcol = 16 * (grp & 1) + 4 * (jj & 3);
#pragma unroll
      for (int sb = 0; sb < S::SI; sb += 16) {
        const int r0 = sb + 8 * (grp >> 1) + (jj >> 2);
        const int d0 = doff + dslot_byte(r0, fcol), d1 = doff + dslot_byte(r0 + 4, fcol);
        const auto dfrag = [&](int m) {
          const u32x2 lo = lds_read_tr16(smem + d0 + m * S::DMAT);
          const u32x2 hi = lds_read_tr16(smem + d1 + m * S::DMAT);
          return as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
        };
        const bf16x8 pda = dfrag(0);
        const bf16x8 pgu = dfrag(2);
        const int t0 = r0 * S::TROW + swz_tr<L::NJ1>(tcol >> 4, r0) * 16 + (tcol & 15);
        const int t1 = (r0 + 4) * S::TROW + swz_tr<L::NJ1>(tcol >> 4, r0 + 4) * 16 + (tcol & 15);
        const u32x2 x0 = lds_read_tr16(xt + t0);
        const u32x2 x1 = lds_read_tr16(xt + t1);
        const u32x2 y0 = lds_read_tr16(xt + S::TILE + t0);
        const u32x2 y1 = lds_read_tr16(xt + S::TILE + t1);
        const bf16x8 xb = as_bf16x8(u32x4{x0[0], x0[1], x1[0], x1[1]});
        const bf16x8 yb = as_bf16x8(u32x4{y0[0], y0[1], y1[0], y1[1]});
        acc1 = mfma32_bf16(pda, xb, acc1);
        if (!GELU) {
          const bf16x8 pdb = dfrag(1);
          acc3 = mfma32_bf16(pdb, xb, acc3);
        }
        acc2 = mfma32_bf16(yb, pgu, acc2);
      }
      // as in phase A: reads two K steps ahead of the MFMAs
      constexpr int NR = GELU ? 8 : 10, NM = GELU ? 2 : 3;
      __builtin_amdgcn_sched_group_barrier(0x100, 2 * NR, 0);
#pragma unroll
      for (int sb = 0; sb < S::SI; sb += 16) {
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
        if (sb + 32 < S::SI) __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
      }
    }
    if constexpr (DMA) {
      if (more) stash_gates(cb ^ 1);
      // the next rows landed, every wavefront is done with this iteration's
      // tiles and da / db / g u
      barrier_vm<0>();
      cb ^= 1;
    } else {
      __syncthreads();  // every wavefront is done with the tiles and da / db / g u
      if (more) stash();
      __syncthreads();
    }
  }

  // acc1/acc3: row f = 8(v/4) + 4(l/32) + v%4 of the chunk, column n = 32 nb
  // + l%32; acc2: row n = 32 nb + 8(v/4) + 4(l/32) + v%4, column f = l%32.
  const int c = lane & 31, g = lane >> 5;
  float* d1 = dW1 + eoff + (int64_t)f0 * DH;
  float* d3 = GELU ? nullptr : dW3 + eoff + (int64_t)f0 * DH;
  float* d2 = dW2 + eoff + f0;
#pragma unroll
  for (int vv = 0; vv < 16; ++vv) {
    const int rr = 8 * (vv >> 2) + 4 * g + (vv & 3);
    d1[(int64_t)rr * DH + 32 * nb + c] = acc1[vv];
    if (!GELU) d3[(int64_t)rr * DH + 32 * nb + c] = acc3[vv];
    d2[(int64_t)(32 * nb + rr) * dff + c] = acc2[vv];
  }
}

// ---------------------------------------------------------------------------
// dW_router[h, e] = sum over the slots of e of dS_slot r[t, h] (Algorithm 2's
// weight gradient; r is the router's input: x itself, or the separate
// routing sub-tokens of Sec. 4.4).  Each (head, expert) pair's slot rows are
// cut into segments of at most kRdwSeg rows (at least one per pair, so an
// expert without slots gets its zeros), one workgroup per segment, so a hot
// expert's rows spread over many workgroups:
//   rdw_plan_kernel: seg_base[p] = segments of the pairs before p (one
//     workgroup; thread t scans a contiguous range of pairs);
//   router_dw_seg_kernel: a segment's sum (thread (q, part) takes rows q,
//     q + Q, ... over 8 columns, U rows in flight, then the Q partials in q
//     order); a one-segment pair's row goes straight to dW_router, a longer
//     pair's partial to part[segment];
//   router_dw_fix_kernel: a longer pair's partials added in segment order.
// Every sum has a fixed order, so the result is deterministic.
// ---------------------------------------------------------------------------
__device__ inline int rdw_segments(const int32_t* offsets, int Ne, int p) {
  const int h = p / Ne, e = p - h * Ne;
  const int c = offsets[(int64_t)h * (Ne + 1) + e + 1] - offsets[(int64_t)h * (Ne + 1) + e];
  return c > kRdwSeg ? (c + kRdwSeg - 1) / kRdwSeg : 1;
}

__global__ __launch_bounds__(256) void rdw_plan_kernel(const int32_t* __restrict__ offsets,
                                                       int Nh, int Ne,
                                                       int32_t* __restrict__ seg_base) {
  __shared__ int32_t sums[256];
  const int P = Nh * Ne, t = threadIdx.x;
  const int lo = (int)((int64_t)P * t / 256), hi = (int)((int64_t)P * (t + 1) / 256);
  int local = 0;
  for (int p = lo; p < hi; ++p) local += rdw_segments(offsets, Ne, p);
  sums[t] = local;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {  // inclusive scan of the 256 partial sums
    const int v = t >= off ? sums[t - off] : 0;
    __syncthreads();
    sums[t] += v;
    __syncthreads();
  }
  int run = t == 0 ? 0 : sums[t - 1];
  for (int p = lo; p < hi; ++p) {
    seg_base[p] = run;
    run += rdw_segments(offsets, Ne, p);
  }
  if (t == 255) seg_base[P] = sums[255];
}

template <int DH, bool XF32>
__global__ __launch_bounds__(256) void router_dw_seg_kernel(
    const void* __restrict__ Rv, const float* __restrict__ dS,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ seg_base, int64_t T, int Nh, int Ne, int k,
    float* __restrict__ part, float* __restrict__ dWr) {
  constexpr int TPR = DH / 8;
  constexpr int Q = 256 / TPR;
  constexpr int U = 8;
  __shared__ float red[Q][DH];
  const int P = Nh * Ne;
  const int g = blockIdx.x;
  if (g >= seg_base[P]) return;  // the grid is an upper bound on the segments
  int lo = 0, hi = P;             // the pair: largest p with seg_base[p] <= g
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (seg_base[mid] <= g) lo = mid; else hi = mid;
  }
  const int pair = lo, h = pair / Ne, e = pair - h * Ne;
  const int nseg = seg_base[pair + 1] - seg_base[pair];
  const int end = offsets[(int64_t)h * (Ne + 1) + e + 1];
  const int row0 = offsets[(int64_t)h * (Ne + 1) + e] + (g - seg_base[pair]) * kRdwSeg;
  const int row1 = row0 + kRdwSeg < end ? row0 + kRdwSeg : end;
  const int q = threadIdx.x / TPR, c8 = (threadIdx.x % TPR) * 8;
  const int32_t* perm_h = perm + (int64_t)h * T * k;
  const DivMagic kmag = div_magic(k);
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int r = row0 + q; r < row1; r += U * Q) {
    float xv[U][8];
    float ds[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ok = r + u * Q < row1;
      const int slot = ok ? perm_h[r + u * Q] : 0;
      const int64_t t = div_by_magic(slot, kmag);
      const int64_t th = t * Nh + h;
      ds[u] = ok ? dS[th * k + (slot - t * k)] : 0.f;
      if (XF32) {
        const float* R = static_cast<const float*>(Rv) + th * DH + c8;
        const f32x4 a = ok ? *reinterpret_cast<const f32x4*>(R) : f32x4{0.f, 0.f, 0.f, 0.f};
        const f32x4 b = ok ? *reinterpret_cast<const f32x4*>(R + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          xv[u][i] = a[i];
          xv[u][4 + i] = b[i];
        }
      } else {
        const uint16_t* R = static_cast<const uint16_t*>(Rv) + th * DH + c8;
        const u32x4 v = ok ? *reinterpret_cast<const u32x4*>(R) : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          xv[u][2 * i] = bf16_bits_to_f32(v[i] & 0xFFFFu);
          xv[u][2 * i + 1] = bf16_bits_to_f32(v[i] >> 16);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] += ds[u] * xv[u][i];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) red[q][c8 + i] = acc[i];
  __syncthreads();
  if (threadIdx.x < DH) {
    float sum = 0.f;
    for (int qq = 0; qq < Q; ++qq) sum += red[qq][threadIdx.x];
    if (nseg == 1)
      dWr[(int64_t)pair * DH + threadIdx.x] = sum;
    else
      part[(int64_t)g * DH + threadIdx.x] = sum;
  }
}

template <int DH>
__global__ __launch_bounds__(DH) void router_dw_fix_kernel(const int32_t* __restrict__ seg_base,
                                                           const float* __restrict__ part,
                                                           float* __restrict__ dWr) {
  const int p = blockIdx.x;
  const int g0 = seg_base[p], g1 = seg_base[p + 1];
  if (g1 - g0 == 1) return;
  float sum = 0.f;
  for (int g = g0; g < g1; ++g) sum += part[(int64_t)g * DH + threadIdx.x];
  dWr[(int64_t)p * DH + threadIdx.x] = sum;
}

// ---------------------------------------------------------------------------
// Algorithm 2 on its own, per (t, h): dS_j = g_j (dgate_j - sum g dgate) and
// dX = sum_j dS_j W_r[h, e_j] in j order (bf16 or fp32 dX).  One thread per
// 8 consecutive dX elements, U slots' router rows in flight.
// ---------------------------------------------------------------------------
template <int DH, bool F32>
__global__ __launch_bounds__(256) void route_bwd_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ gate,
    const float* __restrict__ dgate, const float* __restrict__ W_router, int64_t rows, int Nh,
    int Ne, int k, void* __restrict__ dX, float* __restrict__ dS) {
  constexpr int TPR = DH / 8;
  constexpr int U = 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / TPR;  // t * Nh + h
  const int part = (int)(gid % TPR);
  if (row >= rows) return;
  const int h = (int)(row % Nh);
  const int64_t base = row * k;
  float sgd = 0.f;
#pragma unroll 8
  for (int j = 0; j < k; ++j) sgd += gate[base + j] * dgate[base + j];
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  auto wrow = [&](int j) {
    int e = idx[base + j];
    e = (unsigned)e < (unsigned)Ne ? e : 0;
    return W_router + ((int64_t)h * Ne + e) * DH + part * 8;
  };
  auto add = [&](int j, float gj, float dg, const f32x4& w0, const f32x4& w1) {
    const float ds = gj * (dg - sgd);
    if (part == 0) dS[base + j] = ds;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[i] += ds * w0[i];
      acc[4 + i] += ds * w1[i];
    }
  };
  int j = 0;
  for (; j + U <= k; j += U) {
    float gj[U], dg[U];
    f32x4 w0[U], w1[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      gj[u] = gate[base + j + u];
      dg[u] = dgate[base + j + u];
      const float* wr = wrow(j + u);
      w0[u] = *reinterpret_cast<const f32x4*>(wr);
      w1[u] = *reinterpret_cast<const f32x4*>(wr + 4);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) add(j + u, gj[u], dg[u], w0[u], w1[u]);
  }
  for (; j < k; ++j) {
    const float* wr = wrow(j);
    add(j, gate[base + j], dgate[base + j], *reinterpret_cast<const f32x4*>(wr),
        *reinterpret_cast<const f32x4*>(wr + 4));
  }
  if (F32) {
    float* o = static_cast<float*>(dX) + row * DH + part * 8;
    *reinterpret_cast<f32x4*>(o) = f32x4{acc[0], acc[1], acc[2], acc[3]};
    *reinterpret_cast<f32x4*>(o + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
  } else {
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(dX) + row * DH + part * 8) =
        u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
              pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
  }
}

}  // namespace

hipError_t launch_route_bwd(const int32_t* idx, const float* gate, const float* dgate,
                            const float* W_router, int64_t T, int Nh, int dh, int Ne, int k,
                            bool f32, void* dX, float* dS, hipStream_t s) {
  const int64_t rows = T * Nh;
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)ceil_div(rows * (dh / 8), 256));
#define MHL_ROUTE_BWD(DH, F)                                                                   \
  hipLaunchKernelGGL((route_bwd_kernel<DH, F>), grid, dim3(256), 0, s, idx, gate, dgate,        \
                     W_router, rows, Nh, Ne, k, dX, dS)
  if (dh == 128 && !f32)
    MHL_ROUTE_BWD(128, false);
  else if (dh == 128)
    MHL_ROUTE_BWD(128, true);
  else if (dh == 64 && !f32)
    MHL_ROUTE_BWD(64, false);
  else if (dh == 64)
    MHL_ROUTE_BWD(64, true);
  else
    return hipErrorInvalidValue;
#undef MHL_ROUTE_BWD
  return hipGetLastError();
}

hipError_t launch_bwd_dx(const void* X, const void* dY, const float* gate, const int32_t* perm,
                         const TileInfo* tiles, const int32_t* head_base, const void* W1,
                         const void* W3, const void* W2, int64_t T, int Nh, int dh, int Ne, int k,
                         int dff, void* dxslot, float* dgslot, hipStream_t s) {
  // W3 == NULL: the GELU expert (its loader never reads W3; W1 stands in).
  const bool gelu = W3 == nullptr;
  const uint16_t* w3 = (const uint16_t*)(gelu ? W1 : W3);
#define MHL_BWD_DX(DH, G)                                                                      \
  hipLaunchKernelGGL((bwd_dx_kernel<DH, G>), dim3(kFfnGrid), dim3(kBwdThreads), 0, s,          \
                     (const uint16_t*)X, (const uint16_t*)dY, gate, perm, tiles, head_base,    \
                     (const uint16_t*)W1, w3, (const uint16_t*)W2, T, Nh, Ne, k, dff,          \
                     (uint16_t*)dxslot, dgslot)
  if (dh == 128 && !gelu)
    MHL_BWD_DX(128, false);
  else if (dh == 128)
    MHL_BWD_DX(128, true);
  else if (dh == 64 && !gelu)
    MHL_BWD_DX(64, false);
  else if (dh == 64)
    MHL_BWD_DX(64, true);
  else
    return hipErrorInvalidValue;
#undef MHL_BWD_DX
  return hipGetLastError();
}

hipError_t launch_bwd_combine(const int32_t* idx, const float* gate, const float* dgslot,
                              const void* dxslot, const float* W_router, int64_t T, int Nh,
                              int dh, int Ne, int k, void* dX, void* dR, float* dS,
                              hipStream_t s) {
  const int64_t rows = T * Nh;
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)ceil_div(rows * (dh / 8), 256));
#define MHL_BWD_COMBINE(DH, SPLIT)                                                         \
  do {                                                                                     \
    if (k >= 32)                                                                           \
      hipLaunchKernelGGL((bwd_combine_kernel<DH, SPLIT, 16>), grid, dim3(256), 0, s, idx,   \
                         gate, dgslot, (const uint16_t*)dxslot, W_router, rows, Nh, Ne, k,  \
                         (uint16_t*)dX, (uint16_t*)dR, dS);                                 \
    else                                                                                   \
      hipLaunchKernelGGL((bwd_combine_kernel<DH, SPLIT, 8>), grid, dim3(256), 0, s, idx,    \
                         gate, dgslot, (const uint16_t*)dxslot, W_router, rows, Nh, Ne, k,  \
                         (uint16_t*)dX, (uint16_t*)dR, dS);                                 \
  } while (0)
  if (dh == 128 && dR == nullptr)
    MHL_BWD_COMBINE(128, false);
  else if (dh == 128)
    MHL_BWD_COMBINE(128, true);
  else if (dh == 64 && dR == nullptr)
    MHL_BWD_COMBINE(64, false);
  else if (dh == 64)
    MHL_BWD_COMBINE(64, true);
  else
    return hipErrorInvalidValue;
#undef MHL_BWD_COMBINE
  return hipGetLastError();
}

hipError_t launch_router_dw(const void* R, bool f32, const float* dS, const int32_t* perm,
                            const int32_t* offsets, int64_t T, int Nh, int dh, int Ne, int k,
                            int32_t* seg_base, float* part, float* dWr, hipStream_t s) {
  const int P = Nh * Ne;
  hipLaunchKernelGGL(rdw_plan_kernel, dim3(1), dim3(256), 0, s, offsets, Nh, Ne, seg_base);
  const dim3 grid((unsigned)rdw_max_segments(T, Nh, Ne, k));
#define MHL_RDW(DH, F)                                                                         \
  do {                                                                                         \
    hipLaunchKernelGGL((router_dw_seg_kernel<DH, F>), grid, dim3(256), 0, s, R, dS, perm,       \
                       offsets, seg_base, T, Nh, Ne, k, part, dWr);                            \
    hipLaunchKernelGGL((router_dw_fix_kernel<DH>), dim3((unsigned)P), dim3(DH), 0, s, seg_base, \
                       part, dWr);                                                             \
  } while (0)
  if (dh == 128 && !f32)
    MHL_RDW(128, false);
  else if (dh == 128)
    MHL_RDW(128, true);
  else if (dh == 64 && !f32)
    MHL_RDW(64, false);
  else if (dh == 64)
    MHL_RDW(64, true);
  else
    return hipErrorInvalidValue;
#undef MHL_RDW
  return hipGetLastError();
}

hipError_t launch_bwd_dw(const void* X, const void* dY, const float* gate,
                         const int32_t* perm, const int32_t* offsets, int32_t* order,
                         const void* W1, const void* W3, const void* W2, int64_t T, int Nh,
                         int dh, int Ne, int k, int dff, float* dW1, float* dW3, float* dW2,
                         hipStream_t s) {
  hipLaunchKernelGGL(dw_order_kernel, dim3(1), dim3(kOrderThreads), 0, s, offsets, Nh, Ne, order);
  const int64_t pairs8 = ((int64_t)Nh * Ne + kXcds - 1) / kXcds * kXcds;
  const dim3 grid((unsigned)(pairs8 * (dff / kChunk)));
  // W3 == NULL: the GELU expert (W3 never read, dW3 never written).
  const bool gelu = W3 == nullptr;
  const uint16_t* w3 = (const uint16_t*)(gelu ? W1 : W3);
#define MHL_BWD_DW(DH, G)                                                                      \
  hipLaunchKernelGGL((bwd_dw_kernel<DH, G>), grid, dim3(kBwdThreads), 0, s, (const uint16_t*)X, \
                     (const uint16_t*)dY, gate, perm, offsets, order, (const uint16_t*)W1, w3,  \
                     (const uint16_t*)W2, T, Nh, Ne, k, dff, dW1, dW3, dW2)
  // At d_h 128, an even number of d_ff chunks goes two chunks per workgroup
  // (8 wavefronts share the gathered slot rows), else one.
  const int cpw = (dff / kChunk) % 2 == 0 ? 2 : 1;
  const dim3 grid2((unsigned)(pairs8 * (dff / kChunk / cpw)));
#define MHL_BWD_DW2(G, C)                                                                      \
  hipLaunchKernelGGL((bwd_dw2_kernel<G, C>), grid2, dim3(kBwdThreads * C), 0, s,              \
                     (const uint16_t*)X, (const uint16_t*)dY, gate, perm, offsets, order,       \
                     (const uint16_t*)W1, w3, (const uint16_t*)W2, T, Nh, Ne, k, dff, dW1, dW3, dW2)
  if (dh == 128 && !gelu && cpw == 2)
    MHL_BWD_DW2(false, 2);
  else if (dh == 128 && !gelu)
    MHL_BWD_DW2(false, 1);
  else if (dh == 128 && cpw == 2)
    MHL_BWD_DW2(true, 2);
  else if (dh == 128)
    MHL_BWD_DW2(true, 1);
  else if (dh == 64 && !gelu)
    MHL_BWD_DW(64, false);
  else if (dh == 64)
    MHL_BWD_DW(64, true);
  else
    return hipErrorInvalidValue;
#undef MHL_BWD_DW
#undef MHL_BWD_DW2
  return hipGetLastError();
}

}  // namespace mhl
