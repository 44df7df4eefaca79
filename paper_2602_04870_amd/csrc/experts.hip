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

#include <type_traits>

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
// source and LDS offsets are recomputed per use to save registers.  GELU
// (the two-matrix expert: W1 = W_in, W2 = W_out) neither loads nor stores
// the W3 part.
template <int DH, bool F32, bool GELU = false>
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
      if (GELU && i >= N1 && i < 2 * N1) continue;
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
      if (GELU && i >= N1 && i < 2 * N1) continue;
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
// GELU: A^T = W_in_c X^T only, H^T = gelu(A^T).
template <int DH, bool GELU>
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
    const bf16x8 xb = as_bf16x8(xf.x[s]);
    a = mfma32_bf16(f1, xb, s == 0 ? zero16() : a);
    if (!GELU) {
      const bf16x8 f3 = as_bf16x8(*reinterpret_cast<const u32x4*>(r3 + o));
      b = mfma32_bf16(f3, xb, s == 0 ? zero16() : b);
    }
  }
  u32x4 hp[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = 8 * hh + 2 * i;
      if (GELU)
        hp[hh][i] = pack_bf16x2(gelu_logistic(a[v]), gelu_logistic(a[v + 1]));
      else
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

template <int DH, bool GELU>
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
#pragma unroll
      for (int p = 0; p < 4; ++p) a = mfma32_f32(f1[p], xf.x[s][half][p], a);
      if (!GELU) {
        const f32x4 f3 = *reinterpret_cast<const f32x4*>(r3 + o);
#pragma unroll
        for (int p = 0; p < 4; ++p) b = mfma32_f32(f3[p], xf.x[s][half][p], b);
      }
    }
  }
  float hv[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) hv[v] = GELU ? gelu_logistic(a[v]) : silu_fast(a[v]) * b[v];
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

// Persistent workgroups walk the halves of the compact tile list (work item
// i = half i % 2 of tile i / 2, at most 128 slots): XCD x (workgroups are
// dispatched round-robin over the XCDs) owns the contiguous tile range
// [x n / 8, (x + 1) n / 8), so one expert's adjacent tiles run on one XCD at
// about the same time and share its L2; within it the workgroups stride by
// their count.  While a tile computes, the next tile's descriptor, slot rows,
// X fragments, gate and first weight chunk are fetched, so a tile starts
// without a dependent round trip to memory.  GELU: the two-matrix expert
// (W1 = W_in, W2 = W_out; W3 is not read).
template <int DH, bool F32, bool GELU = false>
__global__ __launch_bounds__(kFfnThreads, 2) void ffn_kernel(
    const void* __restrict__ X, const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const TileInfo* __restrict__ tiles,
    const int32_t* __restrict__ head_base, const void* __restrict__ W1,
    const void* __restrict__ W3, const void* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, int dff, void* __restrict__ yslot) {
  using L = FfnLayout<DH, F32>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * L::STAGE];

  const int ntot = 2 * head_base[Nh];  // half-tile work items
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

  TileInfo ti = half_tile(tiles, tcur);
  TileRows<DH, F32> cur;
  cur.slot = slot_of(ti, cur.ok);
  gather(ti, cur);

  ChunkLoader<DH, F32, GELU> ld;
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
        if (ch == 0) tn = half_tile(tiles, tnext);
        if (ch == (nc > 1 ? 1 : 0)) nxt.slot = slot_of(tn, nxt.ok);
        if (ch == (nc > 2 ? 2 : nc - 1)) gather(tn, nxt);
      }
      if (ch + 1 < nc) {
        ld.load(w1b + eb, w3b + eb, w2b + eb, ch + 1, dff);
      } else if (has_next) {
        const int64_t en = expert_base(tn);
        ld.load(w1b + en, w3b + en, w2b + en, 0, dff);
      }
      if (wave_active) chunk_compute<DH, GELU>(smem + stage * L::STAGE, cur.xf, y, lane);
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

// ---------------------------------------------------------------------------
// Software-pipelined bf16 FFN for d_ff = 32 NC (NC a multiple of 4).  One
// workgroup of 8 wavefronts per CU takes whole tiles (up to 256 slots, 32
// per wavefront) and walks d_ff in NC chunks of 32 rows.  In step c a
// wavefront issues GEMM1 of chunk c+1 and GEMM2 of chunk c-1 (24 MFMAs at
// d_h 128, independent of each other) beside the SwiGLU of chunk c, so the
// matrix cores stay fed while the vector ALU does the elementwise work.  A
// tile's steps are fully unrolled, so the pipeline's two register sets
// alternate and every LDS address is a constant offset.
//
// Everything GEMM1 reads comes from LDS, not registers, leaving the
// register budget of two wavefronts per SIMD to the accumulators:
//  - the tile's gathered sub-token rows X[t, h, :] (256 rows), fetched by
//    global LDS-DMA from the token index of each row; each wavefront
//    fetches its own 32 rows, and the next tile's rows are fetched during
//    the last step of the current one, once no GEMM1 reads them;
//  - W1_c and W3_c (32 rows x d_h each) go by buffer LDS-DMA into a ring of
//    four slots, three chunks ahead of their use; wavefronts 0-3 fill the
//    W1 block, 4-7 the W3 block, each with the same number of 1 KiB DMA
//    instructions, so the issue code has no branches.
// Rows of X, W1_c and W3_c are stored with their 16-byte units XOR-swizzled
// by row (swz), which keeps the fragment reads (row = lane % 32) free of
// bank conflicts; the DMA lanes fetch the units in swizzled order.
//  - W2_c (d_h rows x 32) is loaded into registers two chunks ahead and
//    written to LDS, columns regrouped to GEMM2's K order, at the start of
//    the step before its GEMM2.
// A step ends with one barrier that waits only for the loads issued in the
// step before (s_waitcnt vmcnt(n)), so the step's own prefetches stay in
// flight across it.  Outputs are scaled by the gate and written per slot.
// ---------------------------------------------------------------------------
template <int DH>
struct PipeLayout {
  static constexpr int UPR = DH / 8;               // 16-byte units per row
  static constexpr int RB = DH * 2;                // row bytes (X, W1_c, W3_c)
  static constexpr int RPI = 64 / UPR;             // rows per 1 KiB DMA instruction
  static constexpr int BLOCK = kChunk * RB;        // one W1_c (or W3_c) block
  static constexpr int W13 = 2 * BLOCK;            // one ring slot
  static constexpr int NS = 4;                     // ring slots
  static constexpr int AHEAD = NS - 1;             // chunks DMA'd ahead of the SwiGLU step
  static constexpr int WPB = kPipeWaves / 2;       // wavefronts filling one block
  static constexpr int DMAW = BLOCK / 1024 / WPB;  // W1/W3 DMA instructions per wavefront
  static constexpr int RS2 = kChunk * 2 + 16;      // regrouped W2_c row stride (bytes)
  static constexpr int W2S = DH * RS2;             // one W2_c slot
  static constexpr int W2_OFF = NS * W13;
  static constexpr int X_OFF = W2_OFF + 2 * W2S;
  static constexpr int XW = kFfnRowsPerWave * RB;  // one wavefront's rows of X
  static constexpr int DMAX = XW / 1024;           // X DMA instructions per wavefront
  static constexpr int TOTAL = X_OFF + kPipeWaves * XW;
  static constexpr int THREADS = kPipeWaves * kWave;
  static constexpr int U2 = DH * kChunk / 8;       // 16-byte units of W2_c
  static_assert(DMAW >= 1 && BLOCK % (1024 * WPB) == 0, "uniform W1/W3 DMA split");
  static_assert(XW % 1024 == 0, "uniform X DMA split");
  static_assert(U2 <= THREADS && THREADS % U2 == 0, "W2 staging split");
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Raw buffer resource over one expert's W1 (or W3).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t expert_rsrc(const uint16_t* base, int num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, num_bytes, 0x00020000);
}

// One 16-byte global -> LDS DMA per lane: the lane's bytes land at
// lds + 16 * lane (lds uniform across the wavefront).
__device__ __forceinline__ void dma_global16(const void* src, lds_u8* lds) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// The same from a buffer resource: 16 bytes at byte offset voff + soff.
__device__ __forceinline__ void dma_buffer16(__amdgpu_buffer_rsrc_t rs, lds_u8* lds, uint32_t voff,
                                             int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds, 16, voff, soff, 0, 0);
}

// W2_c staged through registers: every thread issues exactly one 16-byte
// load per chunk (threads beyond the chunk's units repeat one), so each
// wavefront's count of outstanding loads is the same.
template <int DH>
struct PipeW2 {
  using L = PipeLayout<DH>;
  u32x4 r;
  __device__ __forceinline__ void load(const uint16_t* w2e, int ch, int dff) {
    const int uu = threadIdx.x % L::U2;
    const int n = uu / (kChunk / 8), m = uu % (kChunk / 8);
    r = *reinterpret_cast<const u32x4*>(w2e + (int64_t)n * dff + ch * kChunk + m * 8);
  }
  __device__ __forceinline__ void store(uint8_t* slot) const {
    const int uu = threadIdx.x;
    if (L::U2 == L::THREADS || uu < L::U2) {
      const int n = uu / (kChunk / 8), m = uu % (kChunk / 8);
      const int p0 = w2_group_pos(2 * m), p1 = w2_group_pos(2 * m + 1);
      uint8_t* row = slot + n * L::RS2;
      *reinterpret_cast<u32x2*>(row + (p0 >> 1) * 16 + (p0 & 1) * 8) = u32x2{r[0], r[1]};
      *reinterpret_cast<u32x2*>(row + (p1 >> 1) * 16 + (p1 & 1) * 8) = u32x2{r[2], r[3]};
    }
  }
};

// GEMM1 of one chunk: a^T = W1_c x^T, b^T = W3_c x^T, every operand from
// LDS.  off[s] is the lane's swizzled byte offset of k-step s in a row
// block (row c, 16-byte unit 2 s + g).
// (GELU: a only, from the W_in block.)
template <int DH, bool GELU = false>
__device__ __forceinline__ void pipe_gemm1(const uint8_t* slot, const uint8_t* xw,
                                           const uint32_t (&off)[DH / 16], f32x16& a, f32x16& b) {
  using L = PipeLayout<DH>;
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const bf16x8 xb = as_bf16x8(*reinterpret_cast<const u32x4*>(xw + off[s]));
    a = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(slot + off[s])), xb,
                    s == 0 ? zero16() : a);
    if constexpr (!GELU)
      b = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(slot + L::BLOCK + off[s])), xb,
                      s == 0 ? zero16() : b);
  }
}

// GEMM2 of one chunk: y^T += W2_c h^T (K order of h's lane layout).
template <int DH>
__device__ __forceinline__ void pipe_gemm2(const uint8_t* slot, const u32x4 (&hp)[2],
                                           f32x16 (&y)[DH / 32], int lane) {
  using L = PipeLayout<DH>;
  const int g = lane >> 5, c = lane & 31;
  const uint8_t* base = slot + c * L::RS2 + 16 * g;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb)
      y[nb] = mfma32_bf16(
          as_bf16x8(*reinterpret_cast<const u32x4*>(base + nb * 32 * L::RS2 + 32 * hh)),
          as_bf16x8(hp[hh]), y[nb]);
}

// h = silu(a) * b for the lane's 16 d_ff rows, packed to bf16 in GEMM2's K
// order.  Stage by stage over the 16 values, so that dependent instructions
// sit 16 apart and the transcendental latency is hidden.
__device__ __forceinline__ void pipe_swiglu(const f32x16& a, const f32x16& b, u32x4 (&hp)[2]) {
  float t[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = -1.4426950408889634f * a[v];
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = __builtin_amdgcn_exp2f(t[v]);
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = 1.0f + t[v];
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = __builtin_amdgcn_rcpf(t[v]);
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = (a[v] * t[v]) * b[v];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) hp[hh][i] = pack_bf16x2(t[8 * hh + 2 * i], t[8 * hh + 2 * i + 1]);
}

// h = gelu(a) (the two-matrix expert) for the lane's 16 d_ff rows, packed as
// pipe_swiglu packs h.
__device__ __forceinline__ void pipe_gelu(const f32x16& a, u32x4 (&hp)[2]) {
  float t[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) t[v] = gelu_logistic(a[v]);
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) hp[hh][i] = pack_bf16x2(t[8 * hh + 2 * i], t[8 * hh + 2 * i + 1]);
}

// Per-lane facts about its slot row of the tile: token row (t * Nh + h) of
// X, the gate, where the output goes (-1: row past the tile's end).
struct PipeRow {
  int32_t tokrow;
  float gv;
  int64_t out_off;
};

// GELU = true: the paper's two-matrix expert, y = W_out gelu(W_in x) (W1 =
// W_in, W2 = W_out, W3 unused); every wavefront's W1/W3 DMA then fetches
// W_in (the second block of a ring slot holds a copy nobody reads), so the
// DMA counts are those of the SwiGLU kernel.
template <int DH, int NC, bool GELU = false>
__global__ __launch_bounds__(kPipeWaves * kWave) void ffn_pipe_kernel(
    const uint16_t* __restrict__ X, const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const TileInfo* __restrict__ tiles,
    const int32_t* __restrict__ head_base, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W3, const uint16_t* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, uint16_t* __restrict__ yslot) {
  using L = PipeLayout<DH>;
  static_assert(NC % L::NS == 0 && NC >= L::NS, "tiles start on ring slot 0");
  constexpr int DFF = NC * kChunk;
  __shared__ __attribute__((aligned(16))) uint8_t smem[L::TOTAL];
  lds_u8* const smem3 = (lds_u8*)smem;

  const int ntot = head_base[Nh];
  const int xcd = (int)(blockIdx.x % kXcds);
  const int nper = (int)(gridDim.x / kXcds);
  const int t_hi = (int)((int64_t)ntot * (xcd + 1) / kXcds);
  int tcur = (int)((int64_t)ntot * xcd / kXcds) + (int)(blockIdx.x / kXcds);
  if (tcur >= t_hi) return;

  const int tid = threadIdx.x;
  // wave index as a scalar: wave-level branches and DMA bases stay uniform
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int64_t head_slots = T * k;
  constexpr int64_t WEXP = (int64_t)DFF * DH;  // elements of one expert's W1 (= W3 = W2)
  const uint16_t* const W13w = (GELU || wave < L::WPB) ? W1 : W3;  // this wavefront's DMA source

  // Swizzled fragment offsets of this lane in a 32-row block (row c, unit
  // 2 s + g) and the W1/W3 DMA source offsets of its units (row r, unit p
  // of the wavefront's share of a block holds logical unit swz(p, r)).
  uint32_t off[DH / 16];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) off[s] = c * L::RB + 16 * swz<L::UPR>(2 * s + g, c);
  uint32_t doff[L::DMAW];
#pragma unroll
  for (int d = 0; d < L::DMAW; ++d) {
    const int u = ((wave % L::WPB) + L::WPB * d) * 64 + lane;  // unit in the block
    const int r = u / L::UPR, p = u % L::UPR;
    doff[d] = (uint32_t)((r * DH + 8 * swz<L::UPR>(p, r)) * 2);
  }
  const uint8_t* const xw = smem + L::X_OFF + wave * L::XW;  // this wavefront's X rows
  lds_u8* const xw3 = smem3 + L::X_OFF + wave * L::XW;

  auto expert_off = [&](const TileInfo& ti) { return ((int64_t)ti.head * Ne + ti.expert) * WEXP; };
  // The lane's slot row of a tile (rows past the tile re-read its last row,
  // so that every wavefront issues the same loads) and what it needs.
  auto row_of = [&](const TileInfo& ti, int slot, bool ok) {
    PipeRow pr;
    const int t = slot / k;
    const int j = slot - t * k;
    pr.tokrow = t * Nh + ti.head;
    pr.gv = gate[(int64_t)pr.tokrow * k + j];
    pr.out_off = ok ? ((int64_t)pr.tokrow * k + j) * DH : -1;
    return pr;
  };
  auto slot_of = [&](const TileInfo& ti, bool& ok) {
    const int r = ti.row_begin + wave * kFfnRowsPerWave + c;
    ok = r < ti.row_end;
    return perm[(int64_t)ti.head * head_slots + (ok ? r : ti.row_end - 1)];
  };
  // DMA of the wavefront's 32 X rows: instruction d fills rows RPI d ..; the
  // lane's 16 bytes are unit p of row rr, i.e. logical unit swz(p, rr) of
  // token row tokrow(rr) (held by lane rr).
  auto dma_x = [&](int32_t tokrow) {
#pragma unroll
    for (int d = 0; d < L::DMAX; ++d) {
      const int rr = L::RPI * d + lane / L::UPR, p = lane % L::UPR;
      const int32_t src_row = __shfl(tokrow, rr, kWave);
      const uint16_t* src = X + (int64_t)src_row * DH + 8 * swz<L::UPR>(p, rr);
      dma_global16(src, xw3 + d * 1024);
    }
  };
  auto dma_w = [&](int slot, __amdgpu_buffer_rsrc_t rs, int ch) {
    lds_u8* base = smem3 + slot * L::W13 + (wave / L::WPB) * L::BLOCK + (wave % L::WPB) * 1024;
#pragma unroll
    for (int d = 0; d < L::DMAW; ++d)
      dma_buffer16(rs, base + d * L::WPB * 1024, doff[d], ch * kChunk * DH * 2);
  };

  TileInfo ti = tiles[tcur];
  bool ok;
  PipeRow cur = row_of(ti, slot_of(ti, ok), ok);
  int64_t eo = expert_off(ti);
  __amdgpu_buffer_rsrc_t rs = expert_rsrc(W13w + eo, (int)(WEXP * 2));

  // Prologue: the first tile's rows, its W1/W3 chunks 0 .. AHEAD-1 and
  // W2 of its chunks 0 and 1 (register sets 0 and 1).
  PipeW2<DH> w2r[2];
  dma_x(cur.tokrow);
#pragma unroll
  for (int q = 0; q < L::AHEAD; ++q) dma_w(q, rs, q);
  w2r[0].load(W2 + eo, 0, DFF);
  w2r[1].load(W2 + eo, 1, DFF);
  barrier_vm<0>();

  while (true) {
    const int tnext = tcur + nper;
    const bool has_next = tnext < t_hi;
    TileInfo tn = ti;
    int64_t en = eo;
    __amdgpu_buffer_rsrc_t rn = rs;
    int nslot = 0;
    bool nok = false;
    if (has_next) {
      tn = tiles[tnext];
      en = expert_off(tn);
      rn = expert_rsrc(W13w + en, (int)(WEXP * 2));
      nslot = slot_of(tn, nok);
    }
    PipeRow nxt = cur;
    const bool wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;

    f32x16 y[DH / 32];
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) y[nb] = zero16();
    f32x16 A[2], B[2];
    u32x4 H[2][2];
    if (wave_active) pipe_gemm1<DH, GELU>(smem, xw, off, A[0], B[0]);

#pragma unroll
    for (int ch = 0; ch < NC; ++ch) {
      // W2 of this chunk (loaded two steps ago) goes to LDS for the GEMM2
      // of the next step; its register set then takes W2 of chunk ch + 2.
      w2r[ch & 1].store(smem + L::W2_OFF + (ch & 1) * L::W2S);
      // loads: (last step) the next tile's gates and rows, W2 of chunk
      // ch + 2, then W1/W3 of chunk ch + AHEAD, each of this tile or, past
      // its end, of the next one (with no next tile a harmless re-read of
      // this expert into a slot nobody reads again)
      if (ch == NC - 1 && has_next) {
        nxt = row_of(tn, nslot, nok);
        dma_x(nxt.tokrow);
      }
      if (ch + 2 < NC) w2r[ch & 1].load(W2 + eo, ch + 2, DFF);
      else w2r[ch & 1].load(W2 + en, ch + 2 - NC, DFF);
      if (ch + L::AHEAD < NC) dma_w((ch + L::AHEAD) % L::NS, rs, ch + L::AHEAD);
      else dma_w((ch + L::AHEAD) % L::NS, rn, ch + L::AHEAD - NC);
      if (wave_active) {
        if (ch + 1 < NC)
          pipe_gemm1<DH, GELU>(smem + ((ch + 1) % L::NS) * L::W13, xw, off, A[(ch + 1) & 1],
                               B[(ch + 1) & 1]);
        if (ch >= 1)
          pipe_gemm2<DH>(smem + L::W2_OFF + ((ch - 1) & 1) * L::W2S, H[(ch - 1) & 1], y, lane);
        if constexpr (GELU) pipe_gelu(A[ch & 1], H[ch & 1]);
        else pipe_swiglu(A[ch & 1], B[ch & 1], H[ch & 1]);
        {
          // Instruction order of the step: two LDS reads ahead, then per
          // MFMA one LDS read and a share of the activation's VALU work
          // (SwiGLU: three per MFMA; GELU: ten), so the vector ALU works
          // while the matrix core is busy.
          constexpr int NM = (GELU ? 16 : 24) * DH / 128;
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
          for (int i = 0; i < NM; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, GELU ? 10 : 3, 0);
          }
        }
      }
      barrier_vm<L::DMAW + 1>();
    }
    if (wave_active) pipe_gemm2<DH>(smem + L::W2_OFF + ((NC - 1) & 1) * L::W2S, H[(NC - 1) & 1], y, lane);

    // Y^T tile: lane holds slot column c, d_h rows 32 nb + 8 q + 4 g + [0, 4).
    // Lanes c and c + 32 swap halves so that each holds 8 consecutive
    // outputs (groups q = 2 p for g = 0, 2 p + 1 for g = 1) and writes them
    // as one 16-byte piece; the two lanes of a row cover 32 contiguous bytes.
    {
      uint16_t* o = yslot + (cur.out_off >= 0 ? cur.out_off : 0);
#pragma unroll
      for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
        for (int qp = 0; qp < 2; ++qp) {
          const int q0 = 2 * qp, q1 = 2 * qp + 1;
          uint32_t p[2] = {pack_bf16x2(cur.gv * y[nb][4 * q0 + 0], cur.gv * y[nb][4 * q0 + 1]),
                           pack_bf16x2(cur.gv * y[nb][4 * q0 + 2], cur.gv * y[nb][4 * q0 + 3])};
          uint32_t q[2] = {pack_bf16x2(cur.gv * y[nb][4 * q1 + 0], cur.gv * y[nb][4 * q1 + 1]),
                           pack_bf16x2(cur.gv * y[nb][4 * q1 + 2], cur.gv * y[nb][4 * q1 + 3])};
#pragma unroll
          for (int w = 0; w < 2; ++w) {
            const auto r = __builtin_amdgcn_permlane32_swap(p[w], q[w], false, false);
            p[w] = r[0];
            q[w] = r[1];
          }
          if (cur.out_off >= 0)
            *reinterpret_cast<u32x4*>(o + 32 * nb + 16 * qp + 8 * g) = u32x4{p[0], p[1], q[0], q[1]};
        }
    }
    if (!has_next) break;
    ti = tn;
    cur = nxt;
    eo = en;
    rs = rn;
    tcur = tnext;
  }
  // No LDS DMA left in flight when the wavefront ends (vmcnt(0)).
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

// ---------------------------------------------------------------------------
// bf16 FFN at d_h 128 (d_ff = 32 NC), in two shapes.  WAVES = 4: workgroups
// of 4 wavefronts take tiles of up to 128 slots (32 per wavefront), two
// workgroups per CU, so each SIMD runs two wavefronts of different tiles
// whose barriers are independent.  WAVES = 8: one workgroup of 8 wavefronts
// per CU takes tiles of up to 256 slots, so every pass of an expert's
// weights through LDS serves twice the slots (chosen where experts see many
// slots on average: a tile's weight stream, not its slots, sets most of its
// cost).  Per wavefront, d_ff is walked in 32-row chunks; step c issues
//   GEMM1  a^T = W1_c+1 x^T, b^T = W3_c+1 x^T   (32x32x16 MFMAs, K = d_h)
//   GEMM2  y^T += W2_c-1 h_c-1^T                 (K = 32)
// beside h_c = silu(a_c) * b_c (registers), so the matrix core works while
// the vector ALU does the elementwise part; a tile's steps are fully
// unrolled, the two register sets alternating.  The slot rows x (gathered
// from X[t, h, :]) are held in registers as MFMA operands.  Lanes c and
// c + 32 exchange a quarter of h (v_permlane32_swap) so that each lane holds
// 8 consecutive d_ff rows of its slot, GEMM2's operand layout, and W2 is
// used in its natural K order.
//
// W1_c and W3_c (32 rows x d_h, 16 KiB) arrive by buffer LDS-DMA in a ring
// of NS slots AHEAD chunks ahead (2 and 2 with 4 wavefronts, 4 and 3 with
// 8), W2_c (d_h rows x 32, 8 KiB) in a four-slot ring two chunks ahead;
// every wavefront issues the same number of 1 KiB instructions per step.
// Rows have their 16-byte units XOR-swizzled by row so that every fragment
// read is a conflict-free ds_read_b128.  A step ends with a barrier that
// waits for the W1/W3 chunk the next step reads (issued AHEAD - 2 steps
// earlier) and the W2 chunk it reads, and leaves later DMAs in flight.
// ---------------------------------------------------------------------------
template <int WAVES_>
struct Q32Layout {
  static constexpr int DH = 128;
  static constexpr int RB = DH * 2;              // W1_c / W3_c row bytes
  static constexpr int WAVES = WAVES_;
  static constexpr int WPM = WAVES / 2;          // wavefronts per W1 (or W3) DMA
  static constexpr int THREADS = WAVES * kWave;
  static constexpr int MIN_BLOCKS = WAVES == 8 ? 1 : 2;  // workgroups per CU
  static constexpr int WB = kChunk * RB;         // one W1_c (or W3_c) block: 8 KiB
  static constexpr int W2RB = kChunk * 2;        // W2_c row bytes (64)
  static constexpr int W2B = DH * W2RB;          // one W2_c block: 8 KiB
  // W1/W3 ring slots: the DMA of step c (chunk c + AHEAD) goes to the slot
  // of chunk c + AHEAD - NS, whose GEMM1 ran in step c + AHEAD - NS - 1 (the
  // barrier ending that step orders the reads before the overwrite); with a
  // chunk count that NS divides every tile starts at slot 0, so the slots
  // are compile-time offsets
  static constexpr int NS = WAVES == 8 ? 4 : 2;
  static constexpr int AHEAD = WAVES == 8 ? 3 : 2;
  static constexpr int NS2 = 4;                  // W2 ring slots
  static constexpr int AHEAD2 = 2;               // W2 chunks DMA'd ahead of their SwiGLU step
  static constexpr int W2_OFF = NS * 2 * WB;
  static constexpr int TOTAL = W2_OFF + NS2 * W2B;
  static constexpr int DMA13 = WB / 1024 / WPM;  // W1 or W3 instructions per wavefront
  static constexpr int DMA2 = W2B / 1024 / WAVES;  // W2 instructions per wavefront
  static constexpr int NXF = DH / 16;              // loads of a gathered row fragment
  static_assert(WAVES == 4 || WAVES == 8, "two shapes");
  static_assert(WAVES * 32 == (WAVES == 8 ? kTileRows : kPipeTileRows), "tile rows");
  static_assert(DMA13 * WPM * 1024 == WB && DMA2 * WAVES * 1024 == W2B, "uniform DMA split");
  static_assert(TOTAL * MIN_BLOCKS <= 160 * 1024, "LDS per CU");
  static_assert(AHEAD2 == 2 && AHEAD >= 2 && AHEAD <= 3 && NS >= AHEAD, "wait counts");
};

// GELU = false: SwiGLU expert, y = W2 (silu(W1 x) * (W3 x)).  GELU = true:
// the paper's two-matrix expert, y = W2 gelu(W1 x) (W1 = W_in, W2 = W_out,
// W3 unused); the W1/W3 ring slots then hold only the W_in chunk, fetched by
// all the wavefronts.
template <int NC, bool GELU, int WAVES>
__global__ __launch_bounds__(Q32Layout<WAVES>::THREADS,
                             Q32Layout<WAVES>::MIN_BLOCKS) void ffn_q32_kernel(
    const uint16_t* __restrict__ X, const int32_t* __restrict__ perm, const TileInfo* __restrict__ tiles,
    const int32_t* __restrict__ head_base, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W3, const uint16_t* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, uint16_t* __restrict__ yslot) {
  using L = Q32Layout<WAVES>;
  constexpr int DH = L::DH;
  constexpr int DFF = NC * kChunk;
  static_assert(NC % L::NS == 0 && NC % L::NS2 == 0, "every tile starts at ring slot 0");
  __shared__ __attribute__((aligned(16))) uint8_t smem[L::TOTAL];
  lds_u8* const smem3 = (lds_u8*)smem;

  const int ntot = head_base[Nh];
  const int xcd = (int)(blockIdx.x % kXcds);
  const int nper = (int)(gridDim.x / kXcds);
  const int t_hi = (int)((int64_t)ntot * (xcd + 1) / kXcds);
  int tcur = (int)((int64_t)ntot * xcd / kXcds) + (int)(blockIdx.x / kXcds);
  if (tcur >= t_hi) return;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int g = lane >> 5, c = lane & 31;
  const int64_t head_slots = T * k;
  constexpr int64_t WEXP = (int64_t)DFF * DH;  // elements of one expert's W1 (= W3 = W2)
  const uint16_t* const W13w = (GELU || wave < L::WPM) ? W1 : W3;
  // W1/W3 DMA instructions per wavefront (GELU: W_in only, split over all)
  constexpr int D13 = GELU ? L::WB / 1024 / L::WAVES : L::DMA13;
  constexpr int NMAT = GELU ? 1 : 2;  // GEMM1 weight matrices

  // LDS fragment offsets of the lane (the ring slot is added as an
  // immediate).  GEMM1 k-step s: W row c, 16-byte unit 2 s + g, swizzled by
  // the row: (2 s + g) ^ (c & 15) = 2 (s ^ sw1) + (g ^ (c & 1)).  GEMM2
  // half hh: W2 row 32 nb + c, unit 2 hh + g, swizzled by bits 2-3 of the row.
  const int sw1 = (c >> 1) & 7;
  const int sw2 = (c >> 2) & 3;
  uint32_t off1[DH / 16], off2[2];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) off1[s] = c * L::RB + 16 * (g ^ (c & 1)) + 32 * (s ^ sw1);
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) off2[hh] = c * L::W2RB + 16 * ((2 * hh + g) ^ sw2);
  // DMA source offsets.  W1/W3: instruction d fills KiB i = D13 (wave %
  // WPM) + d of the block (GELU: D13 wave + d): rows 4 i + lane / 16,
  // physical unit lane % 16.  W2: KiB j = DMA2 wave + d: rows 16 j + lane /
  // 4, physical unit lane % 4.
  uint32_t doff[D13 + L::DMA2];
#pragma unroll
  for (int d = 0; d < D13; ++d) {
    const int i = D13 * (GELU ? wave : wave % L::WPM) + d;
    const int r = 4 * i + lane / 16, p = lane % 16;
    doff[d] = (uint32_t)((r * DH + 8 * (p ^ (r & 15))) * 2);
  }
#pragma unroll
  for (int d = 0; d < L::DMA2; ++d) {
    const int j = L::DMA2 * wave + d;
    const int n = 16 * j + lane / 4, p = lane % 4;
    doff[D13 + d] = (uint32_t)(n * DFF * 2 + 16 * (p ^ ((n >> 2) & 3)));
  }

  RowFrag<DH, false> xf;  // the lane's gathered slot row (MFMA operand fragments)
  auto expert_off = [&](const TileInfo& ti) { return ((int64_t)ti.head * Ne + ti.expert) * WEXP; };
  auto slot_of = [&](const TileInfo& ti, bool& ok) {
    const int r = ti.row_begin + wave * kFfnRowsPerWave + c;
    ok = r < ti.row_end;
    return perm[(int64_t)ti.head * head_slots + (ok ? r : ti.row_end - 1)];
  };
  // The lane's slot row of a tile: X fragments (every lane loads, rows past
  // the tile re-read its last row: NXF vector loads) and output offset.  A
  // lane past the tile's end takes the last row's slot, so it computes that
  // slot's output bit for bit and writes the same bytes there again: the
  // stores need no lane mask and their number per wavefront is fixed, which
  // the wait counts below rely on.  The slot's gate is applied by the
  // combine kernel.
  auto gather = [&](const TileInfo& ti, int slot, bool ok, RowFrag<DH, false>& xf,
                    int64_t& out_off) {
    (void)ok;
    const int t = slot / k;
    const int j = slot - t * k;
    const int64_t tok_head = (int64_t)t * Nh + ti.head;
    xf.load(X, tok_head, true, g);
    out_off = (tok_head * k + j) * DH;
  };
  auto dma13 = [&](int slot, __amdgpu_buffer_rsrc_t r13, int ch) {
    lds_u8* s3 = smem3 + slot * 2 * L::WB;
#pragma unroll
    for (int d = 0; d < D13; ++d)
      dma_buffer16(r13,
                   s3 + (GELU ? 0 : (wave / L::WPM) * L::WB) +
                       (D13 * (GELU ? wave : wave % L::WPM) + d) * 1024,
                   doff[d], ch * kChunk * DH * 2);
  };
  auto dma2 = [&](int slot, __amdgpu_buffer_rsrc_t r2, int ch) {
    lds_u8* s3 = smem3 + L::W2_OFF + slot * L::W2B;
#pragma unroll
    for (int d = 0; d < L::DMA2; ++d)
      dma_buffer16(r2, s3 + (L::DMA2 * wave + d) * 1024, doff[D13 + d], ch * kChunk * 2);
  };

  f32x16 y[DH / 32];
  f32x16 A[2], B[2];
  u32x4 H[2][2];
  float t[16];
  uint32_t pk[8];

  // The MFMAs of one pipeline step, in issue order: GEMM2 of chunk C2 (8,
  // when C2 >= 0: W2 ring slot C2 % NS2, h of H[C2 & 1]), then GEMM1 of
  // chunk C1 (8 NMAT, when C1 >= 0: ring slot C1 % NS, into A/B[C1 & 1]).
  // Each MFMA's LDS fragment is read P MFMAs ahead into a ring of
  // registers, and the activation work of chunk CA (when CA >= 0) is spread
  // over the MFMAs, a fixed share after each (sched_barrier keeps this
  // order: the compiler would otherwise read each fragment right before its
  // MFMA and stall on the LDS latency).
  auto step = [&](auto C2c, auto C1c, auto CAc) {
    constexpr int C2 = decltype(C2c)::value, C1 = decltype(C1c)::value, CA = decltype(CAc)::value;
    constexpr int N2 = C2 >= 0 ? 8 : 0;
    constexpr int N1 = C1 >= 0 ? 8 * NMAT : 0;
    constexpr int NM = N2 + N1;
    constexpr int P = 4;
    constexpr int NV = CA < 0 ? 0 : GELU ? 16 + 12 : 6 * 16 + 12;
    auto frag = [&](auto Mc) -> u32x4 {
      constexpr int m = decltype(Mc)::value;
      if constexpr (m < N2) {
        constexpr int hh = m / 4, nb = m % 4;
        constexpr uint32_t imm = L::W2_OFF + ((C2 < 0 ? 0 : C2) % L::NS2) * L::W2B + nb * 32 * L::W2RB;
        return *reinterpret_cast<const u32x4*>(smem + off2[hh] + imm);
      } else {
        constexpr int j = m - N2, s = j / NMAT, mat = j % NMAT;
        constexpr uint32_t imm = ((C1 < 0 ? 0 : C1) % L::NS) * 2 * L::WB + mat * L::WB;
        return *reinterpret_cast<const u32x4*>(smem + off1[s] + imm);
      }
    };
    auto mfma = [&](auto Mc, const u32x4& f) {
      constexpr int m = decltype(Mc)::value;
      if constexpr (m < N2) {
        constexpr int hh = m / 4, nb = m % 4;
        y[nb] = mfma32_bf16(as_bf16x8(f), as_bf16x8(H[C2 & 1][hh]), y[nb]);
      } else {
        constexpr int j = m - N2, s = j / NMAT, mat = j % NMAT;
        f32x16& acc = mat == 0 ? A[C1 & 1] : B[C1 & 1];
        acc = mfma32_bf16(as_bf16x8(f), as_bf16x8(xf.x[s]), s == 0 ? zero16() : acc);
      }
    };
    // Activation op o of chunk CA.  SwiGLU, stage-major over the 16
    // accumulator elements v: t = -log2(e) a, 2^t, 1 + t, 1 / t, a t, t b;
    // GELU: t = gelu(a) per element.  Then 8 packs to bf16 and 4 lane swaps
    // (h in GEMM2's operand layout; lane (g, c): slot c, d_ff rows 16 hh +
    // 8 g + [0, 8): the MFMA output holds rows 8 (v / 4) + 4 g + v % 4, so
    // P = rows 16 hh + 4 g + [0, 4) of lane c + 32 trade with Q = rows
    // 16 hh + 8 + 4 g + [0, 4) of lane c).
    auto act = [&](auto Oc) {
      constexpr int o = decltype(Oc)::value;
      constexpr int NE = GELU ? 16 : 96;  // elementwise ops
      const f32x16& a = A[(CA < 0 ? 0 : CA) & 1];
      const f32x16& b = B[(CA < 0 ? 0 : CA) & 1];
      if constexpr (o < NE) {
        constexpr int v = o % 16, st = o / 16;
        if constexpr (GELU) t[v] = gelu_logistic(a[v]);
        else if constexpr (st == 0) t[v] = -1.4426950408889634f * a[v];
        else if constexpr (st == 1) t[v] = __builtin_amdgcn_exp2f(t[v]);
        else if constexpr (st == 2) t[v] = 1.0f + t[v];
        else if constexpr (st == 3) t[v] = __builtin_amdgcn_rcpf(t[v]);
        else if constexpr (st == 4) t[v] = a[v] * t[v];
        else t[v] = t[v] * b[v];
      } else if constexpr (o < NE + 8) {
        constexpr int p = o - NE;
        pk[p] = pack_bf16x2(t[2 * p], t[2 * p + 1]);
      } else {
        constexpr int i = o - NE - 8, hh = i / 2, w = i % 2;
        const auto r = permlane32_swap(pk[4 * hh + w], pk[4 * hh + 2 + w]);
        pk[4 * hh + w] = r[0];
        pk[4 * hh + 2 + w] = r[1];
        if constexpr (w == 1)
          H[CA & 1][hh] = u32x4{pk[4 * hh], pk[4 * hh + 1], pk[4 * hh + 2], pk[4 * hh + 3]};
      }
    };
    u32x4 fr[P];
    static_for<0, (P < NM ? P : NM)>([&](auto I) { fr[decltype(I)::value] = frag(I); });
    static_for<0, NM>([&](auto Mc) {
      constexpr int m = decltype(Mc)::value;
      mfma(Mc, fr[m % P]);
      if constexpr (m + P < NM) fr[m % P] = frag(std::integral_constant<int, m + P>{});
      static_for<m * NV / NM, (m + 1) * NV / NM>(act);
      __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (NM == 0) static_for<0, NV>(act);
  };
  using I_ = std::integral_constant<int, -1>;

  // Y^T tile: lane holds slot column c, d_h rows 32 nb + 8 q + 4 g + [0, 4).
  // Lanes c and c + 32 swap halves so that each holds 8 consecutive
  // outputs (groups q = 2 p for g = 0, 2 p + 1 for g = 1) and writes them
  // as one 16-byte piece; the two lanes of a row cover 32 contiguous bytes.
  // NST stores per lane, issued by every lane of an active wavefront.
  constexpr int NST = DH / 32 * 2;
  // Tiles of at least 8 chunks write their outputs in the next tile's first
  // step (measured: 2-4% faster at d_ff 256); with 4 chunks per tile that
  // step's extra work cost more than the wait it saves (2-6% slower), so
  // those tiles store right after their last step.
  constexpr bool DEFER = NC >= 8;
  auto store_y = [&](int64_t off) {
    uint16_t* o = yslot + off;
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
      for (int qp = 0; qp < 2; ++qp) {
        const int q0_ = 2 * qp, q1_ = 2 * qp + 1;
        uint32_t p[2] = {pack_bf16x2(y[nb][4 * q0_ + 0], y[nb][4 * q0_ + 1]),
                         pack_bf16x2(y[nb][4 * q0_ + 2], y[nb][4 * q0_ + 3])};
        uint32_t r2[2] = {pack_bf16x2(y[nb][4 * q1_ + 0], y[nb][4 * q1_ + 1]),
                          pack_bf16x2(y[nb][4 * q1_ + 2], y[nb][4 * q1_ + 3])};
#pragma unroll
        for (int w = 0; w < 2; ++w) {
          const auto r = permlane32_swap(p[w], r2[w]);
          p[w] = r[0];
          r2[w] = r[1];
        }
        *reinterpret_cast<u32x4*>(o + 32 * nb + 16 * qp + 8 * g) = u32x4{p[0], p[1], r2[0], r2[1]};
      }
  };
  bool pend_store = false;  // (wave-uniform) the previous tile's outputs are still in y
  int64_t pend_off = 0;

  TileInfo ti = tiles[tcur];
  int64_t eo = expert_off(ti);
  __amdgpu_buffer_rsrc_t rs = expert_rsrc(W13w + eo, (int)(WEXP * 2));
  __amdgpu_buffer_rsrc_t rs2 = expert_rsrc(W2 + eo, (int)(WEXP * 2));

  // Prologue: W1/W3 of chunks 0 .. AHEAD-1 and W2 of chunks 0 .. AHEAD2-1
  // of the first tile, then (while they land) its slot rows, whose loads
  // depend on the slot list.
#pragma unroll
  for (int ch = 0; ch < L::AHEAD; ++ch) dma13(ch, rs, ch);
#pragma unroll
  for (int ch = 0; ch < L::AHEAD2; ++ch) dma2(ch, rs2, ch);
  bool ok;
  int64_t out_off;
  gather(ti, slot_of(ti, ok), ok, xf, out_off);
  barrier_vm<0>();
  bool wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;
  if (wave_active) step(I_{}, std::integral_constant<int, 0>{}, I_{});
  // (the ring slot of chunk 0 is refilled in step 0)
  barrier_lds();

  while (true) {
    const int tnext = tcur + nper;
    const bool has_next = tnext < t_hi;
    TileInfo tn = ti;
    int64_t en = eo;
    __amdgpu_buffer_rsrc_t rn = rs, rn2 = rs2;
    int nslot = 0;
    bool nok = false;
    if (has_next) {
      tn = tiles[tnext];
      en = expert_off(tn);
      rn = expert_rsrc(W13w + en, (int)(WEXP * 2));
      rn2 = expert_rsrc(W2 + en, (int)(WEXP * 2));
      nslot = slot_of(tn, nok);
    }
    int64_t nout = out_off;

    // Step ch: GEMM2 of chunk ch - 1, GEMM1 of chunk ch + 1, the activation
    // of chunk ch.  Loads first: W1/W3 of chunk ch + AHEAD (needed in the
    // next step, so waited for at this step's end) and W2 of chunk ch +
    // AHEAD2 (left in flight), each of this tile or, past its end, of the
    // next one (with no next tile a harmless re-read of this expert into a
    // slot nobody reads again).  Step 0 then (DEFER) writes the previous tile's
    // outputs (held in y until now) and clears y: issued after the step's
    // DMAs, the stores are younger than every load a barrier waits for, so
    // no barrier waits for them to reach memory.
    static_for<0, NC>([&](auto CHc) {
      constexpr int ch = decltype(CHc)::value;
      if constexpr (ch + L::AHEAD < NC) dma13((ch + L::AHEAD) % L::NS, rs, ch + L::AHEAD);
      else dma13((ch + L::AHEAD) % L::NS, rn, ch + L::AHEAD - NC);
      if constexpr (ch + L::AHEAD2 < NC) dma2((ch + L::AHEAD2) % L::NS2, rs2, ch + L::AHEAD2);
      else dma2((ch + L::AHEAD2) % L::NS2, rn2, ch + L::AHEAD2 - NC);
      if constexpr (ch == 0) {
        if (DEFER && pend_store) store_y(pend_off);
#pragma unroll
        for (int nb = 0; nb < DH / 32; ++nb) y[nb] = zero16();
      }
      if (wave_active)
        step(std::integral_constant<int, ch - 1>{},
             std::integral_constant<int, (ch + 1 < NC ? ch + 1 : -1)>{},
             std::integral_constant<int, ch>{});
      // last step: the rows are dead after the last GEMM1, so the next
      // tile's are gathered now (issued after this step's DMA, waited for
      // below)
      // The step's end waits for W1/W3 of chunk ch + 2 (issued in step
      // ch + 2 - AHEAD) and W2 of chunk ch (step ch - 2, earlier still):
      // that step's W2 DMA and every later load may stay in flight.
      constexpr int STAY = L::DMA2 + (L::AHEAD - 2) * (D13 + L::DMA2);
      if constexpr (ch == NC - 1) {
        if (has_next) {
          gather(tn, nslot, nok, xf, nout);
          barrier_vm<STAY + L::NXF>();
        } else {
          barrier_vm<STAY>();
        }
      } else if constexpr (ch == 0 && DEFER) {
        if (pend_store) barrier_vm<STAY + NST>();
        else barrier_vm<STAY>();
      } else {
        barrier_vm<STAY>();
      }
    });
    if (wave_active) step(std::integral_constant<int, NC - 1>{}, I_{}, I_{});
    if constexpr (DEFER) {
      pend_store = wave_active;
      pend_off = out_off;
    } else if (wave_active) {
      store_y(out_off);
    }
    if (!has_next) break;
    ti = tn;
    out_off = nout;
    eo = en;
    rs = rn;
    rs2 = rn2;
    tcur = tnext;
    wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;
    // GEMM1 of the new tile's chunk 0, whose ring slot step 0 refills
    if (wave_active) step(I_{}, std::integral_constant<int, 0>{}, I_{});
    barrier_lds();
  }
  if (pend_store) store_y(pend_off);
  // No LDS DMA left in flight when the wavefront ends: vmcnt(0) (bits 3:0
  // and 15:14), expcnt and lgkmcnt left at their maxima.
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

// Y[row] = sum_{j<k} yslot[row][j] in fixed j order (GATED: the per-slot
// outputs are unscaled and the sum is sum_j gate[row][j] yslot[row][j]); one
// thread per 8 consecutive output elements.  All k loads are issued before
// the sums.  Each per-slot row is read exactly once, so the loads are
// non-temporal (they do not displace reusable lines from the caches; 8-23%
// faster at 8-32 slots per row than plain loads).
template <int DH, bool F32, bool GATED>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ yslot,
                                                      const float* __restrict__ gate,
                                                      int64_t rows, int k,
                                                      void* __restrict__ Y) {
  constexpr int TPR = DH / 8;
  constexpr int KU = 16;  // slots loaded per round (at k = 32: 2.8% faster than 8)
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
      float gj[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
          const float* p = reinterpret_cast<const float*>(yslot) + base + (int64_t)(j0 + u) * DH;
          a[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
          b[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
          gj[u] = GATED ? gate[row * k + j0 + u] : 1.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[i] = GATED ? fmaf(gj[u], a[u][i], acc[i]) : acc[i] + a[u][i];
            acc[4 + i] = GATED ? fmaf(gj[u], b[u][i], acc[4 + i]) : acc[4 + i] + b[u][i];
          }
        }
      }
    } else {
      u32x4 v[KU];
      float gj[KU];
#pragma unroll
      for (int u = 0; u < KU; ++u)
        if (j0 + u < k) {
          v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
              reinterpret_cast<const uint16_t*>(yslot) + base + (int64_t)(j0 + u) * DH));
          gj[u] = GATED ? gate[row * k + j0 + u] : 1.0f;
        }
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (j0 + u < k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float lo = bf16_bits_to_f32(v[u][i] & 0xFFFFu);
            const float hi = bf16_bits_to_f32(v[u][i] >> 16);
            acc[2 * i] = GATED ? fmaf(gj[u], lo, acc[2 * i]) : acc[2 * i] + lo;
            acc[2 * i + 1] = GATED ? fmaf(gj[u], hi, acc[2 * i + 1]) : acc[2 * i + 1] + hi;
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
  // d_h 128, bf16, d_ff in {128, 256, 384, 512}: 128-row tiles with two
  // workgroups per CU, or 256-row tiles with one (q32_wide).
  if (q32_eligible(T, Nh, DH, dff, F32)) {
#define MHL_Q32(NC, W)                                                                          \
  hipLaunchKernelGGL((ffn_q32_kernel<NC, false, W>), dim3(W == 8 ? kQ32WideGrid : kQ32Grid),    \
                     dim3(Q32Layout<W>::THREADS), 0, s, (const uint16_t*)X, perm, ti, head_base, \
                     (const uint16_t*)W1, (const uint16_t*)W3, (const uint16_t*)W2, T, Nh, Ne, k,  \
                     (uint16_t*)yslot);                                                         \
  return hipGetLastError()
    const bool wide = q32_wide(T, k, Ne);
    switch (dff / kChunk) {
      case 4: if (wide) { MHL_Q32(4, 8); } else { MHL_Q32(4, 4); }
      case 8: if (wide) { MHL_Q32(8, 8); } else { MHL_Q32(8, 4); }
      case 12: if (wide) { MHL_Q32(12, 8); } else { MHL_Q32(12, 4); }
      case 16: if (wide) { MHL_Q32(16, 8); } else { MHL_Q32(16, 4); }
      default: break;
    }
#undef MHL_Q32
  }
  // The pipelined kernel (d_h 64): bf16, d_ff in {128, 256, 384, 512}, token
  // rows addressable with 32-bit indices.
  if (!F32 && dff % (4 * kChunk) == 0 && T * Nh < (int64_t(1) << 31)) {
#define MHL_PIPE(NC)                                                                           \
  hipLaunchKernelGGL((ffn_pipe_kernel<DH, NC>), dim3(kPipeGrid), dim3(kPipeWaves * kWave), 0, s, \
                     (const uint16_t*)X, gate, perm, ti, head_base, (const uint16_t*)W1,        \
                     (const uint16_t*)W3, (const uint16_t*)W2, T, Nh, Ne, k, (uint16_t*)yslot); \
  return hipGetLastError()
    switch (dff / kChunk) {
      case 4: MHL_PIPE(4);
      case 8: MHL_PIPE(8);
      case 12: MHL_PIPE(12);
      case 16: MHL_PIPE(16);
      default: break;
    }
#undef MHL_PIPE
  }
  hipLaunchKernelGGL((ffn_kernel<DH, F32>), dim3(kFfnGrid), dim3(kFfnThreads), 0, s, X, gate,
                     perm, ti, head_base, W1, W3, W2, T, Nh, Ne, k, dff, yslot);
  return hipGetLastError();
}

template <int DH, bool F32>
hipError_t combine_dispatch(const void* yslot, const float* gate, int64_t T, int Nh, int k,
                            void* Y, hipStream_t s) {
  const int64_t rows = T * Nh;
  const int64_t threads = rows * (DH / 8);
  const dim3 grid((unsigned)ceil_div(threads, 256));
  if (gate)
    hipLaunchKernelGGL((combine_kernel<DH, F32, true>), grid, dim3(256), 0, s, yslot, gate, rows,
                       k, Y);
  else
    hipLaunchKernelGGL((combine_kernel<DH, F32, false>), grid, dim3(256), 0, s, yslot, gate, rows,
                       k, Y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ffn_gelu(const void* X, const float* gate, const int32_t* perm,
                           const TileInfo* tile_info, const int32_t* head_base,
                           const void* W_in, const void* W_out, int64_t T, int Nh, int dh,
                           int Ne, int k, int dff, bool f32, void* yslot, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if ((dh != 64 && dh != 128) || dff < kChunk || dff % kChunk != 0) return hipErrorInvalidValue;
  // fp32, or a d_ff that the pipelined kernels do not take: the generic
  // kernel over half tiles (gate-scaled per-slot outputs)
  if (f32 || dff % (4 * kChunk) != 0 || dff > 16 * kChunk || T * Nh >= (int64_t(1) << 31)) {
#define MHL_FFNG(DH, F)                                                                          \
  hipLaunchKernelGGL((ffn_kernel<DH, F, true>), dim3(kFfnGrid), dim3(kFfnThreads), 0, s, X, gate, \
                     perm, tile_info, head_base, W_in, W_in, W_out, T, Nh, Ne, k, dff, yslot);    \
  return hipGetLastError()
    if (dh == 128 && f32) { MHL_FFNG(128, true); }
    if (dh == 128) { MHL_FFNG(128, false); }
    if (f32) { MHL_FFNG(64, true); }
    MHL_FFNG(64, false);
#undef MHL_FFNG
  }
  if (dh == 64) {
#define MHL_PIPEG(NC)                                                                           \
  hipLaunchKernelGGL((ffn_pipe_kernel<64, NC, true>), dim3(kPipeGrid), dim3(kPipeWaves * kWave), \
                     0, s, (const uint16_t*)X, gate, perm, tile_info, head_base,                 \
                     (const uint16_t*)W_in, (const uint16_t*)W_in, (const uint16_t*)W_out, T,    \
                     Nh, Ne, k, (uint16_t*)yslot);                                               \
  return hipGetLastError()
    switch (dff / kChunk) {
      case 4: MHL_PIPEG(4);
      case 8: MHL_PIPEG(8);
      case 12: MHL_PIPEG(12);
      case 16: MHL_PIPEG(16);
      default: break;
    }
#undef MHL_PIPEG
    return hipErrorInvalidValue;
  }
#define MHL_Q32G(NC, W)                                                                         \
  hipLaunchKernelGGL((ffn_q32_kernel<NC, true, W>), dim3(W == 8 ? kQ32WideGrid : kQ32Grid),     \
                     dim3(Q32Layout<W>::THREADS), 0, s, (const uint16_t*)X, perm, tile_info,     \
                     head_base, (const uint16_t*)W_in, (const uint16_t*)W_in,                   \
                     (const uint16_t*)W_out, T, Nh, Ne, k, (uint16_t*)yslot);                   \
  return hipGetLastError()
  const bool wide = q32_wide(T, k, Ne);
  switch (dff / kChunk) {
    case 4: if (wide) { MHL_Q32G(4, 8); } else { MHL_Q32G(4, 4); }
    case 8: if (wide) { MHL_Q32G(8, 8); } else { MHL_Q32G(8, 4); }
    case 12: if (wide) { MHL_Q32G(12, 8); } else { MHL_Q32G(12, 4); }
    case 16: if (wide) { MHL_Q32G(16, 8); } else { MHL_Q32G(16, 4); }
    default: break;
  }
#undef MHL_Q32G
  return hipErrorInvalidValue;
}

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

hipError_t launch_combine(const void* yslot, const float* gate, int64_t T, int Nh, int dh, int k,
                          bool f32, void* Y, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dh == 128)
    return f32 ? combine_dispatch<128, true>(yslot, gate, T, Nh, k, Y, s)
               : combine_dispatch<128, false>(yslot, gate, T, Nh, k, Y, s);
  if (dh == 64)
    return f32 ? combine_dispatch<64, true>(yslot, gate, T, Nh, k, Y, s)
               : combine_dispatch<64, false>(yslot, gate, T, Nh, k, Y, s);
  return hipErrorInvalidValue;
}

}  // namespace mhl
