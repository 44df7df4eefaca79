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

// Persistent workgroups walk the halves of the compact tile list (work item
// i = half i % 2 of tile i / 2, at most 128 slots): XCD x (workgroups are
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

// ---------------------------------------------------------------------------
// Software-pipelined bf16 FFN (d_ff >= 64).  Per wavefront and d_ff chunk q,
// one step issues GEMM1 of chunk q+1 and GEMM2 of chunk q-1 (24 MFMAs at
// d_h 128, all independent of each other) interleaved with the SwiGLU of
// chunk q (about five VALU instructions per MFMA), so the matrix cores never
// wait for the elementwise work of the same wavefront.  Weight chunks live in
// LDS with padded rows (16 extra bytes) so every fragment read is a
// conflict-free ds_read_b128 at a constant offset from one per-lane base:
// three W1/W3 slots (chunk q+2 is stored while q and q+1 may still be read)
// and two W2 slots.  Loads for step q (W1/W3 of q+2, W2 of q) are issued at
// its start into registers and stored to LDS at its end, before the one
// barrier per step.  Chunk indices q run on across the tiles a workgroup
// processes, so the next tile's first chunks are prefetched by the last steps
// of the current one.
// ---------------------------------------------------------------------------
template <int DH>
struct PipeLayout {
  static constexpr int RS1 = DH * 2 + 16;        // W1_c / W3_c row stride (bytes)
  static constexpr int RS2 = kChunk * 2 + 16;    // regrouped W2_c row stride (bytes)
  // W1_c and W3_c blocks are each padded to whole KiB: one LDS-DMA wave
  // instruction fills 1 KiB (64 lanes x 16 bytes) of one block.
  static constexpr int DMA_PER_BLOCK = (kChunk * RS1 + 1023) / 1024;
  static constexpr int BLOCK = DMA_PER_BLOCK * 1024;
  static constexpr int W13 = 2 * BLOCK;          // one slot: W1_c block, W3_c block
  static constexpr int W2S = DH * RS2;           // one W2 slot
  static constexpr int W2_OFF = 3 * W13;
  static constexpr int TOTAL = 3 * W13 + 2 * W2S;
  static constexpr int THREADS = kPipeWaves * kWave;
  static constexpr int DMA_PER_WAVE = (2 * DMA_PER_BLOCK + kPipeWaves - 1) / kPipeWaves;
  static constexpr int U2 = DH * kChunk / 8;     // 16-byte units of W2_c
  static constexpr int N2 = (U2 + THREADS - 1) / THREADS;
  static_assert(U2 % THREADS == 0 || THREADS % U2 == 0, "uneven chunk split");
};

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Raw buffer resource over one expert's W1 (or W3): reads past num_bytes
// return zeros instead of faulting.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t expert_rsrc(const uint16_t* base, int num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, num_bytes, 0x00020000);
}

template <int DH>
struct PipeLoader {
  using L = PipeLayout<DH>;
  // Per-lane byte offsets of this wave's LDS-DMA instructions inside one
  // chunk of W1 (or W3): instruction i of the slot fills KiB i of it; the
  // lane's 16 bytes land at LDS row u / (RS1 / 16), 16-byte column
  // u % (RS1 / 16) of its block (u = its unit index); pad columns and rows
  // past the chunk load a harmless in-bounds duplicate.
  uint32_t off13[L::DMA_PER_WAVE];
  u32x4 r2[L::N2];

  __device__ __forceinline__ void init(int wave, int lane) {
    constexpr int UPR = L::RS1 / 16;  // 16-byte units per padded row
#pragma unroll
    for (int d = 0; d < L::DMA_PER_WAVE; ++d) {
      const int i = wave + kPipeWaves * d;           // instruction index in the slot
      const int u = (i % L::DMA_PER_BLOCK) * 64 + lane;  // unit inside the block
      const int row = u / UPR, col = u % UPR;
      const bool real = row < kChunk && col < DH / 8;
      off13[d] = real ? (uint32_t)((row * DH + col * 8) * 2) : 0u;
    }
  }
  // Issue the LDS-DMA of W1/W3 rows of chunk ch into one slot: wave w
  // issues instructions w, w + 8, ... (the branch is uniform per wave).
  __device__ __forceinline__ void dma13(lds_u8* slot, __amdgpu_buffer_rsrc_t w1,
                                        __amdgpu_buffer_rsrc_t w3, int ch, int wave) const {
    const int soff = ch * kChunk * DH * 2;
#pragma unroll
    for (int i = 0; i < 2 * L::DMA_PER_BLOCK; ++i) {
      if (i % kPipeWaves == wave) {
        lds_u8* dst = slot + (i / L::DMA_PER_BLOCK) * L::BLOCK + (i % L::DMA_PER_BLOCK) * 1024;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(i < L::DMA_PER_BLOCK ? w1 : w3, dst, 16,
                                                 off13[i / kPipeWaves], soff, 0, 0);
      }
    }
  }
  // W2 columns of chunk ch (W2 is [d_h][d_ff]).
  __device__ __forceinline__ void load2(const uint16_t* w2, int ch, int dff) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < L::N2; ++i) {
      const int uu = tid + L::THREADS * i;
      const int n = uu / (kChunk / 8), m = uu % (kChunk / 8);
      if (uu < L::U2)
        r2[i] = *reinterpret_cast<const u32x4*>(w2 + (int64_t)n * dff + ch * kChunk + m * 8);
    }
  }
  __device__ __forceinline__ void store2(uint8_t* slot) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < L::N2; ++i) {
      const int uu = tid + L::THREADS * i;
      if (uu >= L::U2) continue;
      const int n = uu / (kChunk / 8), m = uu % (kChunk / 8);
      const int p0 = w2_group_pos(2 * m), p1 = w2_group_pos(2 * m + 1);
      uint8_t* row = slot + n * L::RS2;
      *reinterpret_cast<u32x2*>(row + (p0 >> 1) * 16 + (p0 & 1) * 8) = u32x2{r2[i][0], r2[i][1]};
      *reinterpret_cast<u32x2*>(row + (p1 >> 1) * 16 + (p1 & 1) * 8) = u32x2{r2[i][2], r2[i][3]};
    }
  }
};

// GEMM1 of one chunk: a^T = W1_c x^T, b^T = W3_c x^T.
template <int DH>
__device__ __forceinline__ void pipe_gemm1(const uint8_t* slot, const RowFrag<DH, false>& xf,
                                           f32x16& a, f32x16& b, int lane) {
  using L = PipeLayout<DH>;
  const int g = lane >> 5, c = lane & 31;
  const uint8_t* r1 = slot + c * L::RS1 + 16 * g;
  const uint8_t* r3 = r1 + L::BLOCK;
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    const bf16x8 xb = as_bf16x8(xf.x[s]);
    a = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(r1 + 32 * s)), xb,
                    s == 0 ? zero16() : a);
    b = mfma32_bf16(as_bf16x8(*reinterpret_cast<const u32x4*>(r3 + 32 * s)), xb,
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

template <int DH>
__global__ __launch_bounds__(kPipeWaves * kWave) void ffn_pipe_kernel(
    const uint16_t* __restrict__ X, const float* __restrict__ gate,
    const int32_t* __restrict__ perm, const TileInfo* __restrict__ tiles,
    const int32_t* __restrict__ head_base, const uint16_t* __restrict__ W1,
    const uint16_t* __restrict__ W3, const uint16_t* __restrict__ W2, int64_t T,
    int Nh, int Ne, int k, int dff, uint16_t* __restrict__ yslot) {
  using L = PipeLayout<DH>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[L::TOTAL];

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
  const int nc = dff / kChunk;  // >= 2
  const int64_t wexp = (int64_t)dff * DH;  // elements of one expert's W1 (= W3 = W2)

  auto expert_off = [&](const TileInfo& ti) { return ((int64_t)ti.head * Ne + ti.expert) * wexp; };
  auto slot_of = [&](const TileInfo& ti, bool& ok) {
    const int r = ti.row_begin + wave * kFfnRowsPerWave + c;
    ok = r < ti.row_end;
    return ok ? perm[(int64_t)ti.head * head_slots + r] : 0;
  };
  auto gather = [&](const TileInfo& ti, TileRows<DH, false>& tr) {
    const int64_t t = tr.slot / k;
    const int j = tr.slot - (int)t * k;
    const int64_t tok_head = t * Nh + ti.head;
    tr.xf.load(X, tok_head, tr.ok, g);
    tr.gv = tr.ok ? gate[tok_head * k + j] : 0.f;
    tr.out_off = (tok_head * k + j) * DH;
  };

  TileInfo ti = tiles[tcur];
  TileRows<DH, false> cur;
  cur.slot = slot_of(ti, cur.ok);
  gather(ti, cur);
  int64_t eo = expert_off(ti);

  lds_u8* smem3 = (lds_u8*)smem;
  const int wexp_bytes = (int)(wexp * 2);
  __amdgpu_buffer_rsrc_t rs1 = expert_rsrc(W1 + eo, wexp_bytes);
  __amdgpu_buffer_rsrc_t rs3 = expert_rsrc(W3 + eo, wexp_bytes);
  PipeLoader<DH> ld;
  ld.init(wave, lane);
  ld.dma13(smem3, rs1, rs3, 0, wave);
  ld.dma13(smem3 + L::W13, rs1, rs3, 1, wave);
  __syncthreads();
  int q = 0;  // chunk index across this workgroup's tiles

  while (true) {
    const int tnext = tcur + nper;
    const bool has_next = tnext < t_hi;
    TileInfo tn = ti;
    TileRows<DH, false> nxt;
    nxt.ok = false;
    nxt.slot = 0;
    int64_t en = eo;
    __amdgpu_buffer_rsrc_t rn1 = rs1, rn3 = rs3;
    if (has_next) {
      tn = tiles[tnext];
      en = expert_off(tn);
      rn1 = expert_rsrc(W1 + en, wexp_bytes);
      rn3 = expert_rsrc(W3 + en, wexp_bytes);
    }
    const bool wave_active = ti.row_begin + wave * kFfnRowsPerWave < ti.row_end;

    f32x16 y[DH / 32];
#pragma unroll
    for (int nb = 0; nb < DH / 32; ++nb) y[nb] = zero16();
    f32x16 a, b;
    u32x4 hp[2];
    if (wave_active) pipe_gemm1<DH>(smem + (q % 3) * L::W13, cur.xf, a, b, lane);

    // One pipeline step for chunk ch (q = the same chunk's running index).
    // G1: issue GEMM1 of chunk ch+1; G2: issue GEMM2 of chunk ch-1.
    auto step = [&](int ch, auto g1, auto g2) {
      constexpr bool G1 = decltype(g1)::value, G2 = decltype(g2)::value;
      // loads of this step: W1/W3 of chunk q+2, W2 of chunk q
      lds_u8* slot13 = smem3 + ((q + 2) % 3) * L::W13;
      if (ch + 2 < nc) ld.dma13(slot13, rs1, rs3, ch + 2, wave);
      else if (has_next) ld.dma13(slot13, rn1, rn3, ch + 2 - nc, wave);
      ld.load2(W2 + eo, ch, dff);
      if (wave_active) {
        f32x16 a2, b2;
        u32x4 hn[2];
        if (G1) pipe_gemm1<DH>(smem + ((q + 1) % 3) * L::W13, cur.xf, a2, b2, lane);
        if (G2) pipe_gemm2<DH>(smem + L::W2_OFF + ((q - 1) & 1) * L::W2S, hp, y, lane);
        pipe_swiglu(a, b, hn);
        if (G1) {
          a = a2;
          b = b2;
        }
        hp[0] = hn[0];
        hp[1] = hn[1];
      }
      ld.store2(smem + L::W2_OFF + (q & 1) * L::W2S);
      __syncthreads();
      ++q;
    };
    using yes = std::true_type;
    using no = std::false_type;
    if (has_next) nxt.slot = slot_of(tn, nxt.ok);
    step(0, yes{}, no{});
    for (int ch = 1; ch + 1 < nc; ++ch) step(ch, yes{}, yes{});
    // the next tile's rows are gathered only now, when no GEMM1 keeps the
    // current rows live (register budget of two waves per SIMD)
    if (has_next) gather(tn, nxt);
    step(nc - 1, no{}, yes{});
    // last chunk's GEMM2 (its W2 slot was stored before the final barrier)
    if (wave_active) pipe_gemm2<DH>(smem + L::W2_OFF + ((q - 1) & 1) * L::W2S, hp, y, lane);

    // Epilogue through LDS: each wavefront stages its gate-scaled 32 x d_h
    // output tile row-major, 16 rows at a time, then writes whole 16-byte
    // pieces so that d_h / 8 lanes cover one slot's contiguous output row.
    // Staging uses the W1/W3 slot no longer needed ((q + 2) % 3) for waves
    // 0-3 and the two W2 slots for waves 4-7; barriers before (all GEMM2
    // reads done) and after (the next step's loads overwrite these slots).
    __syncthreads();
    {
      constexpr int RSY = DH * 2 + 16;  // staged row stride (bytes)
      constexpr int HALF = 16;          // rows staged at a time
      static_assert(4 * HALF * RSY <= 2 * L::W2S && 4 * HALF * RSY <= L::W13, "staging overflows");
      uint8_t* stage = wave < 4 ? smem + ((q + 2) % 3) * L::W13 + wave * HALF * RSY
                                : smem + L::W2_OFF + (wave - 4) * HALF * RSY;
#pragma unroll
      for (int part = 0; part < 2; ++part) {
        const bool mine = (c >> 4) == part;  // this lane's row is staged now
        if (wave_active && mine) {
          const int rr = c & (HALF - 1);
#pragma unroll
          for (int nb = 0; nb < DH / 32; ++nb)
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
              const int n = 32 * nb + 8 * qq + 4 * g;
              *reinterpret_cast<u32x2*>(stage + rr * RSY + n * 2) =
                  u32x2{pack_bf16x2(cur.gv * y[nb][4 * qq + 0], cur.gv * y[nb][4 * qq + 1]),
                        pack_bf16x2(cur.gv * y[nb][4 * qq + 2], cur.gv * y[nb][4 * qq + 3])};
            }
          // the row's output offset (or -1) goes into its pad bytes
          if (g == 0)
            *reinterpret_cast<int64_t*>(stage + rr * RSY + DH * 2) = cur.ok ? cur.out_off : -1;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (wave_active) {
          constexpr int UPR = DH / 8;  // 16-byte units per row
#pragma unroll
          for (int i = 0; i < HALF * UPR / kWave; ++i) {
            const int u = i * kWave + lane;
            const int r = u / UPR, jj = u % UPR;
            const int64_t o = *reinterpret_cast<const int64_t*>(stage + r * RSY + DH * 2);
            const u32x4 v = *reinterpret_cast<const u32x4*>(stage + r * RSY + jj * 16);
            if (o >= 0) *reinterpret_cast<u32x4*>(yslot + o + jj * 8) = v;
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
    __syncthreads();
    if (!has_next) break;
    ti = tn;
    cur = nxt;
    eo = en;
    rs1 = rn1;
    rs3 = rn3;
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
  if (!F32 && dff >= 2 * kChunk) {
    hipLaunchKernelGGL((ffn_pipe_kernel<DH>), dim3(kPipeGrid), dim3(kPipeWaves * kWave), 0, s,
                       (const uint16_t*)X, gate, perm, ti, head_base, (const uint16_t*)W1,
                       (const uint16_t*)W3, (const uint16_t*)W2, T, Nh, Ne, k, dff,
                       (uint16_t*)yslot);
    return hipGetLastError();
  }
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
