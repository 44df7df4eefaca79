// Internal launch interface between the C ABI (api.cpp) and the kernels.
// Every launcher only enqueues work on `stream` and returns the launch status;
// the shapes it receives have already been validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mhl {

// Tile descriptor of the grouped expert FFN: expert, first and one-past-last
// row of its slice of the head's clustered slot list, and the head.
struct TileInfo {
  int32_t expert;
  int32_t row_begin;
  int32_t row_end;
  int32_t head;
};

constexpr int kXcds = 8;               // accelerator dies; workgroups round-robin over them
constexpr int kTokensPerBlock = 128;   // token block of route/hist/scatter
constexpr int kTileRows = 256;         // most slot rows of one tile of the compact tile list
constexpr int kFfnRowsPerWave = 32;    // slot rows per wavefront (one MFMA column block)
// The pipelined bf16 FFN at d_h 64: 8 wavefronts cover a whole tile, one
// workgroup per CU.
constexpr int kPipeWaves = kTileRows / kFfnRowsPerWave;
constexpr int kPipeGrid = 256;
// The bf16 FFN at d_h 128: tiles of up to 128 rows, 4 wavefronts each, two
// workgroups per CU; or, where the experts see at least kQ32WideMinSlots
// slots on average, tiles of up to kTileRows rows with 8 wavefronts, one
// workgroup per CU (each pass of an expert's weights through LDS then
// serves twice the slots; below that mean, the partly filled last tile of
// each expert costs more than the halved passes save).
constexpr int kPipeTileRows = 128;
constexpr int kQ32Grid = 512;
constexpr int kQ32WideGrid = 256;
constexpr int kQ32WideMinSlots = 768;
// The other expert kernels take a tile in two halves of 4 wavefronts each,
// two workgroups per CU.
constexpr int kFfnWaves = 4;
constexpr int kHalfRows = kFfnRowsPerWave * kFfnWaves;
constexpr int kFfnGrid = 512;
constexpr int kMaxHeadsSupported = 1024;

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t num_token_blocks(int64_t T) { return ceil_div(T, kTokensPerBlock); }
// Upper bound on tiles of one head for tiles of at least kPipeTileRows rows:
// sum_e ceil(c_e / R) <= T*k/R + N_e.
__host__ __device__ inline int64_t max_tiles_per_head(int64_t T, int k, int Ne) {
  return ceil_div(T * k, kPipeTileRows) + Ne;
}

// Half h (0 or 1) of tile list entry item / 2, as a tile of at most
// kHalfRows rows (empty when the tile has no second half).
__host__ __device__ inline TileInfo half_tile(const TileInfo* tiles, int item) {
  TileInfo t = tiles[item >> 1];
  const int rb = t.row_begin + (item & 1) * kHalfRows;
  const int re = t.row_end < rb + kHalfRows ? t.row_end : rb + kHalfRows;
  t.row_begin = rb < re ? rb : re;
  t.row_end = re;
  return t;
}

// Routing forward (Algorithm 1): idx, gate and per-token-block expert
// histograms partial[h][blk][e]; also zeroes *ticket (may be NULL) for the
// clustering kernel that follows.
hipError_t launch_route_fwd(const void* X, const float* W_router,
                            const float* bias, int64_t T, int Nh, int dh,
                            int Ne, int k, bool x_f32, int32_t* idx,
                            float* gate, int32_t* partial, uint32_t* ticket,
                            hipStream_t s);

// Per-token-block expert histograms from an idx tensor; zeroes *ticket.
hipError_t launch_hist(const int32_t* idx, int64_t T, int Nh, int Ne, int k,
                       int32_t* partial, uint32_t* ticket, hipStream_t s);

// counts (always written) and, when base_rel is given, the per-block prefix
// base_rel[h][blk][e]; when offsets is given, the exclusive offsets
// [Nh][Ne+1] and (tile_start non-NULL) the prefix of per-expert tile counts
// [Nh][Ne+1] for tiles of tile_rows slots.  *ticket must be zero on entry
// when offsets is given (the preceding route or hist launch ensures it).
hipError_t launch_count_scan(const int32_t* partial, int64_t T, int Nh, int Ne,
                             int tile_rows, int32_t* counts, int32_t* base_rel,
                             int32_t* offsets, int32_t* tile_start, uint32_t* ticket,
                             hipStream_t s);

// Stable scatter of slot ids into perm[h][...].  When tile_info is given
// the same launch also writes the compact FFN tile list (head h's tiles at
// tile_info[head_base[h] ...], head_base[h] = tiles of the earlier heads,
// written with head_base[Nh] = all tiles): an expert with c slots gets
// ceil(c / tile_rows) tiles of equal size rounded up to whole 32-row blocks.
hipError_t launch_scatter(const int32_t* idx, const int32_t* base_rel,
                          const int32_t* offsets, const int32_t* tile_start,
                          int32_t* head_base, int64_t T, int Nh, int Ne, int k,
                          int tile_rows, int64_t max_tiles, int32_t* perm,
                          TileInfo* tile_info, hipStream_t s);

// Where the bf16 FFN kernel for d_h 128 runs: d_ff a multiple of 128 up to
// 512, token rows addressable with 32-bit indices.
inline bool q32_eligible(int64_t T, int Nh, int dh, int dff, bool f32) {
  return !f32 && dh == 128 && dff % 128 == 0 && dff <= 512 && T * Nh < (int64_t(1) << 31);
}

// Whether the bf16 d_h-128 FFN takes 256-row tiles: T k slots over N_e
// experts per head, at least kQ32WideMinSlots each on average.
inline bool q32_wide(int64_t T, int k, int Ne) {
  return T * k >= (int64_t)kQ32WideMinSlots * Ne;
}

// Rows per tile of the compact tile list that launch_ffn expects for this
// shape: for the bf16 kernel at d_h 128 kPipeTileRows, or kTileRows where
// q32_wide; kTileRows for the other kernels.
inline int ffn_tile_rows(int64_t T, int Nh, int dh, int Ne, int k, int dff, bool f32) {
  return q32_eligible(T, Nh, dh, dff, f32) && !q32_wide(T, k, Ne) ? kPipeTileRows : kTileRows;
}

// Grouped SwiGLU expert FFN over the compact tile list (head_base[Nh] tiles);
// writes per-slot outputs yslot[T][Nh][k][dh] with persistent workgroups,
// scaled by the slot's gate where ffn_slots_gated (the bf16 d_h-128 kernel
// leaves the gate to the combine kernel: fewer vector ALU instructions in
// the FFN, whose combine is HBM-bound anyway).
hipError_t launch_ffn(const void* X, const float* gate, const int32_t* perm,
                      const TileInfo* tile_info, const int32_t* head_base,
                      const void* W1, const void* W3, const void* W2,
                      int64_t T, int Nh, int dh, int Ne, int k, int dff,
                      bool f32, void* yslot, hipStream_t s);

// The same with the paper's two-matrix GELU expert (Sec. 3.4),
// y = W_out gelu(W_in x) (W_in in W1's layout, W_out in W2's), for every
// shape launch_ffn takes; its tile lists use ffn_tile_rows rows and its
// per-slot outputs carry the gate exactly where ffn_slots_gated says.
hipError_t launch_ffn_gelu(const void* X, const float* gate, const int32_t* perm,
                           const TileInfo* tile_info, const int32_t* head_base,
                           const void* W_in, const void* W_out, int64_t T, int Nh, int dh,
                           int Ne, int k, int dff, bool f32, void* yslot, hipStream_t s);

// Whether launch_ffn's (and launch_ffn_gelu's) per-slot outputs already
// carry the gate: false where the bf16 d_h-128 kernel runs.
inline bool ffn_slots_gated(int64_t T, int Nh, int dh, int dff, bool f32) {
  return !q32_eligible(T, Nh, dh, dff, f32);
}

// Y[t][h] = sum_j yslot[t][h][j] in j order (Eq. (1)'s sum); with gate
// non-NULL the per-slot outputs are unscaled and the sum is
// sum_j gate[t][h][j] yslot[t][h][j].
hipError_t launch_combine(const void* yslot, const float* gate, int64_t T, int Nh, int dh, int k,
                          bool f32, void* Y, hipStream_t s);

// Backward, step 1 (bf16): per-slot expert input gradient
// dxslot[T][Nh][k][dh] = W1^T da + W3^T db and dg[T][Nh][k] = <dy, W2 u>,
// recomputing the SwiGLU intermediate, over the compact tile list.  W3 ==
// NULL: the two-matrix GELU expert (dxslot = W_in^T da, u = gelu(W_in x)).
hipError_t launch_bwd_dx(const void* X, const void* dY, const float* gate, const int32_t* perm,
                         const TileInfo* tiles, const int32_t* head_base, const void* W1,
                         const void* W3, const void* W2, int64_t T, int Nh, int dh, int Ne, int k,
                         int dff, void* dxslot, float* dgslot, hipStream_t s);

// Backward, step 2: softmax backward dS[T][Nh][k] and
// dX[t][h] = sum_j dS_j W_r[h, e_j] + dxslot[t][h][j] in j order; with dR
// given (separate routing sub-tokens) the first term goes to dR instead.
hipError_t launch_bwd_combine(const int32_t* idx, const float* gate, const float* dgslot,
                              const void* dxslot, const float* W_router, int64_t T, int Nh,
                              int dh, int Ne, int k, void* dX, void* dR, float* dS,
                              hipStream_t s);

// Backward, step 3: dW1, dW3 and dW2 of every (head, expert), written in
// full (zeros where the expert received no slot).  order (Nh * Ne ints of
// workspace) receives the (head, expert) processing order, experts with the
// most slots first.  W3 == NULL: the GELU expert (dW1 = dW_in, dW2 = dW_out;
// dW3 not written).
hipError_t launch_bwd_dw(const void* X, const void* dY, const float* gate,
                         const int32_t* perm, const int32_t* offsets, int32_t* order,
                         const void* W1, const void* W3, const void* W2, int64_t T, int Nh,
                         int dh, int Ne, int k, int dff, float* dW1, float* dW3, float* dW2,
                         hipStream_t s);

// dW_router[h][e] = sum over e's slots of dS_slot R[t][h] (bf16 R, fp32 when
// f32), every (head, expert) written.  Each pair's rows are cut into segments of at most
// kRdwSeg rows; seg_base (Nh * Ne + 1 ints) and part
// (rdw_max_segments * dh floats) are workspace.
constexpr int kRdwSeg = 1024;
__host__ __device__ inline int64_t rdw_max_segments(int64_t T, int Nh, int Ne, int k) {
  return (int64_t)Nh * Ne + ceil_div((int64_t)Nh * T * k, kRdwSeg);
}
hipError_t launch_router_dw(const void* R, bool f32, const float* dS, const int32_t* perm,
                            const int32_t* offsets, int64_t T, int Nh, int dh, int Ne, int k,
                            int32_t* seg_base, float* part, float* dWr, hipStream_t s);

// Algorithm 2 from the gate gradient: dS[T][Nh][k] and
// dX[t][h] = sum_j dS_j W_r[h, e_j] (dtype bf16, or fp32 when f32).
hipError_t launch_route_bwd(const int32_t* idx, const float* gate, const float* dgate,
                            const float* W_router, int64_t T, int Nh, int dh, int Ne, int k,
                            bool f32, void* dX, float* dS, hipStream_t s);

// Auxiliary-loss-free bias update (Sec. 2.2) of every head, in place.
hipError_t launch_bias_update(const int32_t* counts, int Nh, int Ne, float rate, float* bias,
                              hipStream_t s);

// mhlmoe_route_static's scratch (for callers that cannot allocate): a
// static device array of kStaticScratchBytes that every device the library
// runs on holds until the process ends.  Writes its device address on the
// current device to *ptr (looked up on the first call per device).
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
hipError_t static_scratch(void** ptr);

// Row-major C[M][N] = op(A)[M][K] op(B)[K][N] (+ C when accumulate) through
// hipBLASLt with fp32 accumulation.  A is stored [M][K] (ta false) or [K][M]
// (ta true); B is stored [K][N] (tb false) or [N][K] (tb true).  Inputs are
// bf16 (bf16_in) or fp32; C is fp32 when f32_out, else the input type.
// blas_ws is hipBLASLt's workspace.  K == 0 writes zeros (unless accumulate).
hipError_t gemm_rowmajor(int64_t M, int64_t N, int64_t K, const void* A, bool ta, const void* B,
                         bool tb, bool bf16_in, bool f32_out, bool accumulate, void* C,
                         void* blas_ws, size_t blas_ws_bytes, hipStream_t s);
constexpr size_t kBlasWorkspace = size_t(32) << 20;

}  // namespace mhl
