// Token clustering (Sec. 3.4, Fig. 2) for gfx950: a stable counting sort of
// every head's routed slots by expert, so that each expert's tokens form one
// contiguous run (the block-diagonal layout of the expert computation).
//
//   1. per-token-block expert histograms (written by the routing kernel, or
//      by hist_kernel from an idx tensor);
//   2. count_scan_kernel: counts, exclusive offsets, the absolute scatter base
//      of every (block, expert) and the FFN tile list;
//   3. scatter_kernel: each wavefront ranks its slots in (t, j) order with a
//      ballot-based match of equal experts, so ranks are deterministic and the
//      sort is stable without atomics on the output.

#include "device_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kMaxExperts = 1024;
constexpr int kBucketThreads = 256;
constexpr int kBucketWaves = kBucketThreads / kWave;
static_assert(kBucketWaves * 32 == kTokensPerBlock, "token block mismatch");

__global__ __launch_bounds__(kBucketThreads) void hist_kernel(
    const int32_t* __restrict__ idx, int64_t T, int Nh, int Ne, int k,
    int32_t* __restrict__ partial) {
  __shared__ int hist[kMaxExperts];
  const int blk = blockIdx.x, h = blockIdx.y, nblk = gridDim.x;
  const int tid = threadIdx.x;
  for (int e = tid; e < Ne; e += kBucketThreads) hist[e] = 0;
  __syncthreads();
  const int64_t t0 = (int64_t)blk * kTokensPerBlock;
  const int64_t ntok = (T - t0) < kTokensPerBlock ? (T - t0) : kTokensPerBlock;
  const int nslot = (int)ntok * k;
  for (int q = tid; q < nslot; q += kBucketThreads) {
    const int64_t t = t0 + q / k;
    const int e = idx[(t * Nh + h) * k + q % k];
    if ((unsigned)e < (unsigned)Ne) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  int32_t* out = partial + ((int64_t)h * nblk + blk) * Ne;
  for (int e = tid; e < Ne; e += kBucketThreads) out[e] = hist[e];
}

// Exclusive scan over a 1024-thread block; returns the exclusive prefix of v
// and writes the block total to *total.
__device__ int block_exclusive_scan_1024(int v, int* wave_sums, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int inc = wave_inclusive_scan(v);
  if (lane == 63) wave_sums[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    const int ws = lane < 16 ? wave_sums[lane] : 0;
    const int wi = wave_inclusive_scan(ws);
    if (lane < 16) wave_sums[lane] = wi - ws;
    if (lane == 15) *total = wi;
  }
  __syncthreads();
  const int r = inc - v + wave_sums[wave];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(1024) void count_scan_kernel(
    const int32_t* __restrict__ partial, int nblk, int Ne, int tile_rows,
    int64_t max_tiles, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ base,
    TileInfo* __restrict__ tile_info, int32_t* __restrict__ ntiles) {
  __shared__ int wave_sums[16];
  __shared__ int totals[2];
  const int h = blockIdx.x;
  const int e = threadIdx.x;
  const int32_t* P = partial + (int64_t)h * nblk * Ne;

  int c = 0;
  if (e < Ne)
    for (int b = 0; b < nblk; ++b) c += P[(int64_t)b * Ne + e];
  const int off = block_exclusive_scan_1024(c, wave_sums, &totals[0]);
  const int nt = (tile_rows > 0 && e < Ne) ? (c + tile_rows - 1) / tile_rows : 0;
  const int toff = block_exclusive_scan_1024(nt, wave_sums, &totals[1]);

  if (e < Ne) {
    if (counts) counts[(int64_t)h * Ne + e] = c;
    if (offsets) offsets[(int64_t)h * (Ne + 1) + e] = off;
    if (base) {
      int run = off;
      for (int b = 0; b < nblk; ++b) {
        const int64_t i = (int64_t)b * Ne + e;
        const int pb = P[i];
        base[(int64_t)h * nblk * Ne + i] = run;
        run += pb;
      }
    }
    if (tile_rows > 0) {
      TileInfo* ti = tile_info + (int64_t)h * max_tiles + toff;
      for (int q = 0; q < nt; ++q) {
        const int r0 = off + q * tile_rows;
        const int r1 = (r0 + tile_rows < off + c) ? r0 + tile_rows : off + c;
        ti[q] = TileInfo{e, r0, r1, 0};
      }
    }
  }
  if (e == 0) {
    if (offsets) offsets[(int64_t)h * (Ne + 1) + Ne] = totals[0];
    if (tile_rows > 0) ntiles[h] = totals[1];
  }
}

__global__ __launch_bounds__(kBucketThreads) void scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ base, int64_t T,
    int Nh, int Ne, int k, int ebits, int32_t* __restrict__ perm) {
  __shared__ int whist[kBucketWaves][kMaxExperts];
  const int blk = blockIdx.x, h = blockIdx.y, nblk = gridDim.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  for (int i = tid; i < kBucketWaves * Ne; i += kBucketThreads)
    whist[i / Ne][i % Ne] = 0;
  __syncthreads();

  const int64_t t0 = (int64_t)blk * kTokensPerBlock + wave * 32;
  const int64_t ntok = T - t0 < 32 ? (T - t0 > 0 ? T - t0 : 0) : 32;
  const int nslot = (int)ntok * k;
  const int32_t* idx_h = idx + h * k;
  const int64_t row_stride = (int64_t)Nh * k;

  for (int q = lane; q < nslot; q += kWave) {
    const int e = idx_h[(t0 + q / k) * row_stride + q % k];
    if ((unsigned)e < (unsigned)Ne) atomicAdd(&whist[wave][e], 1);
  }
  __syncthreads();
  for (int e = tid; e < Ne; e += kBucketThreads) {
    int run = base[((int64_t)h * nblk + blk) * Ne + e];
#pragma unroll
    for (int w = 0; w < kBucketWaves; ++w) {
      const int c = whist[w][e];
      whist[w][e] = run;
      run += c;
    }
  }
  __syncthreads();

  int32_t* perm_h = perm + (int64_t)h * T * k;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int q0 = 0; q0 < nslot; q0 += kWave) {
    const int q = q0 + lane;
    const bool ok = q < nslot;
    int e = ok ? idx_h[(t0 + q / k) * row_stride + q % k] : 0;
    const bool valid = ok && (unsigned)e < (unsigned)Ne;
    if (!valid) e = 0;
    uint64_t same = __ballot(valid);
    for (int b = 0; b < ebits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    if (valid) {
      const int rank = __popcll(same & below);
      const int pos = whist[wave][e] + rank;
      perm_h[pos] = (int32_t)((t0 + q / k) * k + q % k);
      if ((same >> lane) == 1ull) whist[wave][e] += __popcll(same);
    }
  }
}

}  // namespace

hipError_t launch_hist(const int32_t* idx, int64_t T, int Nh, int Ne, int k,
                       int32_t* partial, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)num_token_blocks(T), (unsigned)Nh);
  hipLaunchKernelGGL(hist_kernel, grid, dim3(kBucketThreads), 0, s, idx, T, Nh,
                     Ne, k, partial);
  return hipGetLastError();
}

hipError_t launch_count_scan(const int32_t* partial, int64_t T, int Nh, int Ne,
                             int tile_rows, int64_t max_tiles, int32_t* counts,
                             int32_t* offsets, int32_t* base,
                             TileInfo* tile_info, int32_t* ntiles,
                             hipStream_t s) {
  const int nblk = (int)num_token_blocks(T);
  hipLaunchKernelGGL(count_scan_kernel, dim3(Nh), dim3(1024), 0, s, partial,
                     nblk, Ne, tile_rows, max_tiles, counts, offsets, base,
                     tile_info, ntiles);
  return hipGetLastError();
}

hipError_t launch_scatter(const int32_t* idx, const int32_t* base, int64_t T,
                          int Nh, int Ne, int k, int32_t* perm, hipStream_t s) {
  if (T == 0) return hipSuccess;
  int ebits = 0;
  while ((1 << ebits) < Ne) ++ebits;
  const dim3 grid((unsigned)num_token_blocks(T), (unsigned)Nh);
  hipLaunchKernelGGL(scatter_kernel, grid, dim3(kBucketThreads), 0, s, idx,
                     base, T, Nh, Ne, k, ebits, perm);
  return hipGetLastError();
}

}  // namespace mhl
