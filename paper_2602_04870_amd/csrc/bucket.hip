// Token clustering (Sec. 3.4, Fig. 2) for gfx950: a stable counting sort of
// every head's routed slots by expert, so that each expert's tokens form one
// contiguous run (the block-diagonal layout of the expert computation).
//
//   1. per-token-block expert histograms partial[h][blk][e] (written by the
//      routing kernel, or by hist_kernel from an idx tensor);
//   2. count_scan_kernel, one workgroup per (head, 64 experts): counts and the
//      per-block prefix base_rel[h][blk][e] = sum of partial over earlier
//      blocks, then each head's exclusive offsets and, for the expert FFN,
//      the prefix of per-expert tile counts: by the head's own workgroup when
//      it holds every expert (N_e <= 64), else by the last workgroup to finish;
//   3. scatter_kernel: each wavefront ranks its slots in (t, j) order with a
//      ballot-based match of equal experts, so ranks are deterministic and the
//      sort is stable without atomics on the output; each workgroup also
//      writes its share of the compact FFN tile list, placed after the tiles
//      of the earlier heads.

#include "device_common.hpp"
#include "launch.hpp"

namespace mhl {
namespace {

constexpr int kMaxExperts = 1024;
constexpr int kBucketThreads = 256;
constexpr int kBucketWaves = kBucketThreads / kWave;
constexpr int kScanExperts = 64;                       // experts per scan workgroup
constexpr int kScanGroups = kBucketThreads / kScanExperts;  // block groups
constexpr int kStageInts = 8192;  // counts staged per pass of the final scan
constexpr int kCachedBlocks = 16;  // per-block counts a scan thread keeps in registers
constexpr int kSlotRounds = 32 * 32 / kWave;  // 64-slot rounds per wave (32 tokens, k <= 32)
static_assert(kBucketWaves * 32 == kTokensPerBlock, "token block mismatch");

__global__ __launch_bounds__(kBucketThreads) void hist_kernel(
    const int32_t* __restrict__ idx, int64_t T, int Nh, int Ne, int k,
    int32_t* __restrict__ partial, uint32_t* __restrict__ ticket) {
  __shared__ int hist[kMaxExperts];
  const int blk = blockIdx.x, h = blockIdx.y, nblk = gridDim.x;
  const int tid = threadIdx.x;
  if (blk == 0 && h == 0 && tid == 0) *ticket = 0u;
  const int64_t t0 = (int64_t)blk * kTokensPerBlock;
  if (t0 >= T) return;  // T = 0: the launch only resets the counter
  for (int e = tid; e < Ne; e += kBucketThreads) hist[e] = 0;
  __syncthreads();
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

__device__ __forceinline__ void store_agent(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int32_t load_agent(const int32_t* p) {
  return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive offsets and tile prefix of one head from its counts cnt[0..Ne)
// (one wavefront; each lane scans per_lane consecutive experts).
__device__ __forceinline__ void scan_head(const int* cnt, int Ne, int tile_rows,
                                          int32_t* off, int32_t* ts) {
  const int lane = lane_id();
  const int per_lane = (Ne + kWave - 1) / kWave;  // <= 16
  int sc = 0, st = 0;
  for (int i = 0; i < per_lane; ++i) {
    const int ee = lane * per_lane + i;
    const int cv = ee < Ne ? cnt[ee] : 0;
    sc += cv;
    st += tile_rows > 0 ? (cv + tile_rows - 1) / tile_rows : 0;
  }
  const int ic = wave_inclusive_scan(sc), it = wave_inclusive_scan(st);
  int oc = ic - sc, ot = it - st;
  for (int i = 0; i < per_lane; ++i) {
    const int ee = lane * per_lane + i;
    if (ee < Ne) {
      const int cv = cnt[ee];
      off[ee] = oc;
      if (ts) ts[ee] = ot;
      oc += cv;
      ot += tile_rows > 0 ? (cv + tile_rows - 1) / tile_rows : 0;
    }
  }
  if (lane == kWave - 1) {
    off[Ne] = ic;
    if (ts) ts[Ne] = it;
  }
}

// Grid (ceil(Ne / 64), Nh).  Thread (g, c) of a workgroup handles expert
// 64 * blockIdx.x + c over the g-th quarter of the token blocks, keeping up
// to kCachedBlocks of its per-block counts in registers for the prefix pass.
__global__ __launch_bounds__(kBucketThreads) void count_scan_kernel(
    const int32_t* __restrict__ partial, int nblk, int Nh, int Ne, int tile_rows,
    int32_t* __restrict__ counts, int32_t* __restrict__ base_rel,
    int32_t* __restrict__ offsets, int32_t* __restrict__ tile_start,
    uint32_t* __restrict__ ticket) {
  __shared__ int sums[kScanGroups][kScanExperts];
  __shared__ int staged[kStageInts];
  __shared__ bool is_last;
  const int tid = threadIdx.x;
  const int c = tid % kScanExperts, g = tid / kScanExperts;
  const int h = blockIdx.y;
  const int e = blockIdx.x * kScanExperts + c;
  const bool ok = e < Ne;
  const int b0 = (int)((int64_t)g * nblk / kScanGroups);
  const int b1 = (int)((int64_t)(g + 1) * nblk / kScanGroups);
  const int32_t* P = partial + (int64_t)h * nblk * Ne + e;

  int v[kCachedBlocks];
  int s = 0;
  if (ok) {
#pragma unroll
    for (int i = 0; i < kCachedBlocks; ++i) v[i] = b0 + i < b1 ? P[(int64_t)(b0 + i) * Ne] : 0;
#pragma unroll
    for (int i = 0; i < kCachedBlocks; ++i) s += v[i];
    int b = b0 + kCachedBlocks;
    for (; b + 4 <= b1; b += 4) {
      const int v0 = P[(int64_t)b * Ne], v1 = P[(int64_t)(b + 1) * Ne];
      const int v2 = P[(int64_t)(b + 2) * Ne], v3 = P[(int64_t)(b + 3) * Ne];
      s += (v0 + v1) + (v2 + v3);
    }
    for (; b < b1; ++b) s += P[(int64_t)b * Ne];
  }
  sums[g][c] = s;
  __syncthreads();
  if (ok) {
    int before = 0, total = 0;
#pragma unroll
    for (int q = 0; q < kScanGroups; ++q) {
      before += q < g ? sums[q][c] : 0;
      total += sums[q][c];
    }
    if (g == 0) store_agent(&counts[(int64_t)h * Ne + e], total);
    if (base_rel) {
      int32_t* B = base_rel + (int64_t)h * nblk * Ne + e;
      int run = before;
#pragma unroll
      for (int i = 0; i < kCachedBlocks; ++i) {
        if (b0 + i < b1) {
          B[(int64_t)(b0 + i) * Ne] = run;
          run += v[i];
        }
      }
      int b = b0 + kCachedBlocks;
      for (; b + 4 <= b1; b += 4) {
        const int v0 = P[(int64_t)b * Ne], v1 = P[(int64_t)(b + 1) * Ne];
        const int v2 = P[(int64_t)(b + 2) * Ne], v3 = P[(int64_t)(b + 3) * Ne];
        B[(int64_t)b * Ne] = run;
        B[(int64_t)(b + 1) * Ne] = run + v0;
        B[(int64_t)(b + 2) * Ne] = run + v0 + v1;
        B[(int64_t)(b + 3) * Ne] = run + v0 + v1 + v2;
        run += (v0 + v1) + (v2 + v3);
      }
      for (; b < b1; ++b) {
        B[(int64_t)b * Ne] = run;
        run += P[(int64_t)b * Ne];
      }
    }
  }
  if (offsets == nullptr) return;

  if (gridDim.x == 1) {
    // This workgroup holds every expert of head h: scan them here.
    if (tid < kWave) {
      for (int ee = tid; ee < Ne; ee += kWave) {
        int tot = 0;
#pragma unroll
        for (int q = 0; q < kScanGroups; ++q) tot += sums[q][ee];
        staged[ee] = tot;
      }
      scan_head(staged, Ne, tile_rows, offsets + (int64_t)h * (Ne + 1),
                tile_start ? tile_start + (int64_t)h * (Ne + 1) : nullptr);
    }
    return;
  }

  // The last workgroup to arrive scans every head's counts: they are staged
  // in LDS with one burst of loads, then each wavefront scans whole heads.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t n = gridDim.x * gridDim.y;
    is_last = atomicAdd(ticket, 1u) == n - 1;
  }
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  const int wave = tid >> 6;
  const int heads_per_pass = kStageInts / Ne;
  for (int h0 = 0; h0 < Nh; h0 += heads_per_pass) {
    const int nh = Nh - h0 < heads_per_pass ? Nh - h0 : heads_per_pass;
    const int n = nh * Ne;
    const int32_t* src = counts + (int64_t)h0 * Ne;
    for (int i0 = 0; i0 < n; i0 += 8 * kBucketThreads) {
      int w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kBucketThreads + tid;
        w[u] = i < n ? load_agent(src + i) : 0;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kBucketThreads + tid;
        if (i < n) staged[i] = w[u];
      }
    }
    __syncthreads();
    for (int hh = wave; hh < nh; hh += kBucketWaves)
      scan_head(staged + hh * Ne, Ne, tile_rows, offsets + (int64_t)(h0 + hh) * (Ne + 1),
                tile_start ? tile_start + (int64_t)(h0 + hh) * (Ne + 1) : nullptr);
    __syncthreads();
  }
  if (tid == 0) *ticket = 0u;
}

// Grid (token blocks, Nh).  Stable placement of every slot of the block,
// then this block's share of the head's FFN tile list.
__global__ __launch_bounds__(kBucketThreads) void scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ base_rel,
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ tile_start,
    int32_t* __restrict__ head_base, int64_t T, int Nh, int Ne, int k, int ebits,
    int tile_rows, int64_t max_tiles, int32_t* __restrict__ perm,
    TileInfo* __restrict__ tile_info) {
  __shared__ int whist[kBucketWaves][kMaxExperts];
  __shared__ int s_off[kMaxExperts + 1];
  __shared__ int s_ts[kMaxExperts + 1];
  __shared__ int s_base;
  const int blk = blockIdx.x, h = blockIdx.y, nblk = gridDim.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int32_t* off_h = offsets + (int64_t)h * (Ne + 1);

  for (int i = tid; i < kBucketWaves * Ne; i += kBucketThreads)
    whist[i / Ne][i % Ne] = 0;
  for (int e = tid; e <= Ne; e += kBucketThreads) {
    s_off[e] = off_h[e];
    if (tile_info) s_ts[e] = tile_start[(int64_t)h * (Ne + 1) + e];
  }
  if (tile_info && wave == 0) {
    // this head's first tile: the tiles of every earlier head (wavefront 0
    // sums the per-head totals tile_start[h'][Ne]); the first token block of
    // each head publishes it for the FFN, the last head also the total
    int before = 0, all = 0;
    for (int h2 = lane; h2 < Nh; h2 += kWave) {
      const int n2 = tile_start[(int64_t)h2 * (Ne + 1) + Ne];
      before += h2 < h ? n2 : 0;
      all += n2;
    }
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
      before += __shfl_xor(before, d, kWave);
      all += __shfl_xor(all, d, kWave);
    }
    if (lane == 0) {
      s_base = before;
      if (blk == 0) {
        head_base[h] = before;
        if (h == Nh - 1) head_base[Nh] = all;
      }
    }
  }
  __syncthreads();
  if (T == 0) return;  // (launched only to publish the empty tile list)

  const int64_t t0 = (int64_t)blk * kTokensPerBlock + wave * 32;
  const int64_t ntok = T - t0 < 32 ? (T - t0 > 0 ? T - t0 : 0) : 32;
  const int nslot = (int)ntok * k;
  const int32_t* idx_h = idx + h * k;
  const int64_t row_stride = (int64_t)Nh * k;

  // The wave's slots (at most 32 tokens x 32) in registers, loaded at once.
  int ev[kSlotRounds];
#pragma unroll
  for (int r = 0; r < kSlotRounds; ++r) {
    const int q = r * kWave + lane;
    ev[r] = q < nslot ? idx_h[(t0 + q / k) * row_stride + q % k] : -1;
  }
#pragma unroll
  for (int r = 0; r < kSlotRounds; ++r)
    if ((unsigned)ev[r] < (unsigned)Ne) atomicAdd(&whist[wave][ev[r]], 1);
  __syncthreads();
  for (int e = tid; e < Ne; e += kBucketThreads) {
    int run = s_off[e] + base_rel[((int64_t)h * nblk + blk) * Ne + e];
#pragma unroll
    for (int w = 0; w < kBucketWaves; ++w) {
      const int cw = whist[w][e];
      whist[w][e] = run;
      run += cw;
    }
  }
  __syncthreads();

  int32_t* perm_h = perm + (int64_t)h * T * k;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int r = 0; r < kSlotRounds; ++r) {
    if (r * kWave >= nslot) break;
    const int q = r * kWave + lane;
    int e = ev[r];
    const bool valid = (unsigned)e < (unsigned)Ne;
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

  if (tile_info == nullptr) return;
  const int nt = s_ts[Ne];
  TileInfo* tiles_h = tile_info + s_base;
  const int64_t chunk = ceil_div(max_tiles, nblk);
  const int64_t q_end = (blk + 1) * chunk < nt ? (blk + 1) * chunk : nt;
  for (int64_t q = blk * chunk + tid; q < q_end; q += kBucketThreads) {
    // expert e with s_ts[e] <= q < s_ts[e + 1]
    int lo = 0, hi = Ne;  // invariant: s_ts[lo] <= q < s_ts[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_ts[mid] <= q) lo = mid; else hi = mid;
    }
    // the expert's c slots in n = ceil(c / tile_rows) tiles of equal size,
    // rounded up to 32-row blocks (never more than tile_rows, never empty)
    const int c = s_off[lo + 1] - s_off[lo];
    const int n = s_ts[lo + 1] - s_ts[lo];
    const int rpt = (((c + n - 1) / n) + 31) & ~31;
    const int r0 = s_off[lo] + (int)(q - s_ts[lo]) * rpt;
    const int r1 = r0 + rpt < s_off[lo + 1] ? r0 + rpt : s_off[lo + 1];
    tiles_h[q] = TileInfo{lo, r0, r1, h};
  }
}

// ---------------------------------------------------------------------------
// Auxiliary-loss-free load balancing (Sec. 2.2), one workgroup per head:
// the head's total load S = sum_e counts[h][e] is summed exactly in 64-bit
// integers; expert e's bias gains rate when its load is below the mean S / Ne,
// loses it when above and keeps it when equal, the comparison made exactly
// as the sign of S - Ne * counts[h][e].  Each bias changes by one fp32
// addition (round to nearest even).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBucketThreads) void bias_update_kernel(
    const int32_t* __restrict__ counts, int Ne, float rate, float* __restrict__ bias) {
  __shared__ long long sums[kBucketThreads];
  const int64_t base = (int64_t)blockIdx.x * Ne;
  long long part = 0;
  for (int e = threadIdx.x; e < Ne; e += kBucketThreads) part += counts[base + e];
  sums[threadIdx.x] = part;
  __syncthreads();
  for (int w = kBucketThreads / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) sums[threadIdx.x] += sums[threadIdx.x + w];
    __syncthreads();
  }
  const long long S = sums[0];
  for (int e = threadIdx.x; e < Ne; e += kBucketThreads) {
    const long long d = S - (long long)counts[base + e] * Ne;
    float b = bias[base + e];
    if (d > 0)
      b = b + rate;
    else if (d < 0)
      b = b - rate;
    bias[base + e] = b;
  }
}

}  // namespace

hipError_t launch_bias_update(const int32_t* counts, int Nh, int Ne, float rate, float* bias,
                              hipStream_t s) {
  hipLaunchKernelGGL(bias_update_kernel, dim3((unsigned)Nh), dim3(kBucketThreads), 0, s, counts,
                     Ne, rate, bias);
  return hipGetLastError();
}

hipError_t launch_hist(const int32_t* idx, int64_t T, int Nh, int Ne, int k,
                       int32_t* partial, uint32_t* ticket, hipStream_t s) {
  const dim3 grid(T == 0 ? 1u : (unsigned)num_token_blocks(T), T == 0 ? 1u : (unsigned)Nh);
  hipLaunchKernelGGL(hist_kernel, grid, dim3(kBucketThreads), 0, s, idx, T, Nh,
                     Ne, k, partial, ticket);
  return hipGetLastError();
}

hipError_t launch_count_scan(const int32_t* partial, int64_t T, int Nh, int Ne,
                             int tile_rows, int32_t* counts, int32_t* base_rel,
                             int32_t* offsets, int32_t* tile_start, uint32_t* ticket,
                             hipStream_t s) {
  const int nblk = (int)num_token_blocks(T);
  const dim3 grid((unsigned)ceil_div(Ne, kScanExperts), (unsigned)Nh);
  hipLaunchKernelGGL(count_scan_kernel, grid, dim3(kBucketThreads), 0, s, partial,
                     nblk, Nh, Ne, tile_rows, counts, base_rel, offsets, tile_start, ticket);
  return hipGetLastError();
}

hipError_t launch_scatter(const int32_t* idx, const int32_t* base_rel,
                          const int32_t* offsets, const int32_t* tile_start,
                          int32_t* head_base, int64_t T, int Nh, int Ne, int k,
                          int tile_rows, int64_t max_tiles, int32_t* perm,
                          TileInfo* tile_info, hipStream_t s) {
  // With T = 0 only the (empty) tile list's head_base needs writing.
  if (T == 0 && tile_info == nullptr) return hipSuccess;
  int ebits = 0;
  while ((1 << ebits) < Ne) ++ebits;
  const dim3 grid(T == 0 ? 1u : (unsigned)num_token_blocks(T), (unsigned)Nh);
  hipLaunchKernelGGL(scatter_kernel, grid, dim3(kBucketThreads), 0, s, idx,
                     base_rel, offsets, tile_start, head_base, T, Nh, Ne, k, ebits,
                     tile_rows, max_tiles, perm, tile_info);
  return hipGetLastError();
}

}  // namespace mhl
