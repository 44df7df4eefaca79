// Batcher's odd-even merge sort and odd-even merge (K. E. Batcher, "Sorting
// networks and their applications", 1968) as compile-time unrolled
// compare-exchange networks over an array of keys held in registers.
//
// The comparator sequence is fixed by the template arguments, so every
// element index is a constant after unrolling.  cx(a, b) must leave the
// larger key in a and the smaller in b; the networks then sort descending.
// For 8 keys the sort uses 19 compare-exchanges, for 16 keys 63, and the
// merge of two sorted runs of 16 uses 65 (bitonic networks: 24, 80, 80).
//
// The header has no device dependencies so that a host test can check the
// very templates the kernels instantiate (every 0-1 input, which by the 0-1
// principle proves a comparator network sorts all inputs).
#pragma once

#if defined(__HIPCC__)
#define MHL_NET_FN __host__ __device__ inline __attribute__((always_inline))
#else
#define MHL_NET_FN inline __attribute__((always_inline))
#endif

namespace mhl {

// Merge step over v[LO .. HI] (inclusive) taken with stride R: the elements
// at even and at odd multiples of R from LO are merged recursively, then
// neighbours R apart are compared.  With R = 1 and both halves of
// v[LO .. HI] sorted, the range ends sorted.
template <int LO, int HI, int R, typename K, typename CX>
MHL_NET_FN void oe_merge(K* v, const CX& cx) {
  constexpr int STEP = 2 * R;
  if constexpr (STEP < HI - LO) {
    oe_merge<LO, HI, STEP>(v, cx);
    oe_merge<LO + R, HI, STEP>(v, cx);
#pragma unroll
    for (int i = LO + R; i < HI - R; i += STEP) cx(v[i], v[i + R]);
  } else {
    cx(v[LO], v[LO + R]);
  }
}

// Sorts v[LO .. HI] (inclusive; HI - LO + 1 a power of two).
template <int LO, int HI, typename K, typename CX>
MHL_NET_FN void oe_sort(K* v, const CX& cx) {
  if constexpr (HI - LO >= 1) {
    constexpr int MID = LO + (HI - LO) / 2;
    oe_sort<LO, MID>(v, cx);
    oe_sort<MID + 1, HI>(v, cx);
    oe_merge<LO, HI, 1>(v, cx);
  }
}

}  // namespace mhl
