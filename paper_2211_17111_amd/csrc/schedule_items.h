// How a schedule cuts strips into items and shares (device helpers used by
// both schedule builders).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace bevpool {

// Share boundary w, floor(P * w / S), moved to the start or end of the strip
// [a, b) it falls in when within kMinPiece pairs of it, so that no item is
// a small remnant of a strip.
__device__ __forceinline__ int64_t snap_bound(int64_t c, int64_t a, int64_t b) {
  if (c - a < kMinPiece) return a;
  if (b - c < kMinPiece) return b;
  return c;
}

// The items of a strip with pairs [a, b): cut at the (snapped) share
// boundaries inside (a, b), and each piece of L pairs into ceil(L / ip)
// items starting at floor(i * L / K) of the piece (ip: the item size).
// visit(i, first) is called for every item start in order; returns the count.
template <typename F>
__device__ int64_t strip_items(int64_t a, int64_t b, int64_t P, int64_t S, int64_t ip, F visit) {
  // shares w with a < floor(P w / S) < b: floor(P w / S) > a  <=>
  // w >= ceil((a + 1) S / P); floor(P w / S) < b  <=>  w < ceil(b S / P)
  const int64_t w_lo = ((a + 1) * S + P - 1) / P;
  const int64_t w_hi = (b * S + P - 1) / P - 1;
  int64_t n = 0;
  int64_t q = a;
  for (int64_t w = w_lo; w <= w_hi + 1; ++w) {
    const int64_t e = w <= w_hi ? snap_bound((P * w) / S, a, b) : b;  // end of this piece
    const int64_t L = e - q;
    if (L > 0) {
      const int64_t K = (L + ip - 1) / ip;
      for (int64_t i = 0; i < K; ++i) visit(n + i, q + (i * L) / K);
      n += K;
      q = e;
    }
  }
  return n;
}

// Largest index i in [0, n) with a[i] <= v (a ascending, a[0] <= v).
__device__ __forceinline__ int32_t upper_index(const int32_t* __restrict__ a, int32_t n, int32_t v) {
  int32_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (a[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace bevpool
