// Wave-level helpers for CDNA (64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bevpool {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() {
  return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

__device__ __forceinline__ uint64_t wave_ballot(bool pred) {
  return __builtin_amdgcn_ballot_w64(pred);
}

// Number of set bits of `mask` in lanes below the calling lane.
__device__ __forceinline__ int rank_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(v, o, kWave);
    if (lane >= o) v += t;
  }
  return v;
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for the calling wave's outstanding global loads and stores, which
// stalls a barrier behind unrelated stores; callers that exchange data only
// through LDS (or wait for their own global copies explicitly) use this.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Exclusive scan of one int per thread over a block of NT threads.
// `lds` must hold NT/64 ints.  Writes the block total to *total (all threads).
// With LDS_ONLY its barriers leave outstanding global loads in flight.
template <int NT, bool LDS_ONLY = false>
__device__ __forceinline__ int block_exclusive_scan(int v, int* lds, int* total) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int inc = wave_inclusive_scan(v);
  if (lane == kWave - 1) lds[wid] = inc;
  if (LDS_ONLY) lds_barrier(); else __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / kWave; ++w) {
    const int s = lds[w];
    off += (w < wid) ? s : 0;
    tot += s;
  }
  if (LDS_ONLY) lds_barrier(); else __syncthreads();
  *total = tot;
  return off + inc - v;
}

}  // namespace bevpool
