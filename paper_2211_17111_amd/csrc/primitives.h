// Device-wide primitives shared by prepare and the schedule build: exclusive
// scan, ordered compaction and a stable LSD radix sort of (key, value) int32
// pairs.  All are deterministic and order preserving.
//
// Tiles are 4096 elements: 4 waves x 16 rounds x 64 lanes, each wave owning a
// contiguous run of 1024 elements so lane order within a round and round
// order within a wave both follow the element order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_utils.h"
#include "internal.h"

namespace bevpool {
namespace {

constexpr int kWavesPerTile = kPrepThreads / kWave;         // 4
constexpr int kWaveSpan = kPrepRounds * kWave;              // 1024
constexpr int kMaxDigitBits = 8;
constexpr int kMaxBuckets = 1 << kMaxDigitBits;


// ------------------------------------------------------------------ scan
// In-place exclusive scan of int32 data in three launches.

// Each block scans its tile and leaves the tile's total in sums; a scan of
// one tile also writes the total to total_out (if given), with no second pass.
__global__ __launch_bounds__(kScanThreads) void k_scan_local(int32_t* __restrict__ data,
                                                             int64_t cap,
                                                             int32_t* __restrict__ sums,
                                                             int32_t* __restrict__ total_out,
                                                             const int32_t* __restrict__ n_ptr) {
  __shared__ int lds[kScanThreads / kWave];
  const int64_t n = n_ptr != nullptr ? min(cap, (int64_t)max(*n_ptr, 0)) : cap;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int v[kScanItems];
  int s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + k;
    v[k] = (i < n) ? data[i] : 0;
    s += v[k];
  }
  int total;
  int off = block_exclusive_scan<kScanThreads>(s, lds, &total);
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + k;
    if (i < n) data[i] = off;
    off += v[k];
  }
  if (threadIdx.x == 0) {
    sums[blockIdx.x] = total;
    if (gridDim.x == 1 && total_out != nullptr) *total_out = total;
  }
}

__global__ __launch_bounds__(kScanThreads) void k_scan_top(int32_t* __restrict__ sums, int64_t nb,
                                                           int32_t* __restrict__ total_out) {
  __shared__ int lds[kScanThreads / kWave];
  int carry = 0;
  for (int64_t c0 = 0; c0 < nb; c0 += kScanTile) {
    const int64_t base = c0 + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
      const int64_t i = base + k;
      v[k] = (i < nb) ? sums[i] : 0;
      s += v[k];
    }
    int total;
    int off = carry + block_exclusive_scan<kScanThreads>(s, lds, &total);
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
      const int64_t i = base + k;
      if (i < nb) sums[i] = off;
      off += v[k];
    }
    carry += total;
  }
  if (threadIdx.x == 0 && total_out != nullptr) *total_out = carry;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_add(int32_t* __restrict__ data, int64_t cap,
                                                           const int32_t* __restrict__ sums,
                                                           const int32_t* __restrict__ n_ptr) {
  const int64_t n = n_ptr != nullptr ? min(cap, (int64_t)max(*n_ptr, 0)) : cap;
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  const int add = sums[blockIdx.x];
  for (int k = threadIdx.x; k < kScanTile; k += kScanThreads) {
    const int64_t i = base + k;
    if (i < n) data[i] += add;
  }
}

// Exclusive scan of data[0 .. n) in place; with n_ptr, of the first *n_ptr
// elements (n is then the capacity the grid is sized for).
void scan_exclusive(int32_t* data, int64_t n, int32_t* sums, int32_t* total_out,
                    hipStream_t stream, const int32_t* n_ptr = nullptr) {
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  if (nb == 0) {  // (an empty input: only its zero total)
    k_scan_top<<<dim3(1), dim3(kScanThreads), 0, stream>>>(sums, 0, total_out);
    return;
  }
  k_scan_local<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums, total_out,
                                                                       n_ptr);
  if (nb > 1) {
    k_scan_top<<<dim3(1), dim3(kScanThreads), 0, stream>>>(sums, nb, total_out);
    k_scan_add<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums, n_ptr);
  }
}

// ------------------------------------------------------------------ radix sort

__global__ __launch_bounds__(kPrepThreads) void k_radix_hist(const int32_t* __restrict__ keys,
                                                             const int32_t* __restrict__ n_ptr,
                                                             int shift, int nbuckets,
                                                             int32_t* __restrict__ hist,
                                                             int64_t ntiles) {
  __shared__ int h[kMaxBuckets];
  for (int i = threadIdx.x; i < kMaxBuckets; i += kPrepThreads) h[i] = 0;
  __syncthreads();
  const int64_t n = *n_ptr;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile;
  const uint32_t mask = (uint32_t)nbuckets - 1u;
#pragma unroll 4
  for (int k = 0; k < kPrepRounds; ++k) {
    const int64_t e = base + k * kPrepThreads + threadIdx.x;
    if (e < n) atomicAdd(&h[((uint32_t)keys[e] >> shift) & mask], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < nbuckets; d += kPrepThreads)
    hist[(int64_t)d * ntiles + blockIdx.x] = h[d];
}

// Stable scatter of one radix pass.  Within a wave, lanes holding the same
// digit are found with one ballot per digit bit; a per-wave running count per
// digit (in LDS) orders rounds; a prefix over the four waves orders waves;
// the scanned digit-major histogram orders tiles.  When `feat_out` is set
// (last pass) the feature rank of each point is written too.
__global__ __launch_bounds__(kPrepThreads) void k_radix_scatter(
    const int32_t* __restrict__ keys_in, const int32_t* __restrict__ vals_in,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out,
    int32_t* __restrict__ feat_out, const int32_t* __restrict__ n_ptr, int shift, int bits,
    const int32_t* __restrict__ hist_off, int64_t ntiles, int64_t per_view, int64_t hw) {
  __shared__ int cnt[kWavesPerTile][kMaxBuckets];
  __shared__ int s_delta[kMaxBuckets];  // per digit: global offset minus start in the tile
  __shared__ int s_scan[kWavesPerTile];
  __shared__ int32_t s_key[kPrepTile], s_val[kPrepTile];
  const int64_t n = *n_ptr;
  if ((int64_t)blockIdx.x * kPrepTile >= n) return;  // uniform over the block
  const int nbuckets = 1 << bits;
  for (int i = threadIdx.x; i < kWavesPerTile * kMaxBuckets; i += kPrepThreads)
    (&cnt[0][0])[i] = 0;
  __syncthreads();

  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  const uint32_t mask = (uint32_t)nbuckets - 1u;
  int32_t kreg[kPrepRounds], vreg[kPrepRounds], rank[kPrepRounds];
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t e = base + r * kWave + lane;
    const bool valid = e < n;
    const int32_t key = valid ? keys_in[e] : 0;
    const int32_t val = valid ? vals_in[e] : 0;
    const uint32_t digit = ((uint32_t)key >> shift) & mask;
    uint64_t same = wave_ballot(valid);
    for (int b = 0; b < bits; ++b) {
      const bool bit = (digit >> b) & 1u;
      const uint64_t bb = wave_ballot(bit);
      same &= bit ? bb : ~bb;
    }
    const int below = rank_below(same);
    const int prior = cnt[wid][digit];
    if (valid && below == 0) cnt[wid][digit] = prior + __popcll(same);
    rank[r] = prior + below;
    kreg[r] = key;
    vreg[r] = val;
  }
  // The tile is written out sorted by digit through LDS, so that lanes store
  // consecutive positions of one digit's run: element i of the LDS tile goes
  // to its digit's global offset plus i minus the digit's start in the tile.
  // (Positions are those of a direct scatter; only the store order differs.)
  __syncthreads();
  static_assert(kMaxBuckets == kPrepThreads, "one thread per digit");
  const int t = threadIdx.x;
  int tot_d = 0;  // digit t: each wave's offset within the digit, and its tile count
  if (t < nbuckets) {
    for (int w = 0; w < kWavesPerTile; ++w) {
      const int c = cnt[w][t];
      cnt[w][t] = tot_d;
      tot_d += c;
    }
  }
  int tile_total;
  const int start_d = block_exclusive_scan<kPrepThreads>(tot_d, s_scan, &tile_total);
  if (t < nbuckets) {
    for (int w = 0; w < kWavesPerTile; ++w) cnt[w][t] += start_d;
    s_delta[t] = hist_off[(int64_t)t * ntiles + blockIdx.x] - start_d;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t e = base + r * kWave + lane;
    if (e < n) {
      const uint32_t digit = ((uint32_t)kreg[r] >> shift) & mask;
      const int lpos = cnt[wid][digit] + rank[r];
      s_key[lpos] = kreg[r];
      s_val[lpos] = vreg[r];
    }
  }
  __syncthreads();
  const int n_tile = (int)min<int64_t>(kPrepTile, n - (int64_t)blockIdx.x * kPrepTile);
  for (int i = t; i < n_tile; i += kPrepThreads) {
    const int32_t key = s_key[i];
    const int32_t val = s_val[i];
    const int pos = s_delta[((uint32_t)key >> shift) & mask] + i;
    keys_out[pos] = key;
    vals_out[pos] = val;
    if (feat_out != nullptr) {  // (32-bit: p, D*H*W and H*W are below 2^31)
      const uint32_t u = (uint32_t)val, pv = (uint32_t)per_view, h = (uint32_t)hw;
      feat_out[pos] = (int32_t)((u / pv) * h + u % h);
    }
  }
}

// Generic ordered compaction over the same 4096-element tiles as the filter:
// Op provides count(), flag(i), and emit(i, position) (called for flagged i,
// positions in index order).
template <class Op>
__global__ __launch_bounds__(kPrepThreads) void k_compact_count(Op op, int32_t* __restrict__ tile_counts) {
  __shared__ int wave_tot[kWavesPerTile];
  const int64_t n = op.count();
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  int cnt = 0;
#pragma unroll 4
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t i = base + r * kWave + lane;
    cnt += __popcll(wave_ballot(i < n && op.flag(i)));
  }
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < kWavesPerTile; ++w) t += wave_tot[w];
    tile_counts[blockIdx.x] = t;
  }
}

template <class Op>
__global__ __launch_bounds__(kPrepThreads) void k_compact_scatter(Op op,
                                                                  const int32_t* __restrict__ tile_offsets) {
  __shared__ int wave_tot[kWavesPerTile];
  const int64_t n = op.count();
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  uint32_t flags = 0;
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t i = base + r * kWave + lane;
    const bool f = i < n && op.flag(i);
    flags |= (uint32_t)f << r;
    cnt += __popcll(wave_ballot(f));
  }
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  int off = tile_offsets[blockIdx.x];
  for (int w = 0; w < wid; ++w) off += wave_tot[w];
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const bool f = (flags >> r) & 1u;
    const uint64_t m = wave_ballot(f);
    if (f) op.emit(base + r * kWave + lane, off + rank_below(m));
    off += __popcll(m);
  }
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t* __restrict__ a, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) a[i] = v;
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

inline size_t align_up(size_t v) { return (v + 255) & ~size_t(255); }

// returns true when the sorted result ends in (k1, v1)
bool radix_sort_pairs(int32_t* k0, int32_t* v0, int32_t* k1, int32_t* v1, const int32_t* n_ptr,
                      int64_t ntiles, int key_bits, int32_t* hist, int32_t* sums,
                      hipStream_t stream) {
  const int passes = (key_bits + kMaxDigitBits - 1) / kMaxDigitBits;
  const int digit_bits = (key_bits + passes - 1) / passes;
  const dim3 grid((unsigned)ntiles), block(kPrepThreads);
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = pass * digit_bits;
    const int bits = (key_bits - shift) < digit_bits ? (key_bits - shift) : digit_bits;
    int32_t* ik = (pass % 2 == 0) ? k0 : k1;
    int32_t* iv = (pass % 2 == 0) ? v0 : v1;
    int32_t* ok = (pass % 2 == 0) ? k1 : k0;
    int32_t* ov = (pass % 2 == 0) ? v1 : v0;
    k_radix_hist<<<grid, block, 0, stream>>>(ik, n_ptr, shift, 1 << bits, hist, ntiles);
    scan_exclusive(hist, (int64_t(1) << bits) * ntiles, sums, nullptr, stream);
    k_radix_scatter<<<grid, block, 0, stream>>>(ik, iv, ok, ov, nullptr, n_ptr, shift, bits, hist,
                                                ntiles, 1, 1);
  }
  return passes % 2 == 1;
}

int bit_length(int64_t v) {
  int b = 1;
  while ((int64_t(1) << b) < v) ++b;
  return b;
}

}  // namespace
}  // namespace bevpool
