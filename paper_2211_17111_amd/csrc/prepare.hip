// BEVPoolv2 preprocessing (section 2.1): filter frustum points outside the
// voxel grid, sort the rest by voxel (BEV) rank with their frustum index as a
// trace, and find the interval of every occupied voxel.
//
// Every step is deterministic and order preserving:
//   filter      ordered compaction (wave ballot + per-tile offsets)
//   sort        LSD radix sort over the BEV rank, stable per pass (wave
//               ballot multisplit inside a tile, digit-major tile histograms)
//   intervals   wave ballot on rank[i] != rank[i-1], ordered compaction
// Tiles are 4096 elements: 4 waves x 16 rounds x 64 lanes, each wave owning a
// contiguous run of 1024 elements so lane order within a round and round
// order within a wave both follow the element order.

#include <algorithm>

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

__global__ __launch_bounds__(kScanThreads) void k_scan_local(int32_t* __restrict__ data,
                                                             int64_t n,
                                                             int32_t* __restrict__ sums) {
  __shared__ int lds[kScanThreads / kWave];
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
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
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

__global__ __launch_bounds__(kScanThreads) void k_scan_add(int32_t* __restrict__ data, int64_t n,
                                                           const int32_t* __restrict__ sums) {
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  const int add = sums[blockIdx.x];
  for (int k = threadIdx.x; k < kScanTile; k += kScanThreads) {
    const int64_t i = base + k;
    if (i < n) data[i] += add;
  }
}

void scan_exclusive(int32_t* data, int64_t n, int32_t* sums, int32_t* total_out,
                    hipStream_t stream) {
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  k_scan_local<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums);
  k_scan_top<<<dim3(1), dim3(kScanThreads), 0, stream>>>(sums, nb, total_out);
  if (nb > 1) k_scan_add<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums);
}

// ------------------------------------------------------------------ filter

struct Grid {
  int64_t P;          // frustum points
  int64_t per_sample; // N*D*H*W
  int64_t per_view;   // D*H*W
  int64_t hw;         // H*W
  int32_t X, Y, Z;
};

// BEV rank of point p, or -1 when its voxel index lies outside the grid.
__device__ __forceinline__ int32_t bev_rank_or_drop(const int32_t* __restrict__ coor, int64_t p,
                                                    const Grid& g) {
  const int32_t x = coor[3 * p + 0];
  const int32_t y = coor[3 * p + 1];
  const int32_t z = coor[3 * p + 2];
  const bool in = (x >= 0) & (x < g.X) & (y >= 0) & (y < g.Y) & (z >= 0) & (z < g.Z);
  if (!in) return -1;
  const int64_t b = p / g.per_sample;
  return (int32_t)(((b * g.Z + z) * g.Y + y) * g.X + x);
}

__global__ __launch_bounds__(kPrepThreads) void k_filter_count(const int32_t* __restrict__ coor,
                                                               Grid g,
                                                               int32_t* __restrict__ tile_counts) {
  __shared__ int wave_tot[kWavesPerTile];
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  int cnt = 0;
#pragma unroll 4
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t p = base + r * kWave + lane;
    const bool keep = (p < g.P) && bev_rank_or_drop(coor, p, g) >= 0;
    cnt += __popcll(wave_ballot(keep));
  }
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < kWavesPerTile; ++w) s += wave_tot[w];
    tile_counts[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(kPrepThreads) void k_filter_scatter(
    const int32_t* __restrict__ coor, Grid g, const int32_t* __restrict__ tile_offsets,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out) {
  __shared__ int wave_tot[kWavesPerTile];
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  int32_t key[kPrepRounds];
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t p = base + r * kWave + lane;
    key[r] = (p < g.P) ? bev_rank_or_drop(coor, p, g) : -1;
    cnt += __popcll(wave_ballot(key[r] >= 0));
  }
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  int off = tile_offsets[blockIdx.x];
  for (int w = 0; w < wid; ++w) off += wave_tot[w];
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const uint64_t m = wave_ballot(key[r] >= 0);
    if (key[r] >= 0) {
      const int pos = off + rank_below(m);
      keys_out[pos] = key[r];
      vals_out[pos] = (int32_t)(base + r * kWave + lane);
    }
    off += __popcll(m);
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
  __syncthreads();
  if (threadIdx.x < nbuckets) {
    int s = 0;
    for (int w = 0; w < kWavesPerTile; ++w) {
      const int c = cnt[w][threadIdx.x];
      cnt[w][threadIdx.x] = s;
      s += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const int64_t e = base + r * kWave + lane;
    if (e < n) {
      const uint32_t digit = ((uint32_t)kreg[r] >> shift) & mask;
      const int pos = hist_off[(int64_t)digit * ntiles + blockIdx.x] + cnt[wid][digit] + rank[r];
      keys_out[pos] = kreg[r];
      vals_out[pos] = vreg[r];
      if (feat_out != nullptr) {
        const int64_t p = vreg[r];
        feat_out[pos] = (int32_t)((p / per_view) * hw + p % hw);
      }
    }
  }
}

// ------------------------------------------------------------------ intervals

__device__ __forceinline__ bool interval_head(const int32_t* __restrict__ rb, int64_t i, int64_t n) {
  return (i < n) && (i == 0 || rb[i] != rb[i - 1]);
}

__global__ __launch_bounds__(kPrepThreads) void k_interval_count(const int32_t* __restrict__ rb,
                                                                 const int32_t* __restrict__ n_ptr,
                                                                 int32_t* __restrict__ tile_counts) {
  __shared__ int wave_tot[kWavesPerTile];
  const int64_t n = *n_ptr;
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  int cnt = 0;
#pragma unroll 4
  for (int r = 0; r < kPrepRounds; ++r)
    cnt += __popcll(wave_ballot(interval_head(rb, base + r * kWave + lane, n)));
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < kWavesPerTile; ++w) s += wave_tot[w];
    tile_counts[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(kPrepThreads) void k_interval_scatter(
    const int32_t* __restrict__ rb, const int32_t* __restrict__ n_ptr,
    const int32_t* __restrict__ tile_offsets, int32_t* __restrict__ starts) {
  __shared__ int wave_tot[kWavesPerTile];
  const int64_t n = *n_ptr;
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kPrepTile + (int64_t)wid * kWaveSpan;
  uint32_t heads = 0;
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const bool h = interval_head(rb, base + r * kWave + lane, n);
    heads |= (uint32_t)h << r;
    cnt += __popcll(wave_ballot(h));
  }
  if (lane == 0) wave_tot[wid] = cnt;
  __syncthreads();
  int off = tile_offsets[blockIdx.x];
  for (int w = 0; w < wid; ++w) off += wave_tot[w];
#pragma unroll
  for (int r = 0; r < kPrepRounds; ++r) {
    const bool h = (heads >> r) & 1u;
    const uint64_t m = wave_ballot(h);
    if (h) starts[off + rank_below(m)] = (int32_t)(base + r * kWave + lane);
    off += __popcll(m);
  }
}

__global__ __launch_bounds__(256) void k_interval_lengths(const int32_t* __restrict__ starts,
                                                          int32_t* __restrict__ lengths,
                                                          const int32_t* __restrict__ counts) {
  const int64_t n = counts[0];
  const int64_t ni = counts[1];
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < ni) {
    const int64_t next = (j + 1 < ni) ? starts[j + 1] : n;
    lengths[j] = (int32_t)(next - starts[j]);
  }
}

// ------------------------------------------------------------------ schedule
//
// The forward schedule regroups the kept points of a plan by (cell, pixel):
// several depth bins of one pixel often land in the same cell, and their
// depth scores can be summed before the pixel's feature row is read once.
// The regrouping is two more stable radix sorts of the plan (by feature rank,
// then by BEV rank), after which runs of equal (BEV rank, feature rank) are
// "pairs".  Pairs are then cut into tasks that own whole cells: task k owns
// the cells whose first pair lies in [k*T, (k+1)*T).  A task with more than T
// pairs is further split by channels into several work items, which need no
// cross-item reduction because channels are independent.

// Generic ordered compaction over the same 4096-element tiles as the filter:
// Op provides count(), flag(i), visit(i) (called for every i < count) and
// emit(i, position) (called for flagged i, positions in index order).
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
    if (i < n) op.visit(i);
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

__device__ __forceinline__ int32_t pixel_of(int32_t p, int64_t per_view, int64_t hw) {
  return (int32_t)(((int64_t)p / per_view) * hw + (int64_t)p % hw);
}

struct PairHeads {  // runs of equal (BEV rank, pixel) with consecutive depth bins
  const int32_t* rd;
  const int32_t* rb;
  const int32_t* vals;  // plan position of each regrouped point
  const int32_t* hdr;
  int64_t per_view, hw;
  int32_t* pair_rd0;
  int32_t* pair_cell;
  int32_t* head_pos;   // regrouped position of each pair's first point
  __device__ int64_t count() const { return hdr[kHdrValid]; }
  __device__ bool flag(int64_t i) const {
    if (i == 0) return true;
    const int32_t a = vals[i], b = vals[i - 1];
    const int32_t pa = rd[a], pb = rd[b];
    return rb[a] != rb[b] || pixel_of(pa, per_view, hw) != pixel_of(pb, per_view, hw) ||
           (int64_t)pa != (int64_t)pb + hw;
  }
  __device__ void visit(int64_t) const {}
  __device__ void emit(int64_t i, int32_t pos) const {
    const int32_t a = vals[i];
    pair_rd0[pos] = rd[a];
    pair_cell[pos] = rb[a];
    head_pos[pos] = (int32_t)i;
  }
};

struct CellHeads {  // first pair of every occupied cell
  const int32_t* pair_cell;
  const int32_t* hdr;
  int32_t* cell_id;
  int32_t* cell_pair;
  int32_t cap;  // occupied cells the plan declares (n_intervals)
  __device__ int64_t count() const { return hdr[kHdrPairs]; }
  __device__ bool flag(int64_t k) const { return k == 0 || pair_cell[k] != pair_cell[k - 1]; }
  __device__ void visit(int64_t) const {}
  __device__ void emit(int64_t k, int32_t pos) const {
    if (pos >= cap) return;  // plan inconsistent with n_intervals: never write past the arrays
    cell_pair[pos] = (int32_t)k;
    cell_id[pos] = pair_cell[k];
  }
};

__global__ void k_sched_init(int32_t* __restrict__ hdr, int32_t n_valid, int32_t n_occ) {
  if (threadIdx.x < 16) hdr[threadIdx.x] = 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    hdr[kHdrValid] = n_valid;
    hdr[kHdrOcc] = n_occ;
  }
}

__global__ __launch_bounds__(256) void k_sched_rf_keys(const int32_t* __restrict__ rd, int64_t n,
                                                       int64_t per_view, int64_t hw,
                                                       int32_t* __restrict__ keys,
                                                       int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    keys[i] = pixel_of(rd[i], per_view, hw);
    vals[i] = (int32_t)i;
  }
}

__global__ __launch_bounds__(256) void k_sched_rb_keys(const int32_t* __restrict__ rb,
                                                       const int32_t* __restrict__ vals, int64_t n,
                                                       int32_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) keys[i] = rb[vals[i]];
}

__global__ void k_sched_sentinels(int32_t* __restrict__ hdr, int32_t* __restrict__ head_pos,
                                  int32_t* __restrict__ cell_pair) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    const int32_t np = hdr[kHdrPairs];
    head_pos[np] = hdr[kHdrValid];
    cell_pair[min(hdr[kHdrOcc], hdr[kHdrOccFound])] = np;
    hdr[kHdrTasks] = (np + kSchedTaskPairs - 1) / kSchedTaskPairs;
  }
}

__global__ __launch_bounds__(256) void k_pair_npts(const int32_t* __restrict__ head_pos,
                                                   const int32_t* __restrict__ hdr,
                                                   int32_t* __restrict__ pair_npts) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k < hdr[kHdrPairs]) pair_npts[k] = head_pos[k + 1] - head_pos[k];
}

// task_cell[k] = first occupied cell whose first pair is >= k*T.  Nothing
// is written when the plan's cell count disagrees with what was found.
__global__ __launch_bounds__(256) void k_sched_tasks(const int32_t* __restrict__ cell_pair,
                                                     const int32_t* __restrict__ hdr, int32_t n_occ,
                                                     int32_t* __restrict__ task_cell) {
  if (hdr[kHdrOccFound] != n_occ) return;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t T = kSchedTaskPairs;
  const int32_t n_tasks = hdr[kHdrTasks];
  if (j == 0) task_cell[0] = 0;
  if (j >= 1 && j < n_occ) {
    const int32_t hi = min(cell_pair[j] / T, n_tasks);
    for (int32_t k = max(cell_pair[j - 1] / T + 1, 1); k <= hi; ++k) task_cell[k] = (int32_t)j;
  } else if (j == n_occ && n_occ > 0) {
    for (int32_t k = max(cell_pair[n_occ - 1] / T + 1, 1); k <= n_tasks; ++k) task_cell[k] = n_occ;
  }
}

__device__ __forceinline__ int32_t task_chunks(const int32_t* cell_pair, const int32_t* task_cell,
                                               int64_t k, int max_chunks) {
  const int32_t w = cell_pair[task_cell[k + 1]] - cell_pair[task_cell[k]];
  if (w <= 0) return 0;
  const int32_t c = (w + kSchedTaskPairs - 1) / kSchedTaskPairs;
  return c < max_chunks ? c : max_chunks;
}

__global__ __launch_bounds__(256) void k_item_counts(const int32_t* __restrict__ cell_pair,
                                                     const int32_t* __restrict__ task_cell,
                                                     const int32_t* __restrict__ hdr, int64_t cap,
                                                     int max_chunks, int32_t* __restrict__ count) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cap) return;
  const bool ok = hdr[kHdrOccFound] == hdr[kHdrOcc] && k < hdr[kHdrTasks];
  count[k] = ok ? task_chunks(cell_pair, task_cell, k, max_chunks) : 0;
}

// Items in task order; work[i] = pairs of the item's task / its chunk count.
__global__ __launch_bounds__(256) void k_item_scatter(const int32_t* __restrict__ cell_pair,
                                                      const int32_t* __restrict__ task_cell,
                                                      int32_t* __restrict__ hdr, int max_chunks,
                                                      const int32_t* __restrict__ offset,
                                                      int32_t* __restrict__ item_info,
                                                      int32_t* __restrict__ item_chunk,
                                                      int32_t* __restrict__ work) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (hdr[kHdrOccFound] != hdr[kHdrOcc] || k >= hdr[kHdrTasks]) return;
  const int32_t K = task_chunks(cell_pair, task_cell, k, max_chunks);
  if (K == 0) return;
  const int32_t base = offset[k];
  const int32_t cb = task_cell[k], ce = task_cell[k + 1];
  const int32_t pb = cell_pair[cb], pe = cell_pair[ce];
  for (int32_t c = 0; c < K; ++c) {
    int32_t* info = item_info + 4 * (int64_t)(base + c);
    info[0] = cb;
    info[1] = ce;
    info[2] = pb;
    info[3] = pe;
    item_chunk[base + c] = c | (K << 16);
    work[base + c] = (pe - pb + K - 1) / K;
  }
}

__global__ __launch_bounds__(256) void k_item_work_tail(const int32_t* __restrict__ hdr,
                                                        int32_t* __restrict__ work, int64_t cap) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cap && i >= hdr[kHdrItems]) work[i] = 0;
}

// xcd_begin[x] = first item whose exclusive work prefix reaches x/8 of the
// total work, so each die gets a contiguous run of items of about equal work.
// `cum` holds the exclusive prefix of the per-item work.
__global__ __launch_bounds__(256) void k_xcd_bounds(const int32_t* __restrict__ cum,
                                                    const int32_t* __restrict__ hdr,
                                                    int32_t* __restrict__ xcd_begin) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = hdr[kHdrItems];
  const int64_t total = hdr[kHdrWork];
  if (i == 0) {
    xcd_begin[0] = 0;
    xcd_begin[kXcds] = (int32_t)n;
    if (n == 0)
      for (int x = 1; x < kXcds; ++x) xcd_begin[x] = 0;
  }
  if (i >= n) return;
  const int64_t lo = i > 0 ? cum[i - 1] : -1;
  const int64_t hi = cum[i];
  for (int x = 1; x < kXcds; ++x) {
    const int64_t b = (total * x + kXcds - 1) / kXcds;
    if (lo < b && b <= hi) xcd_begin[x] = (int32_t)i;
    if (i == n - 1 && b > hi) xcd_begin[x] = (int32_t)n;
  }
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

PrepareLayout prepare_layout(const Dims& d) {
  PrepareLayout L{};
  L.ntiles = (d.P + kPrepTile - 1) / kPrepTile;
  int kb = 1;
  while ((int64_t(1) << kb) < d.cells) ++kb;
  L.key_bits = kb;
  L.passes = (kb + kMaxDigitBits - 1) / kMaxDigitBits;
  L.digit_bits = (kb + L.passes - 1) / L.passes;
  const int64_t hist_entries = (int64_t(1) << L.digit_bits) * L.ntiles;
  const int64_t scan_n = hist_entries > L.ntiles ? hist_entries : L.ntiles;
  L.nscan = (scan_n + kScanTile - 1) / kScanTile;
  size_t off = 0;
  L.keys_tmp = off;    off += align_up(sizeof(int32_t) * (size_t)d.P);
  L.vals_tmp = off;    off += align_up(sizeof(int32_t) * (size_t)d.P);
  L.tile_counts = off; off += align_up(sizeof(int32_t) * (size_t)(L.ntiles + 1));
  L.hist = off;        off += align_up(sizeof(int32_t) * (size_t)hist_entries);
  L.scan_sums = off;   off += align_up(sizeof(int32_t) * (size_t)(L.nscan + 1));
  L.total = off;
  return L;
}

hipError_t launch_prepare(const Dims& d, const int32_t* coor, int32_t* ranks_depth,
                          int32_t* ranks_feat, int32_t* ranks_bev, int32_t* starts,
                          int32_t* lengths, int32_t* counts, void* workspace,
                          hipStream_t stream) {
  const PrepareLayout L = prepare_layout(d);
  char* ws = static_cast<char*>(workspace);
  int32_t* keys_tmp = reinterpret_cast<int32_t*>(ws + L.keys_tmp);
  int32_t* vals_tmp = reinterpret_cast<int32_t*>(ws + L.vals_tmp);
  int32_t* tiles = reinterpret_cast<int32_t*>(ws + L.tile_counts);
  int32_t* hist = reinterpret_cast<int32_t*>(ws + L.hist);
  int32_t* sums = reinterpret_cast<int32_t*>(ws + L.scan_sums);

  Grid g;
  g.P = d.P;
  g.per_sample = d.N * d.per_view;
  g.per_view = d.per_view;
  g.hw = d.hw;
  g.X = (int32_t)d.X;
  g.Y = (int32_t)d.Y;
  g.Z = (int32_t)d.Z;

  const dim3 grid((unsigned)L.ntiles), block(kPrepThreads);

  // filter: ordered compaction of kept points -> (BEV rank, frustum index)
  k_filter_count<<<grid, block, 0, stream>>>(coor, g, tiles);
  scan_exclusive(tiles, L.ntiles, sums, counts + 0, stream);

  // Radix passes ping-pong between the workspace and the output arrays so
  // that the last pass lands in (ranks_bev, ranks_depth).
  auto stage_keys = [&](int s) { return ((L.passes - s) % 2 == 0) ? ranks_bev : keys_tmp; };
  auto stage_vals = [&](int s) { return ((L.passes - s) % 2 == 0) ? ranks_depth : vals_tmp; };
  k_filter_scatter<<<grid, block, 0, stream>>>(coor, g, tiles, stage_keys(0), stage_vals(0));

  for (int pass = 0; pass < L.passes; ++pass) {
    const int shift = pass * L.digit_bits;
    const int bits = (L.key_bits - shift) < L.digit_bits ? (L.key_bits - shift) : L.digit_bits;
    k_radix_hist<<<grid, block, 0, stream>>>(stage_keys(pass), counts, shift, 1 << bits, hist,
                                             L.ntiles);
    scan_exclusive(hist, (int64_t(1) << bits) * L.ntiles, sums, nullptr, stream);
    const bool last = pass == L.passes - 1;
    k_radix_scatter<<<grid, block, 0, stream>>>(stage_keys(pass), stage_vals(pass),
                                                stage_keys(pass + 1), stage_vals(pass + 1),
                                                last ? ranks_feat : nullptr, counts, shift, bits,
                                                hist, L.ntiles, d.per_view, d.hw);
  }

  // intervals: heads of runs of equal BEV rank
  k_interval_count<<<grid, block, 0, stream>>>(ranks_bev, counts, tiles);
  scan_exclusive(tiles, L.ntiles, sums, counts + 1, stream);
  k_interval_scatter<<<grid, block, 0, stream>>>(ranks_bev, counts, tiles, starts);
  const int64_t cap = d.P < d.cells ? d.P : d.cells;
  k_interval_lengths<<<dim3((unsigned)((cap + 255) / 256)), dim3(256), 0, stream>>>(starts, lengths,
                                                                                   counts);
  return hipGetLastError();
}

}  // namespace bevpool

namespace bevpool {

int schedule_max_chunks(const Dims& d) { return (d.C % 16 == 0) ? (int)(d.C / 16) : 1; }

ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals) {
  ScheduleLayout L{};
  L.n_valid = n_valid;
  L.n_occ = n_intervals;
  L.tasks_cap = (n_valid + kSchedTaskPairs - 1) / kSchedTaskPairs + 1;
  L.items_cap = 2 * L.tasks_cap;
  const size_t nv = (size_t)(n_valid > 0 ? n_valid : 1);
  size_t off = 0;
  auto take = [&](size_t n_ints) {
    const size_t o = off;
    off += align_up(sizeof(int32_t) * n_ints);
    return o;
  };
  L.header = take(16);
  L.pair_rd0 = take(nv);
  L.pair_cell = take(nv);
  L.pair_npts = take(nv);
  L.cell_id = take((size_t)n_intervals + 1);
  L.cell_pair = take((size_t)n_intervals + 1);
  L.task_cell = take((size_t)L.tasks_cap + 1);
  L.item_info = take(4 * (size_t)L.items_cap);
  L.item_chunk = take((size_t)L.items_cap);
  L.xcd_begin = take(kXcds + 1);
  L.total = off;

  L.ntiles = ((int64_t)nv + kPrepTile - 1) / kPrepTile;
  const int64_t scan_n = std::max<int64_t>(256 * L.ntiles, L.items_cap);
  L.nscan = (scan_n + kScanTile - 1) / kScanTile;
  off = 0;
  L.ws_keys_a = take(nv);
  L.ws_vals_a = take(nv);
  L.ws_head = take(nv + 1);
  L.ws_keys_b = take(nv);
  L.ws_vals_b = take(nv);
  L.ws_tiles = take((size_t)std::max<int64_t>(L.ntiles, L.tasks_cap + L.items_cap) + 2);
  L.ws_hist = take((size_t)(256 * L.ntiles));
  L.ws_sums = take((size_t)L.nscan + 1);
  L.ws_total = off;
  L.rf_bits = bit_length(d.rows);
  L.rb_bits = bit_length(d.cells);
  return L;
}

hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream) {
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  char* sc = static_cast<char*>(schedule);
  char* ws = static_cast<char*>(workspace);
  auto S = [&](size_t o) { return reinterpret_cast<int32_t*>(sc + o); };
  auto W = [&](size_t o) { return reinterpret_cast<int32_t*>(ws + o); };
  int32_t* hdr = S(L.header);
  int32_t* tiles = W(L.ws_tiles);
  int32_t* sums = W(L.ws_sums);

  k_sched_init<<<1, 64, 0, stream>>>(hdr, n_valid, n_intervals);
  if (n_valid == 0) return hipGetLastError();

  // regroup by (BEV rank, feature rank, plan position)
  const unsigned g256 = (unsigned)((n_valid + 255) / 256);
  k_sched_rf_keys<<<g256, 256, 0, stream>>>(rd, n_valid, d.per_view, d.hw, W(L.ws_keys_a),
                                            W(L.ws_vals_a));
  const bool in_b = radix_sort_pairs(W(L.ws_keys_a), W(L.ws_vals_a), W(L.ws_keys_b), W(L.ws_vals_b),
                                     hdr + kHdrValid, L.ntiles, L.rf_bits, W(L.ws_hist), sums, stream);
  int32_t* k0 = in_b ? W(L.ws_keys_b) : W(L.ws_keys_a);
  int32_t* v0 = in_b ? W(L.ws_vals_b) : W(L.ws_vals_a);
  int32_t* k1 = in_b ? W(L.ws_keys_a) : W(L.ws_keys_b);
  int32_t* v1 = in_b ? W(L.ws_vals_a) : W(L.ws_vals_b);
  k_sched_rb_keys<<<g256, 256, 0, stream>>>(rb, v0, n_valid, k0);
  const bool in_1 = radix_sort_pairs(k0, v0, k1, v1, hdr + kHdrValid, L.ntiles, L.rb_bits,
                                     W(L.ws_hist), sums, stream);
  const int32_t* vals = in_1 ? v1 : v0;

  // pairs
  const dim3 grid((unsigned)L.ntiles), block(kPrepThreads);
  int32_t* head_pos = W(L.ws_head);
  PairHeads ph{rd, rb, vals, hdr, d.per_view, d.hw, S(L.pair_rd0), S(L.pair_cell), head_pos};
  k_compact_count<<<grid, block, 0, stream>>>(ph, tiles);
  scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrPairs, stream);
  k_compact_scatter<<<grid, block, 0, stream>>>(ph, tiles);

  // occupied cells
  CellHeads ch{S(L.pair_cell), hdr, S(L.cell_id), S(L.cell_pair), n_intervals};
  k_compact_count<<<grid, block, 0, stream>>>(ch, tiles);
  scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrOccFound, stream);
  k_compact_scatter<<<grid, block, 0, stream>>>(ch, tiles);
  k_sched_sentinels<<<1, 64, 0, stream>>>(hdr, head_pos, S(L.cell_pair));
  k_pair_npts<<<g256, 256, 0, stream>>>(head_pos, hdr, S(L.pair_npts));

  // tasks, work items in task order, and the per-die item ranges
  k_sched_tasks<<<(unsigned)((n_intervals + 1 + 255) / 256), 256, 0, stream>>>(
      S(L.cell_pair), hdr, n_intervals, S(L.task_cell));
  const int maxk = schedule_max_chunks(d);
  int32_t* count = tiles;                 // [tasks_cap]: items per task, then their offsets
  int32_t* work = tiles + L.tasks_cap;    // [items_cap]: work per item, then its prefix
  const unsigned gt = (unsigned)((L.tasks_cap + 255) / 256);
  k_item_counts<<<gt, 256, 0, stream>>>(S(L.cell_pair), S(L.task_cell), hdr, L.tasks_cap, maxk,
                                        count);
  scan_exclusive(count, L.tasks_cap, sums, hdr + kHdrItems, stream);
  k_item_scatter<<<gt, 256, 0, stream>>>(S(L.cell_pair), S(L.task_cell), hdr, maxk, count,
                                         S(L.item_info), S(L.item_chunk), work);
  k_item_work_tail<<<(unsigned)((L.items_cap + 255) / 256), 256, 0, stream>>>(hdr, work,
                                                                            L.items_cap);
  scan_exclusive(work, L.items_cap, sums, hdr + kHdrWork, stream);
  k_xcd_bounds<<<(unsigned)((L.items_cap + 255) / 256), 256, 0, stream>>>(work, hdr,
                                                                        S(L.xcd_begin));
  return hipGetLastError();
}

}  // namespace bevpool
