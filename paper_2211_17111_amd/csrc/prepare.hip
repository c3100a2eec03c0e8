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
// The forward schedule regroups the kept points of a plan into pairs, cells,
// tiles and items (see internal.h).  Steps, all on the device:
//   1. stable radix sorts of the plan by feature rank, then by cell key
//      (Morton order of the cell), giving (cell, pixel, depth rank) order;
//   2. pair heads and cell heads by ordered compaction;
//   3. tile heads over the cells;
//   4. the distinct rows of each tile: pairs sorted by (tile, row), heads of
//      equal runs, and each pair's index into its tile's row list;
//   5. the empty cells, by compaction of an occupancy map;
//   6. items per tile, their work, and per-die item ranges;
//   7. the pairs again in pixel-major order (for the backward pass), with
//      the first pair of every feature row.

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

__device__ __forceinline__ int32_t pixel_of(int32_t p, int64_t per_view, int64_t hw) {
  return (int32_t)(((int64_t)p / per_view) * hw + (int64_t)p % hw);
}

// Spreads the low 16 bits of v to the even bit positions.
__device__ __forceinline__ uint32_t spread_bits(uint32_t v) {
  v &= 0xffffu;
  v = (v | (v << 8)) & 0x00ff00ffu;
  v = (v | (v << 4)) & 0x0f0f0f0fu;
  v = (v | (v << 2)) & 0x33333333u;
  v = (v | (v << 1)) & 0x55555555u;
  return v;
}

struct CellKey {  // BEV rank -> sort key of its cell
  int64_t XY;
  int32_t X;
  int32_t level;  // -1: the BEV rank itself
  __device__ int32_t operator()(int32_t rb) const {
    if (level < 0) return rb;
    const int32_t bz = (int32_t)(rb / XY);
    const int32_t r = (int32_t)(rb - (int64_t)bz * XY);
    const int32_t y = r / X, x = r - y * X;
    return (int32_t)(((uint32_t)bz << (2 * level)) | spread_bits((uint32_t)x) |
                     (spread_bits((uint32_t)y) << 1));
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

__global__ __launch_bounds__(256) void k_row_keys(const int32_t* __restrict__ rd, int64_t n,
                                                  int64_t per_view, int64_t hw,
                                                  int32_t* __restrict__ keys,
                                                  int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    keys[i] = pixel_of(rd[i], per_view, hw);
    vals[i] = (int32_t)i;
  }
}

__global__ __launch_bounds__(256) void k_cell_keys(const int32_t* __restrict__ rb,
                                                   const int32_t* __restrict__ vals, int64_t n,
                                                   CellKey key, int32_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) keys[i] = key(rb[vals[i]]);
}

struct PairHeads {  // runs of equal (cell, pixel) over consecutive depth bins
  const int32_t* rd;
  const int32_t* rb;
  const int32_t* vals;  // plan position of each regrouped point
  const int32_t* hdr;
  int64_t per_view, hw;
  int32_t* pair_rb;
  int32_t* pair_row;
  uint32_t* pair_dn;
  int32_t* head_pos;  // regrouped position of each pair's first point
  __device__ int64_t count() const { return hdr[kHdrValid]; }
  __device__ bool flag(int64_t i) const {
    if (i == 0) return true;
    const int32_t a = vals[i], b = vals[i - 1];
    const int32_t pa = rd[a], pb = rd[b];
    return rb[a] != rb[b] || pixel_of(pa, per_view, hw) != pixel_of(pb, per_view, hw) ||
           (int64_t)pa != (int64_t)pb + hw;
  }
  __device__ void emit(int64_t i, int32_t pos) const {
    const int32_t a = vals[i];
    const int32_t p = rd[a];
    pair_rb[pos] = rb[a];
    pair_row[pos] = pixel_of(p, per_view, hw);
    pair_dn[pos] = (uint32_t)(((int64_t)p % per_view) / hw);
    head_pos[pos] = (int32_t)i;
  }
};

__global__ __launch_bounds__(256) void k_pair_points(const int32_t* __restrict__ head_pos,
                                                     const int32_t* __restrict__ hdr,
                                                     uint32_t* __restrict__ pair_dn) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t np = hdr[kHdrPairs];
  if (p < np) {
    const int64_t next = (p + 1 < np) ? head_pos[p + 1] : hdr[kHdrValid];
    pair_dn[p] |= (uint32_t)(next - head_pos[p]) << 16;
  }
}

struct CellHeads {  // first pair of every occupied cell
  const int32_t* pair_rb;
  const int32_t* hdr;
  int32_t* cell_out;
  int32_t* cell_pair;
  int32_t cap;  // occupied cells the plan declares (n_intervals)
  __device__ int64_t count() const { return hdr[kHdrPairs]; }
  __device__ bool flag(int64_t k) const { return k == 0 || pair_rb[k] != pair_rb[k - 1]; }
  __device__ void emit(int64_t k, int32_t pos) const {
    if (pos >= cap) return;  // plan inconsistent with n_intervals: never write past the arrays
    cell_pair[pos] = (int32_t)k;
    cell_out[pos] = pair_rb[k];
  }
};

__global__ void k_cells_end(int32_t* __restrict__ hdr, int32_t* __restrict__ cell_pair) {
  if (threadIdx.x == 0 && blockIdx.x == 0)
    cell_pair[min(hdr[kHdrOcc], hdr[kHdrOccFound])] = hdr[kHdrPairs];
}

struct TileHeads {  // first cell of every tile
  const int32_t* cell_pair;
  const int32_t* hdr;
  int32_t* tile_cell;
  int32_t max_cells;
  __device__ int64_t count() const {
    return hdr[kHdrOccFound] == hdr[kHdrOcc] ? hdr[kHdrOcc] : 0;
  }
  __device__ bool big(int64_t c) const { return cell_pair[c + 1] - cell_pair[c] > kTilePairs / 2; }
  __device__ bool flag(int64_t c) const {
    if (c == 0 || c % max_cells == 0) return true;
    return big(c) || big(c - 1) || cell_pair[c] / (kTilePairs / 2) != cell_pair[c - 1] / (kTilePairs / 2);
  }
  __device__ void emit(int64_t c, int32_t pos) const { tile_cell[pos] = (int32_t)c; }
};

__global__ void k_tiles_end(const int32_t* __restrict__ hdr, int32_t* __restrict__ tile_cell) {
  if (threadIdx.x == 0 && blockIdx.x == 0) tile_cell[hdr[kHdrTiles]] = hdr[kHdrOcc];
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


// Pixel-major pairs: gather the cell and depth run of pair vals[q].
__global__ __launch_bounds__(256) void k_pix_pairs(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ vals,
                                                   const int32_t* __restrict__ pair_rb,
                                                   const uint32_t* __restrict__ pair_dn,
                                                   int32_t* __restrict__ bp_cell,
                                                   uint32_t* __restrict__ bp_dn) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kHdrPairs]) return;
  const int32_t a = vals[q];
  bp_cell[q] = pair_rb[a];
  bp_dn[q] = pair_dn[a];
}

// pix_pair0[f] = first pixel-major pair whose feature row is >= f, for f in
// [0, rows]; `keys` holds the feature row of every pixel-major pair.
__global__ __launch_bounds__(256) void k_pix_offsets(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ keys, int64_t rows,
                                                     int32_t* __restrict__ pix_pair0) {
  const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (f > rows) return;
  int32_t lo = 0, hi = hdr[kHdrPairs];
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if (keys[mid] < f) lo = mid + 1; else hi = mid;
  }
  pix_pair0[f] = lo;
}


__global__ __launch_bounds__(256) void k_pair_row_keys(const int32_t* __restrict__ hdr,
                                                       const int32_t* __restrict__ pair_row,
                                                       int32_t* __restrict__ keys,
                                                       int32_t* __restrict__ vals) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p < hdr[kHdrPairs]) {
    keys[p] = pair_row[p];
    vals[p] = (int32_t)p;
  }
}

// Tile of every pair (into pair_tile) and the (row, pair) keys of the row sort.
__global__ __launch_bounds__(256) void k_pair_tiles(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ cell_pair,
                                                    const int32_t* __restrict__ tile_cell,
                                                    const int32_t* __restrict__ pair_row,
                                                    int32_t* __restrict__ pair_tile,
                                                    int32_t* __restrict__ keys,
                                                    int32_t* __restrict__ vals) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= hdr[kHdrPairs] || hdr[kHdrOccFound] != hdr[kHdrOcc]) return;
  const int32_t c = upper_index(cell_pair, hdr[kHdrOcc], (int32_t)p);
  pair_tile[p] = upper_index(tile_cell, hdr[kHdrTiles], c);
  keys[p] = pair_row[p];
  vals[p] = (int32_t)p;
}

__global__ __launch_bounds__(256) void k_tile_keys(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ vals,
                                                   const int32_t* __restrict__ pair_tile,
                                                   int32_t* __restrict__ keys) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < hdr[kHdrPairs]) keys[q] = pair_tile[vals[q]];
}

__device__ __forceinline__ bool row_head(const int32_t* vals, const int32_t* pair_tile,
                                         const int32_t* pair_row, int64_t q) {
  if (q == 0) return true;
  const int32_t a = vals[q], b = vals[q - 1];
  return pair_tile[a] != pair_tile[b] || pair_row[a] != pair_row[b];
}

// flags[q] = 1 at the first pair of each (tile, row) run, 0 elsewhere (and
// beyond the pairs, up to cap).
__global__ __launch_bounds__(256) void k_row_flags(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ vals,
                                                   const int32_t* __restrict__ pair_tile,
                                                   const int32_t* __restrict__ pair_row,
                                                   int64_t cap, int32_t* __restrict__ flags) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= cap) return;
  flags[q] = (q < hdr[kHdrPairs] && row_head(vals, pair_tile, pair_row, q)) ? 1 : 0;
}

// With flags exclusively scanned: row entry of each sorted pair (kept in
// flags), the row list (feature rank and the pixel's depth rank at bin 0),
// and each tile's first entry.
__global__ __launch_bounds__(256) void k_row_scatter(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ vals,
                                                     const int32_t* __restrict__ pair_tile,
                                                     const int32_t* __restrict__ pair_row,
                                                     int32_t* __restrict__ flags,
                                                     int32_t* __restrict__ rows,
                                                     int32_t* __restrict__ row_dbase,
                                                     int32_t* __restrict__ tile_row0,
                                                     int64_t per_view, int64_t hw) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kHdrPairs]) return;
  const int32_t a = vals[q];
  const bool head = row_head(vals, pair_tile, pair_row, q);
  const int32_t e = flags[q] + (head ? 1 : 0) - 1;
  flags[q] = e;
  if (head) {
    const int64_t row = pair_row[a];
    rows[e] = (int32_t)row;
    row_dbase[e] = (int32_t)((row / hw) * per_view + row % hw);
  }
  if (q == 0 || pair_tile[a] != pair_tile[vals[q - 1]]) tile_row0[pair_tile[a]] = e;
}

__global__ void k_rows_end(const int32_t* __restrict__ hdr, int32_t* __restrict__ tile_row0) {
  if (threadIdx.x == 0 && blockIdx.x == 0) tile_row0[hdr[kHdrTiles]] = hdr[kHdrRowEntries];
}

__global__ __launch_bounds__(256) void k_pair_rl(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ vals,
                                                 const int32_t* __restrict__ pair_tile,
                                                 const int32_t* __restrict__ entry,
                                                 const int32_t* __restrict__ tile_row0,
                                                 uint32_t* __restrict__ pair_rl) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kHdrPairs]) return;
  const int32_t a = vals[q];
  pair_rl[a] = (uint32_t)(entry[q] - tile_row0[pair_tile[a]]);
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t* __restrict__ a, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) a[i] = v;
}

__global__ __launch_bounds__(256) void k_mark_cells(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ cell_out,
                                                    int64_t cells, int32_t* __restrict__ occ) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c < min(hdr[kHdrOcc], hdr[kHdrOccFound])) {
    const int32_t cell = cell_out[c];
    if (cell >= 0 && cell < cells) occ[cell] = 1;
  }
}

struct EmptyCells {  // BEV ranks no kept point maps to, ascending
  const int32_t* occ;
  int64_t cells;
  int32_t* empty;
  int64_t cap;
  __device__ int64_t count() const { return cells; }
  __device__ bool flag(int64_t i) const { return occ[i] == 0; }
  __device__ void emit(int64_t i, int32_t pos) const {
    if (pos < cap) empty[pos] = (int32_t)i;
  }
};

struct SliceCounts {  // channel slice counts a tile may take, ascending
  int32_t k[16];
  int32_t n;
};

// Slices of tile t: the fewest allowed K that bring its staged rows (counted
// at 4 bytes per element) within the per-item target.
__device__ __forceinline__ int32_t tile_slices(const int32_t* tile_row0, int64_t t, int64_t C,
                                               const SliceCounts& sk) {
  const int64_t rows = tile_row0[t + 1] - tile_row0[t];
  for (int i = 0; i < sk.n; ++i)
    if (rows * (C / sk.k[i]) * 4 <= kTileItemBytes) return sk.k[i];
  return sk.k[sk.n - 1];
}

__global__ __launch_bounds__(256) void k_item_counts(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ tile_row0,
                                                     int64_t C, SliceCounts sk, int64_t cap,
                                                     int32_t* __restrict__ count) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= cap) return;
  const bool ok = hdr[kHdrOccFound] == hdr[kHdrOcc] && t < hdr[kHdrTiles];
  count[t] = ok ? tile_slices(tile_row0, t, C, sk) : 0;
}

// Items in tile order; work[i] ~ staged row elements + half the pair-row
// products of the item, in units of 64 elements.
__global__ __launch_bounds__(256) void k_item_scatter(const int32_t* __restrict__ hdr,
                                                      const int32_t* __restrict__ tile_cell,
                                                      const int32_t* __restrict__ cell_pair,
                                                      const int32_t* __restrict__ tile_row0,
                                                      int64_t C, SliceCounts sk,
                                                      const int32_t* __restrict__ offset,
                                                      int32_t* __restrict__ item_tile,
                                                      int32_t* __restrict__ item_slice,
                                                      int32_t* __restrict__ work) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (hdr[kHdrOccFound] != hdr[kHdrOcc] || t >= hdr[kHdrTiles]) return;
  const int32_t K = tile_slices(tile_row0, t, C, sk);
  const int64_t rows = tile_row0[t + 1] - tile_row0[t];
  const int64_t pairs = cell_pair[tile_cell[t + 1]] - cell_pair[tile_cell[t]];
  const int64_t w = ((rows + pairs / 2) * (C / K) + 63) / 64;
  const int32_t base = offset[t];
  for (int32_t k = 0; k < K; ++k) {
    item_tile[base + k] = (int32_t)t;
    item_slice[base + k] = k | (K << 16);
    work[base + k] = (int32_t)(w < 0x3fffffff ? w : 0x3fffffff);
  }
}

__global__ __launch_bounds__(256) void k_item_work_tail(const int32_t* __restrict__ hdr,
                                                        int32_t* __restrict__ work, int64_t cap) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cap && i >= hdr[kHdrItems]) work[i] = 0;
}

// xcd_begin[x] = first item whose preceding work reaches x/8 of the total,
// so each die gets a contiguous run of items of about equal work.
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

int tile_max_cells(const Dims& d) {
  int64_t best = kTileMaxCells;
  for (int vec : {1, 4, 8}) {
    if (d.C % vec != 0) continue;
    const int64_t cs = d.C < 64 * vec ? d.C : 64 * vec;
    const int64_t m = (int64_t)(tile_max_units(vec) - 1) * tile_groups(cs, vec);
    if (m < best) best = m;
  }
  return (int)(best > 0 ? best : 1);
}

namespace {

SliceCounts slice_counts(const Dims& d) {
  SliceCounts sk{};
  sk.n = 0;
  for (int64_t k = 1; k <= d.C && sk.n < 16; ++k)
    if (d.C % k == 0 && (k == 1 || (d.C / k) % 8 == 0)) sk.k[sk.n++] = (int32_t)k;
  return sk;
}

// Morton level L (2^L >= X, Y) when (b*Z + z) << 2L | Morton(y, x) fits 31
// bits, else -1.
int morton_level(const Dims& d) {
  int L = 0;
  while ((int64_t(1) << L) < d.X || (int64_t(1) << L) < d.Y) ++L;
  if (L > 15) return -1;
  if (bit_length(d.B * d.Z) + 2 * L > 31) return -1;
  return L;
}

}  // namespace

ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals) {
  ScheduleLayout L{};
  L.n_valid = n_valid;
  L.n_occ = n_intervals;
  L.n_empty = d.cells > n_intervals ? d.cells - n_intervals : 0;
  const SliceCounts sk = slice_counts(d);
  L.items_cap = (n_intervals + 1) * sk.k[sk.n - 1];
  const size_t nv = (size_t)(n_valid > 0 ? n_valid : 1);
  const size_t nocc = (size_t)n_intervals + 1;
  size_t off = 0;
  auto take = [&](size_t n_ints) {
    const size_t o = off;
    off += align_up(sizeof(int32_t) * n_ints);
    return o;
  };
  L.header = take(16);
  L.pair_rl = take(nv);
  L.pair_dn = take(nv);
  L.cell_out = take(nocc);
  L.cell_pair = take(nocc);
  L.tile_cell = take(nocc);
  L.tile_row0 = take(nocc);
  L.rows = take(nv);
  L.row_dbase = take(nv);
  L.empty = take((size_t)L.n_empty + 1);
  L.bp_cell = take(nv);
  L.bp_dn = take(nv);
  L.pix_pair0 = take((size_t)d.rows + 1);
  L.item_tile = take((size_t)L.items_cap);
  L.item_slice = take((size_t)L.items_cap);
  L.xcd_begin = take(kXcds + 1);
  L.total = off;

  const int64_t span = std::max<int64_t>((int64_t)nv, d.cells);
  L.ntiles = (span + kPrepTile - 1) / kPrepTile;
  const int64_t scan_n = std::max<int64_t>(std::max<int64_t>(256 * L.ntiles, L.items_cap), span);
  L.nscan = (scan_n + kScanTile - 1) / kScanTile;
  off = 0;
  L.ws_ka = take(nv);
  L.ws_va = take(nv);
  L.ws_kb = take(nv);
  L.ws_vb = take(nv);
  L.ws_head = take(nv);
  L.ws_pair_rb = take(nv);
  L.ws_pair_row = take(nv);
  L.ws_flags = take((size_t)span + 1);
  L.ws_tiles = take((size_t)std::max<int64_t>(L.ntiles, nocc + L.items_cap) + 2);
  L.ws_hist = take((size_t)(256 * L.ntiles));
  L.ws_sums = take((size_t)L.nscan + 1);
  L.ws_total = off;
  L.row_bits = bit_length(d.rows);
  L.morton_level = morton_level(d);
  L.key_bits = L.morton_level < 0 ? bit_length(d.cells)
                                  : bit_length(d.B * d.Z) + 2 * L.morton_level;
  L.tile_bits = bit_length(n_intervals + 1);
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
  int32_t* hist = W(L.ws_hist);
  const dim3 grid((unsigned)L.ntiles), block(kPrepThreads);
  const unsigned g_nv = (unsigned)((n_valid + 255) / 256);

  k_sched_init<<<1, 64, 0, stream>>>(hdr, n_valid, n_intervals);

  // empty cells (also when nothing is kept)
  int32_t* occ = W(L.ws_flags);
  k_fill_i32<<<(unsigned)((d.cells + 255) / 256), 256, 0, stream>>>(occ, d.cells, 0);
  if (n_valid > 0) {
    // 1. regroup by (cell key, pixel, plan position)
    k_row_keys<<<g_nv, 256, 0, stream>>>(rd, n_valid, d.per_view, d.hw, W(L.ws_ka), W(L.ws_va));
    const bool in_b = radix_sort_pairs(W(L.ws_ka), W(L.ws_va), W(L.ws_kb), W(L.ws_vb),
                                       hdr + kHdrValid, L.ntiles, L.row_bits, hist, sums, stream);
    int32_t* k0 = in_b ? W(L.ws_kb) : W(L.ws_ka);
    int32_t* v0 = in_b ? W(L.ws_vb) : W(L.ws_va);
    int32_t* k1 = in_b ? W(L.ws_ka) : W(L.ws_kb);
    int32_t* v1 = in_b ? W(L.ws_va) : W(L.ws_vb);
    const CellKey ck{d.X * d.Y, (int32_t)d.X, L.morton_level};
    k_cell_keys<<<g_nv, 256, 0, stream>>>(rb, v0, n_valid, ck, k0);
    const bool in_1 = radix_sort_pairs(k0, v0, k1, v1, hdr + kHdrValid, L.ntiles, L.key_bits, hist,
                                       sums, stream);
    const int32_t* vals = in_1 ? v1 : v0;

    // 2. pairs and cells
    int32_t* head_pos = W(L.ws_head);
    uint32_t* pair_dn = reinterpret_cast<uint32_t*>(S(L.pair_dn));
    PairHeads ph{rd, rb, vals, hdr, d.per_view, d.hw, W(L.ws_pair_rb), W(L.ws_pair_row), pair_dn,
                 head_pos};
    k_compact_count<<<grid, block, 0, stream>>>(ph, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrPairs, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(ph, tiles);
    k_pair_points<<<g_nv, 256, 0, stream>>>(head_pos, hdr, pair_dn);
    CellHeads ch{W(L.ws_pair_rb), hdr, S(L.cell_out), S(L.cell_pair), n_intervals};
    k_compact_count<<<grid, block, 0, stream>>>(ch, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrOccFound, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(ch, tiles);
    k_cells_end<<<1, 64, 0, stream>>>(hdr, S(L.cell_pair));

    // 7 (done here, while each pair's BEV rank is at hand). Stable sort by
    // feature rank keeps the cell-key order within a pixel.
    k_pair_row_keys<<<g_nv, 256, 0, stream>>>(hdr, W(L.ws_pair_row), W(L.ws_ka), W(L.ws_va));
    const bool x_b = radix_sort_pairs(W(L.ws_ka), W(L.ws_va), W(L.ws_kb), W(L.ws_vb),
                                      hdr + kHdrPairs, L.ntiles, L.row_bits, hist, sums, stream);
    k_pix_pairs<<<g_nv, 256, 0, stream>>>(hdr, x_b ? W(L.ws_vb) : W(L.ws_va), W(L.ws_pair_rb),
                                          pair_dn, S(L.bp_cell),
                                          reinterpret_cast<uint32_t*>(S(L.bp_dn)));
    k_pix_offsets<<<(unsigned)((d.rows + 1 + 255) / 256), 256, 0, stream>>>(
        hdr, x_b ? W(L.ws_kb) : W(L.ws_ka), d.rows, S(L.pix_pair0));

    // 3. tiles
    TileHeads th{S(L.cell_pair), hdr, S(L.tile_cell), tile_max_cells(d)};
    k_compact_count<<<grid, block, 0, stream>>>(th, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrTiles, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(th, tiles);
    k_tiles_end<<<1, 64, 0, stream>>>(hdr, S(L.tile_cell));

    // 4. distinct rows per tile
    int32_t* pair_tile = W(L.ws_pair_rb);  // cell ranks are no longer needed
    k_pair_tiles<<<g_nv, 256, 0, stream>>>(hdr, S(L.cell_pair), S(L.tile_cell), W(L.ws_pair_row),
                                           pair_tile, W(L.ws_ka), W(L.ws_va));
    const bool r_b = radix_sort_pairs(W(L.ws_ka), W(L.ws_va), W(L.ws_kb), W(L.ws_vb),
                                      hdr + kHdrPairs, L.ntiles, L.row_bits, hist, sums, stream);
    int32_t* rk0 = r_b ? W(L.ws_kb) : W(L.ws_ka);
    int32_t* rv0 = r_b ? W(L.ws_vb) : W(L.ws_va);
    int32_t* rk1 = r_b ? W(L.ws_ka) : W(L.ws_kb);
    int32_t* rv1 = r_b ? W(L.ws_va) : W(L.ws_vb);
    k_tile_keys<<<g_nv, 256, 0, stream>>>(hdr, rv0, pair_tile, rk0);
    const bool t_1 = radix_sort_pairs(rk0, rv0, rk1, rv1, hdr + kHdrPairs, L.ntiles, L.tile_bits,
                                      hist, sums, stream);
    const int32_t* pvals = t_1 ? rv1 : rv0;
    int32_t* entry = W(L.ws_head);  // pair heads are no longer needed
    k_row_flags<<<g_nv, 256, 0, stream>>>(hdr, pvals, pair_tile, W(L.ws_pair_row), n_valid, entry);
    scan_exclusive(entry, n_valid, sums, hdr + kHdrRowEntries, stream);
    k_row_scatter<<<g_nv, 256, 0, stream>>>(hdr, pvals, pair_tile, W(L.ws_pair_row), entry,
                                            S(L.rows), S(L.row_dbase), S(L.tile_row0),
                                            d.per_view, d.hw);
    k_rows_end<<<1, 64, 0, stream>>>(hdr, S(L.tile_row0));
    k_pair_rl<<<g_nv, 256, 0, stream>>>(hdr, pvals, pair_tile, entry, S(L.tile_row0),
                                        reinterpret_cast<uint32_t*>(S(L.pair_rl)));
    k_mark_cells<<<(unsigned)((n_intervals + 255) / 256 + 1), 256, 0, stream>>>(hdr, S(L.cell_out),
                                                                              d.cells, occ);
  }

  // 5. empty cells
  const dim3 cgrid((unsigned)((d.cells + kPrepTile - 1) / kPrepTile));
  EmptyCells ec{occ, d.cells, S(L.empty), L.n_empty};
  k_compact_count<<<cgrid, block, 0, stream>>>(ec, tiles);
  scan_exclusive(tiles, (int64_t)cgrid.x, sums, hdr + kHdrEmpty, stream);
  k_compact_scatter<<<cgrid, block, 0, stream>>>(ec, tiles);
  if (n_valid == 0) return hipGetLastError();

  // 6. items and per-die ranges
  const SliceCounts sk = slice_counts(d);
  const int64_t tcap = n_intervals + 1;
  int32_t* count = tiles;          // [tcap]: items per tile, then their offsets
  int32_t* work = tiles + tcap;    // [items_cap]: work per item, then its prefix
  const unsigned gt = (unsigned)((tcap + 255) / 256);
  k_item_counts<<<gt, 256, 0, stream>>>(hdr, S(L.tile_row0), d.C, sk, tcap, count);
  scan_exclusive(count, tcap, sums, hdr + kHdrItems, stream);
  k_item_scatter<<<gt, 256, 0, stream>>>(hdr, S(L.tile_cell), S(L.cell_pair), S(L.tile_row0), d.C,
                                         sk, count, S(L.item_tile), S(L.item_slice), work);
  k_item_work_tail<<<(unsigned)((L.items_cap + 255) / 256), 256, 0, stream>>>(hdr, work,
                                                                            L.items_cap);
  scan_exclusive(work, L.items_cap, sums, hdr + kHdrWork, stream);
  k_xcd_bounds<<<(unsigned)((L.items_cap + 255) / 256), 256, 0, stream>>>(work, hdr,
                                                                        S(L.xcd_begin));
  return hipGetLastError();
}

}  // namespace bevpool
