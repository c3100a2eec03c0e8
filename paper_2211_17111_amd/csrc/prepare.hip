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
#include "primitives.h"

namespace bevpool {


namespace {

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
  const int64_t b = (uint32_t)p / (uint32_t)g.per_sample;  // (32-bit: P < 2^31)
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
