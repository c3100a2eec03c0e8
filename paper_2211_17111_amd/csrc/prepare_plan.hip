// BEVPoolv2 preprocessing (section 2.1): drop the frustum points outside the
// voxel grid, sort the kept points by BEV rank with their frustum index as a
// trace (ties in frustum order), and find the interval of every occupied
// cell.
//
//   hist0      per tile of 1024 frustum points: the BEV rank of each point
//              (or drop) and the tile's histogram of the rank's low digit
//   digit scan per digit, the exclusive scan of its tile counts
//   scatter0   the kept points of each tile, stably ranked by the low digit
//              in LDS, stored at their place of the first pass: a filter
//              and a radix pass in one
//   hist1 / digit scan / scatter1   the second (last) radix pass over the
//              kept points, writing the plan's three rank arrays and the
//              point count of every cell
//   (more passes in between for grids of more than 2^16 cells)
//   intervals  one block: the cells with points in ascending order, their
//              first point (exclusive scan of the counts) and their count
//
// Every step is deterministic: tiles are ranked in element order and the
// cell counts are sums.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace bevpool {

namespace {

constexpr int kPT = 256;                 // threads per tile
constexpr int kPW = kPT / kWave;         // 4 waves
constexpr int kPR = 4;                   // rounds of 64 per wave
constexpr int kTile = kPT * kPR;         // 1024 elements per tile
constexpr int kWaveSpan = kPR * kWave;   // 256 consecutive elements per wave
constexpr int kBuckets = 256;            // most digits of a pass (8 bits)

struct PGrid {
  int64_t P;
  int32_t per_sample;  // N*D*H*W (< 2^31)
  int32_t per_view;    // D*H*W
  int32_t hw;          // H*W
  int32_t X, Y, Z;
};

// BEV rank of point p, or -1 when its voxel index lies outside the grid.
__device__ __forceinline__ int32_t rank_or_drop(const int32_t* __restrict__ coor, int64_t p,
                                                const PGrid& g) {
  const int32_t x = coor[3 * p + 0];
  const int32_t y = coor[3 * p + 1];
  const int32_t z = coor[3 * p + 2];
  const bool in = (x >= 0) & (x < g.X) & (y >= 0) & (y < g.Y) & (z >= 0) & (z < g.Z);
  if (!in) return -1;
  const int32_t b = (int32_t)((uint32_t)p / (uint32_t)g.per_sample);
  return ((b * g.Z + z) * g.Y + y) * g.X + x;
}

// Ranks of one tile held in the wave-round layout (element = tile base +
// wave * 256 + round * 64 + lane): pos[r] = the element's place among the
// tile's valid elements ordered by (digit, element), s_start[d] the first
// place of digit d, *n_tile the number of valid elements.  cnt and match are
// LDS scratch; all threads call it.
__device__ void tile_ranks(const uint32_t (&digit)[kPR], const bool (&valid)[kPR],
                           int32_t (*cnt)[kBuckets], uint32_t (*match)[kBuckets][2],
                           int32_t* s_start, int32_t* s_scan, int32_t (&pos)[kPR],
                           int32_t* n_tile) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int t = threadIdx.x;
  for (int i = t; i < kPW * kBuckets; i += kPT) (&cnt[0][0])[i] = 0;
  for (int i = t; i < kPW * kBuckets * 2; i += kPT) (&match[0][0][0])[i] = 0u;
  __syncthreads();
  // lanes with equal digits: each sets its bit in the wave's mask of its
  // digit, reads the mask back and clears it (LDS keeps one wave's order)
  uint2 m[kPR];
#pragma unroll
  for (int r = 0; r < kPR; ++r) {
    uint32_t* w = match[wid][digit[r]];
    m[r] = make_uint2(0u, 0u);
    if (valid[r]) {
      atomicOr(&w[lane >> 5], 1u << (lane & 31));
      m[r] = *reinterpret_cast<const uint2*>(w);
      *reinterpret_cast<uint2*>(w) = make_uint2(0u, 0u);
    }
  }
  // the lowest lane of each digit adds the digit's count to the wave's
  // counter; the returned value is the count in the wave's earlier rounds
  int32_t below[kPR], leader[kPR], old[kPR];
#pragma unroll
  for (int r = 0; r < kPR; ++r) {
    const uint64_t same = (uint64_t)m[r].x | ((uint64_t)m[r].y << 32);
    below[r] = rank_below(same);
    leader[r] = same != 0 ? (int32_t)__builtin_ctzll(same) : lane;
    old[r] = 0;
    if (same != 0 && below[r] == 0) old[r] = atomicAdd(&cnt[wid][digit[r]], __popcll(same));
  }
  int32_t rank[kPR];
#pragma unroll
  for (int r = 0; r < kPR; ++r) rank[r] = __shfl(old[r], leader[r], kWave) + below[r];
  __syncthreads();
  int32_t c[kPW];
  int tot = 0;  // digit t: each wave's offset within the digit, and its count
#pragma unroll
  for (int w = 0; w < kPW; ++w) c[w] = cnt[w][t];
#pragma unroll
  for (int w = 0; w < kPW; ++w) {
    const int x = c[w];
    c[w] = tot;
    tot += x;
  }
  const int start = block_exclusive_scan<kPT>(tot, s_scan, n_tile);
#pragma unroll
  for (int w = 0; w < kPW; ++w) cnt[w][t] = c[w] + start;
  s_start[t] = start;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kPR; ++r) pos[r] = cnt[wid][digit[r]] + rank[r];
}

static_assert(kBuckets == kPT, "one thread per digit");

// Pass 0 histogram over the frustum points; the tiles also clear the cell
// counts, which the last pass adds to.
__global__ __launch_bounds__(kPT) void k_pp_hist0(const int32_t* __restrict__ coor, PGrid g,
                                                  int bits, int32_t* __restrict__ hist,
                                                  int64_t ntiles, int32_t* __restrict__ cell_cnt,
                                                  int64_t cells) {
  __shared__ int32_t h[kBuckets];
  const int t = threadIdx.x;
  h[t] = 0;
  const int64_t per = (cells + ntiles - 1) / ntiles;  // cells cleared by each tile
  for (int64_t c = (int64_t)blockIdx.x * per + t; c < min<int64_t>(cells, (int64_t)(blockIdx.x + 1) * per);
       c += kPT)
    cell_cnt[c] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTile;
  const uint32_t mask = (1u << bits) - 1u;
  int32_t rk[kPR];
#pragma unroll
  for (int k = 0; k < kPR; ++k) {
    const int64_t p = base + k * kPT + t;
    rk[k] = p < g.P ? rank_or_drop(coor, p, g) : -1;
  }
#pragma unroll
  for (int k = 0; k < kPR; ++k)
    if (rk[k] >= 0) atomicAdd(&h[(uint32_t)rk[k] & mask], 1);
  __syncthreads();
  if (t <= (int)mask) hist[(int64_t)t * ntiles + blockIdx.x] = h[t];
}

// Later-pass histogram over the n kept points (tiles past n count nothing).
__global__ __launch_bounds__(kPT) void k_pp_hist(const int32_t* __restrict__ keys,
                                                 const int32_t* __restrict__ n_ptr, int shift,
                                                 int bits, int32_t* __restrict__ hist,
                                                 int64_t ntiles) {
  __shared__ int32_t h[kBuckets];
  const int t = threadIdx.x;
  h[t] = 0;
  __syncthreads();
  const int64_t n = *n_ptr;
  const int64_t base = (int64_t)blockIdx.x * kTile;
  const uint32_t mask = (1u << bits) - 1u;
#pragma unroll
  for (int k = 0; k < kPR; ++k) {
    const int64_t e = base + k * kPT + t;
    if (e < n) atomicAdd(&h[((uint32_t)keys[e] >> shift) & mask], 1);
  }
  __syncthreads();
  if (t <= (int)mask) hist[(int64_t)t * ntiles + blockIdx.x] = h[t];
}

// One block per digit: exclusive scan of the digit's tile counts in place,
// and the digit's total.
__global__ __launch_bounds__(kPT) void k_pp_digit_scan(int32_t* __restrict__ hist, int64_t ntiles,
                                                       int32_t* __restrict__ dtot) {
  __shared__ int32_t s_scan[kPW];
  int32_t* a = hist + (int64_t)blockIdx.x * ntiles;
  constexpr int kPer = 8;
  int32_t carry = 0;
  for (int64_t b0 = 0; b0 < ntiles; b0 += (int64_t)kPT * kPer) {
    const int64_t i0 = b0 + (int64_t)threadIdx.x * kPer;
    int32_t v[kPer];
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      v[k] = i0 + k < ntiles ? a[i0 + k] : 0;
      s += v[k];
    }
    int32_t tot;
    int32_t off = carry + block_exclusive_scan<kPT>(s, s_scan, &tot);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (i0 + k < ntiles) a[i0 + k] = off;
      off += v[k];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) dtot[blockIdx.x] = carry;
}

// Scatter of one radix pass.  Pass 0 reads the frustum points (filter and
// pass in one), later passes the previous pass's keys and values.  Every tile
// goes out sorted by digit through LDS, so that lanes store consecutive
// positions.  The last pass also writes each point's feature rank and counts
// the points of every cell: its LDS tile is sorted by the whole rank, and each
// run of one rank adds its length to the cell's count (the run's first
// element adds -i, its last i + 1), so that every cell takes a few adds.
template <bool FIRST>
__global__ __launch_bounds__(kPT) void k_pp_scatter(
    const int32_t* __restrict__ coor, PGrid g, const int32_t* __restrict__ keys_in,
    const int32_t* __restrict__ vals_in, const int32_t* __restrict__ n_ptr, int shift, int bits,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ dtot, int64_t ntiles,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out,
    int32_t* __restrict__ feat_out, int32_t* __restrict__ count_out,
    int32_t* __restrict__ cell_cnt) {
  __shared__ int32_t cnt[kPW][kBuckets];
  __shared__ uint32_t match[kPW][kBuckets][2];
  __shared__ int32_t s_start[kBuckets];
  __shared__ int32_t s_delta[kBuckets];
  __shared__ int32_t s_scan[kPW];
  __shared__ int32_t s_key[kTile], s_val[kTile];
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int wid = t / kWave;
  const int64_t n = FIRST ? g.P : (int64_t)*n_ptr;
  const int64_t tile0 = (int64_t)blockIdx.x * kTile;
  if (!FIRST && tile0 >= n) return;  // (uniform: a tile past the kept points)
  const int64_t base = tile0 + wid * kWaveSpan;
  const uint32_t mask = (1u << bits) - 1u;
  int32_t key[kPR], val[kPR];
  bool valid[kPR];
  uint32_t digit[kPR];
#pragma unroll
  for (int r = 0; r < kPR; ++r) {
    const int64_t e = base + r * kWave + lane;
    if (FIRST) {
      key[r] = e < n ? rank_or_drop(coor, e, g) : -1;
      val[r] = (int32_t)e;
      valid[r] = key[r] >= 0;
    } else {
      valid[r] = e < n;
      key[r] = valid[r] ? keys_in[e] : 0;
      val[r] = valid[r] ? vals_in[e] : 0;
    }
    digit[r] = ((uint32_t)key[r] >> shift) & mask;
    if (!valid[r]) digit[r] = 0;
  }
  // this tile's first place of each digit: the digit's global start (an
  // exclusive scan of the digit totals) plus the earlier tiles' counts
  const int32_t dt = t <= (int)mask ? dtot[t] : 0;
  const int32_t tile_off = t <= (int)mask ? hist[(int64_t)t * ntiles + blockIdx.x] : 0;
  int32_t n_kept;
  const int32_t dstart = block_exclusive_scan<kPT>(dt, s_scan, &n_kept);
  int32_t pos[kPR];
  int32_t n_valid_tile;
  tile_ranks(digit, valid, cnt, match, s_start, s_scan, pos, &n_valid_tile);
  s_delta[t] = dstart + tile_off - s_start[t];
#pragma unroll
  for (int r = 0; r < kPR; ++r) {
    if (valid[r]) {
      s_key[pos[r]] = key[r];
      s_val[pos[r]] = val[r];
    }
  }
  if (FIRST && blockIdx.x == 0 && t == 0) *count_out = n_kept;
  __syncthreads();
  for (int i = t; i < n_valid_tile; i += kPT) {
    const int32_t k = s_key[i];
    const int32_t v = s_val[i];
    const int32_t q = s_delta[((uint32_t)k >> shift) & mask] + i;
    keys_out[q] = k;
    vals_out[q] = v;
    if (feat_out != nullptr) {  // (last pass; 32-bit: p < 2^31)
      const uint32_t u = (uint32_t)v;
      feat_out[q] = (int32_t)((u / (uint32_t)g.per_view) * (uint32_t)g.hw + u % (uint32_t)g.hw);
      if (i == 0 || s_key[i - 1] != k) atomicAdd(&cell_cnt[k], -i);
      if (i + 1 == n_valid_tile || s_key[i + 1] != k) atomicAdd(&cell_cnt[k], i + 1);
    }
  }
}

// One block: the occupied cells in ascending order with their first point
// and point count, and the number of them.
__global__ __launch_bounds__(1024) void k_pp_intervals(const int32_t* __restrict__ cell_cnt,
                                                       int64_t cells, int64_t cap,
                                                       int32_t* __restrict__ starts,
                                                       int32_t* __restrict__ lengths,
                                                       int32_t* __restrict__ count_out) {
  constexpr int kT = 1024, kPer = 16;
  __shared__ int32_t s_scan[kT / kWave];
  int32_t carry = 0, icarry = 0;
  for (int64_t b0 = 0; b0 < cells; b0 += (int64_t)kT * kPer) {
    const int64_t i0 = b0 + (int64_t)threadIdx.x * kPer;
    int32_t v[kPer];
    if (i0 + kPer <= cells) {
      const int4* q = reinterpret_cast<const int4*>(cell_cnt + i0);
#pragma unroll
      for (int k = 0; k < kPer / 4; ++k) {
        const int4 x = q[k];
        v[4 * k] = x.x;
        v[4 * k + 1] = x.y;
        v[4 * k + 2] = x.z;
        v[4 * k + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int k = 0; k < kPer; ++k) v[k] = i0 + k < cells ? cell_cnt[i0 + k] : 0;
    }
    int32_t s = 0, o = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      s += v[k];
      o += v[k] > 0 ? 1 : 0;
    }
    int32_t tot, otot;
    int32_t off = carry + block_exclusive_scan<kT>(s, s_scan, &tot);
    int32_t ioff = icarry + block_exclusive_scan<kT>(o, s_scan, &otot);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (v[k] > 0) {
        if (ioff < cap) {
          starts[ioff] = off;
          lengths[ioff] = v[k];
        }
        ++ioff;
      }
      off += v[k];
    }
    carry += tot;
    icarry += otot;
  }
  if (threadIdx.x == 0) *count_out = icarry;
}

int bits_for_cells(int64_t cells) {  // bits of the ranks 0 .. cells - 1 (at least 1)
  int b = 1;
  while ((int64_t(1) << b) < cells) ++b;
  return b;
}

}  // namespace

PrepareLayout prepare_layout(const Dims& d) {
  PrepareLayout L{};
  L.ntiles = (d.P + kTile - 1) / kTile;
  L.key_bits = bits_for_cells(d.cells);
  L.passes = (L.key_bits + 7) / 8;
  L.digit_bits = (L.key_bits + L.passes - 1) / L.passes;
  size_t off = 0;
  auto take = [&](size_t n_ints) {
    const size_t o = off;
    off += (sizeof(int32_t) * n_ints + 255) & ~size_t(255);
    return o;
  };
  L.keys_tmp = take((size_t)d.P);
  L.vals_tmp = take((size_t)d.P);
  L.hist = take((size_t)kBuckets * (size_t)L.ntiles);
  L.digit_totals = take(kBuckets);
  L.cell_counts = take((size_t)d.cells);
  L.total = off;
  return L;
}

hipError_t launch_prepare(const Dims& d, const int32_t* coor, int32_t* ranks_depth,
                          int32_t* ranks_feat, int32_t* ranks_bev, int32_t* starts,
                          int32_t* lengths, int32_t* counts, void* workspace,
                          hipStream_t stream) {
  const PrepareLayout L = prepare_layout(d);
  char* ws = static_cast<char*>(workspace);
  auto W = [&](size_t o) { return reinterpret_cast<int32_t*>(ws + o); };
  int32_t* keys_tmp = W(L.keys_tmp);
  int32_t* vals_tmp = W(L.vals_tmp);
  int32_t* hist = W(L.hist);
  int32_t* dtot = W(L.digit_totals);
  int32_t* cell_cnt = W(L.cell_counts);
  PGrid g;
  g.P = d.P;
  g.per_sample = (int32_t)(d.N * d.per_view);
  g.per_view = (int32_t)d.per_view;
  g.hw = (int32_t)d.hw;
  g.X = (int32_t)d.X;
  g.Y = (int32_t)d.Y;
  g.Z = (int32_t)d.Z;
  const unsigned tiles = (unsigned)L.ntiles;
  // The passes alternate between the workspace and the output arrays so
  // that the last lands in (ranks_bev, ranks_depth).
  auto keys_of = [&](int pass) { return ((L.passes - 1 - pass) % 2 == 0) ? ranks_bev : keys_tmp; };
  auto vals_of = [&](int pass) { return ((L.passes - 1 - pass) % 2 == 0) ? ranks_depth : vals_tmp; };
  for (int pass = 0; pass < L.passes; ++pass) {
    const int shift = pass * L.digit_bits;
    const int bits = std::min(L.digit_bits, L.key_bits - shift);
    const bool last = pass == L.passes - 1;
    if (pass == 0)
      k_pp_hist0<<<tiles, kPT, 0, stream>>>(coor, g, bits, hist, L.ntiles, cell_cnt, d.cells);
    else
      k_pp_hist<<<tiles, kPT, 0, stream>>>(keys_of(pass - 1), counts, shift, bits, hist, L.ntiles);
    k_pp_digit_scan<<<1u << bits, kPT, 0, stream>>>(hist, L.ntiles, dtot);
    if (pass == 0)
      k_pp_scatter<true><<<tiles, kPT, 0, stream>>>(coor, g, nullptr, nullptr, nullptr, shift, bits,
                                                    hist, dtot, L.ntiles, keys_of(0), vals_of(0),
                                                    last ? ranks_feat : nullptr, counts + 0,
                                                    cell_cnt);
    else
      k_pp_scatter<false><<<tiles, kPT, 0, stream>>>(
          nullptr, g, keys_of(pass - 1), vals_of(pass - 1), counts, shift, bits, hist, dtot,
          L.ntiles, keys_of(pass), vals_of(pass), last ? ranks_feat : nullptr, nullptr, cell_cnt);
  }
  const int64_t cap = d.P < d.cells ? d.P : d.cells;
  k_pp_intervals<<<1, 1024, 0, stream>>>(cell_cnt, d.cells, cap, starts, lengths, counts + 1);
  return hipGetLastError();
}

}  // namespace bevpool
