// BEVPoolv2 preprocessing (section 2.1): drop the frustum points outside the
// voxel grid, sort the kept points by BEV rank with their frustum index as a
// trace (ties in frustum order), and find the interval of every occupied
// cell.
//
//   hist0      per tile of 1536 frustum points: the BEV rank of each point
//              (or drop) and the tile's histogram of the rank's low digit
//   digit scan per digit, the exclusive scan of its tile counts
//   scatter0   the kept points of each tile, stably ranked by the low digit
//              in LDS, stored at their place of the first pass: a filter
//              and a radix pass in one
//   hist1 / digit scan / scatter1   the second (last) radix pass over the
//              kept points in tiles of 1024, writing the plan's three rank
//              arrays and the point count of every cell
//   (more passes in between for grids of more than 2^16 cells)
//   chunk totals / intervals   per chunk of cells, its point total and
//              occupied-cell count; then the cells with points in ascending
//              order, their first point (exclusive scan of the counts) and
//              their count
//
// Every step is deterministic: tiles are ranked in element order and the
// cell counts are sums.  The first pass's tiles are larger so that its grid
// (a wave per 384 frustum points) fits the GPU at once; the scatter's ranked
// tile reuses the LDS of the ranking's counters for the same reason.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"

namespace bevpool {

namespace {

constexpr int kPT = 256;                 // threads per tile
constexpr int kPW = kPT / kWave;         // 4 waves
constexpr int kR0 = 6;                   // rounds of 64 per wave in the first pass
constexpr int kR1 = 4;                   //   and in later passes
constexpr int kTile0 = kPT * kR0;        // 1536 frustum points per first-pass tile
constexpr int kTile1 = kPT * kR1;        // 1024 kept points per later tile
constexpr int kBuckets = 256;            // most digits of a pass (8 bits)

struct PGrid {
  int64_t P;
  int32_t per_sample;  // N*D*H*W (< 2^31)
  int32_t per_view;    // D*H*W
  int32_t hw;          // H*W
  int32_t X, Y, Z;
};

// BEV rank of point p with voxel index (x, y, z), or -1 when that index lies
// outside the grid.
__device__ __forceinline__ int32_t rank_xyz(int32_t x, int32_t y, int32_t z, int64_t p,
                                            const PGrid& g) {
  const bool in = (x >= 0) & (x < g.X) & (y >= 0) & (y < g.Y) & (z >= 0) & (z < g.Z);
  if (!in) return -1;
  const int32_t b = (int32_t)((uint32_t)p / (uint32_t)g.per_sample);
  return ((b * g.Z + z) * g.Y + y) * g.X + x;
}

__device__ __forceinline__ int32_t rank_or_drop(const int32_t* __restrict__ coor, int64_t p,
                                                const PGrid& g) {
  return rank_xyz(coor[3 * p + 0], coor[3 * p + 1], coor[3 * p + 2], p, g);
}

// Ranks of one tile held in the wave-round layout (element = tile base +
// wave * 64 * R + round * 64 + lane): pos[r] = the element's place among the
// tile's valid elements ordered by (digit, element), s_start[d] the first
// place of digit d, *n_tile the number of valid elements.  cnt and match are
// LDS scratch; all threads call it.  Its barriers order LDS only, so global
// loads issued before it stay in flight.  The lanes of equal digit are found
// with the LDS digit masks, or with BALLOT by one ballot per digit bit (the
// later passes: their digits repeat within a wave much more, and the lanes
// of one digit would queue their ORs on one mask word).
template <int R, bool BALLOT = false>
__device__ void tile_ranks(const uint32_t (&digit)[R], const bool (&valid)[R],
                           int32_t (*cnt)[kBuckets], uint32_t (*match)[kBuckets][2],
                           int32_t* s_start, int32_t* s_scan, int32_t (&pos)[R],
                           int32_t* n_tile, int bits = 8) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int t = threadIdx.x;
  for (int i = t; i < kPW * kBuckets; i += kPT) (&cnt[0][0])[i] = 0;
  for (int i = t; i < kPW * kBuckets * 2; i += kPT) (&match[0][0][0])[i] = 0u;
  lds_barrier();
  // lanes with equal digits: each sets its bit in the wave's mask of its
  // digit, reads the mask back and clears it (LDS keeps one wave's order)
  uint2 m[R];
  if constexpr (BALLOT) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      uint64_t same = wave_ballot(valid[r]);
      for (int b = 0; b < bits; ++b) {
        const bool on = (digit[r] >> b) & 1u;
        const uint64_t x = wave_ballot(on);
        same &= on ? x : ~x;
      }
      if (!valid[r]) same = 0;
      m[r] = make_uint2((uint32_t)same, (uint32_t)(same >> 32));
    }
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      uint32_t* w = match[wid][digit[r]];
      m[r] = make_uint2(0u, 0u);
      if (valid[r]) {
        atomicOr(&w[lane >> 5], 1u << (lane & 31));
        m[r] = *reinterpret_cast<const uint2*>(w);
        *reinterpret_cast<uint2*>(w) = make_uint2(0u, 0u);
      }
    }
  }
  // the lowest lane of each digit adds the digit's count to the wave's
  // counter; the returned value is the count in the wave's earlier rounds
  int32_t below[R], leader[R], old[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint64_t same = (uint64_t)m[r].x | ((uint64_t)m[r].y << 32);
    below[r] = rank_below(same);
    leader[r] = same != 0 ? (int32_t)__builtin_ctzll(same) : lane;
    old[r] = 0;
    if (same != 0 && below[r] == 0) old[r] = atomicAdd(&cnt[wid][digit[r]], __popcll(same));
  }
  int32_t rank[R];
#pragma unroll
  for (int r = 0; r < R; ++r) rank[r] = __shfl(old[r], leader[r], kWave) + below[r];
  lds_barrier();
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
  const int start = block_exclusive_scan<kPT, true>(tot, s_scan, n_tile);
#pragma unroll
  for (int w = 0; w < kPW; ++w) cnt[w][t] = c[w] + start;
  s_start[t] = start;
  lds_barrier();
#pragma unroll
  for (int r = 0; r < R; ++r) pos[r] = cnt[wid][digit[r]] + rank[r];
}

static_assert(kBuckets == kPT, "one thread per digit");

// Pass 0 histogram over the frustum points; the tiles also clear the cell
// counts, which the last pass adds to.  A tile's points are read in groups of
// four consecutive points per thread; with `vec` (coor 16-byte aligned) a
// whole group is three 16-byte loads.
__global__ __launch_bounds__(kPT) void k_pp_hist0(const int32_t* __restrict__ coor, PGrid g,
                                                  bool vec, int bits, int32_t* __restrict__ hist,
                                                  int64_t ntiles, int32_t* __restrict__ cell_cnt,
                                                  int64_t cells) {
  constexpr int kGroups = kTile0 / 4;                 // groups of four points per tile
  constexpr int kGPT = (kGroups + kPT - 1) / kPT;     // per thread
  __shared__ int32_t h[kBuckets];
  const int t = threadIdx.x;
  h[t] = 0;
  const int64_t per = (cells + ntiles - 1) / ntiles;  // cells cleared by each tile
  for (int64_t c = (int64_t)blockIdx.x * per + t; c < min<int64_t>(cells, (int64_t)(blockIdx.x + 1) * per);
       c += kPT)
    cell_cnt[c] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTile0;
  const uint32_t mask = (1u << bits) - 1u;
  int32_t rk[kGPT][4];
#pragma unroll
  for (int j = 0; j < kGPT; ++j) {
    const int grp = t + j * kPT;
    const int64_t p0 = base + 4 * grp;
    if (grp < kGroups && vec && p0 + 4 <= g.P) {
      const int4* q = reinterpret_cast<const int4*>(coor + 3 * p0);
      const int4 a = q[0], b = q[1], c = q[2];
      rk[j][0] = rank_xyz(a.x, a.y, a.z, p0 + 0, g);
      rk[j][1] = rank_xyz(a.w, b.x, b.y, p0 + 1, g);
      rk[j][2] = rank_xyz(b.z, b.w, c.x, p0 + 2, g);
      rk[j][3] = rank_xyz(c.y, c.z, c.w, p0 + 3, g);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        rk[j][k] = grp < kGroups && p0 + k < g.P ? rank_or_drop(coor, p0 + k, g) : -1;
    }
  }
#pragma unroll
  for (int j = 0; j < kGPT; ++j)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (rk[j][k] >= 0) atomicAdd(&h[(uint32_t)rk[j][k] & mask], 1);
  __syncthreads();
  if (t <= (int)mask) hist[(int64_t)t * ntiles + blockIdx.x] = h[t];
}

// Later-pass histogram over the n kept points.  The grid is sized for all
// frustum points; tiles past n return at once (no pass reads their counts).
__global__ __launch_bounds__(kPT) void k_pp_hist(const int32_t* __restrict__ keys,
                                                 const int32_t* __restrict__ n_ptr, int shift,
                                                 int bits, int32_t* __restrict__ hist,
                                                 int64_t ntiles) {
  __shared__ int32_t h[kBuckets];
  const int t = threadIdx.x;
  const int64_t n = *n_ptr;
  const int64_t base = (int64_t)blockIdx.x * kTile1;
  if (base >= n) return;  // (uniform)
  h[t] = 0;
  __syncthreads();
  const uint32_t mask = (1u << bits) - 1u;
#pragma unroll
  for (int k = 0; k < kR1; ++k) {
    const int64_t e = base + k * kPT + t;
    if (e < n) atomicAdd(&h[((uint32_t)keys[e] >> shift) & mask], 1);
  }
  __syncthreads();
  if (t <= (int)mask) hist[(int64_t)t * ntiles + blockIdx.x] = h[t];
}

// One block per digit: exclusive scan of the digit's tile counts in place,
// and the digit's total.  Later passes (n_ptr: the kept count) scan only the
// tiles that hold kept points.
__global__ __launch_bounds__(kPT) void k_pp_digit_scan(int32_t* __restrict__ hist, int64_t row,
                                                       const int32_t* __restrict__ n_ptr,
                                                       int32_t* __restrict__ dtot) {
  __shared__ int32_t s_scan[kPW];
  int32_t* a = hist + (int64_t)blockIdx.x * row;
  const int64_t ntiles =
      n_ptr == nullptr ? row : min<int64_t>(row, ((int64_t)*n_ptr + kTile1 - 1) / kTile1);
  // up to kChunks * kPT * kPer counts loaded at once, then scanned chunk by
  // chunk (the scans' barriers order LDS only, so the loads stay in flight)
  constexpr int kPer = 8, kChunks = 4;
  constexpr int64_t kSpan = (int64_t)kPT * kPer;
  int32_t carry = 0;
  for (int64_t b0 = 0; b0 < ntiles; b0 += kSpan * kChunks) {
    int32_t v[kChunks][kPer];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int64_t i0 = b0 + c * kSpan + (int64_t)threadIdx.x * kPer;
#pragma unroll
      for (int k = 0; k < kPer; ++k) v[c][k] = i0 + k < ntiles ? a[i0 + k] : 0;
    }
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      if (b0 + c * kSpan >= ntiles) break;  // (uniform)
      const int64_t i0 = b0 + c * kSpan + (int64_t)threadIdx.x * kPer;
      int32_t s = 0;
#pragma unroll
      for (int k = 0; k < kPer; ++k) s += v[c][k];
      int32_t tot;
      int32_t off = carry + block_exclusive_scan<kPT, true>(s, s_scan, &tot);
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        if (i0 + k < ntiles) a[i0 + k] = off;
        off += v[c][k];
      }
      carry += tot;
    }
  }
  if (threadIdx.x == 0) dtot[blockIdx.x] = carry;
}

// LDS of the scatter kernels: the ranking's counters and digit masks, which
// the ranked tile (keys, then values) takes over once the ranks are known.
struct ScatterLds {
  int32_t (*cnt)[kBuckets];
  uint32_t (*match)[kBuckets][2];
  int32_t *start, *delta, *scan, *key, *val;
};

#define BEVPOOL_SCATTER_LDS(S, R)                                                   \
  __shared__ __align__(16) int32_t S##_raw[kPW * kBuckets * 3];                    \
  static_assert(2 * kPT * (R) <= kPW * kBuckets * 3, "the ranked tile fits");      \
  __shared__ int32_t S##_start[kBuckets], S##_delta[kBuckets], S##_scan[kPW];       \
  const ScatterLds S {                                                             \
    reinterpret_cast<int32_t(*)[kBuckets]>(S##_raw),                               \
        reinterpret_cast<uint32_t(*)[kBuckets][2]>(S##_raw + kPW * kBuckets),      \
        S##_start, S##_delta, S##_scan, S##_raw, S##_raw + kPT * (R)               \
  }

struct ScatterOut {
  int32_t *keys, *vals;
  int32_t* feat;      // last pass: each point's feature rank, else null
  int32_t* cell_cnt;  // last pass: the point count of every cell
};

// One tile of a radix pass: its valid elements ranked by digit in LDS and
// stored at their places, so that lanes store consecutive positions.  dstart
// is digit t's first place over all tiles and tile_off the earlier tiles'
// count of digit t (thread t).  The last pass also writes each point's
// feature rank and counts the points of every cell: its LDS tile is sorted by
// the whole rank, and each run of one rank adds its length to the cell's count
// (the run's first element adds -i, its last i + 1), so that every cell takes
// a few adds.  (Counting per chunk of cells the same way puts thousands of
// adds on a few addresses, which serialises them.)
template <int R, bool BALLOT = false>
__device__ __forceinline__ void scatter_tile(const ScatterLds& S, const int32_t (&key)[R],
                                             const int32_t (&val)[R], const bool (&valid)[R],
                                             const uint32_t (&digit)[R], int32_t dstart,
                                             int32_t tile_off, int shift, uint32_t mask,
                                             const PGrid& g, const ScatterOut& o) {
  const int t = threadIdx.x;
  int32_t pos[R];
  int32_t n_valid_tile;
  tile_ranks<R, BALLOT>(digit, valid, S.cnt, S.match, S.start, S.scan, pos, &n_valid_tile,
                        __builtin_popcount(mask));
  S.delta[t] = dstart + tile_off - S.start[t];
  lds_barrier();  // (every rank read: the tile takes over the counters)
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (valid[r]) {
      S.key[pos[r]] = key[r];
      S.val[pos[r]] = val[r];
    }
  }
  lds_barrier();
  for (int i = t; i < n_valid_tile; i += kPT) {
    const int32_t k = S.key[i];
    const int32_t v = S.val[i];
    const int32_t q = S.delta[((uint32_t)k >> shift) & mask] + i;
    o.keys[q] = k;
    o.vals[q] = v;
    if (o.feat != nullptr) {  // (last pass; 32-bit: p < 2^31)
      const uint32_t u = (uint32_t)v;
      o.feat[q] = (int32_t)((u / (uint32_t)g.per_view) * (uint32_t)g.hw + u % (uint32_t)g.hw);
      if (i == 0 || S.key[i - 1] != k) atomicAdd(&o.cell_cnt[k], -i);
      if (i + 1 == n_valid_tile || S.key[i + 1] != k) atomicAdd(&o.cell_cnt[k], i + 1);
    }
  }
}

// First radix pass over the frustum points: a filter and a pass in one.
// Element e of a tile is point base + wave * 64 * kR0 + round * 64 + lane.
__global__ __launch_bounds__(kPT) void k_pp_scatter_first(
    const int32_t* __restrict__ coor, PGrid g, int shift, int bits,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ dtot, int64_t ntiles,
    ScatterOut o, int32_t* __restrict__ count_out) {
  BEVPOOL_SCATTER_LDS(S, kR0);
  const int t = threadIdx.x;
  const uint32_t mask = (1u << bits) - 1u;
  const int64_t e0 = (int64_t)blockIdx.x * kTile0 + t / kWave * (kR0 * kWave) + lane_id();
  int32_t x[kR0], y[kR0], z[kR0];
#pragma unroll
  for (int r = 0; r < kR0; ++r) {
    const int64_t e = e0 + r * kWave;
    x[r] = e < g.P ? coor[3 * e + 0] : -1;  // (-1: dropped)
    y[r] = e < g.P ? coor[3 * e + 1] : -1;
    z[r] = e < g.P ? coor[3 * e + 2] : -1;
  }
  // digit t's first place (an exclusive scan of the digit totals) and the
  // earlier tiles' count of it
  const int32_t dt = t <= (int)mask ? dtot[t] : 0;
  const int32_t tile_off = t <= (int)mask ? hist[(int64_t)t * ntiles + blockIdx.x] : 0;
  int32_t n_kept;
  const int32_t dstart = block_exclusive_scan<kPT, true>(dt, S.scan, &n_kept);
  if (blockIdx.x == 0 && t == 0) *count_out = n_kept;
  int32_t key[kR0], val[kR0];
  bool valid[kR0];
  uint32_t digit[kR0];
#pragma unroll
  for (int r = 0; r < kR0; ++r) {
    const int64_t e = e0 + r * kWave;
    key[r] = rank_xyz(x[r], y[r], z[r], e, g);
    val[r] = (int32_t)e;
    valid[r] = key[r] >= 0;
    digit[r] = valid[r] ? ((uint32_t)key[r] >> shift) & mask : 0u;
  }
  scatter_tile<kR0>(S, key, val, valid, digit, dstart, tile_off, shift, mask, g, o);
}

// A later radix pass over the n kept points (tiles past n do nothing).
__global__ __launch_bounds__(kPT) void k_pp_scatter_next(
    PGrid g, const int32_t* __restrict__ keys_in, const int32_t* __restrict__ vals_in,
    const int32_t* __restrict__ n_ptr, int shift, int bits, const int32_t* __restrict__ hist,
    const int32_t* __restrict__ dtot, int64_t ntiles, ScatterOut o) {
  BEVPOOL_SCATTER_LDS(S, kR1);
  const int t = threadIdx.x;
  const int64_t n = *n_ptr;
  const int64_t tile0 = (int64_t)blockIdx.x * kTile1;
  if (tile0 >= n) return;  // (uniform: a tile past the kept points)
  const int64_t base = tile0 + t / kWave * (kR1 * kWave) + lane_id();
  const uint32_t mask = (1u << bits) - 1u;
  int32_t key[kR1], val[kR1];
  bool valid[kR1];
  uint32_t digit[kR1];
#pragma unroll
  for (int r = 0; r < kR1; ++r) {
    const int64_t e = base + r * kWave;
    valid[r] = e < n;
    key[r] = valid[r] ? keys_in[e] : 0;
    val[r] = valid[r] ? vals_in[e] : 0;
    digit[r] = valid[r] ? ((uint32_t)key[r] >> shift) & mask : 0u;
  }
  const int32_t dt = t <= (int)mask ? dtot[t] : 0;
  const int32_t tile_off = t <= (int)mask ? hist[(int64_t)t * ntiles + blockIdx.x] : 0;
  int32_t n_kept;
  const int32_t dstart = block_exclusive_scan<kPT, true>(dt, S.scan, &n_kept);
  scatter_tile<kR1, true>(S, key, val, valid, digit, dstart, tile_off, shift, mask, g, o);
}

// The cells are taken in chunks of 2^chunk_shift >= kIChunk cells, at most
// kMaxIChunks of them.  First the point total and the occupied-cell count of
// every chunk; then each chunk's block adds up those of the chunks before it,
// scans its own cells and stores its intervals through LDS, so that
// consecutive lanes store consecutive entries.
constexpr int kIChunkShift = 10;
constexpr int kIChunk = 1 << kIChunkShift;  // cells per sub-chunk: one int4 per thread
static_assert(kIChunk == 4 * kPT, "one int4 of counts per thread");
constexpr int kMaxIChunks = 1024;

__device__ __forceinline__ int4 load_counts4(const int32_t* __restrict__ cnt, int64_t c0,
                                             int64_t cells) {
  if (c0 + 4 <= cells) return *reinterpret_cast<const int4*>(cnt + c0);  // (c0 % 4 == 0)
  int4 v;
  v.x = c0 + 0 < cells ? cnt[c0 + 0] : 0;
  v.y = c0 + 1 < cells ? cnt[c0 + 1] : 0;
  v.z = c0 + 2 < cells ? cnt[c0 + 2] : 0;
  v.w = c0 + 3 < cells ? cnt[c0 + 3] : 0;
  return v;
}

__global__ __launch_bounds__(kPT) void k_pp_chunk_totals(const int32_t* __restrict__ cell_cnt,
                                                         int64_t cells, int chunk_shift,
                                                         int2* __restrict__ chunk_tot) {
  __shared__ int32_t s_scan[kPW];
  const int64_t c_begin = (int64_t)blockIdx.x << chunk_shift;
  const int64_t c_end = min<int64_t>(cells, c_begin + (int64_t(1) << chunk_shift));
  int32_t s = 0, o = 0;
  for (int64_t c0 = c_begin + 4 * threadIdx.x; c0 < c_end; c0 += kIChunk) {
    const int4 v = load_counts4(cell_cnt, c0, c_end);
    s += v.x + v.y + v.z + v.w;
    o += (v.x > 0) + (v.y > 0) + (v.z > 0) + (v.w > 0);
  }
  int32_t st, ot;
  block_exclusive_scan<kPT>(s, s_scan, &st);
  block_exclusive_scan<kPT>(o, s_scan, &ot);
  if (threadIdx.x == 0) chunk_tot[blockIdx.x] = make_int2(st, ot);
}

__global__ __launch_bounds__(kPT) void k_pp_intervals(const int32_t* __restrict__ cell_cnt,
                                                      int64_t cells, int chunk_shift,
                                                      const int2* __restrict__ chunk_tot,
                                                      int64_t cap, int32_t* __restrict__ starts,
                                                      int32_t* __restrict__ lengths,
                                                      int32_t* __restrict__ count_out) {
  __shared__ int32_t s_scan[kPW];
  __shared__ int32_t s_st[kIChunk], s_ln[kIChunk];
  const int t = threadIdx.x;
  // the points and the occupied cells of the earlier chunks
  int32_t ps = 0, po = 0;
  for (int k = t; k < (int)blockIdx.x; k += kPT) {
    const int2 x = chunk_tot[k];
    ps += x.x;
    po += x.y;
  }
  int32_t carry, icarry;
  block_exclusive_scan<kPT>(ps, s_scan, &carry);
  block_exclusive_scan<kPT>(po, s_scan, &icarry);
  const int64_t c_begin = (int64_t)blockIdx.x << chunk_shift;
  const int64_t c_end = min<int64_t>(cells, c_begin + (int64_t(1) << chunk_shift));
  for (int64_t b0 = c_begin; b0 < c_end; b0 += kIChunk) {
    const int4 x = load_counts4(cell_cnt, b0 + 4 * t, c_end);
    const int32_t v[4] = {x.x, x.y, x.z, x.w};
    int32_t s = 0, o = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      s += v[k];
      o += v[k] > 0 ? 1 : 0;
    }
    int32_t tot, otot;
    int32_t off = carry + block_exclusive_scan<kPT>(s, s_scan, &tot);
    int32_t loc = block_exclusive_scan<kPT>(o, s_scan, &otot);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (v[k] > 0) {
        s_st[loc] = off;
        s_ln[loc] = v[k];
        ++loc;
      }
      off += v[k];
    }
    __syncthreads();
    for (int i = t; i < otot; i += kPT) {
      const int64_t q = (int64_t)icarry + i;
      if (q < cap) {
        starts[q] = s_st[i];
        lengths[q] = s_ln[i];
      }
    }
    __syncthreads();
    carry += tot;
    icarry += otot;
  }
  if (blockIdx.x == gridDim.x - 1 && t == 0) *count_out = icarry;
}

int bits_for_cells(int64_t cells) {  // bits of the ranks 0 .. cells - 1 (at least 1)
  int b = 1;
  while ((int64_t(1) << b) < cells) ++b;
  return b;
}

}  // namespace

PrepareLayout prepare_layout(const Dims& d) {
  PrepareLayout L{};
  L.ntiles0 = (d.P + kTile0 - 1) / kTile0;
  L.ntiles = (d.P + kTile1 - 1) / kTile1;
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
  L.chunk_shift = kIChunkShift;
  while (((d.cells - 1) >> L.chunk_shift) + 1 > kMaxIChunks) ++L.chunk_shift;
  L.nchunks = ((d.cells - 1) >> L.chunk_shift) + 1;
  L.chunk_totals = take(2 * (size_t)L.nchunks);
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
  int2* chunk_tot = reinterpret_cast<int2*>(ws + L.chunk_totals);
  PGrid g;
  g.P = d.P;
  g.per_sample = (int32_t)(d.N * d.per_view);
  g.per_view = (int32_t)d.per_view;
  g.hw = (int32_t)d.hw;
  g.X = (int32_t)d.X;
  g.Y = (int32_t)d.Y;
  g.Z = (int32_t)d.Z;
  const unsigned tiles0 = (unsigned)L.ntiles0;
  const unsigned tiles = (unsigned)L.ntiles;
  const bool vec = reinterpret_cast<uintptr_t>(coor) % 16 == 0;  // 16-byte loads of coor
  // The passes alternate between the workspace and the output arrays so
  // that the last lands in (ranks_bev, ranks_depth).
  auto keys_of = [&](int pass) { return ((L.passes - 1 - pass) % 2 == 0) ? ranks_bev : keys_tmp; };
  auto vals_of = [&](int pass) { return ((L.passes - 1 - pass) % 2 == 0) ? ranks_depth : vals_tmp; };
  for (int pass = 0; pass < L.passes; ++pass) {
    const int shift = pass * L.digit_bits;
    const int bits = std::min(L.digit_bits, L.key_bits - shift);
    const bool last = pass == L.passes - 1;
    const ScatterOut o{keys_of(pass), vals_of(pass), last ? ranks_feat : nullptr, cell_cnt};
    const int64_t nt = pass == 0 ? L.ntiles0 : L.ntiles;  // tiles of this pass
    if (pass == 0)
      k_pp_hist0<<<tiles0, kPT, 0, stream>>>(coor, g, vec, bits, hist, nt, cell_cnt, d.cells);
    else
      k_pp_hist<<<tiles, kPT, 0, stream>>>(keys_of(pass - 1), counts, shift, bits, hist, nt);
    k_pp_digit_scan<<<1u << bits, kPT, 0, stream>>>(hist, nt, pass == 0 ? nullptr : counts, dtot);
    if (pass == 0)
      k_pp_scatter_first<<<tiles0, kPT, 0, stream>>>(coor, g, shift, bits, hist, dtot, nt, o,
                                                     counts + 0);
    else
      k_pp_scatter_next<<<tiles, kPT, 0, stream>>>(g, keys_of(pass - 1), vals_of(pass - 1), counts,
                                                   shift, bits, hist, dtot, nt, o);
  }
  const int64_t cap = d.P < d.cells ? d.P : d.cells;
  const unsigned nchunks = (unsigned)L.nchunks;
  k_pp_chunk_totals<<<nchunks, kPT, 0, stream>>>(cell_cnt, d.cells, L.chunk_shift, chunk_tot);
  k_pp_intervals<<<nchunks, kPT, 0, stream>>>(cell_cnt, d.cells, L.chunk_shift, chunk_tot, cap,
                                              starts, lengths, counts + 1);
  return hipGetLastError();
}

}  // namespace bevpool
