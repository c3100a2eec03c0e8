// Device-wide primitives (exclusive scan, stable LSD radix sort of key/value
// pairs, ordered compaction) and the general schedule builder, which regroups
// a plan (section 2.1) by strips with global sorts; it serves the shapes whose
// strips exceed the bounds of the build in LDS (schedule_local.hip).
//
// Every step is deterministic and order preserving: a radix pass ranks equal
// digits with wave ballots inside a tile and orders tiles with digit-major
// tile histograms.  Tiles are 4096 elements: 4 waves x 16 rounds x 64 lanes,
// each wave owning a contiguous run of 1024 elements so lane order within a
// round and round order within a wave both follow the element order.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"
#include "schedule_items.h"

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
                                                             int64_t n,
                                                             int32_t* __restrict__ sums,
                                                             int32_t* __restrict__ total_out) {
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
  if (nb == 0) {  // (an empty input: only its zero total)
    k_scan_top<<<dim3(1), dim3(kScanThreads), 0, stream>>>(sums, 0, total_out);
    return;
  }
  k_scan_local<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums, total_out);
  if (nb > 1) {
    k_scan_top<<<dim3(1), dim3(kScanThreads), 0, stream>>>(sums, nb, total_out);
    k_scan_add<<<dim3((unsigned)nb), dim3(kScanThreads), 0, stream>>>(data, n, sums);
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

// ------------------------------------------------------------------ schedule
//
// The schedule regroups the kept points of a plan into strips, pairs, items
// and segments (see internal.h).  Steps, all on the device:
//   1. stable radix sorts of the plan by local pixel, then by (strip, BEV
//      rank), giving (strip, cell, pixel, plan position) order;
//   2. pair heads by ordered compaction, and each pair's point count;
//   3. the pairs again in pixel-major order (for the backward pass), with
//      the first pair of every feature row;
//   4. strip heads over the pairs and the items of every strip;
//   5. segment heads (item starts and cell changes) and the pair records;
//   6. segments sorted by cell: a cell covered by several segments gets one
//      slot per segment, consecutive in segment order; the others are
//      written directly by the forward;
//   7. the empty cells, by compaction of an occupancy map.

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

// (32-bit unsigned arithmetic: p, D*H*W and H*W are below 2^31, and 64-bit
// division costs several times more)
__device__ __forceinline__ int32_t pixel_of(int32_t p, int64_t per_view, int64_t hw) {
  const uint32_t u = (uint32_t)p, pv = (uint32_t)per_view, h = (uint32_t)hw;
  return (int32_t)((u / pv) * h + u % h);
}

// Strip and local pixel of a feature row.
struct StripGeom {
  int64_t hw;
  int32_t H, W, bh, bw, nhb, nwb;
  __device__ int32_t strip(int32_t row) const {
    const int32_t bn = (int32_t)((uint32_t)row / (uint32_t)hw);  // (row, H*W < 2^31)
    const int32_t r = row - bn * (int32_t)hw;
    const int32_t h = r / W, w = r - h * W;
    return (bn * nhb + h / bh) * nwb + w / bw;
  }
  __device__ int32_t pixel(int32_t row) const {
    const int32_t bn = (int32_t)((uint32_t)row / (uint32_t)hw);  // (row, H*W < 2^31)
    const int32_t r = row - bn * (int32_t)hw;
    const int32_t h = r / W, w = r - h * W;
    const int32_t w0 = (w / bw) * bw;
    const int32_t bws = min(bw, W - w0);
    return (h % bh) * bws + (w - w0);
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

// keys = local pixel of every kept point, vals = its plan position
__global__ __launch_bounds__(256) void k_pixel_keys(const int32_t* __restrict__ rd, int64_t n,
                                                    int64_t per_view, StripGeom g,
                                                    int32_t* __restrict__ keys,
                                                    int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    keys[i] = g.pixel(pixel_of(rd[i], per_view, g.hw));
    vals[i] = (int32_t)i;
  }
}

// keys[i] for the point at plan position vals[i]: mode 0 (strip << cell_bits)
// | BEV rank, mode 1 the BEV rank, mode 2 the strip.
__global__ __launch_bounds__(256) void k_strip_keys(const int32_t* __restrict__ rd,
                                                    const int32_t* __restrict__ rb,
                                                    const int32_t* __restrict__ vals, int64_t n,
                                                    int64_t per_view, StripGeom g, int cell_bits,
                                                    int mode, int32_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t a = vals[i];
  const int32_t s = g.strip(pixel_of(rd[a], per_view, g.hw));
  keys[i] = mode == 0 ? (int32_t)(((uint32_t)s << cell_bits) | (uint32_t)rb[a])
                      : (mode == 1 ? rb[a] : s);
}

struct PairHeads {  // runs of one cell and pixel over consecutive depth bins
  const int32_t* rd;
  const int32_t* rb;
  const int32_t* vals;  // plan position of each regrouped point
  const int32_t* hdr;
  int64_t per_view, hw;
  int32_t* pair_rb;
  int32_t* pair_row;
  uint32_t* pair_dn;
  int32_t* pair_rd0;
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
    pair_dn[pos] = ((uint32_t)p % (uint32_t)per_view) / (uint32_t)hw;
    pair_rd0[pos] = p;
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

struct StripHeads {  // first pair of every strip that has pairs
  const int32_t* pair_row;
  const int32_t* hdr;
  StripGeom g;
  int32_t* strip_id;
  int32_t* strip_p0;
  __device__ int64_t count() const { return hdr[kHdrPairs]; }
  __device__ bool flag(int64_t k) const {
    return k == 0 || g.strip(pair_row[k]) != g.strip(pair_row[k - 1]);
  }
  __device__ void emit(int64_t k, int32_t pos) const {
    strip_id[pos] = g.strip(pair_row[k]);
    strip_p0[pos] = (int32_t)k;
  }
};

__global__ void k_strips_end(const int32_t* __restrict__ hdr, int32_t* __restrict__ strip_p0) {
  if (threadIdx.x == 0 && blockIdx.x == 0) strip_p0[hdr[kHdrStrips]] = hdr[kHdrPairs];
}

// Items of every listed strip (0 past the last one, up to cap).
__global__ __launch_bounds__(256) void k_item_counts(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ strip_p0,
                                                     int64_t cap, int64_t shares, int64_t ip,
                                                     int32_t* __restrict__ count) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= cap) return;
  int32_t k = 0;
  if (j < hdr[kHdrStrips])
    k = (int32_t)strip_items(strip_p0[j], strip_p0[j + 1], hdr[kHdrPairs], shares, ip,
                             [](int64_t, int64_t) {});
  count[j] = k;
}

// With the item counts exclusively scanned: every item's strip and first
// pair; item_flag marks item starts (item + 1).
__global__ __launch_bounds__(256) void k_item_scatter(const int32_t* __restrict__ hdr,
                                                      const int32_t* __restrict__ strip_id,
                                                      const int32_t* __restrict__ strip_p0,
                                                      const int32_t* __restrict__ offset,
                                                      int64_t items_cap, int64_t shares,
                                                      int64_t ip, int32_t* __restrict__ item_strip,
                                                      int32_t* __restrict__ item_pair0,
                                                      int32_t* __restrict__ item_flag) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= hdr[kHdrStrips]) return;
  const int32_t sid = strip_id[j];
  const int64_t off = offset[j];
  strip_items(strip_p0[j], strip_p0[j + 1], hdr[kHdrPairs], shares, ip, [&](int64_t i, int64_t first) {
    const int64_t item = off + i;
    if (item >= items_cap) return;
    item_strip[item] = sid;
    item_pair0[item] = (int32_t)first;
    item_flag[first] = (int32_t)(item + 1);
  });
}

// First item of every share (an item starts at every share boundary inside
// the pairs), and whether no share holds more than kShareItems items.  One
// block of kShareThreads threads.
constexpr int kShareThreads = 1024;
__global__ __launch_bounds__(kShareThreads) void k_share_items(int32_t* __restrict__ hdr,
                                                               const int32_t* __restrict__ strip_p0,
                                                               const int32_t* __restrict__ item_pair0,
                                                               int64_t items_cap, int32_t shares,
                                                               int32_t ip,
                                                               int32_t* __restrict__ share_item0) {
  __shared__ int32_t s_bad;
  if (threadIdx.x == 0) s_bad = 0;
  const int64_t P = hdr[kHdrPairs];
  const int64_t n_items = min<int64_t>(hdr[kHdrItems], items_cap);
  const int64_t n_strips = hdr[kHdrStrips];
  for (int w = threadIdx.x; w <= shares; w += kShareThreads) {
    int64_t c = (P * w) / shares;
    if (c > 0 && c < P) {  // the strip holding pair c: the last one starting at or before it
      int64_t lo = 0, hi = n_strips;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (strip_p0[mid] <= c) lo = mid; else hi = mid;
      }
      c = snap_bound(c, strip_p0[lo], strip_p0[lo + 1]);
    }
    // lower bound of c among the item starts
    int64_t lo = 0, hi = n_items;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (item_pair0[mid] < c) lo = mid + 1; else hi = mid;
    }
    share_item0[w] = (int32_t)lo;
  }
  __syncthreads();
  for (int w = threadIdx.x; w < shares; w += kShareThreads)
    if (share_item0[w + 1] - share_item0[w] > kShareItems) s_bad = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    hdr[kHdrShares] = shares;
    hdr[kHdrSharesOk] = s_bad ? 0 : 1;
    hdr[kHdrItemPairs] = ip;
  }
}

__global__ void k_items_end(const int32_t* __restrict__ hdr, int64_t items_cap,
                            int32_t* __restrict__ item_pair0) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && hdr[kHdrItems] <= items_cap)
    item_pair0[hdr[kHdrItems]] = hdr[kHdrPairs];
}

__device__ __forceinline__ bool segment_head(int64_t k, const int32_t* item_flag,
                                             const int32_t* pair_rb) {
  return k == 0 || item_flag[k] != 0 || pair_rb[k] != pair_rb[k - 1];
}

struct SegHeads {  // first pair of every segment
  const int32_t* pair_rb;
  const int32_t* item_flag;
  const int32_t* hdr;
  int64_t items_cap;
  int32_t* item_seg0;
  int32_t* seg_cell;  // BEV rank of each segment
  int32_t* seg_id;    // its index (values of the cell sort)
  __device__ int64_t count() const { return hdr[kHdrPairs]; }
  __device__ bool flag(int64_t k) const { return segment_head(k, item_flag, pair_rb); }
  __device__ void emit(int64_t k, int32_t pos) const {
    seg_cell[pos] = pair_rb[k];
    seg_id[pos] = pos;
    const int32_t it = item_flag[k] - 1;
    if (it >= 0 && it < items_cap) item_seg0[it] = pos;
  }
};

__global__ void k_segs_end(const int32_t* __restrict__ hdr, int64_t items_cap,
                           int32_t* __restrict__ item_seg0) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && hdr[kHdrItems] <= items_cap)
    item_seg0[hdr[kHdrItems]] = hdr[kHdrSegs];
}

__global__ __launch_bounds__(256) void k_pair_ln(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ pair_row,
                                                 const int32_t* __restrict__ pair_rb,
                                                 const uint32_t* __restrict__ pair_dn,
                                                 const int32_t* __restrict__ item_flag, StripGeom g,
                                                 uint32_t* __restrict__ pair_ln) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= hdr[kHdrPairs]) return;
  const uint32_t head = segment_head(k, item_flag, pair_rb) ? kPairHead : 0u;
  pair_ln[k] = ((uint32_t)g.pixel(pair_row[k]) & kPairPixel) | head | (pair_dn[k] & 0xffff0000u);
}

// flags[k] = 1 at every segment's first pair, 0 elsewhere (up to cap).
__global__ __launch_bounds__(256) void k_seg_flags(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ pair_rb,
                                                   const int32_t* __restrict__ item_flag,
                                                   int64_t cap, int32_t* __restrict__ flags) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cap) return;
  flags[k] = (k < hdr[kHdrPairs] && segment_head(k, item_flag, pair_rb)) ? 1 : 0;
}

// With the segment flags exclusively scanned into `before`: each pair's
// segment index within its item.
__global__ __launch_bounds__(256) void k_pair_seg(const int32_t* __restrict__ hdr,
                                                  const int32_t* __restrict__ before,
                                                  const int32_t* __restrict__ pair_rb,
                                                  const int32_t* __restrict__ item_flag,
                                                  const int32_t* __restrict__ item_pair0,
                                                  const int32_t* __restrict__ item_seg0,
                                                  int64_t items_cap, uint16_t* __restrict__ pair_seg) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= hdr[kHdrPairs]) return;
  const int32_t n_items = (int32_t)min<int64_t>(hdr[kHdrItems], items_cap);
  if (n_items < 1) return;
  const int32_t seg = before[k] + (segment_head(k, item_flag, pair_rb) ? 1 : 0) - 1;
  const int32_t it = upper_index(item_pair0, n_items, (int32_t)k);
  pair_seg[k] = (uint16_t)(seg - item_seg0[it]);
}

// Over segments sorted by cell: is segment q one of several of its cell?
__device__ __forceinline__ bool shared_cell(const int32_t* keys, int64_t q, int64_t n) {
  return (q > 0 && keys[q - 1] == keys[q]) || (q + 1 < n && keys[q + 1] == keys[q]);
}

__global__ __launch_bounds__(256) void k_slot_flags(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ keys, int64_t cap,
                                                    int32_t* __restrict__ flags) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= cap) return;
  const int64_t n = hdr[kHdrSegs];
  flags[q] = (q < n && shared_cell(keys, q, n)) ? 1 : 0;
}

// With the slot flags exclusively scanned into `slot`.
__global__ __launch_bounds__(256) void k_seg_dest(const int32_t* __restrict__ hdr,
                                                  const int32_t* __restrict__ keys,
                                                  const int32_t* __restrict__ vals,
                                                  const int32_t* __restrict__ slot,
                                                  int32_t* __restrict__ seg_dest) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = hdr[kHdrSegs];
  if (q >= n) return;
  seg_dest[vals[q]] = shared_cell(keys, q, n) ? ~slot[q] : keys[q];
}

struct CombHeads {  // cells with several segments: their first slot
  const int32_t* keys;
  const int32_t* slot;
  const int32_t* hdr;
  int32_t* comb_cell;
  int32_t* comb_slot0;
  int64_t cap;
  __device__ int64_t count() const { return hdr[kHdrSegs]; }
  __device__ bool flag(int64_t q) const {
    return (q == 0 || keys[q - 1] != keys[q]) && shared_cell(keys, q, count());
  }
  __device__ void emit(int64_t q, int32_t pos) const {
    if (pos >= cap) return;
    comb_cell[pos] = keys[q];
    comb_slot0[pos] = slot[q];
  }
};

__global__ void k_comb_end(const int32_t* __restrict__ hdr, int64_t cap,
                           int32_t* __restrict__ comb_slot0) {
  if (threadIdx.x == 0 && blockIdx.x == 0)
    comb_slot0[min<int64_t>(hdr[kHdrComb], cap)] = hdr[kHdrSlots];
}

struct CellRuns {  // occupied cells: runs of equal cell over sorted segments
  const int32_t* keys;
  const int32_t* hdr;
  __device__ int64_t count() const { return hdr[kHdrSegs]; }
  __device__ bool flag(int64_t q) const { return q == 0 || keys[q - 1] != keys[q]; }
  __device__ void emit(int64_t, int32_t) const {}
};

__global__ __launch_bounds__(256) void k_fill_i32(int32_t* __restrict__ a, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) a[i] = v;
}

__global__ __launch_bounds__(256) void k_mark_cells(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ keys,
                                                    int64_t cells, int32_t* __restrict__ occ) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < hdr[kHdrSegs]) {
    const int32_t cell = keys[q];
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

namespace bevpool {

int64_t strip_pixels(int64_t C) {
  const int64_t c = C < 256 ? C : 256;
  const int64_t r = kStripBytes / (4 * c);
  return r > 0 ? r : 1;
}

StripDims strip_dims(const Dims& d) {
  StripDims s{};
  const int64_t R = strip_pixels(d.C);
  s.bh = std::min<int64_t>(d.H, R);
  s.bw = std::max<int64_t>(1, std::min<int64_t>(d.W, R / s.bh));
  s.nhb = (d.H + s.bh - 1) / s.bh;
  s.nwb = (d.W + s.bw - 1) / s.bw;
  s.strips = d.B * d.N * s.nhb * s.nwb;
  s.pixels = s.bh * s.bw;
  return s;
}

ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals) {
  ScheduleLayout L{};
  L.n_valid = n_valid;
  L.n_occ = n_intervals;
  L.n_empty = d.cells > n_intervals ? d.cells - n_intervals : 0;
  L.sd = strip_dims(d);
  // pieces (strips cut at shares) number at most strips + shares - 1, and
  // the sum over pieces of ceil(L / kItemPairs) <= n_pairs / kItemPairs + pieces
  L.items_cap = L.sd.strips + n_valid / kItemPairs + kMaxShares + 2;
  const size_t nv = (size_t)(n_valid > 0 ? n_valid : 1);
  const size_t nocc = (size_t)n_intervals + 1;
  size_t off = 0;
  auto take = [&](size_t n_ints) {
    const size_t o = off;
    off += align_up(sizeof(int32_t) * n_ints);
    return o;
  };
  L.header = take(16);
  L.pair_rd0 = take(nv);
  L.pair_ln = take(nv);
  L.pair_seg = take((nv + 1) / 2);
  L.item_strip = take((size_t)L.items_cap);
  L.item_pair0 = take((size_t)L.items_cap + 1);
  L.item_seg0 = take((size_t)L.items_cap + 1);
  L.seg_dest = take(nv);
  L.comb_cell = take(nocc);
  L.comb_slot0 = take(nocc);
  L.empty = take((size_t)L.n_empty + 1);
  L.bp_cell = take(nv);
  L.bp_dn = take(nv);
  L.pix_pair0 = take((size_t)d.rows + 1);
  L.share_item0 = take((size_t)kMaxShares + 1);
  L.total = off;

  const int64_t span = std::max<int64_t>((int64_t)nv, d.cells);
  L.ntiles = (span + kPrepTile - 1) / kPrepTile;
  const int64_t scan_n = std::max<int64_t>(std::max<int64_t>(256 * L.ntiles, L.sd.strips + 1), span);
  L.nscan = (scan_n + kScanTile - 1) / kScanTile;
  off = 0;
  L.ws_ka = take(nv);
  L.ws_va = take(nv);
  L.ws_kb = take(nv);
  L.ws_vb = take(nv);
  L.ws_head = take(nv);
  L.ws_pair_rb = take(nv);
  L.ws_pair_row = take(nv);
  L.ws_pair_dn = take(nv);
  L.ws_flags = take((size_t)span + 1);
  L.ws_strip = take(3 * ((size_t)L.sd.strips + 1));
  L.ws_tiles = take((size_t)L.ntiles + 2);
  L.ws_hist = take((size_t)(256 * L.ntiles));
  L.ws_sums = take((size_t)L.nscan + 1);
  L.ws_total = off;
  local_schedule_ws(d, L);
  if (schedule_local_ok(d, n_valid)) L.ws_total = std::max(L.ws_total, L.wl_total);
  L.row_bits = bit_length(d.rows);
  L.cell_bits = bit_length(d.cells);
  L.pixel_bits = bit_length(L.sd.pixels);
  L.strip_bits = bit_length(L.sd.strips);
  return L;
}

hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream) {
  if (schedule_local_ok(d, n_valid))
    return launch_schedule_local(d, rd, rb, n_valid, n_intervals, schedule, workspace, stream);
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  char* sc = static_cast<char*>(schedule);
  char* ws = static_cast<char*>(workspace);
  auto S = [&](size_t o) { return reinterpret_cast<int32_t*>(sc + o); };
  auto W = [&](size_t o) { return reinterpret_cast<int32_t*>(ws + o); };
  int32_t* hdr = S(L.header);
  int32_t* tiles = W(L.ws_tiles);
  int32_t* sums = W(L.ws_sums);
  int32_t* hist = W(L.ws_hist);
  int32_t* occ = W(L.ws_flags);
  const dim3 grid((unsigned)L.ntiles), block(kPrepThreads);
  const unsigned g_nv = (unsigned)((n_valid + 255) / 256);
  const unsigned g_cells = (unsigned)((d.cells + 255) / 256);
  StripGeom geom;
  geom.hw = d.hw;
  geom.H = (int32_t)d.H;
  geom.W = (int32_t)d.W;
  geom.bh = (int32_t)L.sd.bh;
  geom.bw = (int32_t)L.sd.bw;
  geom.nhb = (int32_t)L.sd.nhb;
  geom.nwb = (int32_t)L.sd.nwb;

  k_sched_init<<<1, 64, 0, stream>>>(hdr, n_valid, n_intervals);
  if (n_valid > 0) {
    // 1. regroup by (strip, cell, local pixel, plan position)
    int32_t *ck = W(L.ws_ka), *cv = W(L.ws_va), *ak = W(L.ws_kb), *av = W(L.ws_vb);
    auto sort_current = [&](int bits, const int32_t* n_ptr) {
      if (radix_sort_pairs(ck, cv, ak, av, n_ptr, L.ntiles, bits, hist, sums, stream)) {
        std::swap(ck, ak);
        std::swap(cv, av);
      }
    };
    k_pixel_keys<<<g_nv, 256, 0, stream>>>(rd, n_valid, d.per_view, geom, ck, cv);
    sort_current(L.pixel_bits, hdr + kHdrValid);
    if (L.strip_bits + L.cell_bits <= 31) {
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, d.per_view, geom, L.cell_bits, 0,
                                             ck);
      sort_current(L.strip_bits + L.cell_bits, hdr + kHdrValid);
    } else {
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, d.per_view, geom, L.cell_bits, 1,
                                             ck);
      sort_current(L.cell_bits, hdr + kHdrValid);
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, d.per_view, geom, L.cell_bits, 2,
                                             ck);
      sort_current(L.strip_bits, hdr + kHdrValid);
    }
    const int32_t* vals = cv;

    // 2. pairs
    int32_t* pair_rb = W(L.ws_pair_rb);
    int32_t* pair_row = W(L.ws_pair_row);
    uint32_t* pair_dn = reinterpret_cast<uint32_t*>(W(L.ws_pair_dn));
    int32_t* head_pos = W(L.ws_head);
    PairHeads ph{rd, rb, vals, hdr, d.per_view, d.hw, pair_rb, pair_row, pair_dn,
                 S(L.pair_rd0), head_pos};
    k_compact_count<<<grid, block, 0, stream>>>(ph, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrPairs, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(ph, tiles);
    k_pair_points<<<g_nv, 256, 0, stream>>>(head_pos, hdr, pair_dn);

    // 3. pixel-major pairs; a stable sort by feature rank keeps the cell order
    // within a pixel
    ck = W(L.ws_ka); cv = W(L.ws_va); ak = W(L.ws_kb); av = W(L.ws_vb);
    k_pair_row_keys<<<g_nv, 256, 0, stream>>>(hdr, pair_row, ck, cv);
    sort_current(L.row_bits, hdr + kHdrPairs);
    k_pix_pairs<<<g_nv, 256, 0, stream>>>(hdr, cv, pair_rb, pair_dn, S(L.bp_cell),
                                          reinterpret_cast<uint32_t*>(S(L.bp_dn)));
    k_pix_offsets<<<(unsigned)((d.rows + 1 + 255) / 256), 256, 0, stream>>>(hdr, ck, d.rows,
                                                                            S(L.pix_pair0));

    // 4. strips and items
    const int64_t scap = L.sd.strips + 1;
    int32_t* strip_id = W(L.ws_strip);
    int32_t* strip_p0 = strip_id + scap;
    int32_t* icount = strip_p0 + scap;
    StripHeads sh{pair_row, hdr, geom, strip_id, strip_p0};
    k_compact_count<<<grid, block, 0, stream>>>(sh, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrStrips, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(sh, tiles);
    k_strips_end<<<1, 64, 0, stream>>>(hdr, strip_p0);
    const unsigned g_s = (unsigned)((scap + 255) / 256);
    const int32_t shares = (int32_t)std::min<int64_t>(forward_workgroups(), kMaxShares);
    const int32_t ip = schedule_item_pairs(n_valid);
    k_item_counts<<<g_s, 256, 0, stream>>>(hdr, strip_p0, scap, shares, ip, icount);
    scan_exclusive(icount, scap, sums, hdr + kHdrItems, stream);
    int32_t* item_flag = W(L.ws_flags);
    k_fill_i32<<<g_nv, 256, 0, stream>>>(item_flag, n_valid, 0);
    k_item_scatter<<<g_s, 256, 0, stream>>>(hdr, strip_id, strip_p0, icount, L.items_cap, shares,
                                            ip, S(L.item_strip), S(L.item_pair0), item_flag);
    k_items_end<<<1, 64, 0, stream>>>(hdr, L.items_cap, S(L.item_pair0));
    k_share_items<<<1, kShareThreads, 0, stream>>>(hdr, strip_p0, S(L.item_pair0), L.items_cap, shares,
                                                   ip, S(L.share_item0));

    // 5. segments and pair records
    ck = W(L.ws_ka); cv = W(L.ws_va); ak = W(L.ws_kb); av = W(L.ws_vb);
    SegHeads gh{pair_rb, item_flag, hdr, L.items_cap, S(L.item_seg0), ck, cv};
    k_compact_count<<<grid, block, 0, stream>>>(gh, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrSegs, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(gh, tiles);
    k_segs_end<<<1, 64, 0, stream>>>(hdr, L.items_cap, S(L.item_seg0));
    k_pair_ln<<<g_nv, 256, 0, stream>>>(hdr, pair_row, pair_rb, pair_dn, item_flag, geom,
                                        reinterpret_cast<uint32_t*>(S(L.pair_ln)));
    int32_t* seg_before = W(L.ws_head);  // pair heads are no longer needed
    k_seg_flags<<<g_nv, 256, 0, stream>>>(hdr, pair_rb, item_flag, n_valid, seg_before);
    scan_exclusive(seg_before, n_valid, sums, nullptr, stream);
    k_pair_seg<<<g_nv, 256, 0, stream>>>(hdr, seg_before, pair_rb, item_flag, S(L.item_pair0),
                                         S(L.item_seg0), L.items_cap,
                                         reinterpret_cast<uint16_t*>(S(L.pair_seg)));

    // 6. slots of cells with several segments
    sort_current(L.cell_bits, hdr + kHdrSegs);
    int32_t* slot = W(L.ws_head);  // segment flags are no longer needed
    k_slot_flags<<<g_nv, 256, 0, stream>>>(hdr, ck, n_valid, slot);
    scan_exclusive(slot, n_valid, sums, hdr + kHdrSlots, stream);
    k_seg_dest<<<g_nv, 256, 0, stream>>>(hdr, ck, cv, slot, S(L.seg_dest));
    CombHeads mh{ck, slot, hdr, S(L.comb_cell), S(L.comb_slot0), n_intervals};
    k_compact_count<<<grid, block, 0, stream>>>(mh, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrComb, stream);
    k_compact_scatter<<<grid, block, 0, stream>>>(mh, tiles);
    k_comb_end<<<1, 64, 0, stream>>>(hdr, n_intervals, S(L.comb_slot0));
    CellRuns cr{ck, hdr};
    k_compact_count<<<grid, block, 0, stream>>>(cr, tiles);
    scan_exclusive(tiles, L.ntiles, sums, hdr + kHdrOccFound, stream);
    k_fill_i32<<<g_cells, 256, 0, stream>>>(occ, d.cells, 0);  // item flags are done
    k_mark_cells<<<g_nv, 256, 0, stream>>>(hdr, ck, d.cells, occ);
  } else {
    k_fill_i32<<<g_cells, 256, 0, stream>>>(occ, d.cells, 0);
  }

  // 7. empty cells
  const dim3 cgrid((unsigned)((d.cells + kPrepTile - 1) / kPrepTile));
  EmptyCells ec{occ, d.cells, S(L.empty), L.n_empty};
  k_compact_count<<<cgrid, block, 0, stream>>>(ec, tiles);
  scan_exclusive(tiles, (int64_t)cgrid.x, sums, hdr + kHdrEmpty, stream);
  k_compact_scatter<<<cgrid, block, 0, stream>>>(ec, tiles);
  return hipGetLastError();
}

}  // namespace bevpool
