// Schedule build with each image strip regrouped inside one workgroup's LDS.
//
// The schedule (definitions in internal.h) orders the kept points of a plan
// by (strip, BEV rank, local pixel, depth bin).  A strip's points are a small
// set (bh x bw pixels x D bins), so instead of sorting all kept points
// globally, one workgroup per strip gathers its kept points from a map of
// frustum point -> BEV rank, sorts them in LDS and forms its pairs.  What
// needs the whole plan (pair offsets, items and shares, pixel offsets,
// segment offsets, slots, empty cells) is done by single-block scans and two
// flat passes.  The result is bit for bit the schedule of the general
// builder (prepare.hip), which remains for shapes whose strips exceed the
// LDS bounds below.
//
// Launches: init, map, strips, plan, emit, cell totals, cells, segments, slots.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"
#include "schedule_items.h"

namespace bevpool {

namespace {

constexpr int kLT = 1024;                  // threads of the per-strip kernels
constexpr int kLW = kLT / kWave;           // 16 waves
constexpr int kLR = kLocalPoints / kLT;    // 12 rounds of 64 lanes per wave
constexpr int kLBuckets = 256;             // digits of one LDS sort pass (8 bits)
constexpr int kLItems = kMaxShares + kLocalPoints / kItemPairs + 2;  // items of one strip
static_assert(kLocalPoints % kLT == 0, "whole rounds");

struct LGeom {
  int32_t N, D, H, W, bh, bw, nhb, nwb, strips;
  int32_t hw;      // H * W
  int32_t zyx;     // cells of one sample
  int32_t maxpts;  // bh * bw * D: region entries per strip
  int d_bits, lp_bits, rb_bits;
  // strip s: sample-view bn, first row h0 and column w0, its height and width
  __device__ void strip(int32_t s, int32_t& bn, int32_t& h0, int32_t& w0, int32_t& bhs,
                        int32_t& bws) const {
    const int32_t wb = s % nwb;
    const int32_t t = s / nwb;
    const int32_t hb = t % nhb;
    bn = t / nhb;
    h0 = hb * bh;
    w0 = wb * bw;
    bhs = min(bh, H - h0);
    bws = min(bw, W - w0);
  }
};

// Strip of workgroup b: each die (workgroup b runs on die b % kXcds) takes a
// contiguous run of strips, so that neighbouring strips, which read the same
// cache lines of the map, share one L2.  -1 for the padding workgroups.
__device__ __forceinline__ int32_t strip_of_block(int32_t strips) {
  const int32_t per = (strips + kXcds - 1) / kXcds;
  const int32_t b = blockIdx.x;
  const int32_t s = (b % kXcds) * per + b / kXcds;
  return s < strips ? s : -1;
}

// One stable counting pass over the n elements held by a workgroup in the
// wave-round layout (element e = wave * span + round * 64 + lane): returns in
// dest[r] each element's position in the order of digit, then element.  cnt
// is kLW x kLBuckets ints of LDS and match kLW x kLBuckets x 2 words; after
// the pass cnt[0][d] holds the first position of digit d.  Every thread of
// the block must call it.
//
// In a round, the lanes holding one digit are found by each lane setting its
// bit in the wave's 64-bit mask for that digit (one LDS OR), reading the mask
// back and clearing it; LDS applies one wave's operations in order, so the
// rounds need no waits between them.  The lowest lane of each digit then
// adds the digit's count to the wave's counter with a returning LDS add; the
// adds of all rounds are issued before any result is used, and each returns
// the count of that digit in the wave's earlier rounds.
__device__ void local_ranks(const uint32_t (&digit)[kLR], int n, int span,
                            int32_t (*cnt)[kLBuckets], uint32_t (*match)[kLBuckets][2],
                            int32_t* s_scan, int32_t (&dest)[kLR]) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const int t = threadIdx.x;
  for (int i = t; i < kLW * kLBuckets; i += kLT) (&cnt[0][0])[i] = 0;
  for (int i = t; i < kLW * kLBuckets * 2; i += kLT) (&match[0][0][0])[i] = 0u;
  __syncthreads();
  const int rounds = span / kWave;
  uint2 m[kLR];
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= rounds) continue;
    const bool valid = wid * span + r * kWave + lane < n;
    uint32_t* w = match[wid][digit[r]];
    m[r] = make_uint2(0u, 0u);
    if (valid) {
      atomicOr(&w[lane >> 5], 1u << (lane & 31));
      m[r] = *reinterpret_cast<const uint2*>(w);
      *reinterpret_cast<uint2*>(w) = make_uint2(0u, 0u);
    }
  }
  int32_t below[kLR], leader[kLR], old[kLR];
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= rounds) continue;
    const uint64_t same = (uint64_t)m[r].x | ((uint64_t)m[r].y << 32);
    below[r] = rank_below(same);
    leader[r] = same != 0 ? (int32_t)__builtin_ctzll(same) : lane;
    old[r] = 0;
    if (same != 0 && below[r] == 0) old[r] = atomicAdd(&cnt[wid][digit[r]], __popcll(same));
  }
  int32_t rank[kLR];
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= rounds) continue;
    rank[r] = __shfl(old[r], leader[r], kWave) + below[r];
  }
  __syncthreads();
  // digit t: each wave's offset within the digit, and the digit's count
  int32_t c[kLW];
  int tot = 0;
  if (t < kLBuckets) {
#pragma unroll
    for (int w = 0; w < kLW; ++w) c[w] = cnt[w][t];
#pragma unroll
    for (int w = 0; w < kLW; ++w) {
      const int x = c[w];
      c[w] = tot;
      tot += x;
    }
  }
  int total;
  const int start = block_exclusive_scan<kLT>(tot, s_scan, &total);
  if (t < kLBuckets) {
#pragma unroll
    for (int w = 0; w < kLW; ++w) cnt[w][t] = c[w] + start;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= rounds) continue;
    dest[r] = cnt[wid][digit[r]] + rank[r];
  }
}

// Block-wide exclusive scan of per-wave counts: every lane gets the number of
// items counted by earlier waves, and *total the block's count.
__device__ int wave_offsets(int wave_count, int32_t* s_scan, int* total) {
  const int lane = lane_id();
  const int off = block_exclusive_scan<kLT>(lane == 0 ? wave_count : 0, s_scan, total);
  return __shfl(off, 0, kWave);
}

// ---------------------------------------------------------------- kernels

__global__ __launch_bounds__(256) void k_ls_init(int32_t* __restrict__ map, int64_t P,
                                                 int32_t* __restrict__ cnt,
                                                 int32_t* __restrict__ fill, int64_t cells,
                                                 int32_t* __restrict__ hdr, int32_t n_valid,
                                                 int32_t n_occ) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < P) map[i] = -1;
  if (i < cells) {
    cnt[i] = 0;
    fill[i] = 0;
  }
  if (i < 16) hdr[i] = i == kHdrValid ? n_valid : (i == kHdrOcc ? n_occ : 0);
}

// map[q] = BEV rank of kept point p, with q the point's place in its strip's
// region (strip * maxpts + bin * pixels of the strip + local pixel), so that
// a strip reads its points contiguously in frustum order.  Points outside
// the shape's ranges are skipped: the map is never written out of bounds.
__global__ __launch_bounds__(256) void k_ls_map(const int32_t* __restrict__ rd,
                                                const int32_t* __restrict__ rb, int64_t n,
                                                int64_t P, int64_t cells, LGeom g,
                                                int32_t* __restrict__ map) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t p = rd[i], r = rb[i];
  if (p < 0 || p >= P || r < 0 || r >= cells) return;
  // (32-bit unsigned: p < 2^31)
  const uint32_t per_view = (uint32_t)g.D * (uint32_t)g.hw;
  const uint32_t bn = (uint32_t)p / per_view;
  const uint32_t rem = (uint32_t)p - bn * per_view;
  const uint32_t d = rem / (uint32_t)g.hw;
  const uint32_t pix = rem - d * (uint32_t)g.hw;
  const uint32_t h = pix / (uint32_t)g.W, w = pix - h * (uint32_t)g.W;
  const uint32_t hb = h / (uint32_t)g.bh, wb = w / (uint32_t)g.bw;
  const uint32_t h0 = hb * (uint32_t)g.bh, w0 = wb * (uint32_t)g.bw;
  const uint32_t bws = min((uint32_t)g.bw, (uint32_t)g.W - w0);
  const uint32_t bhs = min((uint32_t)g.bh, (uint32_t)g.H - h0);
  const int64_t s = ((int64_t)bn * g.nhb + hb) * g.nwb + wb;
  map[s * g.maxpts + (int64_t)d * (bhs * bws) + (h - h0) * bws + (w - w0)] = r;
}

// One workgroup per strip: its kept points sorted by (BEV rank, local pixel,
// depth bin) in LDS, cut into pairs; the pairs go to the strip's region
// (key = rank within the sample << (lp_bits + d_bits) | pixel << d_bits |
// first bin, and the point count), with the strip's pair count and the pair
// count of each of its pixels.
__global__ __launch_bounds__(kLT) void k_ls_strips(const int32_t* __restrict__ map, LGeom g,
                                                   uint32_t* __restrict__ rkey,
                                                   int32_t* __restrict__ rnpts,
                                                   int32_t* __restrict__ strip_np,
                                                   int32_t* __restrict__ pix_count) {
  __shared__ uint32_t sa[kLocalPoints], sb[kLocalPoints];
  __shared__ int32_t cnt[kLW][kLBuckets];
  __shared__ uint32_t match[kLW][kLBuckets][2];
  __shared__ int32_t s_scan[kLW];
  __shared__ int32_t pc[kLBuckets];
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int wid = t / kWave;
  const int32_t s = strip_of_block(g.strips);
  if (s < 0) return;  // (uniform over the block)
  int32_t bn, h0, w0, bhs, bws;
  g.strip(s, bn, h0, w0, bhs, bws);
  const int32_t npix = bhs * bws;
  const int32_t nf = g.D * npix;  // frustum points of the strip (<= kLocalPoints)
  const int32_t rb_base = (bn / g.N) * g.zyx;
  if (t < kLBuckets) pc[t] = 0;

  // kept points in frustum order (depth bin, then pixel): an ordered
  // compaction, so that the points of one cell and pixel stay in bin order
  const int spanf = ((nf + kLT - 1) / kLT) * kWave;  // frustum points per wave
  const int roundsf = spanf / kWave;
  const int32_t* smap = map + (int64_t)s * g.maxpts;  // the strip's points, in frustum order
  int32_t rv[kLR];
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    const int32_t j = wid * spanf + r * kWave + lane;
    rv[r] = (r < roundsf && j < nf) ? smap[j] : -1;
  }
  int pre[kLR];
  int wkept = 0;
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= roundsf) continue;
    const int32_t rel = rv[r] - rb_base;
    const bool kept = rv[r] >= 0 && rel >= 0 && rel < g.zyx;
    if (!kept) rv[r] = -1;
    const uint64_t m = wave_ballot(kept);
    pre[r] = wkept + rank_below(m);
    wkept += __popcll(m);
  }
  int n;
  const int koff = wave_offsets(wkept, s_scan, &n);
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r >= roundsf) continue;
    if (rv[r] < 0) continue;
    const int32_t j = wid * spanf + r * kWave + lane;
    const int32_t d = j / npix;
    const int32_t lp = j - d * npix;
    sa[koff + pre[r]] = ((uint32_t)(rv[r] - rb_base) << (g.lp_bits + g.d_bits)) |
                        ((uint32_t)lp << g.d_bits) | (uint32_t)d;
  }
  __syncthreads();
  const int span = ((n + kLT - 1) / kLT) * kWave;  // elements per wave
  uint32_t* src = sa;
  uint32_t* dst = sb;
  // stable LSD passes over (cell, pixel); the bins are already in order
  const int sort_bits = g.rb_bits + g.lp_bits;  // + d_bits <= 32
  if (n > 1 && sort_bits > 0) {
    const int passes = (sort_bits + 7) / 8;
    const int pbits = (sort_bits + passes - 1) / passes;
    for (int ps = 0; ps < passes; ++ps) {
      const int shift = g.d_bits + ps * pbits;
      const int bits = min(pbits, sort_bits - ps * pbits);
      const uint32_t mask = (1u << bits) - 1u;
      uint32_t key[kLR], digit[kLR];
      int32_t dest[kLR];
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        if (r * kWave >= span) continue;
        const int e = wid * span + r * kWave + lane;
        key[r] = e < n ? src[e] : 0u;
        digit[r] = (key[r] >> shift) & mask;
      }
      local_ranks(digit, n, span, cnt, match, s_scan, dest);
#pragma unroll
      for (int r = 0; r < kLR; ++r) {
        if (r * kWave >= span) continue;
        const int e = wid * span + r * kWave + lane;
        if (e < n) dst[dest[r]] = key[r];
      }
      __syncthreads();
      uint32_t* tmp = src;
      src = dst;
      dst = tmp;
    }
  }

  // pairs: a head where the cell or pixel changes or the bin is not the next
  const uint32_t dmask = (1u << g.d_bits) - 1u;
  const uint32_t lpmask = (1u << g.lp_bits) - 1u;
  bool hd[kLR];
  int wcount = 0;
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    hd[r] = false;
    if (r * kWave >= span) continue;
    const int e = wid * span + r * kWave + lane;
    const bool valid = e < n;
    const uint32_t k = valid ? src[e] : 0u;
    const uint32_t pk = (valid && e > 0) ? src[e - 1] : 0u;
    hd[r] = valid && (e == 0 || (k >> g.d_bits) != (pk >> g.d_bits) ||
                      (k & dmask) != (pk & dmask) + 1u);
    const uint64_t m = wave_ballot(hd[r]);
    pre[r] = wcount + rank_below(m);
    wcount += __popcll(m);
  }
  int np;
  const int woff = wave_offsets(wcount, s_scan, &np);
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r * kWave >= span) continue;
    const int e = wid * span + r * kWave + lane;
    if (hd[r]) dst[woff + pre[r]] = (uint32_t)e;  // head position of each pair
  }
  __syncthreads();
  const int64_t region = (int64_t)s * g.maxpts;
  for (int j = t; j < np; j += kLT) {
    const int e0 = (int)dst[j];
    const int e1 = j + 1 < np ? (int)dst[j + 1] : n;
    const uint32_t key = src[e0];
    rkey[region + j] = key;
    rnpts[region + j] = e1 - e0;
    atomicAdd(&pc[(key >> g.d_bits) & lpmask], 1);
  }
  __syncthreads();
  for (int lp = t; lp < npix; lp += kLT) {
    const int32_t hl = lp / bws;
    pix_count[(int64_t)bn * g.hw + (int64_t)(h0 + hl) * g.W + w0 + (lp - hl * bws)] = pc[lp];
  }
  if (t == 0) strip_np[s] = np;
}

// Sixteen consecutive ints a[i0 .. i0 + 16) (zero past n), loaded together
// (a and i0 aligned to 16 ints).
__device__ __forceinline__ void load16(const int32_t* __restrict__ a, int64_t i0, int64_t n,
                                       int32_t (&v)[16]) {
  if (i0 + 16 <= n) {
    const int4* q = reinterpret_cast<const int4*>(a + i0);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int4 x = q[k];
      v[4 * k] = x.x;
      v[4 * k + 1] = x.y;
      v[4 * k + 2] = x.z;
      v[4 * k + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = i0 + k < n ? a[i0 + k] : 0;
  }
}

// Exclusive scan of a[0 .. n) by one block of kLT threads, 16 values per
// thread per step; emit(i, exclusive prefix, a[i]) for every i < n, in
// order within a thread.  Returns the total.
template <typename F>
__device__ int32_t block_scan16(const int32_t* __restrict__ a, int64_t n, int32_t* s_scan,
                                F emit) {
  constexpr int64_t kStep = 16 * (int64_t)kLT;
  int32_t carry = 0;
  for (int64_t base = 0; base < n; base += kStep) {
    const int64_t i0 = base + 16 * (int64_t)threadIdx.x;
    int32_t v[16];
    load16(a, i0, n, v);
    int32_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) sum += v[k];
    int32_t tot;
    int32_t off = carry + block_exclusive_scan<kLT>(sum, s_scan, &tot);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if (i0 + k < n) emit(i0 + k, off, v[k]);
      off += v[k];
    }
    carry += tot;
  }
  return carry;
}

constexpr int kPlanStrips = 4096;  // strip offsets kept in LDS up to this many strips
constexpr int kPlanItems = 8192;   // item starts kept in LDS up to this many items

// One block: pair offsets of the strips, the items (cut at the shares) and
// their strips and first pairs, the shares' first items, and the first
// pixel-major pair of every feature row.
__global__ __launch_bounds__(kLT) void k_ls_plan(const int32_t* __restrict__ strip_np,
                                                 int32_t strips, int32_t shares, int32_t ip,
                                                 int64_t items_cap, const int32_t* __restrict__ pix_count,
                                                 int64_t rows, int32_t* __restrict__ strip_p0,
                                                 int32_t* __restrict__ strip_it0,
                                                 int32_t* __restrict__ hdr,
                                                 int32_t* __restrict__ item_strip,
                                                 int32_t* __restrict__ item_pair0,
                                                 int32_t* __restrict__ share_item0,
                                                 int32_t* __restrict__ pix_pair0) {
  __shared__ int32_t s_scan[kLW];
  __shared__ int32_t s_bad;
  __shared__ int32_t s_sp0[kPlanStrips + 1];
  __shared__ int32_t s_ip0[kPlanItems + 1];
  __shared__ int32_t s_rows[17 * kLT];
  const int t = threadIdx.x;
  if (t == 0) s_bad = 0;
  const bool lds_strips = strips <= kPlanStrips;
  // 1. pair offsets (16 consecutive strips per thread and step)
  int32_t P = 0, n_strips = 0;
  {
    int32_t carry = 0, ncarry = 0;
    for (int64_t base = 0; base < strips; base += 16 * kLT) {
      const int64_t i0 = base + 16 * t;
      int32_t v[16];
      load16(strip_np, i0, strips, v);
      int32_t sum = 0, ne = 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        sum += v[k];
        ne += v[k] > 0 ? 1 : 0;
      }
      int32_t tot, ntot;
      int32_t off = carry + block_exclusive_scan<kLT>(sum, s_scan, &tot);
      block_exclusive_scan<kLT>(ne, s_scan, &ntot);
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        if (i0 + k < strips) {
          strip_p0[i0 + k] = off;
          if (lds_strips) s_sp0[i0 + k] = off;
        }
        off += v[k];
      }
      carry += tot;
      ncarry += ntot;
    }
    P = carry;
    n_strips = ncarry;
  }
  if (t == 0) {
    strip_p0[strips] = P;
    if (lds_strips) s_sp0[strips] = P;
  }
  __syncthreads();  // (global and LDS writes above are visible to the block after it)
  const int32_t* sp0 = lds_strips ? s_sp0 : strip_p0;
  // 2. items of every strip (contiguous strips per thread)
  const int32_t per = (strips + kLT - 1) / kLT;
  const int32_t s_lo = min(strips, t * per), s_hi = min(strips, s_lo + per);
  int64_t isum = 0;
  for (int32_t s = s_lo; s < s_hi; ++s) {
    const int32_t a = sp0[s], v = sp0[s + 1] - a;
    if (v > 0) isum += strip_items(a, a + v, P, shares, ip, [](int64_t, int64_t) {});
  }
  int32_t n_items;
  int32_t ioff = block_exclusive_scan<kLT>((int32_t)isum, s_scan, &n_items);
  const bool lds_items = n_items <= kPlanItems && n_items <= items_cap;
  for (int32_t s = s_lo; s < s_hi; ++s) {
    const int32_t a = sp0[s], v = sp0[s + 1] - a;
    strip_it0[s] = ioff;
    if (v > 0) {
      const int32_t first_item = ioff;
      ioff += (int32_t)strip_items(a, a + v, P, shares, ip, [&](int64_t i, int64_t first) {
        const int64_t item = first_item + i;
        if (item < items_cap) {
          item_strip[item] = s;
          item_pair0[item] = (int32_t)first;
          if (lds_items) s_ip0[item] = (int32_t)first;
        }
      });
    }
  }
  if (t == 0) {
    strip_it0[strips] = n_items;
    if (n_items <= items_cap) item_pair0[n_items] = P;
    hdr[kHdrPairs] = P;
    hdr[kHdrItems] = n_items;
    hdr[kHdrStrips] = n_strips;
  }
  __syncthreads();
  const int32_t* ip0 = lds_items ? s_ip0 : item_pair0;
  // 3. shares: boundary w snapped within its strip, then the first item at
  // or after it
  const int32_t n_it = (int32_t)min<int64_t>(n_items, items_cap);
  for (int w = t; w <= shares; w += kLT) {
    int64_t c = ((int64_t)P * w) / shares;
    if (c > 0 && c < P) {  // the last strip starting at or before c holds it
      int32_t lo = 0, hi = strips - 1;
      while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (sp0[mid] <= c) lo = mid; else hi = mid - 1;
      }
      c = snap_bound(c, sp0[lo], sp0[lo + 1]);
    }
    int32_t lo = 0, hi = n_it;
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (ip0[mid] < c) lo = mid + 1; else hi = mid;
    }
    share_item0[w] = lo;
  }
  __syncthreads();
  for (int w = t; w < shares; w += kLT)
    if (share_item0[w + 1] - share_item0[w] > kShareItems) s_bad = 1;
  // 4. first pixel-major pair of every feature row, 16 rows per thread and
  // step; the prefixes go through LDS (17 words per thread, against bank
  // conflicts) so that lanes store consecutive entries
  int32_t rtot = 0;
  for (int64_t base = 0; base < rows; base += 16 * kLT) {
    const int64_t i0 = base + 16 * (int64_t)t;
    int32_t v[16];
    load16(pix_count, i0, rows, v);
    int32_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) sum += v[k];
    int32_t tot;
    int32_t off = rtot + block_exclusive_scan<kLT>(sum, s_scan, &tot);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      s_rows[17 * t + k] = off;
      off += v[k];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int e = j * kLT + t;  // element of this step, staged at 17 * (e / 16) + e % 16
      if (base + e < rows) pix_pair0[base + e] = s_rows[17 * (e >> 4) + (e & 15)];
    }
    __syncthreads();
    rtot += tot;
  }
  if (t == 0) {
    pix_pair0[rows] = rtot;
    hdr[kHdrShares] = shares;
    hdr[kHdrSharesOk] = s_bad ? 0 : 1;
    hdr[kHdrItemPairs] = ip;
  }
}

// One workgroup per strip: the pair records at their global positions, the
// segment index of each pair within its item, the segment count of each
// item, the segment count of each cell, the BEV rank of each segment's first
// pair, and the pixel-major pairs.
__global__ __launch_bounds__(kLT) void k_ls_emit(
    LGeom g, const uint32_t* __restrict__ rkey, const int32_t* __restrict__ rnpts,
    const int32_t* __restrict__ strip_np, const int32_t* __restrict__ strip_p0,
    const int32_t* __restrict__ strip_it0, const int32_t* __restrict__ item_pair0,
    int64_t items_cap, const int32_t* __restrict__ pix_pair0, int32_t* __restrict__ item_nseg,
    int32_t* __restrict__ cell_nseg, int32_t* __restrict__ head_cell,
    int32_t* __restrict__ head_item,
    int32_t* __restrict__ pair_rd0, uint32_t* __restrict__ pair_ln,
    uint16_t* __restrict__ pair_seg, int32_t* __restrict__ bp_cell,
    uint32_t* __restrict__ bp_dn) {
  __shared__ int32_t cnt[kLW][kLBuckets];
  __shared__ uint32_t match[kLW][kLBuckets][2];
  __shared__ int32_t s_scan[kLW];
  __shared__ int32_t s_items[kLItems + 1];
  __shared__ int32_t s_iseg[kLItems + 1];
  __shared__ int32_t s_pix0[kLBuckets];  // first pixel-major pair of each pixel of the strip
  const int t = threadIdx.x;
  const int lane = lane_id();
  const int wid = t / kWave;
  const int32_t s = strip_of_block(g.strips);
  if (s < 0) return;  // (uniform over the block)
  const int np = strip_np[s];
  if (np == 0) return;
  const int32_t P0 = strip_p0[s];
  const int32_t it0 = strip_it0[s];
  const int32_t K = strip_it0[s + 1] - it0;
  if (K < 1 || K > kLItems || (int64_t)it0 + K > items_cap) return;  // (cannot happen)
  int32_t bn, h0, w0, bhs, bws;
  g.strip(s, bn, h0, w0, bhs, bws);
  const int32_t rb_base = (bn / g.N) * g.zyx;
  for (int k = t; k <= K; k += kLT) s_items[k] = item_pair0[it0 + k];
  for (int lp = t; lp < bhs * bws; lp += kLT) {  // (at most kLBuckets pixels)
    const int32_t hl = lp / bws;
    s_pix0[lp] = pix_pair0[(int64_t)bn * g.hw + (int64_t)(h0 + hl) * g.W + w0 + (lp - hl * bws)];
  }
  __syncthreads();

  const int span = ((np + kLT - 1) / kLT) * kWave;
  const int64_t region = (int64_t)s * g.maxpts;
  const int rb_shift = g.lp_bits + g.d_bits;
  const uint32_t dmask = (1u << g.d_bits) - 1u;
  const uint32_t lpmask = (1u << g.lp_bits) - 1u;
  uint32_t key[kLR], digit[kLR];
  int32_t npts[kLR], item[kLR], sin[kLR];
  bool hd[kLR];
  int wcount = 0;
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    hd[r] = false;
    if (r * kWave >= span) continue;
    const int e = wid * span + r * kWave + lane;
    const bool valid = e < np;
    key[r] = valid ? rkey[region + e] : 0u;
    const uint32_t pk = (valid && e > 0) ? rkey[region + e - 1] : 0u;
    npts[r] = valid ? rnpts[region + e] : 0;
    const int32_t gp = P0 + e;
    item[r] = valid ? upper_index(s_items, K, gp) : 0;
    const bool start = valid && s_items[item[r]] == gp;
    hd[r] = valid && (start || (key[r] >> rb_shift) != (pk >> rb_shift));
    const uint64_t m = wave_ballot(hd[r]);
    sin[r] = wcount + rank_below(m) + (hd[r] ? 1 : 0);  // inclusive, within the wave
    wcount += __popcll(m);
    digit[r] = (key[r] >> g.d_bits) & lpmask;
  }
  int nseg;
  const int woff = wave_offsets(wcount, s_scan, &nseg);
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r * kWave >= span) continue;
    sin[r] += woff - 1;  // segment of the pair within the strip
    const int e = wid * span + r * kWave + lane;
    if (e < np && s_items[item[r]] == P0 + e) s_iseg[item[r]] = sin[r];
  }
  __syncthreads();
  for (int k = t; k < K; k += kLT)
    item_nseg[it0 + k] = (k + 1 < K ? s_iseg[k + 1] : nseg) - s_iseg[k];
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r * kWave >= span) continue;
    const int e = wid * span + r * kWave + lane;
    if (e >= np) continue;
    const int32_t gp = P0 + e;
    const uint32_t lp = (key[r] >> g.d_bits) & lpmask;
    const int32_t d0 = (int32_t)(key[r] & dmask);
    const int32_t hl = (int32_t)lp / bws;
    const int32_t cell = rb_base + (int32_t)(key[r] >> rb_shift);
    pair_rd0[gp] = (int32_t)(((int64_t)(bn * g.D + d0) * g.H + h0 + hl) * g.W + w0 +
                             ((int32_t)lp - hl * bws));
    pair_ln[gp] = (lp & kPairPixel) | (hd[r] ? kPairHead : 0u) | ((uint32_t)npts[r] << 16);
    pair_seg[gp] = (uint16_t)(sin[r] - s_iseg[item[r]]);
    if (hd[r]) {
      atomicAdd(&cell_nseg[cell], 1);
      head_cell[gp] = cell;
      head_item[gp] = it0 + item[r];
    }
  }
  // pixel-major pairs: a stable pass by local pixel
  int32_t dest[kLR];
  local_ranks(digit, np, span, cnt, match, s_scan, dest);
#pragma unroll
  for (int r = 0; r < kLR; ++r) {
    if (r * kWave >= span) continue;
    const int e = wid * span + r * kWave + lane;
    if (e >= np) continue;
    const int32_t lp = (int32_t)digit[r];
    const int32_t q = s_pix0[lp] + (dest[r] - cnt[0][lp]);
    bp_cell[q] = rb_base + (int32_t)(key[r] >> rb_shift);
    bp_dn[q] = (key[r] & dmask) | ((uint32_t)npts[r] << 16);
  }
}

// The cells in chunks of 2^chunk_shift >= kCChunk cells, at most
// kMaxCChunks of them.  First each chunk's totals: the slots of its cells with
// several segments, their number, and its number of empty cells.
constexpr int kCT = 256;             // threads of the cell-scan kernels
constexpr int kCChunkShift = 10;
constexpr int kCChunk = 1 << kCChunkShift;  // cells per step of a block: 4 per thread
static_assert(kCChunk == 4 * kCT, "one int4 of counts per thread");
constexpr int kMaxCChunks = 1024;

// a[i0 .. i0 + 4) with in-range flags (a and i0 aligned to 4 ints)
__device__ __forceinline__ int4 load4(const int32_t* __restrict__ a, int64_t i0, int64_t n) {
  if (i0 + 4 <= n) return *reinterpret_cast<const int4*>(a + i0);
  return make_int4(i0 < n ? a[i0] : 0, i0 + 1 < n ? a[i0 + 1] : 0, i0 + 2 < n ? a[i0 + 2] : 0,
                   i0 + 3 < n ? a[i0 + 3] : 0);
}

__global__ __launch_bounds__(kCT) void k_ls_cell_totals(const int32_t* __restrict__ cell_nseg,
                                                        int64_t cells, int chunk_shift,
                                                        int4* __restrict__ chunk_tot) {
  __shared__ int32_t s_scan[kCT / kWave];
  const int64_t c_begin = (int64_t)blockIdx.x << chunk_shift;
  const int64_t c_end = min<int64_t>(cells, c_begin + (int64_t(1) << chunk_shift));
  int32_t ss = 0, sc = 0, se = 0;
  for (int64_t c0 = c_begin + 4 * threadIdx.x; c0 < c_end; c0 += kCChunk) {
    const int4 x = load4(cell_nseg, c0, c_end);
    const int32_t v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      ss += v[k] > 1 ? v[k] : 0;
      sc += v[k] > 1 ? 1 : 0;
      se += (c0 + k < c_end && v[k] == 0) ? 1 : 0;
    }
  }
  int32_t ts, tc, te;
  block_exclusive_scan<kCT>(ss, s_scan, &ts);
  block_exclusive_scan<kCT>(sc, s_scan, &tc);
  block_exclusive_scan<kCT>(se, s_scan, &te);
  if (threadIdx.x == 0) chunk_tot[blockIdx.x] = make_int4(ts, tc, te, 0);
}

// Blocks 0 .. nchunks - 1: the first slot of each cell with several segments,
// the list of those cells with their first slots, and the list of empty
// cells, each chunk adding the totals of the chunks before it; the lists go
// through LDS so that lanes store consecutive entries.  Block nchunks: the
// first segment of every item (an exclusive scan of the items' segment
// counts) and the segment count.
__global__ __launch_bounds__(kCT) void k_ls_cells(
    int32_t* __restrict__ hdr, const int32_t* __restrict__ item_nseg, int64_t items_cap,
    const int32_t* __restrict__ cell_nseg, int64_t cells, int chunk_shift,
    const int4* __restrict__ chunk_tot, int32_t nchunks, int32_t* __restrict__ item_seg0,
    int32_t* __restrict__ slot0, int32_t* __restrict__ comb_cell,
    int32_t* __restrict__ comb_slot0, int64_t comb_cap, int32_t* __restrict__ empty,
    int64_t empty_cap) {
  __shared__ int32_t s_scan[kCT / kWave];
  __shared__ int32_t s_a[kCChunk], s_b[kCChunk], s_e[kCChunk];
  const int t = threadIdx.x;
  if ((int32_t)blockIdx.x == nchunks) {  // (uniform)
    const int64_t n_items = min<int64_t>(hdr[kHdrItems], items_cap);
    int32_t carry = 0;
    for (int64_t b0 = 0; b0 < n_items; b0 += kCChunk) {
      const int4 x = load4(item_nseg, b0 + 4 * t, n_items);
      const int32_t v[4] = {x.x, x.y, x.z, x.w};
      int32_t tot;
      int32_t off = carry + block_exclusive_scan<kCT>(v[0] + v[1] + v[2] + v[3], s_scan, &tot);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        s_a[4 * t + k] = off;
        off += v[k];
      }
      __syncthreads();
      for (int i = t; i < kCChunk; i += kCT)
        if (b0 + i < n_items) item_seg0[b0 + i] = s_a[i];
      __syncthreads();
      carry += tot;
    }
    if (t == 0) {
      if (n_items == hdr[kHdrItems]) item_seg0[n_items] = carry;
      hdr[kHdrSegs] = carry;
    }
    return;
  }
  // the totals of the chunks before this one
  int32_t ps = 0, pc = 0, pe = 0;
  for (int k = t; k < (int)blockIdx.x; k += kCT) {
    const int4 x = chunk_tot[k];
    ps += x.x;
    pc += x.y;
    pe += x.z;
  }
  int32_t cs, cc, ce;
  block_exclusive_scan<kCT>(ps, s_scan, &cs);
  block_exclusive_scan<kCT>(pc, s_scan, &cc);
  block_exclusive_scan<kCT>(pe, s_scan, &ce);
  const int64_t c_begin = (int64_t)blockIdx.x << chunk_shift;
  const int64_t c_end = min<int64_t>(cells, c_begin + (int64_t(1) << chunk_shift));
  for (int64_t b0 = c_begin; b0 < c_end; b0 += kCChunk) {
    const int64_t c0 = b0 + 4 * t;
    const int4 x = load4(cell_nseg, c0, c_end);
    const int32_t v[4] = {x.x, x.y, x.z, x.w};
    int32_t ss = 0, sc = 0, se = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      ss += v[k] > 1 ? v[k] : 0;
      sc += v[k] > 1 ? 1 : 0;
      se += (c0 + k < c_end && v[k] == 0) ? 1 : 0;
    }
    int32_t ts, tc, te;
    int32_t so = cs + block_exclusive_scan<kCT>(ss, s_scan, &ts);
    int32_t co = block_exclusive_scan<kCT>(sc, s_scan, &tc);
    int32_t eo = block_exclusive_scan<kCT>(se, s_scan, &te);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t c = c0 + k;
      if (c >= c_end) continue;
      if (v[k] > 1) {
        slot0[c] = so;
        s_a[co] = (int32_t)c;
        s_b[co] = so;
        so += v[k];
        ++co;
      } else if (v[k] == 0) {
        s_e[eo] = (int32_t)c;
        ++eo;
      }
    }
    __syncthreads();
    for (int i = t; i < tc; i += kCT) {
      const int64_t q = (int64_t)cc + i;
      if (q < comb_cap) {
        comb_cell[q] = s_a[i];
        comb_slot0[q] = s_b[i];
      }
    }
    for (int i = t; i < te; i += kCT) {
      const int64_t q = (int64_t)ce + i;
      if (q < empty_cap) empty[q] = s_e[i];
    }
    __syncthreads();
    cs += ts;
    cc += tc;
    ce += te;
  }
  if ((int32_t)blockIdx.x == nchunks - 1 && t == 0) {
    comb_slot0[min<int64_t>(cc, comb_cap)] = cs;
    hdr[kHdrSlots] = cs;
    hdr[kHdrComb] = cc;
    hdr[kHdrEmpty] = ce;
    hdr[kHdrOccFound] = (int32_t)(cells - ce);
  }
}

// Every segment: its destination when its cell has no other segment; else
// its index joins its cell's list of slots (in any order; ranked below).
__global__ __launch_bounds__(256) void k_ls_segments(
    const int32_t* __restrict__ hdr, const uint32_t* __restrict__ pair_ln,
    const uint16_t* __restrict__ pair_seg, const int32_t* __restrict__ head_cell,
    const int32_t* __restrict__ head_item, const int32_t* __restrict__ item_seg0,
    const int32_t* __restrict__ cell_nseg, const int32_t* __restrict__ slot0,
    int32_t* __restrict__ fill, int32_t* __restrict__ slot_seg, int32_t* __restrict__ seg_dest) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= hdr[kHdrPairs] || !(pair_ln[k] & kPairHead)) return;
  const int32_t seg = item_seg0[head_item[k]] + pair_seg[k];
  const int32_t cell = head_cell[k];
  if (cell_nseg[cell] == 1) {
    seg_dest[seg] = cell;
  } else {
    slot_seg[slot0[cell] + atomicAdd(&fill[cell], 1)] = seg;
  }
}

// Every slot: the cells with several segments list their segments (in any
// order); a segment's slot is its cell's first slot plus the number of the
// cell's segments with a smaller index, so the segments of a cell get its
// slots in ascending order.
__global__ __launch_bounds__(256) void k_ls_slots(const int32_t* __restrict__ hdr,
                                                  const int32_t* __restrict__ comb_slot0,
                                                  int64_t comb_cap,
                                                  const int32_t* __restrict__ slot_seg,
                                                  int32_t* __restrict__ seg_dest) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kHdrSlots]) return;
  const int32_t n_comb = (int32_t)min<int64_t>(hdr[kHdrComb], comb_cap);
  if (n_comb < 1) return;
  const int32_t j = upper_index(comb_slot0, n_comb, (int32_t)q);
  const int32_t s0 = comb_slot0[j], s1 = comb_slot0[j + 1];
  const int32_t v = slot_seg[q];
  int32_t rank = 0;
  int32_t i = s0;
  for (; i + 8 <= s1; i += 8) {
    int32_t a[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) a[k] = slot_seg[i + k];
#pragma unroll
    for (int k = 0; k < 8; ++k) rank += a[k] < v ? 1 : 0;
  }
  for (; i < s1; ++i) rank += slot_seg[i] < v ? 1 : 0;
  seg_dest[v] = ~(s0 + rank);
}

int bits_for(int64_t n) {  // bits of the values 0 .. n - 1
  int b = 0;
  while ((int64_t(1) << b) < n) ++b;
  return b;
}

}  // namespace

bool schedule_local_ok(const Dims& d, int64_t n_valid) {
  const StripDims sd = strip_dims(d);
  if (n_valid <= 0) return false;
  if (sd.pixels > kLBuckets || sd.pixels * d.D > kLocalPoints) return false;
  if (sd.strips > INT32_MAX - 1) return false;
  const int64_t zyx = d.Z * d.Y * d.X;
  return bits_for(zyx) + bits_for(sd.pixels) + bits_for(d.D) <= 32;
}

void local_schedule_ws(const Dims& d, ScheduleLayout& L) {
  size_t off = 0;
  auto take = [&](size_t n_ints) {
    const size_t o = off;
    off += (sizeof(int32_t) * n_ints + 255) & ~size_t(255);
    return o;
  };
  const size_t nv = (size_t)(L.n_valid > 0 ? L.n_valid : 1);
  const size_t region = (size_t)L.sd.strips * (size_t)(L.sd.pixels * d.D);
  L.wl_map = take(region);
  L.wl_rkey = take(region);
  L.wl_rnpts = take(region);
  L.wl_strip_np = take((size_t)L.sd.strips + 1);
  L.wl_strip_p0 = take((size_t)L.sd.strips + 1);
  L.wl_strip_it0 = take((size_t)L.sd.strips + 1);
  L.wl_pix_count = take((size_t)d.rows);
  L.wl_item_nseg = take((size_t)L.items_cap + 1);
  L.wl_cell_nseg = take((size_t)d.cells);
  L.wl_fill = take((size_t)d.cells);
  L.wl_slot0 = take((size_t)d.cells);
  L.wl_head_cell = take(nv);
  L.wl_head_item = take(nv);
  L.wl_slot_seg = take(nv);
  L.wl_cell_shift = kCChunkShift;
  while (((d.cells - 1) >> L.wl_cell_shift) + 1 > kMaxCChunks) ++L.wl_cell_shift;
  L.wl_cell_chunks = ((d.cells - 1) >> L.wl_cell_shift) + 1;
  L.wl_cell_tot = take(4 * (size_t)L.wl_cell_chunks);
  L.wl_total = off;
}

hipError_t launch_schedule_local(const Dims& d, const int32_t* rd, const int32_t* rb,
                                 int32_t n_valid, int32_t n_intervals, void* schedule,
                                 void* workspace, hipStream_t stream) {
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  char* sc = static_cast<char*>(schedule);
  char* ws = static_cast<char*>(workspace);
  auto S = [&](size_t o) { return reinterpret_cast<int32_t*>(sc + o); };
  auto W = [&](size_t o) { return reinterpret_cast<int32_t*>(ws + o); };
  int32_t* hdr = S(L.header);
  LGeom g{};
  g.N = (int32_t)d.N;
  g.D = (int32_t)d.D;
  g.H = (int32_t)d.H;
  g.W = (int32_t)d.W;
  g.bh = (int32_t)L.sd.bh;
  g.bw = (int32_t)L.sd.bw;
  g.nhb = (int32_t)L.sd.nhb;
  g.nwb = (int32_t)L.sd.nwb;
  g.strips = (int32_t)L.sd.strips;
  g.hw = (int32_t)d.hw;
  g.zyx = (int32_t)(d.Z * d.Y * d.X);
  g.maxpts = (int32_t)(L.sd.pixels * d.D);
  g.d_bits = bits_for(d.D);
  g.lp_bits = bits_for(L.sd.pixels);
  g.rb_bits = bits_for(g.zyx);
  const int32_t shares = (int32_t)std::min<int64_t>(forward_workgroups(), kMaxShares);
  int32_t* map = W(L.wl_map);
  uint32_t* rkey = reinterpret_cast<uint32_t*>(W(L.wl_rkey));
  int32_t* rnpts = W(L.wl_rnpts);
  int32_t* strip_np = W(L.wl_strip_np);
  int32_t* strip_p0 = W(L.wl_strip_p0);
  int32_t* strip_it0 = W(L.wl_strip_it0);
  int32_t* pix_count = W(L.wl_pix_count);
  int32_t* item_nseg = W(L.wl_item_nseg);
  int32_t* cell_nseg = W(L.wl_cell_nseg);
  int32_t* fill = W(L.wl_fill);
  int32_t* slot0 = W(L.wl_slot0);
  int32_t* head_cell = W(L.wl_head_cell);
  int32_t* head_item = W(L.wl_head_item);
  int32_t* slot_seg = W(L.wl_slot_seg);

  const int64_t region = L.sd.strips * (L.sd.pixels * d.D);
  const int64_t span = std::max<int64_t>(std::max<int64_t>(region, d.cells), 16);
  k_ls_init<<<(unsigned)((span + 255) / 256), 256, 0, stream>>>(map, region, cell_nseg, fill,
                                                                 d.cells, hdr, n_valid, n_intervals);
  const unsigned g_nv = (unsigned)((n_valid + 255) / 256);
  k_ls_map<<<g_nv, 256, 0, stream>>>(rd, rb, n_valid, d.P, d.cells, g, map);
  const unsigned strip_blocks = (unsigned)((L.sd.strips + kXcds - 1) / kXcds * kXcds);
  k_ls_strips<<<strip_blocks, kLT, 0, stream>>>(map, g, rkey, rnpts, strip_np, pix_count);
  k_ls_plan<<<1, kLT, 0, stream>>>(strip_np, g.strips, shares, schedule_item_pairs(n_valid),
                                   L.items_cap, pix_count, d.rows,
                                   strip_p0, strip_it0, hdr, S(L.item_strip), S(L.item_pair0),
                                   S(L.share_item0), S(L.pix_pair0));
  k_ls_emit<<<strip_blocks, kLT, 0, stream>>>(
      g, rkey, rnpts, strip_np, strip_p0, strip_it0, S(L.item_pair0), L.items_cap, S(L.pix_pair0),
      item_nseg, cell_nseg, head_cell, head_item, S(L.pair_rd0), reinterpret_cast<uint32_t*>(S(L.pair_ln)),
      reinterpret_cast<uint16_t*>(S(L.pair_seg)), S(L.bp_cell),
      reinterpret_cast<uint32_t*>(S(L.bp_dn)));
  int4* cell_tot = reinterpret_cast<int4*>(ws + L.wl_cell_tot);
  const int32_t nchunks = (int32_t)L.wl_cell_chunks;
  k_ls_cell_totals<<<(unsigned)nchunks, kCT, 0, stream>>>(cell_nseg, d.cells, L.wl_cell_shift,
                                                         cell_tot);
  k_ls_cells<<<(unsigned)nchunks + 1, kCT, 0, stream>>>(
      hdr, item_nseg, L.items_cap, cell_nseg, d.cells, L.wl_cell_shift, cell_tot, nchunks,
      S(L.item_seg0), slot0, S(L.comb_cell), S(L.comb_slot0), L.n_occ, S(L.empty), L.n_empty);
  k_ls_segments<<<g_nv, 256, 0, stream>>>(hdr, reinterpret_cast<const uint32_t*>(S(L.pair_ln)),
                                          reinterpret_cast<const uint16_t*>(S(L.pair_seg)),
                                          head_cell, head_item, S(L.item_seg0), cell_nseg, slot0,
                                          fill, slot_seg, S(L.seg_dest));
  k_ls_slots<<<g_nv, 256, 0, stream>>>(hdr, S(L.comb_slot0), L.n_occ, slot_seg, S(L.seg_dest));
  return hipGetLastError();
}

}  // namespace bevpool
