// Scheduled BEVPoolv2 pooling: the same sum as bevpool_forward (section 2.1),
// driven by a strip schedule built once from the plan (prepare.hip; the
// layout is described in internal.h).
//
// A strip is a block of image pixels, normally whole pixel columns of one
// camera.  The frustum points of a pixel column lie in one vertical plane, so
// a strip's kept points fall into few BEV cells, and the strip's feature rows
// are few enough to sit in LDS.  The work is therefore organised around the
// image instead of the grid: every feature row is read from memory once per
// item, every pair (one cell, one pixel, a run of consecutive depth bins)
// reads its row from LDS, and only the cells a strip shares with its
// neighbours need a second pass.
//
//   k_fwd_strips   one persistent workgroup per compute unit and channel
//                  chunk (up to 64 vectors), taking one share of the items
//                  (a contiguous run of strips) and two LDS item buffers:
//     1. loading waves fill one buffer with the next item: the strip's feature
//        rows (this chunk; 16-byte vectors go straight from memory into
//        LDS), the item's pair records, each pair's weight (the sum of its
//        points' depth scores, gathered) and the segment destinations;
//     2. meanwhile walking waves sum the current item from the other buffer:
//        its pairs are cut into equal ranges, one per lane group (one lane per
//        vector of the chunk); each group sums weight x feature row over its
//        range, reading both from LDS, and stores each segment it holds whole;
//     3. a segment cut by range boundaries is added up in range order by the
//        loading waves from partial sums the walkers leave in the walked
//        buffer.  Each segment's sum is stored once: into `out` when the
//        segment alone covers its cell, else into its slot.
//   k_fwd_combine  one lane group per cell covered by several segments (adds
//                  its slots in segment order and stores the cell) or per
//                  empty cell (stores zeros).
//
// Every element of `out` is written exactly once and no atomics are used;
// the summation order depends only on the schedule, so results are bitwise
// reproducible.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

#include <algorithm>
#include <atomic>
#include <mutex>
#include <type_traits>

namespace bevpool {

namespace {

// 16 bytes per lane from memory straight into LDS (global_load_lds_dwordx4):
// lane i of the wave writes at lds + 16 i, lds being the same for the wave.
// (A plain device function: inside the kernel template the builtin keeps the
// host pass from emitting the kernel's launch stub.)
__device__ __forceinline__ void global_to_lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// One workgroup per CU: kLoadWaves waves fetch the next item into one LDS
// buffer while the other waves walk the current item in the other.
constexpr int kNT = 1024;
constexpr int kWaves = kNT / kWave;
constexpr int kLoadWaves = 4;
constexpr int kWalkWaves = kWaves - kLoadWaves;
constexpr int kLoadThreads = kLoadWaves * kWave;
constexpr int kDepthBurst = 2;  // depth scores per pair loaded before any is summed
constexpr int kRowBatch = 8;    // row vectors per loading thread in flight
constexpr int kPairBatch = 8;   // pair records per loading thread in flight
// LDS of one item buffer for items of up to ip pairs: rows | pair records |
// destinations
constexpr int buf_bytes(int ip) { return kStripBytes + ip * 12; }
constexpr int kHdrCache = 128;  // item headers of a workgroup kept in LDS
constexpr int kCombThreads = 256;
static_assert(kStripBytes % (16 * kLoadThreads) == 0, "row vectors split evenly over the loading threads");
static_assert(kItemPairs % kNT == 0 && kItemPairs % kLoadThreads == 0 &&
                  kItemPairsBig % kNT == 0 && kItemPairsBig % kLoadThreads == 0,
              "pair records split evenly over the loading threads");
static_assert(kItemPairsBig <= 65536, "segment index fits 16 bits");
static_assert(2 * buf_bytes(kItemPairsBig) + 16 * 1024 <= 160 * 1024, "two big item buffers fit LDS");
static_assert(kShareItems <= kHdrCache, "a share's item headers fit the cache");

struct StripArgs {
  const int32_t* hdr;
  const int32_t* pair_rd0;
  const uint32_t* pair_ln;
  const uint16_t* pair_seg;
  const int32_t* item_strip;
  const int32_t* item_pair0;
  const int32_t* item_seg0;
  const int32_t* seg_dest;
  const int32_t* comb_cell;
  const int32_t* comb_slot0;
  const int32_t* empty;
  const int32_t* share_item0;
  float* slots;
  int64_t slot_cap;  // slots the workspace holds
  int32_t n_valid, n_occ, n_slots, items_cap;  // counts the launch was sized from
  int32_t item_pairs;  // the item size the launch's kernel holds (schedule_item_pairs)
  const double* lse;  // fused depth softmax: per-pixel log-sum-exp of the logits (else unused)
  int32_t dhw;       // D * H * W (points of one view)
  int32_t C, H, W, bh, bw, nhb, nwb, strips;
  int32_t hw32;    // H * W
  int64_t P, cells, n_empty;
};

// The schedule's header must hold the counts the launch was sized from.
__device__ __forceinline__ bool header_ok(const StripArgs& a) {
  const int32_t* hdr = a.hdr;
  return hdr[kHdrOcc] == a.n_occ && hdr[kHdrOccFound] == a.n_occ && hdr[kHdrValid] == a.n_valid &&
         hdr[kHdrSlots] == a.n_slots && hdr[kHdrItemPairs] == a.item_pairs;
}

struct PairRec {
  float w;      // summed depth score
  uint32_t ps;  // row offset (local pixel * vectors per row) | segment << 19 | kRecHead
};
constexpr uint32_t kRecHead = 1u << 31;  // first pair of a segment
constexpr int kRecSegShift = 19;
constexpr uint32_t kRecOff = (1u << kRecSegShift) - 1;
static_assert(kItemPairsBig <= (1 << (31 - kRecSegShift)), "segment index fits its field");
static_assert(kStripBytes / 2 <= (int)kRecOff + 1, "row offset (in staged elements) fits its field");

// Raw element vector moved between memory and LDS without conversion.
template <typename T, int VEC>
struct Raw {
  typedef T type;
};
template <>
struct Raw<float, 4> {
  typedef float4_t type;
};
template <>
struct Raw<half_t, 8> {
  typedef half8_t type;
};
template <>
struct Raw<float, 8> {  // two 16-byte vectors per lane
  typedef float4_t type;
};
// 16-byte (or scalar) vectors of one lane's VEC elements
template <typename T, int VEC>
constexpr int raw_parts() {
  return VEC * (int)sizeof(T) > 16 ? VEC * (int)sizeof(T) / 16 : 1;
}
// Lanes of a channel chunk: a chunk holds at most 1 KB of each pixel's row,
// the budget the strip size is computed with.
template <typename T, int VEC>
constexpr int chunk_lanes() {
  return 1024 / (VEC * (int)sizeof(T)) < kWave ? 1024 / (VEC * (int)sizeof(T)) : kWave;
}

template <typename T, int VEC>
__device__ __forceinline__ void raw_to_float(const typename Raw<T, VEC>::type& r, float* v);
template <>
__device__ __forceinline__ void raw_to_float<float, 1>(const float& r, float* v) { v[0] = r; }
template <>
__device__ __forceinline__ void raw_to_float<half_t, 1>(const half_t& r, float* v) {
  v[0] = (float)r;
}
template <>
__device__ __forceinline__ void raw_to_float<float, 4>(const float4_t& r, float* v) {
  v[0] = r.x; v[1] = r.y; v[2] = r.z; v[3] = r.w;
}
template <>
__device__ __forceinline__ void raw_to_float<half_t, 8>(const half8_t& r, float* v) {
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)r[e];
}
template <>
__device__ __forceinline__ void raw_to_float<float, 8>(const float4_t& r, float* v) {
  v[0] = r.x; v[1] = r.y; v[2] = r.z; v[3] = r.w;
}
// A lane's VEC elements of a staged row: kNV parts at row + part * cvc.
template <typename TIn, int VEC>
__device__ __forceinline__ void lane_row(const typename Raw<TIn, VEC>::type* p, int cvc, float* v) {
  constexpr int kNV = raw_parts<TIn, VEC>();
  constexpr int kPer = VEC / kNV;
#pragma unroll
  for (int h = 0; h < kNV; ++h) raw_to_float<TIn, VEC>(p[h * cvc], v + h * kPer);
}

// The largest batch of at most m loads that divides n loads.
constexpr int whole_batch(int n, int m) {
  int b = n < m ? n : m;
  while (b > 1 && n % b != 0) --b;
  return b > 0 ? b : 1;
}

// An item's header, the same for the whole workgroup.
struct ItemHdr {
  int32_t strip, p0, np, g0, nseg;
};

// SM: `depth` holds depth logits, and a point's depth score is
// exp(logit - lse[pixel]) (the softmax over the pixel's depth bins, with the
// log-sum-exp from k_depth_lse), formed as the points are gathered.
template <typename TIn, typename TOut, int VEC, bool SM, int IP>
__global__ __launch_bounds__(kNT) void k_fwd_strips(const TIn* __restrict__ depth,
                                                    const TIn* __restrict__ feat,
                                                    TOut* __restrict__ out, StripArgs a) {
  typedef typename Raw<TIn, VEC>::type RawT;
  constexpr int kUnroll = VEC >= 8 ? 2 : 4;    // pairs per step of the accumulation walk
  constexpr int kNV = raw_parts<TIn, VEC>();  // staged vectors per lane and row
  constexpr int kPer = VEC / kNV;            // elements per staged vector
  // two buffers of [rows, then partial sums | pair records | segment destinations]
  constexpr int kBufBytes = buf_bytes(IP);
  __shared__ __attribute__((aligned(16))) char smem[2 * kBufBytes];
  __shared__ int32_t s_hdr[3][kHdrCache + 1];  // strip, first pair, first segment
  __shared__ int4 s_meta[kWalkWaves * kWave];  // each lane group's last walked range
  __shared__ int32_t s_lsync;                  // arrivals of the loading waves (loader_sync)

  static_assert((int64_t)kWaves * kWave * 8 * sizeof(float) <= kStripBytes, "partial sums fit the row area");
  static_assert(IP <= 65535, "pair indices fit 16 bits");
  auto buf_rows = [&](int b) { return reinterpret_cast<RawT*>(smem + b * kBufBytes); };
  auto buf_pr = [&](int b) { return reinterpret_cast<PairRec*>(smem + b * kBufBytes + kStripBytes); };
  auto buf_dest = [&](int b) {
    return reinterpret_cast<int32_t*>(smem + b * kBufBytes + kStripBytes + IP * sizeof(PairRec));
  };

  // This workgroup's items.  Workgroup w = (die, slot) of a die-major
  // numbering takes share w when the schedule's items were cut at this
  // launch's workgroups (the same pair count for each), else an equal count
  // of its die's items; either way a die holds a contiguous run of strips,
  // so its L2 serves neighbouring strips' shared depth lines.
  const int xcd = blockIdx.x % kXcds;
  const int slot = blockIdx.x / kXcds;
  const int nslots = gridDim.x / kXcds;
  const int w_idx = xcd * nslots + slot;
  const int32_t* hdr = a.hdr;
  // (the share bounds are read with the counts; used only if they apply)
  const int32_t sh_lo = a.share_item0[min(w_idx, kMaxShares)];
  const int32_t sh_hi = a.share_item0[min(w_idx + 1, kMaxShares)];
  if (!header_ok(a)) return;  // (uniform; k_fwd_combine writes NaN everywhere)
  const int32_t n_items = min(hdr[kHdrItems], a.items_cap);
  const int32_t n_pairs = min(hdr[kHdrPairs], a.n_valid);
  const int32_t n_segs = min(hdr[kHdrSegs], a.n_valid);
  int i_begin, i_end;
  if (hdr[kHdrSharesOk] == 1 && hdr[kHdrShares] == (int32_t)gridDim.x) {
    i_begin = min(max(sh_lo, 0), n_items);
    i_end = min(max(sh_hi, i_begin), n_items);
  } else {
    const int per_die = (n_items + kXcds - 1) / kXcds;
    const int d_lo = min(xcd * per_die, n_items);
    const int d_cnt = min(n_items, d_lo + per_die) - d_lo;
    i_begin = d_lo + (int)(((int64_t)slot * d_cnt) / nslots);
    i_end = d_lo + (int)(((int64_t)(slot + 1) * d_cnt) / nslots);
  }
  if (i_begin >= i_end) return;

  const int C = a.C;
  const int CV = C / VEC;
  constexpr int kLanes = chunk_lanes<TIn, VEC>();
  const int cbase = blockIdx.y * kLanes;
  const int cvc = min(kLanes, CV - cbase);
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int64_t hw = a.hw32;
  const TIn* const fchunk = feat + (int64_t)cbase * VEC;
  // depth score of a gathered point: the stored score, or exp(logit - lse)
  // of the point's pixel (SM)
  auto score = [&](TIn x, double lse) -> float {
    if constexpr (SM) return expf((float)((double)to_float(x) - lse));  // (exponent in double)
    return to_float(x);
  };
  // log-sum-exp of the pixel of frustum point p (all points of a pair share
  // it); 0 outside the index range (the pair's points then read nothing)
  auto pixel_lse = [&](int32_t p) -> double {
    if (p < 0 || (int64_t)p >= a.P) return 0.0;
    const int32_t view = p / a.dhw;
    return a.lse[(int64_t)view * hw + (p - view * a.dhw) % a.hw32];
  };

  // Item headers, copied to LDS once (the launch gives no workgroup more
  // than kHdrCache items; scalar loads share their wait counter with LDS
  // reads, so loading headers inside the pipeline would stall every walk).
  const int n_my = min(i_end - i_begin, kHdrCache);
  for (int j = tid; j <= n_my; j += kNT) {
    s_hdr[0][j] = j < n_my ? a.item_strip[i_begin + j] : 0;
    s_hdr[1][j] = a.item_pair0[i_begin + j];
    s_hdr[2][j] = a.item_seg0[i_begin + j];
  }
  if (tid == 0) s_lsync = 0;
  lds_barrier();
  // item i's header (i clamped to this workgroup's items)
  auto header = [&](int i) {
    i = min(max(i - i_begin, 0), n_my - 1);
    int32_t v[5];
    v[0] = s_hdr[0][i]; v[1] = s_hdr[1][i]; v[2] = s_hdr[1][i + 1];
    v[3] = s_hdr[2][i]; v[4] = s_hdr[2][i + 1];
    ItemHdr h;
    h.strip = __builtin_amdgcn_readfirstlane(v[0]);
    h.p0 = __builtin_amdgcn_readfirstlane(v[1]);
    h.np = __builtin_amdgcn_readfirstlane(v[2]) - h.p0;
    h.g0 = __builtin_amdgcn_readfirstlane(v[3]);
    h.nseg = __builtin_amdgcn_readfirstlane(v[4]) - h.g0;
    // (bitwise or: no branches)
    const bool bad = (h.strip < 0) | (h.strip >= a.strips) | (h.p0 < 0) | (h.np < 1) |
                     (h.np > IP) | (h.p0 + h.np > n_pairs) | (h.g0 < 0) | (h.nseg < 1) |
                     (h.nseg > h.np) | (h.g0 + h.nseg > n_segs);
    if (bad) h = ItemHdr{0, 0, 0, 0, 0};  // an inconsistent header becomes an empty item
    return h;
  };
  struct Geo {
    int64_t origin;
    int bws, npix;
  };
  auto geometry = [&](int strip) {
    const int32_t sper = a.nhb * a.nwb;
    const int32_t bn = strip / sper;
    const int32_t sr = strip - bn * sper;
    const int32_t hb = sr / a.nwb, wb = sr - hb * a.nwb;
    const int32_t h0 = hb * a.bh, w0 = wb * a.bw;
    Geo g;
    g.bws = min(a.bw, a.W - w0);
    g.npix = min(a.bh, a.H - h0) * g.bws;
    g.origin = ((int64_t)bn * a.H + h0) * a.W + w0;
    return g;
  };
  // staged vector idx of a strip (pixel-major, then each pixel's chunk in
  // memory order): its address, and its LDS slot [pixel][part][lane]
  const int rowvec = cvc * kNV;  // staged vectors per pixel
  auto vec_addr = [&](const Geo& g, int idx) {
    const int lp = idx / rowvec;
    const int v = idx - lp * rowvec;
    const int lh = lp / g.bws;
    const int64_t row = g.origin + (int64_t)lh * a.W + (lp - lh * g.bws);
    return reinterpret_cast<const RawT*>(fchunk + row * C + (int64_t)v * kPer);
  };
  auto vec_slot = [&](int idx) {
    if (kNV == 1) return idx;
    const int lp = idx / rowvec;
    const int v = idx - lp * rowvec;
    const int vi = v / kNV;
    return lp * rowvec + (v - vi * kNV) * cvc + vi;
  };

  // ---- an item's rows, destinations and pair records into LDS buffer b, by
  // threads 0 .. NT - 1 (the loading waves; the whole workgroup for the first
  // item, which nothing could overlap).  Loads are unconditional where they
  // can be, surplus lanes repeating an in-range address: a load under a branch
  // makes the compiler wait for it where the branch joins.
  const int lt = tid;
  // Rows of 16-byte vectors, one per staged slot, go from memory straight into
  // LDS (global_load_lds_dwordx4: lane i of a wave writes its 16 bytes at the
  // wave's LDS address + 16 i, the staged layout).  They take no registers and
  // are issued before the item's other loads, so that rows, records and
  // destinations share one round trip to memory; a strip's vectors fill at
  // most kStripBytes, so kStripBytes / 16 / NT rounds cover them.  The wait
  // for the loads after them (memory loads complete in order) also waits for
  // these.  Other widths go through registers.
  constexpr bool kDirectRows = kNV == 1 && sizeof(RawT) == 16;
  auto stage_rows_direct = [&](const Geo& g, int b, auto nt_tag) {
    constexpr int NT = decltype(nt_tag)::value;
    constexpr int kLoadRows = kStripBytes / 16 / NT;
    static_assert(NT % kWave == 0 && kLoadRows * NT * 16 == kStripBytes, "whole waves and rounds");
    const int nvec = g.npix * rowvec;
    RawT* const s_rows = buf_rows(b);
#pragma unroll
    for (int r = 0; r < kLoadRows; ++r) {
      const int idx = r * NT + lt;  // (a wave's lanes take consecutive slots)
      global_to_lds16(vec_addr(g, min(idx, nvec - 1)), s_rows + (idx & ~(kWave - 1)));
    }
  };
  // the depth scores of a pair's points kDepthBurst .. n - 1 added to sum in
  // point order, four loads at a time (clamped indices; runs longer than
  // kDepthBurst points are few)
  auto depth_tail = [&](float& sum, int32_t rd0, int n, double lq) {
    for (int j0 = kDepthBurst; j0 < n; j0 += 4) {
      TIn x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t p = (int64_t)rd0 + (int64_t)min(j0 + u, n - 1) * hw;
        x[u] = depth[min(max(p, (int64_t)0), a.P - 1)];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t p = (int64_t)rd0 + (int64_t)(j0 + u) * hw;
        if (j0 + u < n && p >= 0 && p < a.P) sum += score(x[u], lq);
      }
    }
  };
  auto load_item = [&](const ItemHdr& h, int b, auto nt_tag) {
    constexpr int NT = decltype(nt_tag)::value;
    constexpr int kLoadRows = kStripBytes / 16 / NT;  // 16-byte row vectors per thread
    constexpr int kRB = whole_batch(kLoadRows, kRowBatch);
    constexpr int kLP = IP / NT;  // pairs per thread
    constexpr int kPB = whole_batch(kLP, kPairBatch);
    static_assert(kLoadRows % kRB == 0 && kLP % kPB == 0, "whole batches");
    const Geo g = geometry(h.strip);
    const int nvec = g.npix * rowvec;
    RawT* const s_rows = buf_rows(b);
    PairRec* const s_pr = buf_pr(b);
    int32_t* const s_dest = buf_dest(b);
    if constexpr (kDirectRows) {
      stage_rows_direct(g, b, nt_tag);
    } else {
      // rows, kRB vectors per thread in flight
      for (int r0 = 0; r0 < kLoadRows; r0 += kRB) {
        RawT rv[kRB];
#pragma unroll
        for (int u = 0; u < kRB; ++u)
          rv[u] = *vec_addr(g, min((r0 + u) * NT + lt, nvec - 1));
#pragma unroll
        for (int u = 0; u < kRB; ++u) {
          const int idx = (r0 + u) * NT + lt;
          if (idx < nvec) s_rows[vec_slot(idx)] = rv[u];
        }
      }
      for (int idx = kLoadRows * NT + lt; idx < nvec; idx += NT)
        s_rows[vec_slot(idx)] = *vec_addr(g, idx);
    }
    // pair records and their depth scores, kPB pairs per thread at a time;
    // the destinations are loaded between a batch's records and its depth
    // scores (the records have arrived once the destinations have)
    for (int q0 = 0; q0 < kLP; q0 += kPB) {
      int32_t rd0[kPB];
      uint32_t ln[kPB];
      uint32_t sg[kPB];
#pragma unroll
      for (int q = 0; q < kPB; ++q) {
        const int k = h.p0 + min((q0 + q) * NT + lt, max(h.np - 1, 0));
        rd0[q] = a.pair_rd0[k];
        ln[q] = a.pair_ln[k];
        sg[q] = a.pair_seg[k];
      }
      if (q0 == 0)
        for (int j = lt; j < h.nseg; j += NT) s_dest[j] = a.seg_dest[h.g0 + j];
      float dv[kPB][kDepthBurst];
      double lq[kPB];
#pragma unroll
      for (int q = 0; q < kPB; ++q) {
        const int n = (q0 + q) * NT + lt < h.np ? (int)(ln[q] >> 16) : 0;
        if constexpr (SM) lq[q] = pixel_lse(rd0[q]);
#pragma unroll
        for (int j = 0; j < kDepthBurst; ++j) {
          const int64_t p = (int64_t)rd0[q] + j * hw;
          float v = 0.f;
          if (j < n && p >= 0 && p < a.P) v = score(depth[p], lq[q]);
          dv[q][j] = v;
        }
      }
#pragma unroll
      for (int q = 0; q < kPB; ++q) {
        const int k = (q0 + q) * NT + lt;
        if (k < h.np) {
          const int n = (int)(ln[q] >> 16);
          // (no constant start: an add of 0.f would be folded into the load's branch)
          float sum = dv[q][0];
#pragma unroll
          for (int j = 1; j < kDepthBurst; ++j) sum += dv[q][j];
          depth_tail(sum, rd0[q], n, lq[q]);
          const uint32_t lp = ln[q] & kPairPixel;
          const bool ok = lp < (uint32_t)g.npix;
          const uint32_t sgc = min(sg[q], (uint32_t)(h.nseg - 1));
          PairRec rec;
          rec.w = ok ? sum : 0.f;
          rec.ps = (ok ? lp * (uint32_t)rowvec : 0u) | (sgc << kRecSegShift) |
                   ((ln[q] & kPairHead) ? kRecHead : 0u);
          s_pr[k] = rec;
        }
      }
    }
    if constexpr (kDirectRows) __builtin_amdgcn_s_waitcnt(0);  // (the rows are in LDS)
  };

  // ---- the loading waves' item loads, with the item's pair records (depth
  // rank, pixel and run) read one item ahead into registers (fetch_pairs):
  // the depth gathers, which need them, then go out first, beside the row
  // loads, and the LDS stores follow.
  constexpr int kLPL = IP / kLoadThreads;  // pairs per loading thread
  constexpr int kRowsL = kStripBytes / 16 / kLoadThreads;  // row vectors per loading thread
  constexpr int kRowsH = kRowsL / 2;  // row vectors per batch
  static_assert(kRowsL % 2 == 0, "two row batches");
  struct PairPf {
    int32_t rd0[kLPL];
    uint32_t ln[kLPL];
  };
  auto fetch_pairs = [&](const ItemHdr& h, PairPf& pf) {
#pragma unroll
    for (int q = 0; q < kLPL; ++q) {
      const int k = h.p0 + min(q * kLoadThreads + lt, max(h.np - 1, 0));
      pf.rd0[q] = a.pair_rd0[k];
      pf.ln[q] = a.pair_ln[k];
    }
  };
  auto load_item_pf = [&](const ItemHdr& h, int b, const PairPf& pf) {
    const Geo g = geometry(h.strip);
    const int nvec = g.npix * rowvec;
    RawT* const s_rows = buf_rows(b);
    PairRec* const s_pr = buf_pr(b);
    int32_t* const s_dest = buf_dest(b);
    if constexpr (kDirectRows) stage_rows_direct(g, b, std::integral_constant<int, kLoadThreads>{});
    float dv[kLPL][kDepthBurst];
    double lq[kLPL];
#pragma unroll
    for (int q = 0; q < kLPL; ++q) {
      const int n = q * kLoadThreads + lt < h.np ? (int)(pf.ln[q] >> 16) : 0;
      if constexpr (SM) lq[q] = pixel_lse(pf.rd0[q]);
#pragma unroll
      for (int j = 0; j < kDepthBurst; ++j) {
        const int64_t p = (int64_t)pf.rd0[q] + j * hw;
        float v = 0.f;
        if (j < n && p >= 0 && p < a.P) v = score(depth[p], lq[q]);
        dv[q][j] = v;
      }
    }
    uint32_t sg[kLPL];
#pragma unroll
    for (int q = 0; q < kLPL; ++q) sg[q] = a.pair_seg[h.p0 + min(q * kLoadThreads + lt, max(h.np - 1, 0))];
    if constexpr (!kDirectRows) {
#pragma unroll
      for (int r0 = 0; r0 < kRowsL; r0 += kRowsH) {
        RawT rv[kRowsH];
#pragma unroll
        for (int u = 0; u < kRowsH; ++u) rv[u] = *vec_addr(g, min((r0 + u) * kLoadThreads + lt, nvec - 1));
#pragma unroll
        for (int u = 0; u < kRowsH; ++u) {
          const int idx = (r0 + u) * kLoadThreads + lt;
          if (idx < nvec) s_rows[vec_slot(idx)] = rv[u];
        }
      }
      for (int idx = kRowsL * kLoadThreads + lt; idx < nvec; idx += kLoadThreads)
        s_rows[vec_slot(idx)] = *vec_addr(g, idx);
    }
    for (int j = lt; j < h.nseg; j += kLoadThreads) s_dest[j] = a.seg_dest[h.g0 + j];
#pragma unroll
    for (int q = 0; q < kLPL; ++q) {
      const int k = q * kLoadThreads + lt;
      if (k < h.np) {
        const int n = (int)(pf.ln[q] >> 16);
        // (no constant start: an add of 0.f would be folded into the load's branch)
        float sum = dv[q][0];
#pragma unroll
        for (int j = 1; j < kDepthBurst; ++j) sum += dv[q][j];
        depth_tail(sum, pf.rd0[q], n, lq[q]);
        const uint32_t lp = pf.ln[q] & kPairPixel;
        const bool ok = lp < (uint32_t)g.npix;
        const uint32_t sgc = min(sg[q], (uint32_t)(h.nseg - 1));
        PairRec rec;
        rec.w = ok ? sum : 0.f;
        rec.ps = (ok ? lp * (uint32_t)rowvec : 0u) | (sgc << kRecSegShift) |
                 ((pf.ln[q] & kPairHead) ? kRecHead : 0u);
        s_pr[k] = rec;
      }
    }
    if constexpr (kDirectRows) __builtin_amdgcn_s_waitcnt(0);  // (the rows are in LDS)
  };

  // ---- walking waves: lane group lg of walking wave wv owns an equal range
  // of each item's pairs
  const int gpw = kWave / cvc;
  const int G = kWalkWaves * gpw;
  const int wv = wave - kLoadWaves;
  const int lg = lane / cvc;
  const int vi = lane - lg * cvc;
  const int g = wv * gpw + lg;
  const bool walker = wave >= kLoadWaves;
  const bool active = walker && lg < gpw;
  const int64_t col = (int64_t)(cbase + vi) * VEC;

  int kb = 0, ke = 0, last_seg = -1, first_seg = -1;
  int32_t last_dest = 0;
  bool prev_cont = false, next_cont = false;
  float first_sum[VEC], last_sum[VEC];

  // a segment's sum to its destination: a cell of `out`, or (~d) a slot
  auto store_dest = [&](int32_t d, const float* v) {
    if (d >= 0) {
      if (d < a.cells) Vec<TOut, VEC>::store(out + (int64_t)d * C + col, v);
    } else {
      const int64_t sl = (int64_t)(~d);
      if (sl < a.slot_cap) Vec<float, VEC>::store(a.slots + sl * C + col, v);
    }
  };

  // sums this group's range of an item's pairs from LDS buffer b; segments
  // wholly inside the range are stored, the parts of cut ones kept
  auto walk_item = [&](const ItemHdr& h, int b) {
    const RawT* const s_lane = buf_rows(b) + vi;
    const PairRec* const s_pr = buf_pr(b);
    const int32_t* const s_dest = buf_dest(b);
    const int np = h.np;
    auto is_head = [&](int k) { return (s_pr[k].ps & kRecHead) != 0; };
    auto seg_at = [&](int k) { return (int)((s_pr[k].ps & ~kRecHead) >> kRecSegShift); };
    kb = ke = 0;
    prev_cont = next_cont = false;
    last_seg = first_seg = -1;
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = first_sum[e] = last_sum[e] = 0.f;
    if (active) {
      kb = (g * np) / G;  // below 2^31: G <= kNT
      ke = ((g + 1) * np) / G;
    }
    if (kb < ke) {
      // a range that starts inside a segment owes that segment's part to the
      // group holding its start (kept in first_sum); one that ends inside a
      // segment keeps the part in last_sum and adds the other groups' parts
      prev_cont = !is_head(kb);
      next_cont = ke < np && !is_head(ke);
      last_seg = seg_at(ke - 1);
      first_seg = seg_at(kb);
      last_dest = s_dest[min(last_seg, h.nseg - 1)];
      int cur = first_seg;
      bool pend_first = prev_cont;
      auto end_segment = [&]() {  // segment `cur` has no more pairs in this range
        if (pend_first) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) first_sum[e] = acc[e];
          pend_first = false;
        } else {
          store_dest(s_dest[min(cur, h.nseg - 1)], acc);
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
        ++cur;
      };
      {
        // the range's first pair never ends a segment
        const PairRec r = s_pr[kb];
        float x[VEC];
        lane_row<TIn, VEC>(s_lane + (r.ps & kRecOff), cvc, x);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = fmaf(r.w, x[e], acc[e]);
      }
      int k0 = kb + 1;
      for (; k0 + kUnroll <= ke; k0 += kUnroll) {
        // records first, then rows: two LDS round trips per kUnroll pairs
        PairRec r[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) r[u] = s_pr[k0 + u];
        float x[kUnroll][VEC];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) lane_row<TIn, VEC>(s_lane + (r[u].ps & kRecOff), cvc, x[u]);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          if (r[u].ps & kRecHead) end_segment();
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] = fmaf(r[u].w, x[u][e], acc[e]);
        }
      }
      for (; k0 < ke; ++k0) {
        const PairRec r = s_pr[k0];
        float x[VEC];
        lane_row<TIn, VEC>(s_lane + (r.ps & kRecOff), cvc, x);
        if (r.ps & kRecHead) end_segment();
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = fmaf(r.w, x[e], acc[e]);
      }
      // the range's last segment
      if (pend_first) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) first_sum[e] = acc[e];
      } else if (next_cont) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) last_sum[e] = acc[e];
      } else {
        store_dest(s_dest[min(cur, h.nseg - 1)], acc);
      }
    }
  };

  // ---- segments cut by range boundaries, added in range order.  After a
  // walk every group publishes, in the walked buffer (its rows and records
  // are no longer read): the part of the segment its range starts inside
  // (part_first, over the rows), the part of the one it ends inside when it
  // holds that segment's start (part_last, over the pair records and
  // destinations), and a record of its range.  The loading waves add the
  // parts up while the walking waves go on to the next item.
  constexpr int kMetaPrev = 1, kMetaNext = 2, kMetaLast = 4, kMetaEmpty = 8;
  static_assert((int64_t)kWalkWaves * kWave * 8 * sizeof(float) <= IP * 12,
                "last parts fit the pair records and destinations");
  auto part_first = [&](int b) { return reinterpret_cast<float*>(smem + b * kBufBytes); };
  auto part_last = [&](int b) { return reinterpret_cast<float*>(smem + b * kBufBytes + kStripBytes); };
  auto publish = [&](int b) {
    if (!active) return;
    int flags = kMetaEmpty;
    if (kb < ke) {
      const bool has_last = next_cont && !(prev_cont && first_seg == last_seg);
      flags = (prev_cont ? kMetaPrev : 0) | (next_cont ? kMetaNext : 0) | (has_last ? kMetaLast : 0);
      if (prev_cont) Vec<float, VEC>::store(part_first(b) + ((int64_t)g * cvc + vi) * VEC, first_sum);
      if (has_last) Vec<float, VEC>::store(part_last(b) + ((int64_t)g * cvc + vi) * VEC, last_sum);
    }
    if (vi == 0) s_meta[g] = make_int4(last_seg, last_dest, flags, 0);
  };
  // group gg's segment that continues past its range: its part plus the
  // following ranges' first parts, up to the range where that segment ends;
  // handled by the lane groups of threads 0 .. nthreads - 1
  auto combine_parts = [&](int b, int nthreads) {
    if (lg >= gpw) return;
    const int n_h = (nthreads / kWave) * gpw;
    for (int gg = wave * gpw + lg; gg < G; gg += n_h) {
      // the range's record and part and the following ranges' records and
      // parts, kChain at a time, are read together (whether or not the
      // range holds a cut segment; past the chain's end they are not used)
      constexpr int kChain = 4;
      const int4 m = s_meta[gg];
      float sum[VEC];
      Vec<float, VEC>::load(part_last(b) + ((int64_t)gg * cvc + vi) * VEC, sum);
      bool go = true;
      for (int g2 = gg + 1; go && g2 < G; g2 += kChain) {
        int4 m2[kChain];
        float t[kChain][VEC];
#pragma unroll
        for (int u = 0; u < kChain; ++u) {
          const int gi = min(g2 + u, G - 1);
          m2[u] = s_meta[gi];
          Vec<float, VEC>::load(part_first(b) + ((int64_t)gi * cvc + vi) * VEC, t[u]);
        }
        if (!(m.z & kMetaLast)) break;
#pragma unroll
        for (int u = 0; u < kChain; ++u) {
          if (!go || g2 + u >= G || (m2[u].z & kMetaEmpty)) continue;
          if (!(m2[u].z & kMetaPrev)) {  // range g2 + u starts a segment
            go = false;
            continue;
          }
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] += t[u][e];
          // on to the next range only if this one lies wholly inside the segment
          if (!(m2[u].x == m.x && (m2[u].z & kMetaNext))) go = false;
        }
      }
      if (m.z & kMetaLast) store_dest(m.y, sum);
    }
  };

  // The loading waves wait for each other (the walking waves are walking,
  // so no workgroup barrier can be used): each wave's lane 0 counts its
  // arrival in LDS, then the wave waits until all kLoadWaves have arrived.
  // Every loading wave runs the same item loop, so every wait ends.
  int lsync_target = 0;
  auto loader_sync = [&]() {
    lsync_target += kLoadWaves;
    if (lane == 0) __hip_atomic_fetch_add(&s_lsync, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    while (__hip_atomic_load(&s_lsync, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < lsync_target)
      __builtin_amdgcn_s_sleep(1);
  };

  // ---- the pipeline: item i is walked from buffer b while the loading
  // waves add up the cut segments of item i - 1 (published in buffer b ^ 1)
  // and then fill buffer b ^ 1 with item i + 1
  // (records are read ahead where the walk leaves the registers for them;
  // not in the fused softmax forms, whose per-pair lse already takes them,
  // nor for big items, whose records would not fit)
  constexpr bool kPrefetch = VEC < 8 && !SM && IP <= kItemPairs;
  load_item(header(i_begin), 0, std::integral_constant<int, kNT>{});
  PairPf pf;  // the second item's records
  if (kPrefetch && !walker && i_begin + 1 < i_begin + n_my) fetch_pairs(header(i_begin + 1), pf);
  lds_barrier();
  int b = 0;
  for (int i = i_begin; i < i_begin + n_my; ++i) {
    if (!walker) {
      if (i > i_begin) {
        combine_parts(b ^ 1, kLoadThreads);
        loader_sync();  // every part read before buffer b ^ 1 is refilled
      }
      if (kPrefetch) {
        if (i + 1 < i_begin + n_my) load_item_pf(header(i + 1), b ^ 1, pf);
        if (i + 2 < i_begin + n_my) fetch_pairs(header(i + 2), pf);
      } else if (i + 1 < i_begin + n_my) {
        load_item(header(i + 1), b ^ 1, std::integral_constant<int, kLoadThreads>{});
      }
    } else {
      walk_item(header(i), b);
    }
    lds_barrier();  // item i walked, item i - 1 combined, item i + 1 loaded
    if (walker) publish(b);
    lds_barrier();  // item i's parts published
    b ^= 1;
  }
  combine_parts(b ^ 1, kNT);  // the last item's, by every wave
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(kCombThreads) void k_fwd_combine(TOut* __restrict__ out,
                                                              StripArgs a) {
  const int32_t* hdr = a.hdr;
  const bool ok = header_ok(a);
  const int lane = lane_id();
  const int C = a.C;
  const int CV = C / VEC;
  const int cbase = blockIdx.y * kWave;
  const int cvc = min(kWave, CV - cbase);
  const int gpw = kWave / cvc;
  const int lg = lane / cvc;
  const int vi = lane - lg * cvc;
  if (lg >= gpw) return;
  const int64_t j = ((int64_t)blockIdx.x * (kCombThreads / kWave) + threadIdx.x / kWave) * gpw + lg;
  if (!ok) {
    // a schedule that does not hold the launch's counts: every cell is NaN
    // (the grid has a lane group per cell and channel chunk)
    if (j < a.cells) {
      float nan[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) nan[e] = __builtin_nanf("");
      Vec<TOut, VEC>::store(out + j * C + (int64_t)(cbase + vi) * VEC, nan);
    }
    return;
  }
  const int64_t n_comb = min(hdr[kHdrComb], a.n_occ);
  const int64_t n_empty = min<int64_t>(hdr[kHdrEmpty], a.n_empty);
  const int64_t col = (int64_t)(cbase + vi) * VEC;
  if (j >= n_comb + n_empty) return;
  // Both roles' records are read at once, unconditionally (clamped index),
  // so that a cell and its slot range arrive together: a load behind a test
  // of the cell would cost another round trip.
  const int64_t jc = min(j, n_comb > 0 ? n_comb - 1 : 0);
  const int64_t cell_c = a.comb_cell[jc];
  const int64_t s0 = a.comb_slot0[jc], s1 = a.comb_slot0[jc + 1];
  const int64_t cell_e = a.empty[min(max(j - n_comb, (int64_t)0), n_empty > 0 ? n_empty - 1 : 0)];
  // (an empty asm reading all four values: the compiler would otherwise move
  // each load into the branch that uses it, behind the previous one's test)
  asm volatile("" ::"v"((int32_t)cell_c), "v"((int32_t)s0), "v"((int32_t)s1), "v"((int32_t)cell_e));
  if (j < n_comb) {
    if (cell_c < 0 || cell_c >= a.cells) return;
    float sum[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) sum[e] = 0.f;
    if (s0 < 0 || s1 <= s0 || s1 > a.slot_cap) {
      // the workspace does not hold this cell's slots: make that visible
#pragma unroll
      for (int e = 0; e < VEC; ++e) sum[e] = __builtin_nanf("");
    } else {
      int64_t s = s0;
      for (; s + 4 <= s1; s += 4) {
        float t[4][VEC];
#pragma unroll
        for (int k = 0; k < 4; ++k) Vec<float, VEC>::load(a.slots + (s + k) * C + col, t[k]);
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] += t[k][e];
      }
      // the last 1-3 slots (most cells have 2 or 3), loaded together
      const int rest = (int)(s1 - s);
      float t[3][VEC];
#pragma unroll
      for (int k = 0; k < 3; ++k) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) t[k][e] = 0.f;
        if (k < rest) Vec<float, VEC>::load(a.slots + (s + k) * C + col, t[k]);
      }
#pragma unroll
      for (int k = 0; k < 3; ++k)
        if (k < rest)
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] += t[k][e];
    }
    Vec<TOut, VEC>::store(out + cell_c * C + col, sum);
  } else if (cell_e >= 0 && cell_e < a.cells) {
    store_zero<TOut, VEC>(out + cell_e * C + col);
  }
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero_out(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

template <typename TIn, typename TOut, int VEC, bool SM>
hipError_t run(const Dims& d, const StripDims& sd, const void* depth, const void* feat,
               StripArgs a, void* out, hipStream_t stream) {
  TOut* o = static_cast<TOut*>(out);
  const int CV = (int)(d.C / VEC);
  constexpr int kLanes = chunk_lanes<TIn, VEC>();
  const unsigned chunks = (unsigned)((CV + kLanes - 1) / kLanes);
  // one persistent workgroup per CU (a whole number per die), more when a
  // workgroup would otherwise get more than kHdrCache items
  const int64_t per_die_slots = std::max<int64_t>(forward_workgroups() / kXcds,
                                                  a.items_cap / ((int64_t)kXcds * kHdrCache) + 1);
  const int blocks = (int)(per_die_slots * kXcds);
  if (a.item_pairs == kItemPairsBig)
    k_fwd_strips<TIn, TOut, VEC, SM, kItemPairsBig><<<dim3((unsigned)blocks, chunks), dim3(kNT), 0, stream>>>(
        static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), o, a);
  else
    k_fwd_strips<TIn, TOut, VEC, SM, kItemPairs><<<dim3((unsigned)blocks, chunks), dim3(kNT), 0, stream>>>(
        static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), o, a);
  const int64_t gpw = kWave / (CV < kWave ? CV : kWave);
  const int64_t entries = (int64_t)a.n_occ + a.n_empty;
  const int64_t per_block = gpw * (kCombThreads / kWave);
  const int64_t cblocks = (entries + per_block - 1) / per_block;
  const unsigned cchunks = (unsigned)((CV + kWave - 1) / kWave);
  if (cblocks > 0)
    k_fwd_combine<TOut, VEC><<<dim3((unsigned)cblocks, cchunks), dim3(kCombThreads), 0, stream>>>(
        o, a);
  return hipGetLastError();
}

template <typename TOut, int VEC>
hipError_t zero_fill(const Dims& d, void* out, hipStream_t stream) {
  const int64_t nvec = d.cells * (d.C / VEC);
  k_zero_out<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(
      static_cast<TOut*>(out), nvec);
  return hipGetLastError();
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

int device_cus() {
  static int cached[64];  // per device; 0 = not yet queried
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  cached[dev] = cus;
  return cus;
}

int forward_workgroups() { return (device_cus() + kXcds - 1) / kXcds * kXcds; }

size_t forward_scheduled_workspace_bytes(const Dims& d, int64_t n_slots) {
  return (size_t)(n_slots > 0 ? n_slots : 0) * (size_t)d.C * sizeof(float);
}

template <bool SM>
hipError_t dispatch_scheduled(const Dims& d, const StripDims& sd, bool half_in, bool half_out,
                              int vec, const void* depth, const void* feat, const StripArgs& a,
                              void* out, hipStream_t stream) {
  if (!half_in) {
    if (vec == 4) return run<float, float, 4, SM>(d, sd, depth, feat, a, out, stream);
    return run<float, float, 1, SM>(d, sd, depth, feat, a, out, stream);
  }
  if (half_out) {
    if (vec == 8) return run<half_t, half_t, 8, SM>(d, sd, depth, feat, a, out, stream);
    return run<half_t, half_t, 1, SM>(d, sd, depth, feat, a, out, stream);
  }
  if (vec == 8) return run<half_t, float, 8, SM>(d, sd, depth, feat, a, out, stream);
  return run<half_t, float, 1, SM>(d, sd, depth, feat, a, out, stream);
}

hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                    const void* depth, const void* feat, const void* schedule,
                                    int32_t n_valid, int32_t n_intervals, int32_t n_slots,
                                    void* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, const double* lse) {
  const bool al = aligned16(feat) && aligned16(out) && aligned16(workspace);
  const bool half_in = in_dtype == BEVPOOL_F16;
  const bool half_out = out_dtype == BEVPOOL_F16;
  const int vec = half_in ? ((al && d.C % 8 == 0) ? 8 : 1) : ((al && d.C % 4 == 0) ? 4 : 1);
  if (n_valid == 0 || n_intervals == 0) {
    if (half_out) return vec == 8 ? zero_fill<half_t, 8>(d, out, stream) : zero_fill<half_t, 1>(d, out, stream);
    if (vec == 4) return zero_fill<float, 4>(d, out, stream);
    if (vec == 8) return zero_fill<float, 8>(d, out, stream);
    return zero_fill<float, 1>(d, out, stream);
  }
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  const char* sc = static_cast<const char*>(schedule);
  auto S = [&](size_t o) { return reinterpret_cast<const int32_t*>(sc + o); };
  StripArgs a;
  a.hdr = S(L.header);
  a.pair_rd0 = S(L.pair_rd0);
  a.pair_ln = reinterpret_cast<const uint32_t*>(S(L.pair_ln));
  a.pair_seg = reinterpret_cast<const uint16_t*>(S(L.pair_seg));
  a.item_strip = S(L.item_strip);
  a.item_pair0 = S(L.item_pair0);
  a.item_seg0 = S(L.item_seg0);
  a.seg_dest = S(L.seg_dest);
  a.comb_cell = S(L.comb_cell);
  a.comb_slot0 = S(L.comb_slot0);
  a.empty = S(L.empty);
  a.share_item0 = S(L.share_item0);
  a.slots = static_cast<float*>(workspace);
  a.slot_cap = workspace == nullptr ? 0 : (int64_t)(workspace_bytes / ((size_t)d.C * sizeof(float)));
  a.n_valid = n_valid;
  a.n_occ = n_intervals;
  a.n_slots = n_slots;
  a.items_cap = (int32_t)L.items_cap;
  // (the item size every schedule of n_valid kept points is cut at; a
  // schedule cut otherwise fails the header check)
  a.item_pairs = schedule_item_pairs(n_valid);
  a.C = (int32_t)d.C;
  a.H = (int32_t)d.H;
  a.W = (int32_t)d.W;
  a.bh = (int32_t)L.sd.bh;
  a.bw = (int32_t)L.sd.bw;
  a.nhb = (int32_t)L.sd.nhb;
  a.nwb = (int32_t)L.sd.nwb;
  a.strips = (int32_t)L.sd.strips;
  a.hw32 = (int32_t)d.hw;
  a.P = d.P;
  a.cells = d.cells;
  a.n_empty = L.n_empty;
  a.lse = lse;
  a.dhw = (int32_t)(d.D * d.hw);
  if (lse != nullptr)
    return dispatch_scheduled<true>(d, L.sd, half_in, half_out, vec, depth, feat, a, out, stream);
  return dispatch_scheduled<false>(d, L.sd, half_in, half_out, vec, depth, feat, a, out, stream);
}

// ---- allocation-free forward: the slots live in a file-scope device array.
// Each device holds its own copy from the first call on it until the
// process ends; every call on a device shares it.
namespace {

static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

hipError_t forward_noalloc_scratch(void** addr) {
  *addr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    // (once per device, with that device current: the array's device
    // address; in host code `scratch` itself is only a stand-in)
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (p == nullptr) return hipErrorInvalidSymbol;
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *addr = p;
  return hipSuccess;
}

}  // namespace bevpool
