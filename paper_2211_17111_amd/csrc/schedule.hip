// Block schedule build (terms and device layout in internal.h).
//
// Built once per plan, like the plan itself (section 2.1: the indices are
// fixed parameters, preprocessed offline).  Every step runs on the device,
// reads its counts from the schedule header, and is deterministic: sorts are
// stable, compactions order preserving, minima and maxima over a TC or a
// piece are taken by one thread over its own range, and the only atomics are
// integer maxima of four header counts (order independent).
//   1. pairs: the plan regrouped by (strip, cell, pixel, depth) with two or
//      three stable radix sorts; a pair starts where the cell or pixel
//      changes or the depth bin does not follow on;
//   2. the pairs again in feature-row order (for the scheduled backward);
//   3. TCs (runs of one strip and cell), ranked by (strip, least depth bin)
//      and cut into pieces at every tcmax-th TC of a strip and where the
//      strip's running pair count crosses a multiple of kSchedPairs;
//   4. CCs (a TC's pairs in one column) with their least depth bin and row
//      range, sorted by (piece, column, least depth bin, TC) and cut into
//      blocks of kSchedK; each block's row range gives its weight entries;
//   5. destinations: cells reached from one strip are written directly,
//      the others get one slot per TC, in (cell, strip) order;
//   6. pieces: row and depth ranges, the pairs as records in (local pixel,
//      depth) order, and each local pixel's first record.

#include <algorithm>

#include "device_utils.h"
#include "internal.h"
#include "primitives.h"

namespace bevpool {

namespace {

constexpr int kStride = 1024;  // workgroups of kernels that loop over a device-side count

// Strip geometry of feature rows and frustum points (32-bit unsigned
// arithmetic: p, D*H*W and H*W are below 2^31).
struct Geo {
  uint32_t per_view, hw;
  int32_t H, W, nsw;
  __device__ int32_t row_of(int32_t p) const {
    const uint32_t u = (uint32_t)p;
    return (int32_t)((u / per_view) * hw + u % hw);
  }
  __device__ int32_t d_of(int32_t p) const { return (int32_t)(((uint32_t)p % per_view) / hw); }
  __device__ int32_t strip(int32_t row) const {
    const int32_t bn = (int32_t)((uint32_t)row / hw);
    const int32_t w = (int32_t)((uint32_t)row % hw) % W;
    return bn * nsw + w / kSchedSW;
  }
  __device__ int32_t h(int32_t row) const { return (int32_t)((uint32_t)row % hw) / W; }
  __device__ int32_t col(int32_t row) const { return ((int32_t)((uint32_t)row % hw) % W) % kSchedSW; }
  __device__ int32_t lp_strip(int32_t row) const { return h(row) * kSchedSW + col(row); }
};

// scratch counters of the build (workspace)
constexpr int kCntStrips = 0, kCntGroups = 1, kCntEntries = 2, kCntPieceBlocks = 3;

__global__ void k_sched_init(int32_t* __restrict__ hdr, int32_t* __restrict__ cnt,
                             int32_t n_valid, int32_t n_occ) {
  if (threadIdx.x < 16) {
    hdr[threadIdx.x] = 0;
    cnt[threadIdx.x] = 0;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    hdr[kSHdrValid] = n_valid;
    hdr[kSHdrOcc] = n_occ;
  }
}

// a[*idx] = *val (an end sentinel after a compaction)
__global__ void k_set_end(int32_t* __restrict__ a, const int32_t* __restrict__ idx,
                          const int32_t* __restrict__ val, int64_t cap) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && *idx >= 0 && *idx <= cap) a[*idx] = *val;
}

// ---- 1. pairs ------------------------------------------------------------------

// keys = pixel of every kept point within its strip, vals = plan position
__global__ __launch_bounds__(256) void k_pixel_keys(const int32_t* __restrict__ rd, int64_t n,
                                                    Geo g, int32_t* __restrict__ keys,
                                                    int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    keys[i] = g.lp_strip(g.row_of(rd[i]));
    vals[i] = (int32_t)i;
  }
}

// keys[i] for the point at plan position vals[i]: mode 0 (strip << cell_bits)
// | BEV rank, mode 1 the BEV rank, mode 2 the strip.
__global__ __launch_bounds__(256) void k_strip_keys(const int32_t* __restrict__ rd,
                                                    const int32_t* __restrict__ rb,
                                                    const int32_t* __restrict__ vals, int64_t n,
                                                    Geo g, int cell_bits, int mode,
                                                    int32_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t a = vals[i];
  const int32_t s = g.strip(g.row_of(rd[a]));
  keys[i] = mode == 0 ? (int32_t)(((uint32_t)s << cell_bits) | (uint32_t)rb[a])
                      : (mode == 1 ? rb[a] : s);
}

struct PairHeads {  // runs of one cell and pixel over consecutive depth bins
  const int32_t* rd;
  const int32_t* rb;
  const int32_t* vals;  // plan position of each regrouped point
  const int32_t* hdr;
  Geo g;
  int32_t* pair_rb;
  int32_t* pair_row;
  uint32_t* pair_dn;
  int32_t* head_pos;  // regrouped position of each pair's first point
  __device__ int64_t count() const { return hdr[kSHdrValid]; }
  __device__ bool flag(int64_t i) const {
    if (i == 0) return true;
    const int32_t a = vals[i], b = vals[i - 1];
    const int32_t pa = rd[a], pb = rd[b];
    return rb[a] != rb[b] || g.row_of(pa) != g.row_of(pb) ||
           (int64_t)pa != (int64_t)pb + (int64_t)g.hw;
  }
  __device__ void emit(int64_t i, int32_t pos) const {
    const int32_t a = vals[i];
    const int32_t p = rd[a];
    pair_rb[pos] = rb[a];
    pair_row[pos] = g.row_of(p);
    pair_dn[pos] = (uint32_t)g.d_of(p);
    head_pos[pos] = (int32_t)i;
  }
};

__global__ __launch_bounds__(256) void k_pair_points(const int32_t* __restrict__ head_pos,
                                                     const int32_t* __restrict__ hdr,
                                                     uint32_t* __restrict__ pair_dn) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t np = hdr[kSHdrPairs];
  if (p < np) {
    const int64_t next = (p + 1 < np) ? head_pos[p + 1] : hdr[kSHdrValid];
    pair_dn[p] |= (uint32_t)(next - head_pos[p]) << 16;
  }
}

// ---- 2. pixel-major pairs ------------------------------------------------------

__global__ __launch_bounds__(256) void k_pair_row_keys(const int32_t* __restrict__ hdr,
                                                       const int32_t* __restrict__ pair_row,
                                                       int32_t* __restrict__ keys,
                                                       int32_t* __restrict__ vals) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p < hdr[kSHdrPairs]) {
    keys[p] = pair_row[p];
    vals[p] = (int32_t)p;
  }
}

__global__ __launch_bounds__(256) void k_pix_pairs(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ vals,
                                                   const int32_t* __restrict__ pair_rb,
                                                   const uint32_t* __restrict__ pair_dn,
                                                   int32_t* __restrict__ bp_cell,
                                                   uint32_t* __restrict__ bp_dn) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kSHdrPairs]) return;
  const int32_t a = vals[q];
  bp_cell[q] = pair_rb[a];
  bp_dn[q] = pair_dn[a];
}

// pix_pair0[f] = first pixel-major pair whose feature row is >= f, f in [0, rows]
__global__ __launch_bounds__(256) void k_pix_offsets(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ keys, int64_t rows,
                                                     int32_t* __restrict__ pix_pair0) {
  const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (f > rows) return;
  int32_t lo = 0, hi = hdr[kSHdrPairs];
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if (keys[mid] < f) lo = mid + 1; else hi = mid;
  }
  pix_pair0[f] = lo;
}

// ---- 3. TCs and pieces ---------------------------------------------------------

struct TCHeads {  // first pair of every (strip, cell) run
  const int32_t* pair_rb;
  const int32_t* pair_row;
  const int32_t* hdr;
  Geo g;
  int32_t* tc_p0;
  __device__ int64_t count() const { return hdr[kSHdrPairs]; }
  __device__ bool flag(int64_t k) const {
    return k == 0 || pair_rb[k] != pair_rb[k - 1] ||
           g.strip(pair_row[k]) != g.strip(pair_row[k - 1]);
  }
  __device__ void emit(int64_t k, int32_t pos) const { tc_p0[pos] = (int32_t)k; }
};

// Per TC (one thread over its pairs): pair count, sort key (strip, least
// depth bin; mode 0 joined, mode 1 the depth bin alone, the strip following
// in a second sort), row and depth range, and per column of the strip its
// CC's least depth bin and row range (dense arrays at TC * SW + column; row
// range -1 for a column without pairs).
__global__ __launch_bounds__(256) void k_tc_keys(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ tc_p0,
                                                 const int32_t* __restrict__ pair_row,
                                                 const uint32_t* __restrict__ pair_dn, Geo g,
                                                 int mode, int32_t* __restrict__ tc_np,
                                                 int32_t* __restrict__ tc_rng,
                                                 int32_t* __restrict__ ccd,
                                                 int32_t* __restrict__ cchlo,
                                                 int32_t* __restrict__ cchhi,
                                                 int32_t* __restrict__ keys,
                                                 int32_t* __restrict__ vals) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < ntc;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int32_t a = tc_p0[t], b = tc_p0[t + 1];
    int32_t dmin = kSchedMaxD - 1, dmax = 0, hmin = INT32_MAX, hmax = -1;
    int32_t cd[kSchedSW], clo[kSchedSW], chi[kSchedSW];
#pragma unroll
    for (int c = 0; c < kSchedSW; ++c) {
      cd[c] = INT32_MAX;
      clo[c] = INT32_MAX;
      chi[c] = -1;
    }
    for (int32_t k = a; k < b; ++k) {
      const uint32_t dn = pair_dn[k];
      const int32_t d0 = (int32_t)(dn & 0xFFFFu);
      const int32_t row = pair_row[k];
      const int32_t h = g.h(row), c = g.col(row);
      dmin = min(dmin, d0);
      dmax = max(dmax, d0 + (int32_t)(dn >> 16) - 1);
      hmin = min(hmin, h);
      hmax = max(hmax, h);
#pragma unroll
      for (int cc = 0; cc < kSchedSW; ++cc)
        if (cc == c) {
          cd[cc] = min(cd[cc], d0);
          clo[cc] = min(clo[cc], h);
          chi[cc] = max(chi[cc], h);
        }
    }
#pragma unroll
    for (int c = 0; c < kSchedSW; ++c) {
      ccd[t * kSchedSW + c] = cd[c];
      cchlo[t * kSchedSW + c] = clo[c];
      cchhi[t * kSchedSW + c] = chi[c];
    }
    const int32_t s = g.strip(pair_row[a]);
    tc_np[t] = b - a;
    tc_rng[4 * t + 0] = hmin;
    tc_rng[4 * t + 1] = hmax;
    tc_rng[4 * t + 2] = dmin;
    tc_rng[4 * t + 3] = dmax;
    keys[t] = mode == 0 ? (int32_t)(((uint32_t)s << 11) | (uint32_t)dmin) : dmin;
    vals[t] = (int32_t)t;
  }
}

__global__ __launch_bounds__(256) void k_tc_strip_keys(const int32_t* __restrict__ hdr,
                                                       const int32_t* __restrict__ tc_p0,
                                                       const int32_t* __restrict__ pair_row,
                                                       const int32_t* __restrict__ vals, Geo g,
                                                       int32_t* __restrict__ keys) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < ntc;
       r += (int64_t)gridDim.x * blockDim.x)
    keys[r] = g.strip(pair_row[tc_p0[vals[r]]]);
}

// TCs in rank order: TC of each rank, rank of each TC, strip and pair count
// of each rank (the counts to be scanned in rk_cum).
__global__ __launch_bounds__(256) void k_tc_rank(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ vals,
                                                 const int32_t* __restrict__ tc_np,
                                                 const int32_t* __restrict__ tc_p0,
                                                 const int32_t* __restrict__ pair_row, Geo g,
                                                 int32_t* __restrict__ tord,
                                                 int32_t* __restrict__ rank_of_tc,
                                                 int32_t* __restrict__ rk_strip,
                                                 int32_t* __restrict__ rk_cum) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < ntc;
       r += (int64_t)gridDim.x * blockDim.x) {
    const int32_t t = vals[r];
    tord[r] = t;
    rank_of_tc[t] = (int32_t)r;
    rk_strip[r] = g.strip(pair_row[tc_p0[t]]);
    rk_cum[r] = tc_np[t];
  }
}

struct RunHeads {  // positions where a key array changes (a run's first element)
  const int32_t* key;
  const int32_t* n_ptr;
  int32_t* first;
  int64_t cap;  // entries `first` holds
  __device__ int64_t count() const { return *n_ptr; }
  __device__ bool flag(int64_t i) const { return i == 0 || key[i] != key[i - 1]; }
  __device__ void emit(int64_t i, int32_t pos) const {
    if (pos < cap) first[pos] = (int32_t)i;
  }
};

// Piece boundaries over ranked TCs (see internal.h).
__global__ __launch_bounds__(256) void k_piece_flags(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ rk_cum,
                                                     const int32_t* __restrict__ ss,
                                                     const int32_t* __restrict__ cnt, int32_t tcmax,
                                                     int32_t* __restrict__ flags) {
  const int64_t ntc = hdr[kSHdrTCs];
  const int32_t nss = cnt[kCntStrips];
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < ntc;
       r += (int64_t)gridDim.x * blockDim.x) {
    const int32_t st = ss[upper_index(ss, nss, (int32_t)r)];
    const int32_t rin = (int32_t)r - st;
    const int32_t cin = rk_cum[r] - rk_cum[st];
    bool f = rin == 0 || rin % tcmax == 0;
    if (!f) {
      const int32_t prev = rk_cum[r - 1] - rk_cum[st];
      f = cin / kSchedPairs != prev / kSchedPairs;
    }
    flags[r] = f ? 1 : 0;
  }
}

struct FlagHeads {  // positions with flag != 0
  const int32_t* flags;
  const int32_t* n_ptr;
  int32_t* first;
  int64_t cap;  // entries `first` holds
  __device__ int64_t count() const { return *n_ptr; }
  __device__ bool flag(int64_t i) const { return flags[i] != 0; }
  __device__ void emit(int64_t i, int32_t pos) const {
    if (pos < cap) first[pos] = (int32_t)i;
  }
};

// ---- 4. CCs and blocks -----------------------------------------------------------

struct CCHeads {  // dense (TC, column) entries that hold pairs, in TC order
  const int32_t* hdr;
  const int32_t* cchhi;
  const int32_t* ccd;
  const int32_t* pc_rank0;
  const int32_t* rank_of_tc;
  int mode;  // 0: key (piece, column, least bin); 1: (column, least bin)
  int32_t* cc_dense;
  int32_t* keys;
  int32_t* vals;
  __device__ int64_t count() const { return (int64_t)hdr[kSHdrTCs] * kSchedSW; }
  __device__ bool flag(int64_t i) const { return cchhi[i] >= 0; }
  __device__ void emit(int64_t i, int32_t pos) const {
    const int32_t t = (int32_t)(i / kSchedSW), c = (int32_t)(i % kSchedSW);
    const int32_t pc = upper_index(pc_rank0, hdr[kSHdrPieces], rank_of_tc[t]);
    const uint32_t low = ((uint32_t)c << 11) | (uint32_t)ccd[i];
    cc_dense[pos] = (int32_t)i;
    keys[pos] = mode == 0 ? (int32_t)(((uint32_t)pc << 13) | low) : (int32_t)low;
    vals[pos] = pos;
  }
};

__global__ __launch_bounds__(256) void k_cc_piece_keys(const int32_t* __restrict__ hdr,
                                                       const int32_t* __restrict__ cc_dense,
                                                       const int32_t* __restrict__ pc_rank0,
                                                       const int32_t* __restrict__ rank_of_tc,
                                                       const int32_t* __restrict__ vals,
                                                       int32_t* __restrict__ keys) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kSHdrCCs]) return;
  keys[q] = upper_index(pc_rank0, hdr[kSHdrPieces], rank_of_tc[cc_dense[vals[q]] / kSchedSW]);
}

// CCs in sorted order: dense index, piece and (piece, column) group
__global__ __launch_bounds__(256) void k_cc_sorted(const int32_t* __restrict__ hdr,
                                                   const int32_t* __restrict__ vals,
                                                   const int32_t* __restrict__ cc_dense,
                                                   const int32_t* __restrict__ pc_rank0,
                                                   const int32_t* __restrict__ rank_of_tc,
                                                   int32_t* __restrict__ q_dense,
                                                   int32_t* __restrict__ q_piece,
                                                   int32_t* __restrict__ q_grp) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kSHdrCCs]) return;
  const int32_t i = cc_dense[vals[q]];
  const int32_t pc = upper_index(pc_rank0, hdr[kSHdrPieces], rank_of_tc[i / kSchedSW]);
  q_dense[q] = i;
  q_piece[q] = pc;
  q_grp[q] = pc * kSchedSW + i % kSchedSW;
}

struct BlockHeads {  // every K-th CC of a (piece, column) group
  const int32_t* hdr;
  const int32_t* gs;  // group starts
  const int32_t* cnt;
  int32_t* bpos0;
  __device__ int64_t count() const { return hdr[kSHdrCCs]; }
  __device__ bool flag(int64_t q) const {
    const int32_t g0 = gs[upper_index(gs, cnt[kCntGroups], (int32_t)q)];
    return ((int32_t)q - g0) % kSchedK == 0;
  }
  __device__ void emit(int64_t q, int32_t pos) const { bpos0[pos] = (int32_t)q; }
};

__global__ __launch_bounds__(256) void k_block_info(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ bpos0,
                                                    const int32_t* __restrict__ gs,
                                                    const int32_t* __restrict__ cnt,
                                                    const int32_t* __restrict__ q_dense,
                                                    const int32_t* __restrict__ q_piece,
                                                    const int32_t* __restrict__ q_grp,
                                                    const int32_t* __restrict__ cchlo,
                                                    const int32_t* __restrict__ cchhi,
                                                    int32_t* __restrict__ blk,
                                                    int32_t* __restrict__ b_sz,
                                                    int32_t* __restrict__ b_piece) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= hdr[kSHdrBlocks]) return;
  const int32_t q0 = bpos0[b];
  const int32_t ng = cnt[kCntGroups];
  const int32_t j = upper_index(gs, ng, q0);
  const int32_t gend = j + 1 < ng ? gs[j + 1] : hdr[kSHdrCCs];
  const int32_t q1 = min(q0 + kSchedK, gend);
  int32_t hlo = INT32_MAX, hhi = -1;
  for (int32_t q = q0; q < q1; ++q) {
    hlo = min(hlo, cchlo[q_dense[q]]);
    hhi = max(hhi, cchhi[q_dense[q]]);
  }
  const int32_t pc = q_piece[q0];
  const int32_t c = q_grp[q0] - pc * kSchedSW;
  blk[4 * b + 0] = c | ((q1 - q0) << 8);
  blk[4 * b + 1] = hlo;
  blk[4 * b + 2] = hhi - hlo + 1;
  b_sz[b] = kSchedK * (hhi - hlo + 1);
  b_piece[b] = pc;
}

__global__ __launch_bounds__(256) void k_block_ebase(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ b_piece,
                                                     const int32_t* __restrict__ bcum,
                                                     const int32_t* __restrict__ pc_blk0,
                                                     int32_t* __restrict__ blk) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= hdr[kSHdrBlocks]) return;
  blk[4 * b + 3] = bcum[b] - bcum[pc_blk0[b_piece[b]]];
}

// Piece CC table and, per dense (rank, column): the CC's partial row in the
// piece (block in piece * K + k) | its index in the piece's CC table << 8.
__global__ __launch_bounds__(256) void k_cc_tab(const int32_t* __restrict__ hdr,
                                                const int32_t* __restrict__ bpos0,
                                                const int32_t* __restrict__ blk,
                                                const int32_t* __restrict__ q_dense,
                                                const int32_t* __restrict__ q_piece,
                                                const int32_t* __restrict__ pc_blk0,
                                                const int32_t* __restrict__ pc_cc0,
                                                int32_t* __restrict__ cc,
                                                int32_t* __restrict__ ccref) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= hdr[kSHdrCCs]) return;
  const int32_t b = upper_index(bpos0, hdr[kSHdrBlocks], (int32_t)q);
  const int32_t k = (int32_t)q - bpos0[b];
  const int32_t pc = q_piece[q];
  cc[q] = (blk[4 * b + 3] + k) | (blk[4 * b + 1] << 16);
  ccref[q_dense[q]] = ((b - pc_blk0[pc]) * kSchedK + k) | (((int32_t)q - pc_cc0[pc]) << 8);
}

// ---- 5. destinations -------------------------------------------------------------

__global__ __launch_bounds__(256) void k_tc_cell_keys(const int32_t* __restrict__ hdr,
                                                      const int32_t* __restrict__ tc_p0,
                                                      const int32_t* __restrict__ pair_rb,
                                                      int32_t* __restrict__ keys,
                                                      int32_t* __restrict__ vals) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < ntc;
       t += (int64_t)gridDim.x * blockDim.x) {
    keys[t] = pair_rb[tc_p0[t]];
    vals[t] = (int32_t)t;
  }
}

// Over TCs sorted by cell: is TC q one of several of its cell?
__device__ __forceinline__ bool shared_cell(const int32_t* keys, int64_t q, int64_t n) {
  return (q > 0 && keys[q - 1] == keys[q]) || (q + 1 < n && keys[q + 1] == keys[q]);
}

__global__ __launch_bounds__(256) void k_slot_flags(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ keys,
                                                    int32_t* __restrict__ flags) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < ntc;
       q += (int64_t)gridDim.x * blockDim.x)
    flags[q] = shared_cell(keys, q, ntc) ? 1 : 0;
}

__global__ __launch_bounds__(256) void k_tc_dest(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ keys,
                                                 const int32_t* __restrict__ vals,
                                                 const int32_t* __restrict__ slot,
                                                 int32_t* __restrict__ dest,
                                                 int32_t* __restrict__ occ, int64_t cells) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < ntc;
       q += (int64_t)gridDim.x * blockDim.x) {
    dest[vals[q]] = shared_cell(keys, q, ntc) ? ~slot[q] : keys[q];
    if (keys[q] >= 0 && keys[q] < cells) occ[keys[q]] = 1;
  }
}

struct CombHeads {  // cells with several TCs: their first slot
  const int32_t* keys;
  const int32_t* slot;
  const int32_t* hdr;
  int32_t* comb_cell;
  int32_t* comb_slot0;
  int64_t cap;
  __device__ int64_t count() const { return hdr[kSHdrTCs]; }
  __device__ bool flag(int64_t q) const {
    return (q == 0 || keys[q - 1] != keys[q]) && shared_cell(keys, q, count());
  }
  __device__ void emit(int64_t q, int32_t pos) const {
    if (pos >= cap) return;
    comb_cell[pos] = keys[q];
    comb_slot0[pos] = slot[q];
  }
};

struct CellRuns {  // occupied cells: runs of equal cell over sorted TCs
  const int32_t* keys;
  const int32_t* hdr;
  __device__ int64_t count() const { return hdr[kSHdrTCs]; }
  __device__ bool flag(int64_t q) const { return q == 0 || keys[q - 1] != keys[q]; }
  __device__ void emit(int64_t, int32_t) const {}
};

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

// TC table in rank order: destination and each column's partial row
__global__ __launch_bounds__(256) void k_tc_tab(const int32_t* __restrict__ hdr,
                                                const int32_t* __restrict__ tord,
                                                const int32_t* __restrict__ dest,
                                                const int32_t* __restrict__ cchhi,
                                                const int32_t* __restrict__ ccref,
                                                int32_t* __restrict__ tc) {
  const int64_t ntc = hdr[kSHdrTCs];
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < ntc;
       r += (int64_t)gridDim.x * blockDim.x) {
    uint32_t prs = 0;
    const int64_t t = tord[r];
#pragma unroll
    for (int c = 0; c < kSchedSW; ++c) {
      const int64_t i = t * kSchedSW + c;
      const uint32_t pr = cchhi[i] >= 0 ? (uint32_t)(ccref[i] & 0xFF) : 0xFFu;
      prs |= pr << (8 * c);
    }
    tc[2 * r] = dest[t];
    tc[2 * r + 1] = (int32_t)prs;
  }
}

// ---- 6. pieces and records -------------------------------------------------------

// Row and depth range of every piece, from its TCs' ranges.
__global__ __launch_bounds__(256) void k_piece_range(const int32_t* __restrict__ hdr,
                                                     const int32_t* __restrict__ pc_rank0,
                                                     const int32_t* __restrict__ tord,
                                                     const int32_t* __restrict__ tc_rng,
                                                     int32_t* __restrict__ plo, int32_t* __restrict__ phi,
                                                     int32_t* __restrict__ dlo, int32_t* __restrict__ dhi) {
  const int64_t n = hdr[kSHdrPieces];
  for (int64_t pc = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; pc < n;
       pc += (int64_t)gridDim.x * blockDim.x) {
    const int32_t r0 = pc_rank0[pc], r1 = pc + 1 < n ? pc_rank0[pc + 1] : hdr[kSHdrTCs];
    int32_t hl = INT32_MAX, hh = -1, dl = INT32_MAX, dh = -1;
    for (int32_t r = r0; r < r1; ++r) {
      const int32_t* rg = tc_rng + 4 * (int64_t)tord[r];
      hl = min(hl, rg[0]);
      hh = max(hh, rg[1]);
      dl = min(dl, rg[2]);
      dh = max(dh, rg[3]);
    }
    plo[pc] = hl;
    phi[pc] = hh;
    dlo[pc] = dl;
    dhi[pc] = dh;
  }
}

// Each pair's piece and its CC's index in the piece's CC table.
__global__ __launch_bounds__(256) void k_pair_piece(const int32_t* __restrict__ hdr,
                                                    const int32_t* __restrict__ tc_p0,
                                                    const int32_t* __restrict__ rank_of_tc,
                                                    const int32_t* __restrict__ pc_rank0,
                                                    const int32_t* __restrict__ pair_row, Geo g,
                                                    const int32_t* __restrict__ ccref,
                                                    int32_t* __restrict__ pair_pc,
                                                    int32_t* __restrict__ pair_ccl) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= hdr[kSHdrPairs]) return;
  const int32_t t = upper_index(tc_p0, hdr[kSHdrTCs], (int32_t)k);
  pair_pc[k] = upper_index(pc_rank0, hdr[kSHdrPieces], rank_of_tc[t]);
  pair_ccl[k] = (ccref[(int64_t)t * kSchedSW + g.col(pair_row[k])] >> 8) & 0xFF;
}

// record sort keys: mode 0 (piece, local pixel, d0) joined, mode 1 (local
// pixel, d0), mode 2 the piece
__global__ __launch_bounds__(256) void k_rec_keys(const int32_t* __restrict__ hdr,
                                                  const int32_t* __restrict__ vals_in,
                                                  const int32_t* __restrict__ pair_pc,
                                                  const int32_t* __restrict__ pair_row,
                                                  const uint32_t* __restrict__ pair_dn,
                                                  const int32_t* __restrict__ plo, Geo g, int lp_bits,
                                                  int mode, int32_t* __restrict__ keys,
                                                  int32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= hdr[kSHdrPairs]) return;
  const int32_t k = vals_in != nullptr ? vals_in[i] : (int32_t)i;
  const int32_t pc = pair_pc[k];
  const int32_t row = pair_row[k];
  const uint32_t lp = (uint32_t)((g.h(row) - plo[pc]) * kSchedSW + g.col(row));
  const uint32_t low = (lp << 11) | (pair_dn[k] & 0x7FFu);
  keys[i] = mode == 0 ? (int32_t)(((uint32_t)pc << (lp_bits + 11)) | low)
                      : (mode == 1 ? (int32_t)low : pc);
  vals[i] = k;
}

__global__ __launch_bounds__(256) void k_records(const int32_t* __restrict__ hdr,
                                                 const int32_t* __restrict__ vals,
                                                 const int32_t* __restrict__ pair_pc,
                                                 const int32_t* __restrict__ pair_row,
                                                 const uint32_t* __restrict__ pair_dn,
                                                 const int32_t* __restrict__ pair_ccl,
                                                 const int32_t* __restrict__ plo,
                                                 const int32_t* __restrict__ dlo, Geo g,
                                                 uint32_t* __restrict__ rec,
                                                 int32_t* __restrict__ rec_pc,
                                                 int32_t* __restrict__ rec_lp) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= hdr[kSHdrPairs]) return;
  const int32_t k = vals[i];
  const int32_t pc = pair_pc[k];
  const uint32_t dn = pair_dn[k];
  const int32_t row = pair_row[k];
  rec[i] = ((dn & 0xFFFFu) - (uint32_t)dlo[pc]) | (((dn >> 16) - 1u) << 11) |
           ((uint32_t)pair_ccl[k] << 24);
  rec_pc[i] = pc;
  rec_lp[i] = (g.h(row) - plo[pc]) * kSchedSW + g.col(row);
}

struct PieceWords {  // the arrays a piece row is assembled from
  const int32_t* pc_rank0;
  const int32_t* pc_blk0;
  const int32_t* pc_cc0;
  const int32_t* pc_rec0;
  const int32_t* rk_strip;
  const int32_t* bcum;
  const int32_t* plo;
  const int32_t* phi;
  const int32_t* dlo;
  const int32_t* dhi;
};

__global__ __launch_bounds__(256) void k_piece_table(int32_t* __restrict__ hdr, PieceWords pw,
                                                     int32_t W, int32_t nsw,
                                                     int32_t* __restrict__ piece,
                                                     int32_t* __restrict__ npix) {
  const int64_t n = hdr[kSHdrPieces];
  int32_t m[4] = {0, 0, 0, 0};  // this thread's maxima of nent, nblk, pixels, records
  for (int64_t pc = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; pc < n;
       pc += (int64_t)gridDim.x * blockDim.x) {
    const int32_t r0 = pw.pc_rank0[pc], r1 = pc + 1 < n ? pw.pc_rank0[pc + 1] : hdr[kSHdrTCs];
    const int32_t b0 = pw.pc_blk0[pc], b1 = pc + 1 < n ? pw.pc_blk0[pc + 1] : hdr[kSHdrBlocks];
    const int32_t c0 = pw.pc_cc0[pc], c1 = pc + 1 < n ? pw.pc_cc0[pc + 1] : hdr[kSHdrCCs];
    const int32_t e0 = pw.pc_rec0[pc], e1 = pc + 1 < n ? pw.pc_rec0[pc + 1] : hdr[kSHdrPairs];
    const int32_t strip = pw.rk_strip[r0];
    const int32_t nh = pw.phi[pc] - pw.plo[pc] + 1;
    const int32_t nent = pw.bcum[b1] - pw.bcum[b0];
    int32_t* p = piece + pc * kPieceWords;
    p[0] = strip;
    p[1] = pw.plo[pc];
    p[2] = nh;
    p[3] = pw.dlo[pc];
    p[4] = pw.dhi[pc] - pw.dlo[pc] + 1;
    p[5] = b0;
    p[6] = b1 - b0;
    p[7] = e0;
    p[8] = e1 - e0;
    p[9] = r0;
    p[10] = r1 - r0;
    p[11] = c0;
    p[12] = c1 - c0;
    p[13] = nent;
    p[15] = min(kSchedSW, W - (strip % nsw) * kSchedSW);
    npix[pc] = nh * kSchedSW + 1;
    m[0] = max(m[0], nent);
    m[1] = max(m[1], b1 - b0);
    m[2] = max(m[2], nh * kSchedSW);
    m[3] = max(m[3], e1 - e0);
  }
  // block maxima, then one atomic per block and count
  __shared__ int32_t s_m[4][256 / kWave];
  const int lane = lane_id(), wid = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int32_t v = m[j];
    for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, kWave));
    if (lane == 0) s_m[j][wid] = v;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    int32_t v = 0;
    for (int w = 0; w < 256 / kWave; ++w) v = max(v, s_m[threadIdx.x][w]);
    const int word[4] = {kSHdrMaxEnt, kSHdrMaxBlk, kSHdrMaxPix, kSHdrMaxRec};
    if (v > 0) atomicMax(&hdr[word[threadIdx.x]], v);
  }
}

// Each piece's pixel table (one workgroup per piece at a time): the first
// record of every local pixel, relative to the piece's first record.
__global__ __launch_bounds__(256) void k_pixrec(const int32_t* __restrict__ hdr,
                                                int32_t* __restrict__ piece,
                                                const int32_t* __restrict__ pix0,
                                                const int32_t* __restrict__ rec_lp,
                                                int32_t* __restrict__ pixrec, int64_t cap) {
  const int64_t n = hdr[kSHdrPieces];
  for (int64_t pc = blockIdx.x; pc < n; pc += gridDim.x) {
    int32_t* p = piece + pc * kPieceWords;
    const int32_t base = pix0[pc];
    const int32_t npx = p[2] * kSchedSW;
    const int32_t e0 = p[7], ne = p[8];
    if (threadIdx.x == 0) p[14] = base;
    for (int32_t lp = threadIdx.x; lp <= npx; lp += blockDim.x) {
      int32_t lo = 0, hi = ne;  // first record with local pixel >= lp
      while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (rec_lp[e0 + mid] < lp) lo = mid + 1; else hi = mid;
      }
      if ((int64_t)base + lp < cap) pixrec[base + lp] = lo;
    }
  }
}

template <class Op>
void compact(const Op& op, int64_t ntiles, int32_t* tiles, int32_t* sums, int32_t* count_out,
             hipStream_t stream) {
  const dim3 grid((unsigned)ntiles), block(kPrepThreads);
  k_compact_count<<<grid, block, 0, stream>>>(op, tiles);
  scan_exclusive(tiles, ntiles, sums, count_out, stream);
  k_compact_scatter<<<grid, block, 0, stream>>>(op, tiles);
}

}  // namespace

int64_t sched_tc_max(int64_t H) {
  const int64_t blocks_per_col = std::min<int64_t>(4, kSchedEntries / (kSchedSW * kSchedK * H));
  return kSchedK * std::max<int64_t>(0, blocks_per_col);
}

namespace {

// Build workspace: one int32 array per intermediate.
enum WsArray {
  kWsKa, kWsVa, kWsKb, kWsVb,                  // sort ping-pong
  kWsHeadPos, kWsPairRb, kWsPairRow, kWsPairDn,
  kWsTcP0, kWsTcNp, kWsTcRng, kWsTord, kWsRankOfTc, kWsRkStrip, kWsRkCum, kWsStripStarts, kWsFlags,
  kWsPcRank0, kWsCcD, kWsCcHlo, kWsCcHhi, kWsCcRef,
  kWsCcDense, kWsQDense, kWsQPiece, kWsQGrp, kWsGroupStarts, kWsBpos0, kWsBcum, kWsBPiece,
  kWsPcBlk0, kWsPcCc0, kWsSlot, kWsDest, kWsOcc, kWsPlo, kWsPhi, kWsDlo, kWsDhi, kWsNpix,
  kWsPairPc, kWsPairCcl, kWsRecPc, kWsRecLp, kWsPcRec0, kWsCounters, kWsTiles, kWsHist, kWsSums,
  kWsCount
};

struct WsLayout {
  size_t off[kWsCount];
  size_t total;
  int64_t ntiles;
};

WsLayout ws_layout(const Dims& d, int64_t nv, int64_t pcap) {
  const int64_t span = std::max<int64_t>(nv * kSchedSW, d.cells);
  WsLayout w{};
  w.ntiles = (span + kPrepTile - 1) / kPrepTile;
  const int64_t scan_n = std::max<int64_t>(256 * w.ntiles, span);
  const int64_t nscan = (scan_n + kScanTile - 1) / kScanTile;
  int64_t n[kWsCount];
  for (int i = 0; i < kWsCount; ++i) n[i] = nv + 1;
  n[kWsPcRank0] = n[kWsPcBlk0] = n[kWsPcCc0] = n[kWsPcRec0] = pcap + 1;
  n[kWsPlo] = n[kWsPhi] = n[kWsDlo] = n[kWsDhi] = n[kWsNpix] = pcap + 1;
  n[kWsCcD] = n[kWsCcHlo] = n[kWsCcHhi] = n[kWsCcRef] = (int64_t)kSchedSW * nv;
  n[kWsTcRng] = 4 * nv;
  n[kWsOcc] = d.cells + 1;
  n[kWsCounters] = 16;
  n[kWsTiles] = w.ntiles + 2;
  n[kWsHist] = 256 * w.ntiles;
  n[kWsSums] = nscan + 1;
  size_t off = 0;
  for (int i = 0; i < kWsCount; ++i) {
    w.off[i] = off;
    off += align_up(sizeof(int32_t) * (size_t)n[i]);
  }
  w.total = off;
  return w;
}

}  // namespace

ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals) {
  ScheduleLayout L{};
  L.n_valid = n_valid;
  L.n_occ = n_intervals;
  L.n_empty = d.cells > n_intervals ? d.cells - n_intervals : 0;
  L.nsw = (d.W + kSchedSW - 1) / kSchedSW;
  L.strips = d.B * d.N * L.nsw;
  const int64_t nv = n_valid > 0 ? n_valid : 1;
  // pieces: at most one per strip start, per tcmax-th TC and per kSchedPairs pairs
  const int64_t tcmax = std::max<int64_t>(sched_tc_max(d.H), 1);
  L.piece_cap = std::min<int64_t>(nv, 2 * L.strips + nv / tcmax + nv / kSchedPairs + 2);
  size_t off = 0;
  auto take = [&](int64_t n_ints) {
    const size_t o = off;
    off += align_up(sizeof(int32_t) * (size_t)n_ints);
    return o;
  };
  L.header = take(16);
  L.piece = take((int64_t)kPieceWords * L.piece_cap);
  L.block = take(4 * nv);
  L.cc = take(nv);
  L.tc = take(2 * nv);
  L.pixrec_cap = L.piece_cap * (d.H * kSchedSW + 1);  // a piece's pixel rows: at most H
  L.pixrec = take(L.pixrec_cap);
  L.rec = take(nv);
  L.comb_cell = take(n_intervals + 1);
  L.comb_slot0 = take(n_intervals + 1);
  L.empty = take(L.n_empty + 1);
  L.bp_cell = take(nv);
  L.bp_dn = take(nv);
  L.pix_pair0 = take(d.rows + 1);
  L.total = off;
  L.ws_total = ws_layout(d, nv, L.piece_cap).total;
  return L;
}

hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream) {
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  const int64_t nv = std::max<int64_t>(n_valid, 1);
  const WsLayout wl = ws_layout(d, nv, L.piece_cap);
  char* sc = static_cast<char*>(schedule);
  char* wsb = static_cast<char*>(workspace);
  auto S = [&](size_t o) { return reinterpret_cast<int32_t*>(sc + o); };
  auto W = [&](WsArray a) { return reinterpret_cast<int32_t*>(wsb + wl.off[a]); };
  int32_t* hdr = S(L.header);
  int32_t* tiles = W(kWsTiles);
  int32_t* sums = W(kWsSums);
  int32_t* hist = W(kWsHist);
  int32_t* cnt = W(kWsCounters);
  const int64_t ntiles = wl.ntiles;
  const unsigned g_nv = (unsigned)((nv + 255) / 256);
  const unsigned g_cells = (unsigned)((d.cells + 255) / 256);
  const unsigned g_str = kStride;
  Geo geo;
  geo.per_view = (uint32_t)d.per_view;
  geo.hw = (uint32_t)d.hw;
  geo.H = (int32_t)d.H;
  geo.W = (int32_t)d.W;
  geo.nsw = (int32_t)L.nsw;
  const int32_t tcmax = (int32_t)sched_tc_max(d.H);
  const int row_bits = bit_length(d.rows);
  const int cell_bits = bit_length(d.cells);
  const int lp_bits = bit_length(d.H * kSchedSW + 1);
  const int strip_bits = bit_length(L.strips);
  const int piece_bits = bit_length(L.piece_cap + 1);

  k_sched_init<<<1, 64, 0, stream>>>(hdr, cnt, n_valid, n_intervals);
  int32_t* occ = W(kWsOcc);
  k_fill_i32<<<g_cells, 256, 0, stream>>>(occ, d.cells, 0);
  if (n_valid > 0) {
    int32_t *ck = W(kWsKa), *cv = W(kWsVa), *ak = W(kWsKb), *av = W(kWsVb);
    auto sort_current = [&](int bits, const int32_t* n_ptr) {
      if (radix_sort_pairs(ck, cv, ak, av, n_ptr, ntiles, bits, hist, sums, stream)) {
        std::swap(ck, ak);
        std::swap(cv, av);
      }
    };
    auto reset_sort = [&]() {
      ck = W(kWsKa); cv = W(kWsVa); ak = W(kWsKb); av = W(kWsVb);
    };

    // 1. points by (strip, cell, pixel, plan position) -> pairs
    k_pixel_keys<<<g_nv, 256, 0, stream>>>(rd, n_valid, geo, ck, cv);
    sort_current(lp_bits, hdr + kSHdrValid);
    if (strip_bits + cell_bits <= 31) {
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, geo, cell_bits, 0, ck);
      sort_current(strip_bits + cell_bits, hdr + kSHdrValid);
    } else {
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, geo, cell_bits, 1, ck);
      sort_current(cell_bits, hdr + kSHdrValid);
      k_strip_keys<<<g_nv, 256, 0, stream>>>(rd, rb, cv, n_valid, geo, cell_bits, 2, ck);
      sort_current(strip_bits, hdr + kSHdrValid);
    }
    int32_t* pair_rb = W(kWsPairRb);
    int32_t* pair_row = W(kWsPairRow);
    uint32_t* pair_dn = reinterpret_cast<uint32_t*>(W(kWsPairDn));
    int32_t* head_pos = W(kWsHeadPos);
    compact(PairHeads{rd, rb, cv, hdr, geo, pair_rb, pair_row, pair_dn, head_pos}, ntiles, tiles,
            sums, hdr + kSHdrPairs, stream);
    k_pair_points<<<g_nv, 256, 0, stream>>>(head_pos, hdr, pair_dn);

    // 2. pixel-major pairs (stable by feature row: cell order within a pixel)
    reset_sort();
    k_pair_row_keys<<<g_nv, 256, 0, stream>>>(hdr, pair_row, ck, cv);
    sort_current(row_bits, hdr + kSHdrPairs);
    k_pix_pairs<<<g_nv, 256, 0, stream>>>(hdr, cv, pair_rb, pair_dn, S(L.bp_cell),
                                          reinterpret_cast<uint32_t*>(S(L.bp_dn)));
    k_pix_offsets<<<(unsigned)((d.rows + 1 + 255) / 256), 256, 0, stream>>>(hdr, ck, d.rows,
                                                                            S(L.pix_pair0));

    // 3. TCs ranked by (strip, least depth bin) and cut into pieces
    int32_t* tc_p0 = W(kWsTcP0);
    compact(TCHeads{pair_rb, pair_row, hdr, geo, tc_p0}, ntiles, tiles, sums, hdr + kSHdrTCs,
            stream);
    k_set_end<<<1, 64, 0, stream>>>(tc_p0, hdr + kSHdrTCs, hdr + kSHdrPairs, nv);
    int32_t* tc_np = W(kWsTcNp);
    reset_sort();
    const bool tc_joined = strip_bits + 11 <= 31;
    int32_t* tc_rng = W(kWsTcRng);
    int32_t* ccd = W(kWsCcD);
    int32_t* cchlo = W(kWsCcHlo);
    int32_t* cchhi = W(kWsCcHhi);
    int32_t* ccref = W(kWsCcRef);
    k_tc_keys<<<g_str, 256, 0, stream>>>(hdr, tc_p0, pair_row, pair_dn, geo, tc_joined ? 0 : 1,
                                         tc_np, tc_rng, ccd, cchlo, cchhi, ck, cv);
    sort_current(tc_joined ? strip_bits + 11 : 11, hdr + kSHdrTCs);
    if (!tc_joined) {
      k_tc_strip_keys<<<g_str, 256, 0, stream>>>(hdr, tc_p0, pair_row, cv, geo, ck);
      sort_current(strip_bits, hdr + kSHdrTCs);
    }
    int32_t* tord = W(kWsTord);
    int32_t* rank_of_tc = W(kWsRankOfTc);
    int32_t* rk_strip = W(kWsRkStrip);
    int32_t* rk_cum = W(kWsRkCum);
    k_tc_rank<<<g_str, 256, 0, stream>>>(hdr, cv, tc_np, tc_p0, pair_row, geo, tord, rank_of_tc,
                                         rk_strip, rk_cum);
    scan_exclusive(rk_cum, nv, sums, nullptr, stream, hdr + kSHdrTCs);
    int32_t* ss = W(kWsStripStarts);
    compact(RunHeads{rk_strip, hdr + kSHdrTCs, ss, nv + 1}, ntiles, tiles, sums, cnt + kCntStrips, stream);
    int32_t* flags = W(kWsFlags);
    k_piece_flags<<<g_str, 256, 0, stream>>>(hdr, rk_cum, ss, cnt, tcmax, flags);
    int32_t* pc_rank0 = W(kWsPcRank0);
    compact(FlagHeads{flags, hdr + kSHdrTCs, pc_rank0, L.piece_cap}, ntiles, tiles, sums, hdr + kSHdrPieces,
            stream);

    // 4. CCs and blocks
    reset_sort();
    int32_t* cc_dense = W(kWsCcDense);
    const bool cc_joined = piece_bits + 13 <= 31;
    compact(CCHeads{hdr, cchhi, ccd, pc_rank0, rank_of_tc, cc_joined ? 0 : 1, cc_dense, ck, cv}, ntiles,
            tiles, sums, hdr + kSHdrCCs, stream);
    sort_current(cc_joined ? piece_bits + 13 : 13, hdr + kSHdrCCs);
    if (!cc_joined) {
      k_cc_piece_keys<<<g_nv, 256, 0, stream>>>(hdr, cc_dense, pc_rank0, rank_of_tc, cv, ck);
      sort_current(piece_bits, hdr + kSHdrCCs);
    }
    int32_t* q_dense = W(kWsQDense);
    int32_t* q_piece = W(kWsQPiece);
    int32_t* q_grp = W(kWsQGrp);
    k_cc_sorted<<<g_nv, 256, 0, stream>>>(hdr, cv, cc_dense, pc_rank0, rank_of_tc, q_dense, q_piece,
                                          q_grp);
    int32_t* gs = W(kWsGroupStarts);
    compact(RunHeads{q_grp, hdr + kSHdrCCs, gs, nv + 1}, ntiles, tiles, sums, cnt + kCntGroups, stream);
    int32_t* bpos0 = W(kWsBpos0);
    compact(BlockHeads{hdr, gs, cnt, bpos0}, ntiles, tiles, sums, hdr + kSHdrBlocks, stream);
    int32_t* blk = S(L.block);
    int32_t* bcum = W(kWsBcum);
    int32_t* b_piece = W(kWsBPiece);
    k_block_info<<<g_nv, 256, 0, stream>>>(hdr, bpos0, gs, cnt, q_dense, q_piece, q_grp, cchlo,
                                           cchhi, blk, bcum, b_piece);
    scan_exclusive(bcum, nv, sums, cnt + kCntEntries, stream, hdr + kSHdrBlocks);
    k_set_end<<<1, 64, 0, stream>>>(bcum, hdr + kSHdrBlocks, cnt + kCntEntries, nv);
    int32_t* pc_blk0 = W(kWsPcBlk0);
    compact(RunHeads{b_piece, hdr + kSHdrBlocks, pc_blk0, L.piece_cap}, ntiles, tiles, sums,
            cnt + kCntPieceBlocks, stream);
    k_block_ebase<<<g_nv, 256, 0, stream>>>(hdr, b_piece, bcum, pc_blk0, blk);
    int32_t* pc_cc0 = W(kWsPcCc0);
    compact(RunHeads{q_piece, hdr + kSHdrCCs, pc_cc0, L.piece_cap}, ntiles, tiles, sums, nullptr, stream);
    k_cc_tab<<<g_nv, 256, 0, stream>>>(hdr, bpos0, blk, q_dense, q_piece, pc_blk0, pc_cc0,
                                       S(L.cc), ccref);

    // 5. destinations: one slot per TC of a cell reached from several strips
    reset_sort();
    k_tc_cell_keys<<<g_str, 256, 0, stream>>>(hdr, tc_p0, pair_rb, ck, cv);
    sort_current(cell_bits, hdr + kSHdrTCs);
    int32_t* slot = W(kWsSlot);
    k_slot_flags<<<g_str, 256, 0, stream>>>(hdr, ck, slot);
    scan_exclusive(slot, nv, sums, hdr + kSHdrSlots, stream, hdr + kSHdrTCs);
    int32_t* dest = W(kWsDest);
    k_tc_dest<<<g_str, 256, 0, stream>>>(hdr, ck, cv, slot, dest, occ, d.cells);
    compact(CombHeads{ck, slot, hdr, S(L.comb_cell), S(L.comb_slot0), n_intervals}, ntiles, tiles,
            sums, hdr + kSHdrComb, stream);
    k_set_end<<<1, 64, 0, stream>>>(S(L.comb_slot0), hdr + kSHdrComb, hdr + kSHdrSlots,
                                    n_intervals);
    compact(CellRuns{ck, hdr}, ntiles, tiles, sums, hdr + kSHdrOccFound, stream);
    k_tc_tab<<<g_str, 256, 0, stream>>>(hdr, tord, dest, cchhi, ccref, S(L.tc));

    // 6. pieces and records
    int32_t* plo = W(kWsPlo);
    int32_t* phi = W(kWsPhi);
    int32_t* dlo = W(kWsDlo);
    int32_t* dhi = W(kWsDhi);
    int32_t* pair_pc = W(kWsPairPc);
    int32_t* pair_ccl = W(kWsPairCcl);
    k_piece_range<<<g_str, 256, 0, stream>>>(hdr, pc_rank0, tord, tc_rng, plo, phi, dlo, dhi);
    k_pair_piece<<<g_nv, 256, 0, stream>>>(hdr, tc_p0, rank_of_tc, pc_rank0, pair_row, geo, ccref,
                                           pair_pc, pair_ccl);
    reset_sort();
    const bool rec_joined = piece_bits + lp_bits + 11 <= 31;
    k_rec_keys<<<g_nv, 256, 0, stream>>>(hdr, nullptr, pair_pc, pair_row, pair_dn, plo, geo,
                                         lp_bits, rec_joined ? 0 : 1, ck, cv);
    sort_current(rec_joined ? piece_bits + lp_bits + 11 : lp_bits + 11, hdr + kSHdrPairs);
    if (!rec_joined) {
      k_rec_keys<<<g_nv, 256, 0, stream>>>(hdr, cv, pair_pc, pair_row, pair_dn, plo, geo, lp_bits,
                                           2, ck, av);
      std::swap(cv, av);
      sort_current(piece_bits, hdr + kSHdrPairs);
    }
    int32_t* rec_pc = W(kWsRecPc);
    int32_t* rec_lp = W(kWsRecLp);
    k_records<<<g_nv, 256, 0, stream>>>(hdr, cv, pair_pc, pair_row, pair_dn, pair_ccl, plo, dlo,
                                        geo, reinterpret_cast<uint32_t*>(S(L.rec)), rec_pc,
                                        rec_lp);
    int32_t* pc_rec0 = W(kWsPcRec0);
    compact(RunHeads{rec_pc, hdr + kSHdrPairs, pc_rec0, L.piece_cap}, ntiles, tiles, sums, nullptr, stream);
    int32_t* npix = W(kWsNpix);
    PieceWords pw{pc_rank0, pc_blk0, pc_cc0, pc_rec0, rk_strip, bcum, plo, phi, dlo, dhi};
    k_piece_table<<<g_str, 256, 0, stream>>>(hdr, pw, geo.W, geo.nsw, S(L.piece), npix);
    scan_exclusive(npix, L.piece_cap, sums, hdr + kSHdrPixrec, stream, hdr + kSHdrPieces);
    k_pixrec<<<g_str, 256, 0, stream>>>(hdr, S(L.piece), npix, rec_lp, S(L.pixrec), L.pixrec_cap);
  }

  // empty cells (all of them when the plan is empty)
  const dim3 cgrid((unsigned)((d.cells + kPrepTile - 1) / kPrepTile));
  EmptyCells ec{occ, d.cells, S(L.empty), L.n_empty};
  compact(ec, (int64_t)cgrid.x, tiles, sums, hdr + kSHdrEmpty, stream);
  return hipGetLastError();
}

}  // namespace bevpool
