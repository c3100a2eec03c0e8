// BEVPoolv2 pooling (section 2.1, paragraph 2): every occupied BEV cell sums
// depth[rank_depth] * feat[rank_feat, :] over the points of its interval,
// reading both operands through the frustum-index trace, so the frustum
// feature is never formed.
//
// Interval lengths are very uneven (mean 89, longest 4520 points at the
// 640x1600 / D=118 shape), so work is not assigned per interval.  Instead the
// sorted points are cut into equal ranges of RG points (a merge-path style
// partition: every range costs the same).
//
//   k_fwd_ranges   A 64-lane wavefront is split into G lane groups of CV
//                  lanes, CV = 16-byte vectors per feature row, and each
//                  group owns one range.  The wave first loads the ranks of
//                  all its G*RG points (coalesced, one point per lane), gathers
//                  their depth scores and stages (depth, feature rank, BEV
//                  rank) in LDS.  Each group then walks its range reading that
//                  metadata as LDS broadcasts and keeps kUnroll feature-row
//                  loads in flight.  When the BEV rank changes the group
//                  flushes its sum: a cell lying inside the range is stored
//                  once; the part of a cell cut by a range boundary goes to
//                  one of the range's two partial slots.
//   k_fwd_cells    One lane group per interval: combines the partial slots of
//                  cells that span several ranges (in range order, so the
//                  result is deterministic) and zero-fills the empty cells
//                  between consecutive occupied cells.
//
// Every element of `out` is written exactly once and no atomics are used.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

constexpr int kFwdThreads = 256;
constexpr int kFwdWaves = kFwdThreads / kWave;
constexpr int kUnroll = 8;
constexpr int kMetaPerWave = 256;  // points staged in LDS per wavefront

struct FwdArgs {
  const int32_t* rd;
  const int32_t* rf;
  const int32_t* rb;
  const int32_t* starts;
  const int32_t* lengths;
  float* part_a;  // [n_ranges][C]: first segment of a range, continued from the previous range
  float* part_b;  // [n_ranges][C]: last segment of a range, continued in the next range
  int32_t n_valid;
  int32_t n_intervals;
  int32_t C;
  int32_t RG;     // points per range
  int64_t cells;
  int64_t P;
  int64_t rows;
};

struct PointMeta {
  float depth;
  int32_t row;   // feature rank
  int32_t cell;  // BEV rank
};

template <typename TOut, int VEC>
__device__ __forceinline__ void zero_rows(TOut* __restrict__ out, int64_t r0, int64_t r1, int C,
                                          int cbase, int cvc, int lane, int width) {
  if (r1 <= r0) return;
  const int64_t total = (r1 - r0) * cvc;
  for (int64_t idx = lane; idx < total; idx += width) {
    const int64_t r = r0 + idx / cvc;
    const int v = (int)(idx % cvc);
    store_zero<TOut, VEC>(out + r * C + (int64_t)(cbase + v) * VEC);
  }
}

template <typename TIn, typename TOut, int VEC>
__global__ __launch_bounds__(kFwdThreads) void k_fwd_ranges(const TIn* __restrict__ depth,
                                                            const TIn* __restrict__ feat,
                                                            TOut* __restrict__ out, FwdArgs a) {
  __shared__ PointMeta meta_all[kFwdWaves][kMetaPerWave];
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  PointMeta* meta = meta_all[wid];

  const int C = a.C;
  const int CV = C / VEC;
  const int cbase = blockIdx.y * kWave;
  const int cvc = min(kWave, CV - cbase);
  const int RG = a.RG;
  // groups per wave, capped so the wave's points fit the LDS staging area
  const int G = min(kWave / cvc, kMetaPerWave / RG);
  const int g = lane / cvc;
  const int vi = lane - g * cvc;

  // this wave's points: ranges w*G .. w*G+G-1.  Workgroup b runs on die
  // b % kXcds; consecutive blocks of ranges are given to the same die so its
  // L2 holds the feature rows of one region of the grid.
  const int64_t per_die = gridDim.x / kXcds;
  const int64_t lb = (int64_t)(blockIdx.x % kXcds) * per_die + blockIdx.x / kXcds;
  const int64_t w = lb * kFwdWaves + wid;
  const int64_t wb = w * G * RG;
  if (wb >= a.n_valid) return;
  const int wn = (int)min<int64_t>((int64_t)G * RG, a.n_valid - wb);

  // stage (depth, feature rank, BEV rank) of the wave's points in LDS
  for (int k = lane; k < wn; k += kWave) {
    const int32_t pa = a.rd[wb + k];
    const int32_t pf = a.rf[wb + k];
    PointMeta m;
    m.cell = a.rb[wb + k];
    m.depth = 0.f;
    m.row = 0;
    if (pa >= 0 && pa < a.P && pf >= 0 && pf < a.rows) {
      m.depth = to_float(depth[pa]);
      m.row = pf;
    }
    meta[k] = m;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  if (g >= G) return;  // idle lanes past the last group
  const int k_begin = g * RG;
  const int k_end = min(k_begin + RG, wn);
  if (k_begin >= k_end) return;
  const int64_t range = w * G + g;
  const int64_t gs = wb + k_begin, ge = wb + k_end;
  const int32_t prev_c = gs > 0 ? a.rb[gs - 1] : -1;
  const int32_t next_c = ge < a.n_valid ? a.rb[ge] : -1;
  const TIn* fbase = feat + (int64_t)(cbase + vi) * VEC;
  const int64_t col = (int64_t)(cbase + vi) * VEC;

  float acc0[VEC], acc1[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc0[e] = acc1[e] = 0.f;
  int32_t cur = meta[k_begin].cell;

  auto flush = [&]() {
    float s[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      s[e] = acc0[e] + acc1[e];
      acc0[e] = acc1[e] = 0.f;
    }
    if (cur == prev_c) {
      Vec<float, VEC>::store(a.part_a + range * C + col, s);
    } else if (cur == next_c) {
      Vec<float, VEC>::store(a.part_b + range * C + col, s);
    } else if (cur >= 0 && cur < a.cells) {
      Vec<TOut, VEC>::store(out + (int64_t)cur * C + col, s);
    }
  };

  for (int k0 = k_begin; k0 < k_end; k0 += kUnroll) {
    float d[kUnroll];
    int32_t c[kUnroll];
    float v[kUnroll][VEC];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int k = k0 + u;
      if (k < k_end) {
        const PointMeta m = meta[k];
        d[u] = m.depth;
        c[u] = m.cell;
        Vec<TIn, VEC>::load(fbase + (int64_t)m.row * C, v[u]);
      } else {
        d[u] = 0.f;
        c[u] = -1;  // padding past the range end: never a cell change
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[u][e] = 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (k0 + u < k_end && c[u] != cur) {
        flush();
        cur = c[u];
      }
      float* acc = (u & 1) ? acc1 : acc0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = fmaf(d[u], v[u][e], acc[e]);
    }
  }
  flush();
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(kFwdThreads) void k_fwd_cells(TOut* __restrict__ out, FwdArgs a) {
  const int lane = lane_id();
  const int C = a.C;
  const int CV = C / VEC;
  const int cbase = blockIdx.y * kWave;
  const int cvc = min(kWave, CV - cbase);
  const int G = kWave / cvc;
  const int g = lane / cvc;
  const int vi = lane - g * cvc;
  if (g >= G) return;
  const int64_t j = ((int64_t)blockIdx.x * kFwdWaves + threadIdx.x / kWave) * G + g;
  if (j >= a.n_intervals) return;

  const int64_t s = a.starts[j];
  const int64_t len = a.lengths[j];
  if (s < 0 || len <= 0 || s + len > a.n_valid) return;
  const int64_t cell = a.rb[s];
  if (cell < 0 || cell >= a.cells) return;
  int64_t prev = -1;
  if (j > 0) {
    const int64_t ps = a.starts[j - 1];
    if (ps >= 0 && ps < a.n_valid) prev = a.rb[ps];
    prev = max<int64_t>(-1, min<int64_t>(prev, a.cells - 1));
  }
  zero_rows<TOut, VEC>(out, prev + 1, cell, C, cbase, cvc, vi, cvc);
  if (j == a.n_intervals - 1) zero_rows<TOut, VEC>(out, cell + 1, a.cells, C, cbase, cvc, vi, cvc);

  const int64_t r0 = s / a.RG, r1 = (s + len - 1) / a.RG;
  if (r0 != r1) {
    const int64_t col = (int64_t)(cbase + vi) * VEC;
    // partials added in range order; eight loads in flight per step
    float sum[VEC];
    Vec<float, VEC>::load(a.part_b + r0 * C + col, sum);
    int64_t r = r0 + 1;
    for (; r + 8 <= r1 + 1; r += 8) {
      float t[8][VEC];
#pragma unroll
      for (int k = 0; k < 8; ++k) Vec<float, VEC>::load(a.part_a + (r + k) * C + col, t[k]);
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int e = 0; e < VEC; ++e) sum[e] += t[k][e];
    }
    for (; r <= r1; ++r) {
      float t[VEC];
      Vec<float, VEC>::load(a.part_a + r * C + col, t);
#pragma unroll
      for (int e = 0; e < VEC; ++e) sum[e] += t[e];
    }
    Vec<TOut, VEC>::store(out + cell * C + col, sum);
  }
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

// Points per range for a row of cv 16-byte vectors: the wave's G groups
// together stage kMetaPerWave points.
inline int range_points(int64_t cv) {
  const int64_t cvc = cv < kWave ? cv : kWave;
  const int64_t G = kWave / cvc;
  return (int)(kMetaPerWave / G);
}

template <typename TIn, typename TOut, int VEC>
hipError_t run(const Dims& d, const void* depth, const void* feat, FwdArgs a, void* out,
               hipStream_t stream) {
  const int CV = (int)d.C / VEC;
  TOut* o = static_cast<TOut*>(out);
  if (a.n_intervals == 0 || a.n_valid == 0) {
    const int64_t nvec = d.cells * CV;
    k_zero<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(o, nvec);
    return hipGetLastError();
  }
  a.RG = range_points(CV);
  const unsigned chunks = (unsigned)((CV + kWave - 1) / kWave);
  // The first chunk has the most lanes per group, hence the fewest groups
  // per wave (G = kMetaPerWave / RG exactly); every chunk partitions the
  // points into the same ranges of RG, and a chunk with more groups per wave
  // leaves its surplus waves idle.
  const int64_t G = kWave / (CV < kWave ? CV : kWave);
  const int64_t n_ranges = (a.n_valid + a.RG - 1) / a.RG;
  const int64_t waves = (n_ranges + G - 1) / G;
  const int64_t blocks = (waves + kFwdWaves - 1) / kFwdWaves;
  const int64_t padded = ((blocks + kXcds - 1) / kXcds) * kXcds;  // surplus blocks exit
  k_fwd_ranges<TIn, TOut, VEC>
      <<<dim3((unsigned)padded, chunks), dim3(kFwdThreads), 0, stream>>>(
          static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), o, a);
  const int64_t cwaves = (a.n_intervals + G - 1) / G;
  k_fwd_cells<TOut, VEC>
      <<<dim3((unsigned)((cwaves + kFwdWaves - 1) / kFwdWaves), chunks), dim3(kFwdThreads), 0,
         stream>>>(o, a);
  return hipGetLastError();
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

// Smallest range length any kernel variant uses for this C (the 16-byte
// fp16 path has the most groups per wave), so the workspace fits them all.
int64_t min_range_points(const Dims& d) {
  int64_t rg = range_points(d.C);            // scalar path
  rg = rg < range_points((d.C + 3) / 4) ? rg : range_points((d.C + 3) / 4);
  rg = rg < range_points((d.C + 7) / 8) ? rg : range_points((d.C + 7) / 8);
  return rg;
}

size_t forward_workspace_bytes(const Dims& d) {
  const int64_t n_ranges = (d.P + min_range_points(d) - 1) / min_range_points(d);
  return 2 * sizeof(float) * (size_t)n_ranges * (size_t)d.C;
}

hipError_t launch_forward(const Dims& d, int in_dtype, int out_dtype, const void* depth,
                          const void* feat, const int32_t* rd, const int32_t* rf,
                          const int32_t* rb, const int32_t* starts, const int32_t* lengths,
                          int32_t n_valid, int32_t n_intervals, void* out, void* workspace,
                          hipStream_t stream) {
  FwdArgs a;
  a.rd = rd;
  a.rf = rf;
  a.rb = rb;
  a.starts = starts;
  a.lengths = lengths;
  const int64_t n_ranges = (d.P + min_range_points(d) - 1) / min_range_points(d);
  a.part_a = static_cast<float*>(workspace);
  a.part_b = a.part_a + n_ranges * d.C;
  a.n_valid = n_valid;
  a.n_intervals = n_intervals;
  a.C = (int32_t)d.C;
  a.RG = 0;  // set per kernel variant
  a.cells = d.cells;
  a.P = d.P;
  a.rows = d.rows;

  const bool al = aligned16(feat) && aligned16(out) && aligned16(workspace);
  if (in_dtype == BEVPOOL_F32) {
    if (al && d.C % 4 == 0) return run<float, float, 4>(d, depth, feat, a, out, stream);
    return run<float, float, 1>(d, depth, feat, a, out, stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0) return run<half_t, half_t, 8>(d, depth, feat, a, out, stream);
    return run<half_t, half_t, 1>(d, depth, feat, a, out, stream);
  }
  if (al && d.C % 8 == 0) return run<half_t, float, 8>(d, depth, feat, a, out, stream);
  return run<half_t, float, 1>(d, depth, feat, a, out, stream);
}

}  // namespace bevpool
