// BEVPoolv2 pooling (section 2.1, paragraph 2): every occupied BEV cell sums
// depth[rank_depth] * feat[rank_feat, :] over the points of its interval,
// reading both operands through the frustum-index trace, so the frustum
// feature is never formed.
//
// Mapping on CDNA: one 64-lane wavefront per interval (per channel chunk of
// up to 64 vectors).  Lanes are split into G groups of CV lanes, CV = number
// of 16-byte vectors in a feature row; each group takes every G-th point, so
// a wave keeps G feature rows in flight per step with fully coalesced row
// loads.  The interval's ranks are loaded cooperatively, one point per lane,
// and the depth scalar and feature rank of each point are broadcast to its
// group with a cross-lane shuffle.  Partial sums are blocked per 64 points
// and the G group sums are combined with a shuffle tree, then each cell is
// stored exactly once.  The wave also zero-fills the empty cells between the
// previous interval's cell and its own (and after the last), so the output
// is written in full with no atomics and no separate memset.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

constexpr int kFwdThreads = 256;
constexpr int kFwdWaves = kFwdThreads / kWave;
constexpr int kUnroll = 4;

template <typename TOut, int VEC>
__device__ __forceinline__ void zero_rows(TOut* __restrict__ out, int64_t r0, int64_t r1, int C,
                                          int cbase, int cvc, int lane) {
  if (r1 <= r0) return;
  const int64_t total = (r1 - r0) * cvc;
  for (int64_t idx = lane; idx < total; idx += kWave) {
    const int64_t r = r0 + idx / cvc;
    const int v = (int)(idx % cvc);
    store_zero<TOut, VEC>(out + r * C + (int64_t)(cbase + v) * VEC);
  }
}

template <typename TIn, typename TOut, int VEC>
__global__ __launch_bounds__(kFwdThreads) void k_forward(
    const TIn* __restrict__ depth, const TIn* __restrict__ feat, const int32_t* __restrict__ rd,
    const int32_t* __restrict__ rf, const int32_t* __restrict__ rb,
    const int32_t* __restrict__ starts, const int32_t* __restrict__ lengths, int32_t n_valid,
    int32_t n_intervals, TOut* __restrict__ out, int32_t C, int64_t cells, int64_t P,
    int64_t rows) {
  const int lane = lane_id();
  const int64_t j = (int64_t)blockIdx.x * kFwdWaves + threadIdx.x / kWave;
  if (j >= n_intervals) return;

  const int CV = C / VEC;
  const int cbase = blockIdx.y * kWave;
  const int cvc = min(kWave, CV - cbase);
  const int G = kWave / cvc;
  const int g = lane / cvc;
  const int vi = lane - g * cvc;
  const bool lane_active = g < G;

  const int64_t start = starts[j];
  const int64_t len = lengths[j];
  const int64_t cell = (start >= 0 && start < n_valid && len > 0) ? (int64_t)rb[start] : -1;
  const bool ok = cell >= 0 && cell < cells;

  // zero-fill the empty cells this interval is responsible for
  int64_t prev = -1;
  if (j > 0) {
    const int64_t ps = starts[j - 1];
    if (ps >= 0 && ps < n_valid) prev = rb[ps];
    prev = max<int64_t>(-1, min<int64_t>(prev, cells - 1));
  }
  if (ok) {
    if (prev < cell) zero_rows<TOut, VEC>(out, prev + 1, cell, C, cbase, cvc, lane);
    if (j == n_intervals - 1) zero_rows<TOut, VEC>(out, cell + 1, cells, C, cbase, cvc, lane);
  } else {
    return;
  }

  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.f;

  const int64_t end = min<int64_t>(start + len, n_valid);
  const TIn* fbase = feat + (int64_t)(cbase + vi) * VEC;
  for (int64_t base = start; base < end; base += kWave) {
    const int cnt = (int)min<int64_t>(kWave, end - base);
    int my_f = 0;
    float my_d = 0.f;
    if (lane < cnt) {
      const int32_t a = rd[base + lane];
      const int32_t f = rf[base + lane];
      if (a >= 0 && a < P && f >= 0 && f < rows) {
        my_d = to_float(depth[a]);
        my_f = f;
      }
    }
    float blk[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) blk[e] = 0.f;
    for (int q0 = 0; q0 < cnt; q0 += G * kUnroll) {
      float dq[kUnroll];
      float v[kUnroll][VEC];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int q = q0 + u * G + g;
        dq[u] = __shfl(my_d, q & (kWave - 1));
        const int fq = __shfl(my_f, q & (kWave - 1));
        if (lane_active && q < cnt) {
          Vec<TIn, VEC>::load(fbase + (int64_t)fq * C, v[u]);
        } else {
          dq[u] = 0.f;
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[u][e] = 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
#pragma unroll
        for (int e = 0; e < VEC; ++e) blk[e] = fmaf(dq[u], v[u][e], blk[e]);
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] += blk[e];
  }

  // combine the G group sums into group 0 with a shuffle tree
  for (int off = 1; off < G; off <<= 1) {
    float t[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) t[e] = __shfl_down(acc[e], off * cvc);
    if ((g % (2 * off)) == 0 && g + off < G) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += t[e];
    }
  }
  if (g == 0) Vec<TOut, VEC>::store(out + cell * C + (int64_t)(cbase + vi) * VEC, acc);
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

template <typename TIn, typename TOut, int VEC>
hipError_t run(const Dims& d, const void* depth, const void* feat, const int32_t* rd,
               const int32_t* rf, const int32_t* rb, const int32_t* starts,
               const int32_t* lengths, int32_t n_valid, int32_t n_intervals, void* out,
               hipStream_t stream) {
  const int CV = (int)d.C / VEC;
  TOut* o = static_cast<TOut*>(out);
  if (n_intervals == 0) {
    const int64_t nvec = d.cells * CV;
    k_zero<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(o, nvec);
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((n_intervals + kFwdWaves - 1) / kFwdWaves),
                  (unsigned)((CV + kWave - 1) / kWave));
  k_forward<TIn, TOut, VEC><<<grid, dim3(kFwdThreads), 0, stream>>>(
      static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), rd, rf, rb, starts, lengths,
      n_valid, n_intervals, o, (int32_t)d.C, d.cells, d.P, d.rows);
  return hipGetLastError();
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

hipError_t launch_forward(const Dims& d, int in_dtype, int out_dtype, const void* depth,
                          const void* feat, const int32_t* rd, const int32_t* rf,
                          const int32_t* rb, const int32_t* starts, const int32_t* lengths,
                          int32_t n_valid, int32_t n_intervals, void* out, hipStream_t stream) {
  const bool al = aligned16(feat) && aligned16(out);
  if (in_dtype == BEVPOOL_F32) {
    if (al && d.C % 4 == 0)
      return run<float, float, 4>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals, out,
                                  stream);
    return run<float, float, 1>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals, out,
                                stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0)
      return run<half_t, half_t, 8>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals,
                                    out, stream);
    return run<half_t, half_t, 1>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals, out,
                                  stream);
  }
  if (al && d.C % 8 == 0)
    return run<half_t, float, 8>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals, out,
                                 stream);
  return run<half_t, float, 1>(d, depth, feat, rd, rf, rb, starts, lengths, n_valid, n_intervals, out,
                               stream);
}

}  // namespace bevpool
