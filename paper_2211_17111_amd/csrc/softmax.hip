// Per-pixel log-sum-exp of depth logits, the pre-pass of the fused
// depth-softmax forward.  Section 2.1 treats the depth score of a pixel as a
// distribution over its D depth bins; when a network gives the logits, the
// score of bin d is exp(logit_d - lse) with lse = log sum_d exp(logit_d).
// This kernel writes lse (float64, one per pixel of (B, N, H, W)); the
// scheduled forward then forms each kept point's score on the fly, so the
// (B, N, D, H, W) score tensor is never written or read.
//
// The logits of a pixel are D values H*W apart; lanes take neighbouring
// pixels, so every step of the loops over d reads consecutive addresses
// across a wave.  lse = m + log(sum
// exp(logit - m)) with m the pixel's largest logit (no overflow; the largest
// term is exp(0) = 1).  The terms come from the device library's expf
// (float32, about 1 ulp) and are summed and logged in double, so lse is
// good to about 2^-23 absolute whatever D is (a float32 sum of D terms could
// lose up to D ulps), and it is kept in double: a float32 lse would carry
// |lse| * 2^-24 of rounding into every score, too much for logits in the
// tens.  The forward forms the exponent logit - lse in double and rounds
// only it to float32, so a score's relative error is about (|logit - lse|
// + 4) * 2^-24: a few 1e-6 for the scores that carry weight.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

// A block takes 64 pixels; its eight waves split each pixel's depth bins
// into eight ranges (lane = pixel, so every load of a wave reads 64
// consecutive logits) and combine their partial maxima and sums in LDS, in
// wave order.  When a range fits kLseRegs bins it is loaded once, into
// registers, for both the maximum and the sum.
constexpr int kLseWaves = 8;
constexpr int kLseThreads = kLseWaves * kWave;
constexpr int kLseBatch = 8;  // logits in flight per thread (two-pass form)
constexpr int kLseRegs = 16;  // a wave share of at most this many bins stays in registers

template <typename TIn>
__global__ __launch_bounds__(kLseThreads) void k_depth_lse(const TIn* __restrict__ logits,
                                                           double* __restrict__ lse, int64_t rows,
                                                           int32_t D, int64_t hw) {
  __shared__ float s_max[kLseWaves][kWave];
  __shared__ double s_sum[kLseWaves][kWave];
  const int lane = threadIdx.x % kWave;
  const int wv = threadIdx.x / kWave;
  const int64_t px = (int64_t)blockIdx.x * kWave + lane;
  const bool on = px < rows;
  const int64_t pxc = on ? px : rows - 1;  // (lanes past the end repeat the last pixel)
  const int64_t view = pxc / hw;
  const TIn* p = logits + view * (int64_t)D * hw + (pxc - view * hw);
  const int d0 = (int)((int64_t)D * wv / kLseWaves), d1 = (int)((int64_t)D * (wv + 1) / kLseWaves);
  float m = -INFINITY;
  double s = 0.0;
  if ((D + kLseWaves - 1) / kLseWaves <= kLseRegs) {  // (the same for every wave: both forms hold a barrier)
    // the wave's share, loaded once: its largest logit, then (with the
    // pixel's largest) the sum of exp(logit - m) in double
    float v[kLseRegs];
#pragma unroll
    for (int u = 0; u < kLseRegs; ++u) v[u] = d0 + u < d1 ? to_float(p[(int64_t)(d0 + u) * hw]) : -INFINITY;
#pragma unroll
    for (int u = 0; u < kLseRegs; ++u) m = fmaxf(m, v[u]);
    s_max[wv][lane] = m;
    __syncthreads();
    m = s_max[0][lane];
#pragma unroll
    for (int w = 1; w < kLseWaves; ++w) m = fmaxf(m, s_max[w][lane]);
#pragma unroll
    for (int u = 0; u < kLseRegs; ++u)
      if (d0 + u < d1) s += (double)expf(v[u] - m);
  } else {
    // this wave's share of the largest logit
    int d = d0;
    for (; d + kLseBatch <= d1; d += kLseBatch) {
      float v[kLseBatch];
#pragma unroll
      for (int u = 0; u < kLseBatch; ++u) v[u] = to_float(p[(int64_t)(d + u) * hw]);
#pragma unroll
      for (int u = 0; u < kLseBatch; ++u) m = fmaxf(m, v[u]);
    }
    for (; d < d1; ++d) m = fmaxf(m, to_float(p[(int64_t)d * hw]));
    s_max[wv][lane] = m;
    __syncthreads();
    m = s_max[0][lane];
#pragma unroll
    for (int w = 1; w < kLseWaves; ++w) m = fmaxf(m, s_max[w][lane]);
    // this wave's share of the sum of exp(logit - m), in double
    d = d0;
    for (; d + kLseBatch <= d1; d += kLseBatch) {
      float v[kLseBatch];
#pragma unroll
      for (int u = 0; u < kLseBatch; ++u) v[u] = to_float(p[(int64_t)(d + u) * hw]);
#pragma unroll
      for (int u = 0; u < kLseBatch; ++u) s += (double)expf(v[u] - m);
    }
    for (; d < d1; ++d) s += (double)expf(to_float(p[(int64_t)d * hw]) - m);
  }
  s_sum[wv][lane] = s;
  __syncthreads();
  if (wv == 0 && on) {
    double t = s_sum[0][lane];
#pragma unroll
    for (int w = 1; w < kLseWaves; ++w) t += s_sum[w][lane];
    lse[px] = (double)m + log(t);
  }
}

}  // namespace

hipError_t launch_depth_lse(const Dims& d, int in_dtype, const void* logits, double* lse,
                            hipStream_t stream) {
  if (d.rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((d.rows + kWave - 1) / kWave)), block(kLseThreads);
  if (in_dtype == BEVPOOL_F16)
    k_depth_lse<half_t><<<grid, block, 0, stream>>>(static_cast<const half_t*>(logits), lse, d.rows,
                                                    (int32_t)d.D, d.hw);
  else
    k_depth_lse<float><<<grid, block, 0, stream>>>(static_cast<const float*>(logits), lse, d.rows,
                                                   (int32_t)d.D, d.hw);
  return hipGetLastError();
}

}  // namespace bevpool
