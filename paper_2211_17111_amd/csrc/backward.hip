// Gradients of the BEVPoolv2 pooling (the paper gives none; chain rule):
//   grad_depth[p]  = <grad_out[cell(p), :], feat[pixel(p), :]>   (0 if p dropped)
//   grad_feat[f,:] = sum over kept p of pixel f of depth[p] * grad_out[cell(p), :]
//
// Two implementations, both writing every output element exactly once and
// without atomics (deterministic).
//
// From the plan alone (bevpool_backward):
//   1. k_fill + k_point_map scatter the plan back into frustum-index order,
//      map[p] = BEV rank of p, or -1 when p was dropped;
//   2. k_backward gives each feature-map pixel to a group of GS lanes (GS a
//      power of two covering the row's 16-byte vectors).  The group keeps the
//      pixel's feature row in registers, walks its D depth points, gathers the
//      upstream-gradient row of each kept point's cell, reduces the dot
//      product across the group for grad_depth and accumulates
//      depth * grad_out for grad_feat.
//
// From a schedule (bevpool_backward_scheduled), which lists every pixel's
// pairs (a cell and a run of consecutive depth bins):
//   1. k_zero_vec clears grad_depth (coalesced), so dropped points are 0 (in
//      a launch too small to fill the GPU, k_bwd_pixels writes those zeros
//      itself instead, from a mask of the depth bins its pairs cover);
//   2. k_bwd_pixels gives each pixel to a group of GS lanes holding its
//      feature row; lane l of the group takes pair l of the current chunk
//      and sums that pair's depth scores; the group then walks the chunk U
//      pairs at a time, reading one grad_out row per pair (a pair's points
//      share their cell), adding the pair's depth sum times the row to
//      grad_feat, and reducing the U dot products with the feature row across
//      the group in one butterfly reduce-scatter; each total is grad_depth of
//      every point of its pair.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

constexpr int kBwdThreads = 256;
constexpr int kBwdWaves = kBwdThreads / kWave;
constexpr int kBwdUnroll = 4;

__global__ __launch_bounds__(256) void k_fill(int32_t* __restrict__ map, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) map[i] = v;
}

__global__ __launch_bounds__(256) void k_point_map(const int32_t* __restrict__ rd,
                                                   const int32_t* __restrict__ rb, int64_t n_valid,
                                                   int32_t* __restrict__ map, int64_t P,
                                                   int64_t cells) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_valid) {
    const int32_t p = rd[i];
    const int32_t c = rb[i];
    if (p >= 0 && p < P) map[p] = (c >= 0 && c < cells) ? c : -1;
  }
}

template <typename TIn, typename TG, int VEC, int NV>
__global__ __launch_bounds__(kBwdThreads) void k_backward(
    const TG* __restrict__ grad_out, const TIn* __restrict__ depth, const TIn* __restrict__ feat,
    const int32_t* __restrict__ map, TIn* __restrict__ grad_depth, TIn* __restrict__ grad_feat,
    int32_t C, int32_t D, int64_t hw, int64_t rows, int GS) {
  const int lane = lane_id();
  const int G = kWave / GS;
  const int g = lane / GS;
  const int vi = lane - g * GS;
  const int64_t f = ((int64_t)blockIdx.x * kBwdWaves + threadIdx.x / kWave) * G + g;
  const bool pix_ok = f < rows;
  const int CV = C / VEC;

  float fv[NV][VEC];
  float acc[NV][VEC];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int v = vi + k * GS;
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[k][e] = 0.f;
    if (pix_ok && v < CV) {
      Vec<TIn, VEC>::load(feat + f * C + (int64_t)v * VEC, fv[k]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) fv[k][e] = 0.f;
    }
  }

  const int64_t bn = pix_ok ? f / hw : 0;
  const int64_t p0 = bn * D * hw + (pix_ok ? f % hw : 0);  // point at depth 0

  for (int d0 = 0; d0 < D; d0 += GS) {
    // one depth point per lane: cell and depth score, zero grad for drops
    const int dl = d0 + vi;
    int my_cell = -1;
    float my_dep = 0.f;
    if (pix_ok && dl < D) {
      const int64_t p = p0 + (int64_t)dl * hw;
      my_cell = map[p];
      if (my_cell >= 0) {
        my_dep = to_float(depth[p]);
      } else {
        grad_depth[p] = (TIn)0.f;
      }
    }
    const int nd = min(GS, D - d0);
    for (int k0 = 0; k0 < nd; k0 += kBwdUnroll) {
      int cell[kBwdUnroll];
      float dep[kBwdUnroll];
      float gv[kBwdUnroll][NV][VEC];
#pragma unroll
      for (int u = 0; u < kBwdUnroll; ++u) {
        const int src = g * GS + ((k0 + u) & (GS - 1));
        cell[u] = __shfl(my_cell, src);
        dep[u] = __shfl(my_dep, src);
        if (k0 + u >= nd) cell[u] = -1;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int v = vi + k * GS;
          if (cell[u] >= 0 && v < CV) {
            Vec<TG, VEC>::load(grad_out + (int64_t)cell[u] * C + (int64_t)v * VEC, gv[u][k]);
          } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) gv[u][k][e] = 0.f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kBwdUnroll; ++u) {
        float part = 0.f;
#pragma unroll
        for (int k = 0; k < NV; ++k)
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            part = fmaf(gv[u][k][e], fv[k][e], part);
            acc[k][e] = fmaf(dep[u], gv[u][k][e], acc[k][e]);
          }
        for (int o = GS >> 1; o > 0; o >>= 1) part += __shfl_xor(part, o);
        if (vi == 0 && cell[u] >= 0)
          grad_depth[p0 + (int64_t)(d0 + k0 + u) * hw] = (TIn)part;
      }
    }
  }

  if (pix_ok) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int v = vi + k * GS;
      if (v < CV) Vec<TIn, VEC>::store(grad_feat + f * C + (int64_t)v * VEC, acc[k]);
    }
  }
}

template <typename TIn, typename TG, int VEC, int NV>
hipError_t run(const Dims& d, const void* grad_out, const void* depth, const void* feat,
               const int32_t* map, void* grad_depth, void* grad_feat, hipStream_t stream) {
  const int CV = (int)d.C / VEC;
  const int per_lane = (CV + NV - 1) / NV;
  int GS = 1;
  while (GS < per_lane) GS <<= 1;
  const int G = kWave / GS;
  const int64_t pix_per_block = (int64_t)G * kBwdWaves;
  const dim3 grid((unsigned)((d.rows + pix_per_block - 1) / pix_per_block));
  k_backward<TIn, TG, VEC, NV><<<grid, dim3(kBwdThreads), 0, stream>>>(
      static_cast<const TG*>(grad_out), static_cast<const TIn*>(depth),
      static_cast<const TIn*>(feat), map, static_cast<TIn*>(grad_depth),
      static_cast<TIn*>(grad_feat), (int32_t)d.C, (int32_t)d.D, d.hw, d.rows, GS);
  return hipGetLastError();
}

template <typename TIn, typename TG, int VEC>
hipError_t run_nv(const Dims& d, const void* grad_out, const void* depth, const void* feat,
                  const int32_t* map, void* grad_depth, void* grad_feat, hipStream_t stream) {
  const int64_t CV = d.C / VEC;
  if (CV <= 64) return run<TIn, TG, VEC, 1>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  if (CV <= 128) return run<TIn, TG, VEC, 2>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  if (CV <= 256) return run<TIn, TG, VEC, 4>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  if (CV <= 512) return run<TIn, TG, VEC, 8>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  return run<TIn, TG, VEC, 16>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
}


template <typename T, int VEC>
__global__ __launch_bounds__(256) void k_zero_vec(T* __restrict__ a, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<T, VEC>(a + i * VEC);
}

struct PixArgs {
  const int32_t* pix_pair0;
  const int32_t* bp_cell;
  const uint32_t* bp_dn;
  int32_t C, D, hw;
  int32_t n_pairs;
  int64_t per_view, rows, cells;
  int32_t blocks;  // logical blocks (the grid is rounded up to a multiple of kXcds)
};

// Pixel order and block placement.  Blocks take consecutive pixels of an
// image row; the XCD-aware mapping gives each XCD a contiguous run of blocks,
// so that the grad_depth lines written by neighbouring pixels (adjacent in
// memory) and the grad_out rows of neighbouring rays stay in one L2.
// (Column-major pixel order was measured slower.)
constexpr bool kPixXcdMap = true;
// grad_out rows in flight per group: up to umax, within 64 registers of row
// data (always a power of two).  umax is 4 when the launch has waves enough
// to fill every SIMD several times over (kPixManyWaves per CU): then the
// extra waves that fewer registers allow hide the load latency better than
// longer steps; else 8.
constexpr int kPixManyWaves = 8;
// Depth bins the pixel kernel tracks itself (one bit each, in registers): for
// D up to this, in a launch too small to fill the GPU, each pixel's lane group
// also writes the zeros of its dropped points, so that no separate clearing
// launch is needed (in a large launch the extra registers would cost more
// waves than that launch saves).
constexpr int kPixMaskWords = 4;
constexpr int kPixMaskBits = 32 * kPixMaskWords;
constexpr int pix_unroll(int vec, int nv, int umax) {
  return vec * nv >= 64 ? 1 : (64 / (vec * nv) < umax ? 64 / (vec * nv) : umax);
}
constexpr int kDepthBurst = 2;  // depth scores of a pair loaded before any is summed

// Butterfly reduce-scatter of U per-lane partial sums over a group of GS
// lanes (both powers of two).  Lane offsets O = GS/2, GS/4, ... : while a lane
// holds M > 1 values it keeps one half (the upper half when bit O of its group
// index is set) and adds the partner's copy of that half; once it holds one
// value the remaining offsets all-reduce it.  Afterwards v[i], i < max(1, U/GS),
// is the group total of value base + i; lanes that share base differ only in
// their low bits.  U - 1 + log2(GS/U) shuffles instead of U * log2(GS).
template <int O, int M, int U>
struct ReduceScatter {
  static __device__ __forceinline__ void run(float (&v)[U], int vi, int& base) {
    if constexpr (O >= 1) {
      if constexpr (M > 1) {
        const bool up = (vi & O) != 0;
#pragma unroll
        for (int i = 0; i < M / 2; ++i) {
          const float send = up ? v[i] : v[i + M / 2];
          const float keep = up ? v[i + M / 2] : v[i];
          v[i] = keep + __shfl_xor(send, O);
        }
        if (up) base += M / 2;
        ReduceScatter<O / 2, M / 2, U>::run(v, vi, base);
      } else {
        v[0] += __shfl_xor(v[0], O);
        ReduceScatter<O / 2, 1, U>::run(v, vi, base);
      }
    }
  }
};

// The large-launch form (UMAX 4) of one-part rows is held to 5 waves per
// SIMD (96 VGPRs): float16 rows of 8 channels need 104 and would run 4 (large:
// 251 -> 230 us, at most 4 registers spilled); wider rows (NV > 1) would spill
// heavily and are left to the compiler.
template <typename TIn, typename TG, int VEC, int NV, int GS, int UMAX, int MW>
__global__ __launch_bounds__(kBwdThreads)
__attribute__((amdgpu_waves_per_eu(UMAX == 4 && NV == 1 ? 5 : 1))) void k_bwd_pixels(
    const TG* __restrict__ grad_out, const TIn* __restrict__ depth, const TIn* __restrict__ feat,
    TIn* __restrict__ grad_depth, TIn* __restrict__ grad_feat, PixArgs a) {
  constexpr int G = kWave / GS;
  constexpr int U = pix_unroll(VEC, NV, UMAX);
  constexpr int M = U > GS ? U / GS : 1;  // pair totals a lane holds after the reduction
  constexpr int LPU = GS * M / U;         // lanes holding the same pair totals
  const int lane = lane_id();
  const int g = lane / GS;
  const int vi = lane - g * GS;
  int64_t blk = blockIdx.x;
  if (kPixXcdMap) {  // hardware block b runs on XCD b % kXcds
    const int64_t per_xcd = gridDim.x / kXcds;
    blk = (blk % kXcds) * per_xcd + blk / kXcds;
    if (blk >= a.blocks) return;
  }
  const int64_t f = (blk * kBwdWaves + threadIdx.x / kWave) * G + g;
  if (f >= a.rows) return;  // whole groups leave together
  const int C = a.C;
  const int CV = C / VEC;

  float fv[NV][VEC], acc[NV][VEC];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int v = vi + k * GS;
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[k][e] = fv[k][e] = 0.f;
    if (v < CV) Vec<TIn, VEC>::load(feat + f * C + (int64_t)v * VEC, fv[k]);
  }
  const int32_t p_begin = max(a.pix_pair0[f], 0);
  const int32_t p_end = min(a.pix_pair0[f + 1], a.n_pairs);
  const int64_t dbase = (f / a.hw) * a.per_view + f % a.hw;  // depth rank at bin 0
  // (MW > 0) the depth bins this pixel's pairs cover: each lane marks its own
  // pairs' runs; the other bins are dropped points, cleared at the end
  uint32_t kept[MW > 0 ? MW : 1];
#pragma unroll
  for (int w = 0; w < (MW > 0 ? MW : 1); ++w) kept[w] = 0u;

  for (int32_t pb = p_begin; pb < p_end; pb += GS) {
    // lane vi: pair pb + vi -- its cell, depth run and summed depth score
    int32_t my_cell = -1;
    uint32_t my_dn = 0;
    float my_w = 0.f;
    if (pb + vi < p_end) {
      const int32_t c = a.bp_cell[pb + vi];
      const uint32_t dn = a.bp_dn[pb + vi];
      const int32_t d0 = (int32_t)(dn & 0xffffu), n = (int32_t)(dn >> 16);
      // (bitwise: a short-circuit test of c first would delay the load of dn)
      if ((c >= 0) & (c < a.cells) & (n >= 1) & (d0 + n <= a.D)) {
        my_cell = c;
        my_dn = dn;
#pragma unroll
        for (int w = 0; w < MW; ++w) {  // bins [d0, d0 + n) of word w
          const int lo = max(d0, 32 * w), hi = min(d0 + n, 32 * w + 32);
          const int len = hi - lo;
          if (len > 0) kept[w] |= (len >= 32 ? ~0u : ((1u << len) - 1u)) << (lo - 32 * w);
        }
        // the first kDepthBurst scores loaded together, the rest (rare) after
        float dq[kDepthBurst];
#pragma unroll
        for (int q = 0; q < kDepthBurst; ++q)  // clamped to the run: always in range
          dq[q] = to_float(depth[dbase + (int64_t)(d0 + min(q, n - 1)) * a.hw]);
#pragma unroll
        for (int q = 1; q < kDepthBurst; ++q) dq[q] = q < n ? dq[q] : 0.f;
        float wsum = dq[0];  // (no constant start: it would be folded into a load's branch)
#pragma unroll
        for (int q = 1; q < kDepthBurst; ++q) wsum += dq[q];
        for (int32_t q = kDepthBurst; q < n; ++q) wsum += to_float(depth[dbase + (int64_t)(d0 + q) * a.hw]);
        my_w = wsum;
      }
    }
    const int cnt = min(GS, p_end - pb);
    for (int j0 = 0; j0 < cnt; j0 += U) {
      int32_t cell[U];
      uint32_t dn[U];
      float w[U];
      float gv[U][NV][VEC];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int src = g * GS + ((j0 + u) & (GS - 1));
        cell[u] = __shfl(my_cell, src);
        dn[u] = (uint32_t)__shfl((int32_t)my_dn, src);
        w[u] = __shfl(my_w, src);
        if (j0 + u >= cnt) cell[u] = -1;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int v = vi + k * GS;
#pragma unroll
          for (int e = 0; e < VEC; ++e) gv[u][k][e] = 0.f;
          if (cell[u] >= 0 && v < CV)
            Vec<TG, VEC>::load(grad_out + (int64_t)cell[u] * C + (int64_t)v * VEC, gv[u][k]);
        }
      }
      float part[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float p = 0.f;
#pragma unroll
        for (int k = 0; k < NV; ++k)
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            p = fmaf(gv[u][k][e], fv[k][e], p);
            acc[k][e] = fmaf(w[u], gv[u][k][e], acc[k][e]);
          }
        part[u] = p;
      }
      int base = 0;
      ReduceScatter<GS / 2, U, U>::run(part, vi, base);
      // lane vi holds the dot products of pairs j0 + base + i; the LPU lanes
      // sharing them write the pairs' points in turn
#pragma unroll
      for (int i = 0; i < M; ++i) {
        int32_t c = -1;
        uint32_t d = 0;
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (u == base + i) c = cell[u], d = dn[u];
        if (c >= 0) {
          const int32_t d0 = (int32_t)(d & 0xffffu), n = (int32_t)(d >> 16);
          for (int32_t q = vi & (LPU - 1); q < n; q += LPU)
            grad_depth[dbase + (int64_t)(d0 + q) * a.hw] = (TIn)part[i];
        }
      }
    }
  }
  if (MW > 0) {
    // the group's covered bins (an OR over its lanes), then lane vi clears
    // the uncovered bins vi, vi + GS, ...: addresses no pair writes
#pragma unroll
    for (int w = 0; w < MW; ++w)
#pragma unroll
      for (int o = GS / 2; o > 0; o >>= 1) kept[w] |= (uint32_t)__shfl_xor((int)kept[w], o);
    for (int b = vi; b < a.D; b += GS) {
      uint32_t word = 0u;
#pragma unroll
      for (int w = 0; w < MW; ++w) word = (b >> 5) == w ? kept[w] : word;
      if (!((word >> (b & 31)) & 1u)) grad_depth[dbase + (int64_t)b * a.hw] = (TIn)0.f;
    }
  }
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int v = vi + k * GS;
    if (v < CV) Vec<TIn, VEC>::store(grad_feat + f * C + (int64_t)v * VEC, acc[k]);
  }
}

template <typename T>
hipError_t zero_fill(T* a, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(a) & 15u) == 0 && n % (16 / sizeof(T)) == 0) {
    constexpr int V = 16 / sizeof(T);
    const int64_t nvec = n / V;
    k_zero_vec<T, V><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(a, nvec);
  } else {
    k_zero_vec<T, 1><<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream>>>(a, n);
  }
  return hipGetLastError();
}

template <typename TIn, typename TG, int VEC, int NV, int GS>
hipError_t run_pixels(const Dims& d, const void* grad_out, const void* depth, const void* feat,
                      const PixArgs& a, void* grad_depth, void* grad_feat, hipStream_t stream) {
  constexpr int G = kWave / GS;
  const int64_t pix_per_block = (int64_t)G * kBwdWaves;
  PixArgs b = a;
  b.blocks = (int32_t)((d.rows + pix_per_block - 1) / pix_per_block);
  const int64_t nb = kPixXcdMap ? (b.blocks + kXcds - 1) / kXcds * kXcds : b.blocks;
  const bool many = (d.rows + G - 1) / G >= (int64_t)kPixManyWaves * device_cus();
  auto launch = [&](auto kern) {
    kern<<<dim3((unsigned)nb), dim3(kBwdThreads), 0, stream>>>(
        static_cast<const TG*>(grad_out), static_cast<const TIn*>(depth),
        static_cast<const TIn*>(feat), static_cast<TIn*>(grad_depth), static_cast<TIn*>(grad_feat), b);
  };
  // dropped points: zeros written by the pixel kernel (small launch, D within
  // its bin mask), else by a clearing launch before it
  const bool mask = !many && d.D <= kPixMaskBits;
  if (!mask) {
    const hipError_t e = zero_fill(static_cast<TIn*>(grad_depth), d.P, stream);
    if (e != hipSuccess) return e;
  }
  if (many)
    launch(k_bwd_pixels<TIn, TG, VEC, NV, GS, 4, 0>);
  else if (mask)
    launch(k_bwd_pixels<TIn, TG, VEC, NV, GS, 8, kPixMaskWords>);
  else
    launch(k_bwd_pixels<TIn, TG, VEC, NV, GS, 8, 0>);
  return hipGetLastError();
}

// A group of GS lanes (the smallest power of two with GS * NV >= C / VEC)
// holds a pixel's row; C <= 1024 keeps GS <= 64 for NV = 16.
template <typename TIn, typename TG, int VEC>
hipError_t run_pixels_nv(const Dims& d, const void* grad_out, const void* depth, const void* feat,
                         const PixArgs& a, void* grad_depth, void* grad_feat, hipStream_t stream) {
  const int64_t CV = d.C / VEC;
#define BWD_RUN(NV, GS) \
  return run_pixels<TIn, TG, VEC, NV, GS>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream)
  if (CV <= 1) BWD_RUN(1, 1);
  if (CV <= 2) BWD_RUN(1, 2);
  if (CV <= 4) BWD_RUN(1, 4);
  if (CV <= 8) BWD_RUN(1, 8);
  if (CV <= 16) BWD_RUN(1, 16);
  if (CV <= 32) BWD_RUN(1, 32);
  if (CV <= 64) BWD_RUN(1, 64);
  if (CV <= 128) BWD_RUN(2, 64);
  if (CV <= 256) BWD_RUN(4, 64);
  if (CV <= 512) BWD_RUN(8, 64);
  BWD_RUN(16, 64);
#undef BWD_RUN
}


inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

size_t backward_workspace_bytes(const Dims& d) { return sizeof(int32_t) * (size_t)d.P; }

hipError_t launch_backward(const Dims& d, int in_dtype, int out_dtype, const void* grad_out,
                           const void* depth, const void* feat, const int32_t* rd,
                           const int32_t* rb, int32_t n_valid, void* grad_depth,
                           void* grad_feat, void* workspace, hipStream_t stream) {
  int32_t* map = static_cast<int32_t*>(workspace);
  k_fill<<<dim3((unsigned)((d.P + 255) / 256)), dim3(256), 0, stream>>>(map, d.P, -1);
  if (n_valid > 0)
    k_point_map<<<dim3((unsigned)((n_valid + 255) / 256)), dim3(256), 0, stream>>>(
        rd, rb, n_valid, map, d.P, d.cells);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  const bool al = aligned16(grad_out) && aligned16(feat) && aligned16(grad_feat);
  if (in_dtype == BEVPOOL_F32) {
    if (al && d.C % 4 == 0)
      return run_nv<float, float, 4>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
    return run_nv<float, float, 1>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0)
      return run_nv<half_t, half_t, 8>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
    return run_nv<half_t, half_t, 1>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  }
  if (al && d.C % 8 == 0)
    return run_nv<half_t, float, 8>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
  return run_nv<half_t, float, 1>(d, grad_out, depth, feat, map, grad_depth, grad_feat, stream);
}


hipError_t launch_backward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                     const void* grad_out, const void* depth, const void* feat,
                                     const void* schedule, int32_t n_valid, int32_t n_intervals,
                                     void* grad_depth, void* grad_feat, hipStream_t stream) {
  const bool f32 = in_dtype == BEVPOOL_F32;
  if (n_valid == 0 || n_intervals == 0) {  // no kept point: both gradients are zero
    hipError_t e = f32 ? zero_fill(static_cast<float*>(grad_depth), d.P, stream)
                       : zero_fill(static_cast<half_t*>(grad_depth), d.P, stream);
    if (e != hipSuccess) return e;
    return f32 ? zero_fill(static_cast<float*>(grad_feat), d.rows * d.C, stream)
               : zero_fill(static_cast<half_t*>(grad_feat), d.rows * d.C, stream);
  }
  // (grad_depth's dropped points are cleared by run_pixels)
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  const char* sc = static_cast<const char*>(schedule);
  PixArgs a;
  a.pix_pair0 = reinterpret_cast<const int32_t*>(sc + L.pix_pair0);
  a.bp_cell = reinterpret_cast<const int32_t*>(sc + L.bp_cell);
  a.bp_dn = reinterpret_cast<const uint32_t*>(sc + L.bp_dn);
  a.C = (int32_t)d.C;
  a.D = (int32_t)d.D;
  a.hw = (int32_t)d.hw;
  a.blocks = 0;
  a.n_pairs = n_valid;  // pairs never outnumber kept points
  a.per_view = d.per_view;
  a.rows = d.rows;
  a.cells = d.cells;
  const bool al = aligned16(grad_out) && aligned16(feat) && aligned16(grad_feat);
  if (f32) {
    // 8 channels per lane where C allows: smaller lane groups, so more pixels
    // (and their independent load chains) per wave
    if (al && d.C % 8 == 0)
      return run_pixels_nv<float, float, 8>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
    if (al && d.C % 4 == 0)
      return run_pixels_nv<float, float, 4>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
    return run_pixels_nv<float, float, 1>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0)
      return run_pixels_nv<half_t, half_t, 8>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
    return run_pixels_nv<half_t, half_t, 1>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
  }
  if (al && d.C % 8 == 0)
    return run_pixels_nv<half_t, float, 8>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
  return run_pixels_nv<half_t, float, 1>(d, grad_out, depth, feat, a, grad_depth, grad_feat, stream);
}

}  // namespace bevpool
