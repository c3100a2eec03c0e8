// Voxel index of every frustum point from camera parameters: section 2.1's
// offline step (the index "computed from the camera intrinsics and
// extrinsics"), on the device, for training where augmentation or ego
// motion changes the geometry every sample.
//
// Pinhole model, in float64: feature cell (h, w) looks through the pixel
// centre (u, v) = ((w + 0.5) s, (h + 0.5) s) for stride s; depth bin k is at
// depth_start + k depth_step along the optical axis; the camera point is
// ((u - cx) dep / fx, (v - cy) dep / fy, dep); the ego point is R cam + t
// with each coordinate summed as (R0 X + R1 Y) + R2 Z + t; the voxel index
// is floor((e - lo) / res), clipped to +-2^30.  Out-of-grid points keep
// their index; bevpool_prepare's filter drops them.  Every operation is a
// correctly rounded IEEE double operation taken in a fixed order, with no
// contraction into fused multiply-adds, so the indices are reproducible
// bit for bit on any IEEE double implementation that takes the same order.
//
// Point p = (((b N + n) D + d) H + h) W + w gets its three int32 indices
// from the thread of its pixel (h, w) in view (b, n) that takes depth bins
// d0 .. d0 + kGeoBins - 1: blocks cover a view's H W pixels (grid x), the
// runs of depth bins (y) and the views (z; larger counts are walked in
// strides).  A thread finds (h, w) with one 32-bit division (64-bit
// divisions of p cost more than the float64 arithmetic) and reuses its
// pixel's (u, v) for every bin; the 16 camera words of (b, n) are shared by
// the threads of a view and come from cache.

#include "internal.h"

#include <math.h>

#include <algorithm>

namespace bevpool {

namespace {

constexpr int kGeoThreads = 256;
constexpr int kGeoMaxGrid = 65535;  // grid y and z limit
constexpr int kGeoBins = 8;         // depth bins per thread

struct GeoParams {
  double stride, depth_start, depth_step;
  double lo[3], res[3];
  int64_t views;  // B * N
  int32_t D, H, W;
};

__global__ __launch_bounds__(kGeoThreads) void k_geometry(const double* __restrict__ cams,
                                                          GeoParams g, int32_t* __restrict__ coor) {
#pragma clang fp contract(off)
  const int32_t hw = g.H * g.W;  // (< 2^31: P is)
  const int32_t t = (int32_t)blockIdx.x * kGeoThreads + (int32_t)threadIdx.x;
  if (t >= hw) return;
  const int32_t h = t / g.W;
  const int32_t w = t - h * g.W;
  const double u = ((double)w + 0.5) * g.stride;
  const double v = ((double)h + 0.5) * g.stride;
  for (int64_t view = blockIdx.z; view < g.views; view += gridDim.z) {
    const double* c = cams + view * kCameraWords;
    for (int32_t d0 = blockIdx.y * kGeoBins; d0 < g.D; d0 += gridDim.y * kGeoBins) {
      const int32_t d_end = min(d0 + kGeoBins, g.D);
      for (int32_t d = d0; d < d_end; ++d) {
        const int64_t p = (view * g.D + d) * hw + t;
        const double dep = g.depth_start + (double)d * g.depth_step;
        const double xc = ((u - c[2]) * dep) / c[0];
        const double yc = ((v - c[3]) * dep) / c[1];
        const double zc = dep;
#pragma unroll
        for (int i = 0; i < 3; ++i) {
          const double e =
              ((c[4 + 3 * i] * xc + c[5 + 3 * i] * yc) + c[6 + 3 * i] * zc) + c[13 + i];
          double idx = floor((e - g.lo[i]) / g.res[i]);
          idx = fmin(fmax(idx, -1073741824.0), 1073741824.0);  // (+-2^30; a NaN stays NaN)
          coor[p * 3 + i] = idx == idx ? (int32_t)idx : (int32_t)-1073741824;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_geometry(const Dims& d, const bevpool_frustum& f, const double* cams,
                           int32_t* coor, hipStream_t stream) {
  if (d.P == 0) return hipSuccess;
  GeoParams g;
  g.stride = f.stride;
  g.depth_start = f.depth_start;
  g.depth_step = f.depth_step;
  for (int i = 0; i < 3; ++i) {
    g.lo[i] = f.lo[i];
    g.res[i] = f.res[i];
  }
  g.views = d.B * d.N;
  g.D = (int32_t)d.D;
  g.H = (int32_t)d.H;
  g.W = (int32_t)d.W;
  const dim3 grid((unsigned)((d.hw + kGeoThreads - 1) / kGeoThreads),
                  (unsigned)std::min<int64_t>((d.D + kGeoBins - 1) / kGeoBins, kGeoMaxGrid),
                  (unsigned)std::min<int64_t>(g.views, kGeoMaxGrid));
  k_geometry<<<grid, dim3(kGeoThreads), 0, stream>>>(cams, g, coor);
  return hipGetLastError();
}

}  // namespace bevpool
