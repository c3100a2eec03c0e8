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
// One thread per point p = (((b N + n) D + d) H + h) W + w, writing its
// three int32 indices; the 16 camera words of (b, n) are shared by the
// threads of a view and come from cache.

#include "internal.h"

#include <math.h>

namespace bevpool {

namespace {

constexpr int kGeoThreads = 256;

struct GeoParams {
  double stride, depth_start, depth_step;
  double lo[3], res[3];
  int64_t P;
  int32_t D, H, W;
};

__global__ __launch_bounds__(kGeoThreads) void k_geometry(const double* __restrict__ cams,
                                                          GeoParams g, int32_t* __restrict__ coor) {
#pragma clang fp contract(off)
  const int64_t p = (int64_t)blockIdx.x * kGeoThreads + threadIdx.x;
  if (p >= g.P) return;
  const int64_t hw = (int64_t)g.H * g.W;
  const int w = (int)(p % g.W);
  const int h = (int)((p / g.W) % g.H);
  const int d = (int)((p / hw) % g.D);
  const int64_t view = p / (hw * g.D);
  const double* c = cams + view * kCameraWords;
  const double u = ((double)w + 0.5) * g.stride;
  const double v = ((double)h + 0.5) * g.stride;
  const double dep = g.depth_start + (double)d * g.depth_step;
  const double xc = ((u - c[2]) * dep) / c[0];
  const double yc = ((v - c[3]) * dep) / c[1];
  const double zc = dep;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const double e = ((c[4 + 3 * i] * xc + c[5 + 3 * i] * yc) + c[6 + 3 * i] * zc) + c[13 + i];
    double idx = floor((e - g.lo[i]) / g.res[i]);
    idx = fmin(fmax(idx, -1073741824.0), 1073741824.0);  // (+-2^30; a NaN stays NaN)
    coor[p * 3 + i] = idx == idx ? (int32_t)idx : (int32_t)-1073741824;
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
  g.P = d.P;
  g.D = (int32_t)d.D;
  g.H = (int32_t)d.H;
  g.W = (int32_t)d.W;
  k_geometry<<<dim3((unsigned)((d.P + kGeoThreads - 1) / kGeoThreads)), dim3(kGeoThreads), 0,
               stream>>>(cams, g, coor);
  return hipGetLastError();
}

}  // namespace bevpool
