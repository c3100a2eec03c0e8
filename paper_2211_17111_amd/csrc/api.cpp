// C ABI of the BEVPoolv2 path: argument validation, workspace sizing and
// dispatch to the HIP launchers.  Validation runs before any HIP API call, so
// every error path can be exercised on a machine without a GPU.

#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "bevpool.h"
#include "internal.h"

namespace bevpool {

Dims dims_of(const bevpool_shape& s) {
  Dims d;
  d.B = s.B; d.N = s.N; d.D = s.D; d.H = s.H; d.W = s.W; d.C = s.C;
  d.X = s.X; d.Y = s.Y; d.Z = s.Z;
  d.hw = d.H * d.W;
  d.per_view = d.D * d.hw;
  d.P = d.B * d.N * d.per_view;
  d.rows = d.B * d.N * d.hw;
  d.cells = d.B * d.Z * d.Y * d.X;
  return d;
}

}  // namespace bevpool

namespace {

thread_local std::string g_last_error;

constexpr int64_t kIndexLimit = int64_t(1) << 31;
constexpr int64_t kMaxC = 1024;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return BEVPOOL_OK;
}

int check_shape(const bevpool_shape* s, bevpool::Dims* out) {
  if (s == nullptr) return fail(BEVPOOL_EINVAL, "shape is NULL");
  const int32_t v[9] = {s->B, s->N, s->D, s->H, s->W, s->C, s->X, s->Y, s->Z};
  const char* names = "BNDHWCXYZ";
  for (int i = 0; i < 9; ++i)
    if (v[i] <= 0) return fail(BEVPOOL_EINVAL, "shape.%c = %d must be >= 1", names[i], v[i]);
  const bevpool::Dims d = bevpool::dims_of(*s);
  if (d.P >= kIndexLimit)
    return fail(BEVPOOL_EOVERFLOW, "B*N*D*H*W = %lld frustum points exceeds 2^31-1",
                (long long)d.P);
  if (d.cells * d.C >= kIndexLimit)
    return fail(BEVPOOL_EOVERFLOW, "B*Z*Y*X*C = %lld exceeds 2^31-1", (long long)(d.cells * d.C));
  if (d.rows * d.C >= kIndexLimit)
    return fail(BEVPOOL_EOVERFLOW, "B*N*H*W*C = %lld exceeds 2^31-1", (long long)(d.rows * d.C));
  if (d.C > kMaxC) return fail(BEVPOOL_EOVERFLOW, "C = %lld exceeds 1024", (long long)d.C);
  *out = d;
  return BEVPOOL_OK;
}

int check_dtypes(int in_dtype, int out_dtype) {
  const bool in_ok = in_dtype == BEVPOOL_F32 || in_dtype == BEVPOOL_F16;
  const bool out_ok = out_dtype == BEVPOOL_F32 || out_dtype == BEVPOOL_F16;
  if (!in_ok || !out_ok)
    return fail(BEVPOOL_EDTYPE, "unknown dtype (in %d, out %d)", in_dtype, out_dtype);
  if (in_dtype == BEVPOOL_F32 && out_dtype == BEVPOOL_F16)
    return fail(BEVPOOL_EDTYPE, "float32 inputs with a float16 output are not supported");
  return BEVPOOL_OK;
}

#define REQUIRE_PTR(p)                                          \
  do {                                                          \
    if ((p) == nullptr) return fail(BEVPOOL_EINVAL, #p " is NULL"); \
  } while (0)

int from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(BEVPOOL_ELAUNCH, "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
}

int check_counts(const bevpool::Dims& d, int32_t n_valid, int32_t n_intervals) {
  if (n_valid < 0 || n_valid > d.P)
    return fail(BEVPOOL_EINVAL, "n_valid = %d outside [0, %lld]", n_valid, (long long)d.P);
  const int64_t cap = d.P < d.cells ? d.P : d.cells;
  if (n_intervals < 0 || n_intervals > cap || n_intervals > n_valid ||
      (n_valid > 0 && n_intervals == 0))
    return fail(BEVPOOL_EINVAL, "n_intervals = %d inconsistent with n_valid = %d (cells %lld)",
                n_intervals, n_valid, (long long)d.cells);
  return BEVPOOL_OK;
}

// Checks shared by the two scheduled forwards (everything but the workspace).
int check_forward_scheduled(const bevpool_shape* shape, int in_dtype, int out_dtype,
                            const void* depth, const void* feat, const void* schedule,
                            size_t schedule_bytes, int32_t n_valid, int32_t n_intervals,
                            int32_t n_slots, void* out, bevpool::Dims* d) {
  int st = check_shape(shape, d);
  if (st != BEVPOOL_OK) return st;
  st = check_dtypes(in_dtype, out_dtype);
  if (st != BEVPOOL_OK) return st;
  st = check_counts(*d, n_valid, n_intervals);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(out);
  if (n_intervals > 0) {
    REQUIRE_PTR(depth);
    REQUIRE_PTR(feat);
    REQUIRE_PTR(schedule);
    const size_t need = bevpool::schedule_layout(*d, n_valid, n_intervals).total;
    if (schedule_bytes < need)
      return fail(BEVPOOL_EINVAL, "schedule of %zu bytes is smaller than the %zu this plan needs",
                  schedule_bytes, need);
    // (each slot holds part of a cell's pairs, so there are at most n_valid)
    if (n_slots < 0 || n_slots > n_valid)
      return fail(BEVPOOL_EINVAL, "n_slots = %d outside [0, n_valid = %d]", n_slots, n_valid);
  }
  return BEVPOOL_OK;
}

}  // namespace

extern "C" {

int bevpool_version(void) { return BEVPOOL_VERSION; }

const char* bevpool_strerror(int status) {
  switch (status) {
    case BEVPOOL_OK: return "success";
    case BEVPOOL_EINVAL: return "invalid argument";
    case BEVPOOL_EOVERFLOW: return "size exceeds the supported index range";
    case BEVPOOL_EDTYPE: return "unsupported dtype";
    case BEVPOOL_EWORKSPACE: return "workspace missing or too small";
    case BEVPOOL_ELAUNCH: return "HIP launch failed";
    default: return "unknown status";
  }
}

const char* bevpool_last_error(void) { return g_last_error.c_str(); }

int bevpool_prepare_workspace_size(const bevpool_shape* shape, size_t* bytes) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(bytes);
  *bytes = bevpool::prepare_layout(d).total;
  return ok();
}

int bevpool_prepare(const bevpool_shape* shape, const int32_t* coor, int32_t* ranks_depth,
                    int32_t* ranks_feat, int32_t* ranks_bev, int32_t* interval_starts,
                    int32_t* interval_lengths, int32_t* counts, void* workspace,
                    size_t workspace_bytes, void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(coor);
  REQUIRE_PTR(ranks_depth);
  REQUIRE_PTR(ranks_feat);
  REQUIRE_PTR(ranks_bev);
  REQUIRE_PTR(interval_starts);
  REQUIRE_PTR(interval_lengths);
  REQUIRE_PTR(counts);
  const size_t need = bevpool::prepare_layout(d).total;
  if (workspace == nullptr || workspace_bytes < need)
    return fail(BEVPOOL_EWORKSPACE, "prepare needs %zu workspace bytes, got %zu at %p", need,
                workspace_bytes, workspace);
  return from_hip(bevpool::launch_prepare(d, coor, ranks_depth, ranks_feat, ranks_bev,
                                          interval_starts, interval_lengths, counts, workspace,
                                          static_cast<hipStream_t>(stream)),
                  "bevpool_prepare");
}

int bevpool_forward_workspace_size(const bevpool_shape* shape, size_t* bytes) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(bytes);
  *bytes = bevpool::forward_workspace_bytes(d);
  return ok();
}

int bevpool_forward(const bevpool_shape* shape, int in_dtype, int out_dtype, const void* depth,
                    const void* feat, const int32_t* ranks_depth, const int32_t* ranks_feat,
                    const int32_t* ranks_bev, const int32_t* interval_starts,
                    const int32_t* interval_lengths, int32_t n_valid, int32_t n_intervals,
                    void* out, void* workspace, size_t workspace_bytes, void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_dtypes(in_dtype, out_dtype);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(out);
  if (n_valid < 0 || n_valid > d.P)
    return fail(BEVPOOL_EINVAL, "n_valid = %d outside [0, %lld]", n_valid, (long long)d.P);
  const int64_t cap = d.P < d.cells ? d.P : d.cells;
  if (n_intervals < 0 || n_intervals > cap || n_intervals > n_valid)
    return fail(BEVPOOL_EINVAL, "n_intervals = %d outside [0, min(%lld, n_valid = %d)]",
                n_intervals, (long long)cap, n_valid);
  if (n_intervals > 0) {
    REQUIRE_PTR(depth);
    REQUIRE_PTR(feat);
    REQUIRE_PTR(ranks_depth);
    REQUIRE_PTR(ranks_feat);
    REQUIRE_PTR(ranks_bev);
    REQUIRE_PTR(interval_starts);
    REQUIRE_PTR(interval_lengths);
  }
  const size_t need = bevpool::forward_workspace_bytes(d);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(BEVPOOL_EWORKSPACE, "forward needs %zu workspace bytes, got %zu at %p", need,
                workspace_bytes, workspace);
  return from_hip(bevpool::launch_forward(d, in_dtype, out_dtype, depth, feat, ranks_depth,
                                          ranks_feat, ranks_bev, interval_starts,
                                          interval_lengths, n_valid, n_intervals, out, workspace,
                                          static_cast<hipStream_t>(stream)),
                  "bevpool_forward");
}

int bevpool_schedule_size(const bevpool_shape* shape, int32_t n_valid, int32_t n_intervals,
                          size_t* schedule_bytes, size_t* workspace_bytes) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_counts(d, n_valid, n_intervals);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(schedule_bytes);
  REQUIRE_PTR(workspace_bytes);
  const bevpool::ScheduleLayout L = bevpool::schedule_layout(d, n_valid, n_intervals);
  *schedule_bytes = L.total;
  *workspace_bytes = L.ws_total;
  return ok();
}

int bevpool_schedule(const bevpool_shape* shape, const int32_t* ranks_depth,
                     const int32_t* ranks_bev, int32_t n_valid, int32_t n_intervals,
                     void* schedule, size_t schedule_bytes, void* workspace,
                     size_t workspace_bytes, void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_counts(d, n_valid, n_intervals);
  if (st != BEVPOOL_OK) return st;
  if (n_valid > 0) {
    REQUIRE_PTR(ranks_depth);
    REQUIRE_PTR(ranks_bev);
  }
  REQUIRE_PTR(schedule);
  if (d.D > 65535)
    return fail(BEVPOOL_EINVAL, "the schedule stores depth bins in 16 bits: D = %lld > 65535",
                (long long)d.D);
  const bevpool::ScheduleLayout L = bevpool::schedule_layout(d, n_valid, n_intervals);
  if (schedule_bytes < L.total)
    return fail(BEVPOOL_EINVAL, "schedule needs %zu bytes, got %zu", L.total, schedule_bytes);
  if (workspace == nullptr || workspace_bytes < L.ws_total)
    return fail(BEVPOOL_EWORKSPACE, "schedule build needs %zu workspace bytes, got %zu at %p",
                L.ws_total, workspace_bytes, workspace);
  return from_hip(bevpool::launch_schedule(d, ranks_depth, ranks_bev, n_valid, n_intervals,
                                           schedule, workspace, static_cast<hipStream_t>(stream)),
                  "bevpool_schedule");
}

int bevpool_forward_scheduled_workspace_size(const bevpool_shape* shape, int32_t n_slots,
                                              size_t* bytes) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(bytes);
  if (n_slots < 0) return fail(BEVPOOL_EINVAL, "n_slots = %d is negative", n_slots);
  *bytes = bevpool::forward_scheduled_workspace_bytes(d, n_slots);
  return ok();
}

int bevpool_forward_scheduled(const bevpool_shape* shape, int in_dtype, int out_dtype,
                              const void* depth, const void* feat, const void* schedule,
                              size_t schedule_bytes, int32_t n_valid, int32_t n_intervals,
                              int32_t n_slots, void* out, void* workspace, size_t workspace_bytes,
                              void* stream) {
  bevpool::Dims d;
  int st = check_forward_scheduled(shape, in_dtype, out_dtype, depth, feat, schedule,
                                   schedule_bytes, n_valid, n_intervals, n_slots, out, &d);
  if (st != BEVPOOL_OK) return st;
  if (n_intervals > 0) {
    const size_t ws_need = bevpool::forward_scheduled_workspace_bytes(d, n_slots);
    if (ws_need > 0 && (workspace == nullptr || workspace_bytes < ws_need))
      return fail(BEVPOOL_EWORKSPACE, "%d slots need %zu workspace bytes, got %zu at %p", n_slots,
                  ws_need, workspace_bytes, workspace);
  }
  return from_hip(bevpool::launch_forward_scheduled(d, in_dtype, out_dtype, depth, feat, schedule,
                                                    n_valid, n_intervals, n_slots, out, workspace,
                                                    workspace_bytes,
                                                    static_cast<hipStream_t>(stream)),
                  "bevpool_forward_scheduled");
}

int bevpool_geometry(const bevpool_shape* shape, const bevpool_frustum* frustum,
                     const double* cams, int32_t* coor, void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(frustum);
  REQUIRE_PTR(cams);
  REQUIRE_PTR(coor);
  const bevpool_frustum& f = *frustum;
  bool ok = std::isfinite(f.stride) && f.stride > 0 && std::isfinite(f.depth_start) &&
            std::isfinite(f.depth_step) && f.depth_step > 0;
  for (int i = 0; i < 3; ++i) ok = ok && std::isfinite(f.lo[i]) && std::isfinite(f.res[i]) && f.res[i] > 0;
  if (!ok)
    return fail(BEVPOOL_EINVAL, "frustum: stride, depth step and cell sizes must be finite and "
                                "positive, depth start and bounds finite");
  return from_hip(bevpool::launch_geometry(d, f, cams, coor, static_cast<hipStream_t>(stream)),
                  "bevpool_geometry");
}

int bevpool_depth_lse(const bevpool_shape* shape, int in_dtype, const void* logits, double* lse,
                      void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_dtypes(in_dtype, BEVPOOL_F32);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(logits);
  REQUIRE_PTR(lse);
  return from_hip(bevpool::launch_depth_lse(d, in_dtype, logits, lse,
                                            static_cast<hipStream_t>(stream)),
                  "bevpool_depth_lse");
}

int bevpool_forward_scheduled_softmax(const bevpool_shape* shape, int in_dtype, int out_dtype,
                                      const void* logits, const double* lse, const void* feat,
                                      const void* schedule, size_t schedule_bytes,
                                      int32_t n_valid, int32_t n_intervals, int32_t n_slots,
                                      void* out, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  bevpool::Dims d;
  int st = check_forward_scheduled(shape, in_dtype, out_dtype, logits, feat, schedule,
                                   schedule_bytes, n_valid, n_intervals, n_slots, out, &d);
  if (st != BEVPOOL_OK) return st;
  if (n_intervals > 0) {
    REQUIRE_PTR(lse);
    const size_t ws_need = bevpool::forward_scheduled_workspace_bytes(d, n_slots);
    if (ws_need > 0 && (workspace == nullptr || workspace_bytes < ws_need))
      return fail(BEVPOOL_EWORKSPACE, "%d slots need %zu workspace bytes, got %zu at %p", n_slots,
                  ws_need, workspace_bytes, workspace);
  }
  return from_hip(bevpool::launch_forward_scheduled(d, in_dtype, out_dtype, logits, feat, schedule,
                                                    n_valid, n_intervals, n_slots, out, workspace,
                                                    workspace_bytes,
                                                    static_cast<hipStream_t>(stream), lse),
                  "bevpool_forward_scheduled_softmax");
}

int bevpool_forward_scheduled_noalloc(const bevpool_shape* shape, int in_dtype, int out_dtype,
                                      const void* depth, const void* feat, const void* schedule,
                                      size_t schedule_bytes, int32_t n_valid, int32_t n_intervals,
                                      int32_t n_slots, void* out, void* stream) {
  bevpool::Dims d;
  int st = check_forward_scheduled(shape, in_dtype, out_dtype, depth, feat, schedule,
                                   schedule_bytes, n_valid, n_intervals, n_slots, out, &d);
  if (st != BEVPOOL_OK) return st;
  const size_t ws_need =
      n_intervals > 0 ? bevpool::forward_scheduled_workspace_bytes(d, n_slots) : 0;
  if (ws_need > bevpool::kNoAllocScratchBytes)
    return fail(BEVPOOL_EWORKSPACE,
                "%d slots need %zu bytes; the allocation-free forward holds at most %zu "
                "(use bevpool_forward_scheduled with a workspace)",
                n_slots, ws_need, bevpool::kNoAllocScratchBytes);
  void* scratch = nullptr;
  st = from_hip(bevpool::forward_noalloc_scratch(&scratch), "bevpool_forward_scheduled_noalloc");
  if (st != BEVPOOL_OK) return st;
  return from_hip(bevpool::launch_forward_scheduled(d, in_dtype, out_dtype, depth, feat, schedule,
                                                    n_valid, n_intervals, n_slots, out, scratch,
                                                    bevpool::kNoAllocScratchBytes,
                                                    static_cast<hipStream_t>(stream)),
                  "bevpool_forward_scheduled_noalloc");
}

int bevpool_backward_workspace_size(const bevpool_shape* shape, size_t* bytes) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(bytes);
  *bytes = bevpool::backward_workspace_bytes(d);
  return ok();
}

int bevpool_backward(const bevpool_shape* shape, int in_dtype, int out_dtype,
                     const void* grad_out, const void* depth, const void* feat,
                     const int32_t* ranks_depth, const int32_t* ranks_bev, int32_t n_valid,
                     void* grad_depth, void* grad_feat, void* workspace, size_t workspace_bytes,
                     void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_dtypes(in_dtype, out_dtype);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(grad_out);
  REQUIRE_PTR(depth);
  REQUIRE_PTR(feat);
  REQUIRE_PTR(grad_depth);
  REQUIRE_PTR(grad_feat);
  if (n_valid < 0 || n_valid > d.P)
    return fail(BEVPOOL_EINVAL, "n_valid = %d outside [0, %lld]", n_valid, (long long)d.P);
  if (n_valid > 0) {
    REQUIRE_PTR(ranks_depth);
    REQUIRE_PTR(ranks_bev);
  }
  const size_t need = bevpool::backward_workspace_bytes(d);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(BEVPOOL_EWORKSPACE, "backward needs %zu workspace bytes, got %zu at %p", need,
                workspace_bytes, workspace);
  return from_hip(bevpool::launch_backward(d, in_dtype, out_dtype, grad_out, depth, feat,
                                           ranks_depth, ranks_bev, n_valid, grad_depth,
                                           grad_feat, workspace,
                                           static_cast<hipStream_t>(stream)),
                  "bevpool_backward");
}

int bevpool_backward_scheduled(const bevpool_shape* shape, int in_dtype, int out_dtype,
                               const void* grad_out, const void* depth, const void* feat,
                               const void* schedule, size_t schedule_bytes, int32_t n_valid,
                               int32_t n_intervals, void* grad_depth, void* grad_feat,
                               void* stream) {
  bevpool::Dims d;
  int st = check_shape(shape, &d);
  if (st != BEVPOOL_OK) return st;
  st = check_dtypes(in_dtype, out_dtype);
  if (st != BEVPOOL_OK) return st;
  st = check_counts(d, n_valid, n_intervals);
  if (st != BEVPOOL_OK) return st;
  REQUIRE_PTR(grad_out);
  REQUIRE_PTR(depth);
  REQUIRE_PTR(feat);
  REQUIRE_PTR(grad_depth);
  REQUIRE_PTR(grad_feat);
  if (n_valid > 0 && n_intervals > 0) {
    REQUIRE_PTR(schedule);
    const size_t need = bevpool::schedule_layout(d, n_valid, n_intervals).total;
    if (schedule_bytes < need)
      return fail(BEVPOOL_EINVAL, "schedule of %zu bytes is smaller than the %zu this plan needs",
                  schedule_bytes, need);
  }
  return from_hip(bevpool::launch_backward_scheduled(d, in_dtype, out_dtype, grad_out, depth, feat,
                                                     schedule, n_valid, n_intervals, grad_depth,
                                                     grad_feat, static_cast<hipStream_t>(stream)),
                  "bevpool_backward_scheduled");
}

}  // extern "C"
