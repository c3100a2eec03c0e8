/*
 * bevpool.h -- C ABI of the BEVPoolv2 view-transformation path for AMD
 * Instinct MI355X (gfx950).
 *
 * BEVPoolv2 (section 2.1) turns the Lift-Splat-Shoot view transformer into
 * two stages:
 *   1. an offline preprocessing of the voxel index of every frustum point:
 *      drop points outside the scope of all voxels and sort the rest by
 *      voxel index, carrying each point's frustum index along as a trace;
 *   2. an online pooling that, for every voxel, reads the depth score and the
 *      image feature of each of its points through that trace and sums their
 *      products, so the (N, D, H, W, C) frustum feature is never formed.
 * bevpool_prepare is stage 1, bevpool_forward is stage 2 and
 * bevpool_backward gives the gradients of stage 2 (which the paper does not
 * describe; they follow from the chain rule).
 *
 * Shapes and layouts (all arrays dense, row-major, no padding):
 *   depth     (B, N, D, H, W)   depth score, element type in_dtype
 *   feat      (B, N, H, W, C)   image feature, channels last, in_dtype
 *   coor      (P, 3) int32      voxel index (x, y, z) of every frustum point
 *   out       (B, Z, Y, X, C)   BEV feature, channels last, out_dtype
 * with P = B*N*D*H*W frustum points enumerated
 *   p = (((b*N + n)*D + d)*H + h)*W + w,
 * the same order as the depth score.  A point is kept when
 * 0 <= x < X, 0 <= y < Y and 0 <= z < Z.  For a kept point
 *   depth rank   = p
 *   feature rank = ((b*N + n)*H + h)*W + w          (row of feat)
 *   BEV rank     = ((b*Z + z)*Y + y)*X + x          (row of out)
 *
 * Conventions shared by every call:
 *   - All array pointers are device pointers (hipMalloc'd or equivalent),
 *     owned by the caller.  The library never allocates or frees device
 *     memory and never synchronises the stream, except where stated.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *     Work is enqueued asynchronously; results are visible after the stream
 *     is synchronised.
 *   - Every call validates its arguments before any HIP call and returns
 *     BEVPOOL_OK (0) or a negative bevpool_status.  No C++ exception crosses
 *     the ABI.  bevpool_last_error() gives a message for the calling thread.
 *   - Limits: every dimension >= 1; P < 2^31; B*Z*Y*X*C < 2^31;
 *     B*N*H*W*C < 2^31; C <= 1024.
 *   - 16-byte aligned depth/feat/out/grad pointers with C a multiple of the
 *     vector width (4 for f32, 8 for f16) take the vectorised kernels; any
 *     other alignment or C takes the scalar kernels (not an error).
 *   - Accumulation is always in float32.
 *   - Kernels bounds-check every index they read from a plan, so a plan that
 *     does not satisfy the documented invariants cannot cause out-of-bounds
 *     accesses; the numerical result is then unspecified.
 */
#ifndef BEVPOOL_H
#define BEVPOOL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BEVPOOL_VERSION 1

typedef struct bevpool_shape {
  int32_t B; /* samples */
  int32_t N; /* camera views */
  int32_t D; /* depth classes */
  int32_t H; /* feature-map height */
  int32_t W; /* feature-map width */
  int32_t C; /* feature channels */
  int32_t X; /* BEV cells along ego x */
  int32_t Y; /* BEV cells along ego y */
  int32_t Z; /* BEV cells along ego z */
} bevpool_shape;

enum bevpool_dtype {
  BEVPOOL_F32 = 0, /* IEEE binary32 */
  BEVPOOL_F16 = 1  /* IEEE binary16 */
};

enum bevpool_status {
  BEVPOOL_OK = 0,
  BEVPOOL_EINVAL = -1,     /* null pointer, non-positive dimension, bad count */
  BEVPOOL_EOVERFLOW = -2,  /* a size exceeds the int32 index range or C > 1024 */
  BEVPOOL_EDTYPE = -3,     /* unknown dtype or unsupported dtype combination */
  BEVPOOL_EWORKSPACE = -4, /* workspace pointer NULL or smaller than required */
  BEVPOOL_ELAUNCH = -5     /* a HIP call or kernel launch failed */
};

/* Library version (BEVPOOL_VERSION of the build). */
int bevpool_version(void);

/* Static description of a status code; never NULL. */
const char* bevpool_strerror(int status);

/* Message describing the last failure of a call on this thread (for
 * BEVPOOL_ELAUNCH it includes the HIP error string); "" if none. */
const char* bevpool_last_error(void);

/*
 * Geometry (section 2.1, paragraph 1: each frustum point's voxel index,
 * computed from the camera intrinsics and extrinsics), on the device, for
 * geometry that changes per sample (augmentation, ego motion).
 *
 * cams: device float64 (B, N, BEVPOOL_CAMERA_WORDS), per camera fx, fy, cx,
 * cy, then the camera-to-ego rotation R (row-major 3x3) and translation t
 * (ego = R cam + t; camera frame x right, y down, z forward).  Feature cell
 * (h, w) looks through the pixel centre ((w + 0.5) stride, (h + 0.5) stride);
 * depth bin k lies at depth_start + k depth_step along the optical axis.
 * bevpool_geometry writes coor (P x 3 int32, the layout bevpool_prepare
 * reads, points enumerated like the depth score): floor((e - lo) / res) of
 * each ego coordinate e, clipped to +-2^30.  Points outside the grid keep
 * their index (bevpool_prepare filters them).  All arithmetic is float64 in
 * a fixed order with no fused multiply-add, so the indices match a float64
 * evaluation of the same expressions bit for bit.  EINVAL for NULL pointers,
 * a non-positive or non-finite stride, step or cell size, or non-finite
 * bounds.
 */
#define BEVPOOL_CAMERA_WORDS 16
typedef struct bevpool_frustum {
  double stride;      /* input pixels per feature cell */
  double depth_start; /* depth of bin 0 along the optical axis (metres) */
  double depth_step;  /* depth between neighbouring bins (metres) */
  double lo[3];       /* grid lower bounds x, y, z in the ego frame (metres) */
  double res[3];      /* cell sizes x, y, z (metres) */
} bevpool_frustum;
int bevpool_geometry(const bevpool_shape* shape, const bevpool_frustum* frustum,
                     const double* cams, int32_t* coor, void* stream);

/*
 * Preprocessing (section 2.1, paragraphs 1-2): filter, sort, intervals.
 *
 * bevpool_prepare_workspace_size writes to *bytes the device scratch size
 * bevpool_prepare needs for `shape` (radix ping-pong buffers, digit
 * histograms of the tiles, the point count of every cell and the totals of
 * every chunk of cells).
 *
 * bevpool_prepare reads coor (P x 3 int32) and writes:
 *   ranks_depth, ranks_feat, ranks_bev   capacity P each; the first n_valid
 *       entries hold the kept points sorted by BEV rank, ties in ascending
 *       frustum index (a stable sort), so the order is unique;
 *   interval_starts, interval_lengths    capacity min(P, B*Z*Y*X) each; the
 *       first n_intervals entries give, for every occupied BEV cell in
 *       ascending cell order, the position of its first point in the sorted
 *       ranks and its number of points;
 *   counts[0] = n_valid, counts[1] = n_intervals  (device int32[2]).
 * Points outside the grid are filtered, not errors.  The caller reads
 * `counts` after synchronising the stream.  Entries beyond the counts are
 * left unspecified.  The workspace must stay untouched until the stream has
 * executed the call.  Deterministic: the same coor always gives the same
 * bytes.
 */
int bevpool_prepare_workspace_size(const bevpool_shape* shape, size_t* bytes);
int bevpool_prepare(const bevpool_shape* shape, const int32_t* coor,
                    int32_t* ranks_depth, int32_t* ranks_feat, int32_t* ranks_bev,
                    int32_t* interval_starts, int32_t* interval_lengths,
                    int32_t* counts, void* workspace, size_t workspace_bytes,
                    void* stream);

/*
 * Pooling (section 2.1, paragraph 2): for every occupied cell j,
 *   out[cell_j, c] = sum over i in [start_j, start_j + length_j) of
 *                    depth[ranks_depth[i]] * feat[ranks_feat[i], c],
 * with cell_j = ranks_bev[start_j]; every other cell of out is +0.0.
 * The plan arrays are those of bevpool_prepare (or any plan with the same
 * invariants: ranks_bev non-decreasing, intervals covering maximal runs of
 * equal ranks_bev in ascending order); n_valid is the number of entries of
 * the ranks arrays and n_intervals that of the interval arrays.  out is
 * written in full, exactly once per element, without atomics; results are
 * bitwise reproducible.  out must not alias any input.  in_dtype applies to
 * depth and feat, out_dtype to out; both F32 or both F16, or F16 in with F32
 * out.  n_intervals == 0 writes an all-zero out.
 *
 * Work is split into equal ranges of sorted points, one wavefront each;
 * cells cut by a range boundary are summed from per-range partials held in
 * the workspace (bevpool_forward_workspace_size bytes, float32 partial rows).
 * The workspace contents are scratch: one forward at a time per workspace.
 */
int bevpool_forward_workspace_size(const bevpool_shape* shape, size_t* bytes);
int bevpool_forward(const bevpool_shape* shape, int in_dtype, int out_dtype,
                    const void* depth, const void* feat,
                    const int32_t* ranks_depth, const int32_t* ranks_feat,
                    const int32_t* ranks_bev, const int32_t* interval_starts,
                    const int32_t* interval_lengths, int32_t n_valid,
                    int32_t n_intervals, void* out, void* workspace,
                    size_t workspace_bytes, void* stream);

/*
 * Schedule (optional): a regrouping of the plan of section 2.1, built once
 * offline like the plan itself.
 *
 * The schedule regroups the kept points of a plan by image strips: blocks of
 * bh x bw feature pixels of one camera image, normally whole pixel columns
 * (the frustum points of a pixel column lie in one vertical plane, so a
 * strip's points fall into few BEV cells).  Within a strip, kept points of one
 * pixel in one cell over consecutive depth bins form a pair: their depth
 * scores are summed first and the pixel's feature row is read once.  The
 * pairs are cut into equal shares, one per workgroup of the scheduled forward
 * on the device the schedule is built on (its compute units); a strip's pairs
 * are cut at those shares and into items of at most a few thousand pairs, and
 * an item's pairs into segments (one per cell).  A schedule built on one
 * device gives the same results on another; only the balance of the work
 * over the workgroups depends on the device.  A cell covered by one segment
 * is written directly; a cell covered by several has one partial-sum slot per
 * segment in the forward's workspace, added in a fixed order.
 *
 * bevpool_schedule_size gives the schedule buffer size and the build
 * workspace size for a plan with n_valid kept points and n_intervals
 * occupied cells.  bevpool_schedule reads the first n_valid entries of
 * ranks_depth and ranks_bev of a plan from bevpool_prepare and writes the
 * schedule (device memory owned by the caller).  Enqueued on `stream`;
 * deterministic.  The schedule starts with BEVPOOL_SCHEDULE_HEADER int32
 * counts, indexed by bevpool_schedule_count; the rest is opaque.  A caller
 * reads the header back once (after the build has completed) to size the
 * forward's workspace.
 *
 * bevpool_forward_scheduled computes exactly what bevpool_forward computes
 * (same layouts, dtypes and zero-filled empty cells, every element of `out`
 * written once, no atomics, bitwise reproducible) from the schedule alone.
 * n_valid and n_intervals are the values the schedule was built with, and
 * n_slots is its header's BEVPOOL_SCHEDULE_SLOTS count (read back once by
 * the caller).  Its workspace holds the slots: at least
 * bevpool_forward_scheduled_workspace_size(shape, n_slots) bytes (float32
 * rows of C; may be 0 bytes and NULL when n_slots is 0), else
 * BEVPOOL_EWORKSPACE before anything is enqueued.  The workspace contents
 * are scratch: one forward at a time per workspace; the schedule is only
 * read, so concurrent forwards may share it.  If the schedule's header does
 * not hold these three counts (a schedule of another plan, or one not yet
 * built), every element of `out` is written as NaN; nothing is read or
 * written outside the schedule, the inputs, `out` and the workspace.
 */
#define BEVPOOL_SCHEDULE_HEADER 16
enum bevpool_schedule_count {
  BEVPOOL_SCHEDULE_PAIRS = 0,
  BEVPOOL_SCHEDULE_ITEMS = 1,
  BEVPOOL_SCHEDULE_SEGMENTS = 2,
  BEVPOOL_SCHEDULE_KEPT = 3,        /* n_valid the schedule was built with */
  BEVPOOL_SCHEDULE_CELLS = 4,       /* n_intervals the schedule was built with */
  BEVPOOL_SCHEDULE_CELLS_FOUND = 5, /* occupied cells found in the plan */
  BEVPOOL_SCHEDULE_EMPTY = 6,
  BEVPOOL_SCHEDULE_SLOTS = 7
};
int bevpool_schedule_size(const bevpool_shape* shape, int32_t n_valid,
                          int32_t n_intervals, size_t* schedule_bytes,
                          size_t* workspace_bytes);
int bevpool_schedule(const bevpool_shape* shape, const int32_t* ranks_depth,
                     const int32_t* ranks_bev, int32_t n_valid, int32_t n_intervals,
                     void* schedule, size_t schedule_bytes, void* workspace,
                     size_t workspace_bytes, void* stream);
int bevpool_forward_scheduled_workspace_size(const bevpool_shape* shape, int32_t n_slots,
                                              size_t* bytes);
int bevpool_forward_scheduled(const bevpool_shape* shape, int in_dtype, int out_dtype,
                              const void* depth, const void* feat, const void* schedule,
                              size_t schedule_bytes, int32_t n_valid, int32_t n_intervals,
                              int32_t n_slots, void* out, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * Fused depth softmax (section 2.1: a pixel's depth score is a distribution
 * over its D depth bins).  When the scores come from logits, the score of
 * point (b, n, d, h, w) is exp(logit[b,n,d,h,w] - lse[b,n,h,w]) with
 * lse[b,n,h,w] = log sum_d exp(logit[b,n,d,h,w]).
 *
 * bevpool_depth_lse reads logits (B, N, D, H, W; in_dtype) and writes lse
 * (B, N, H, W; float64, caller's device memory): one double per pixel,
 * m + log(sum exp(logit - m)) with m the pixel's largest logit.
 *
 * bevpool_forward_scheduled_softmax is bevpool_forward_scheduled with the
 * depth scores formed on the fly from the logits and that lse (exponent in
 * double, the device library's float32 expf), so the (B, N, D, H, W) score
 * tensor is never written or read.  Arguments, workspace, results and
 * errors as bevpool_forward_scheduled; lse may be NULL only when
 * n_intervals is 0.  Logits must be finite.  There is no fused backward:
 * a training step materialises the scores and uses bevpool_backward_scheduled.
 */
int bevpool_depth_lse(const bevpool_shape* shape, int in_dtype, const void* logits, double* lse,
                      void* stream);
int bevpool_forward_scheduled_softmax(const bevpool_shape* shape, int in_dtype, int out_dtype,
                                      const void* logits, const double* lse, const void* feat,
                                      const void* schedule, size_t schedule_bytes,
                                      int32_t n_valid, int32_t n_intervals, int32_t n_slots,
                                      void* out, void* workspace, size_t workspace_bytes,
                                      void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * bevpool_forward_scheduled without a workspace.  The slots live in a
 * static device array of BEVPOOL_NOALLOC_SCRATCH_BYTES bytes that the
 * library holds on each device it runs on from the first call there until
 * the process ends; nothing is allocated or freed by the call (the first
 * call on a device looks the array's address up).  Arguments, results and
 * errors as bevpool_forward_scheduled, except that a schedule whose n_slots
 * float32 rows of C exceed BEVPOOL_NOALLOC_SCRATCH_BYTES is refused with
 * BEVPOOL_EWORKSPACE.  Every call on a device uses the same array: calls
 * that may overlap on one device (on different streams, or from different
 * threads without ordering) race and give undefined results.
 */
#define BEVPOOL_NOALLOC_SCRATCH_BYTES (32u << 20)
int bevpool_forward_scheduled_noalloc(const bevpool_shape* shape, int in_dtype, int out_dtype,
                                      const void* depth, const void* feat, const void* schedule,
                                      size_t schedule_bytes, int32_t n_valid,
                                      int32_t n_intervals, int32_t n_slots, void* out,
                                      void* stream);

/*
 * Gradients of bevpool_forward (not in the paper; chain rule):
 *   grad_depth[p]  = sum_c grad_out[rank_bev(p), c] * feat[rank_feat(p), c]
 *                    for a kept point p, and +0.0 for a dropped point;
 *   grad_feat[f,c] = sum over kept points p of pixel f of
 *                    depth[p] * grad_out[rank_bev(p), c], +0.0 if none.
 * grad_out has out's shape and out_dtype; grad_depth and grad_feat have the
 * shapes and in_dtype of depth and feat.  The backward reads ranks_depth and
 * ranks_bev (first n_valid entries) to map every frustum point to its cell;
 * a point's feature row is its pixel, as bevpool_prepare's ranks_feat
 * records.  Both gradients are written in full, exactly once per element,
 * without atomics (deterministic).  Workspace: bevpool_backward_workspace_size
 * bytes (one int32 per frustum point).
 */
int bevpool_backward_workspace_size(const bevpool_shape* shape, size_t* bytes);
int bevpool_backward(const bevpool_shape* shape, int in_dtype, int out_dtype,
                     const void* grad_out, const void* depth, const void* feat,
                     const int32_t* ranks_depth, const int32_t* ranks_bev,
                     int32_t n_valid, void* grad_depth, void* grad_feat,
                     void* workspace, size_t workspace_bytes, void* stream);

/* The same gradients from a schedule (bevpool_schedule of the same plan and
 * shape), which lists every pixel's pairs of kept points: each pixel's
 * feature row is read once and each pair (a cell and a run of consecutive
 * depth bins of the pixel) reads its grad_out row once.  Dropped points of
 * grad_depth get +0.0 and kept points their gradient; in launches large
 * enough to fill the device all of grad_depth is cleared first and the kept
 * points are written again, in smaller ones each element is written once.
 * grad_feat is written once per element.  No workspace; no atomics (deterministic).  Arguments as for
 * bevpool_backward and bevpool_forward_scheduled; an all-zero result when
 * n_valid or n_intervals is 0 (schedule may then be NULL). */
int bevpool_backward_scheduled(const bevpool_shape* shape, int in_dtype, int out_dtype,
                               const void* grad_out, const void* depth, const void* feat,
                               const void* schedule, size_t schedule_bytes, int32_t n_valid,
                               int32_t n_intervals, void* grad_depth, void* grad_feat,
                               void* stream);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* BEVPOOL_H */
