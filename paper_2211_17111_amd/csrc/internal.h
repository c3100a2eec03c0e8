// Internal interface between the C ABI (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

// Sizes derived from a validated shape, all in int64 to avoid overflow while
// checking limits.
struct Dims {
  int64_t B, N, D, H, W, C, X, Y, Z;
  int64_t P;      // frustum points B*N*D*H*W
  int64_t rows;   // image-feature rows B*N*H*W
  int64_t cells;  // BEV cells B*Z*Y*X
  int64_t per_view;  // D*H*W
  int64_t hw;        // H*W
};

Dims dims_of(const bevpool_shape& s);

// ---- prepare ---------------------------------------------------------------
constexpr int kPrepThreads = 256;               // 4 waves
constexpr int kPrepRounds = 16;                 // 64-lane rounds per wave
constexpr int kPrepTile = kPrepThreads * kPrepRounds;  // 4096 elements per block
constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;   // 2048

struct PrepareLayout {
  size_t keys_tmp, vals_tmp;   // int32[P] each (radix ping-pong)
  size_t tile_counts;          // int32[ntiles + 1]
  size_t hist;                 // int32[256 * ntiles]
  size_t scan_sums;            // int32[nscan + 1]
  size_t total;                // bytes
  int64_t ntiles;
  int64_t nscan;
  int key_bits, passes, digit_bits;
};
PrepareLayout prepare_layout(const Dims& d);

hipError_t launch_prepare(const Dims& d, const int32_t* coor, int32_t* ranks_depth,
                          int32_t* ranks_feat, int32_t* ranks_bev, int32_t* starts,
                          int32_t* lengths, int32_t* counts, void* workspace,
                          hipStream_t stream);

// ---- schedule ----------------------------------------------------------------
// Device layout of a forward schedule (all int32), built from a plan:
//   header[16]            runtime counts, see kHdr*
//   pair_rd0[n_valid]     depth rank of the first point of each pair
//   pair_cell[n_valid]    BEV rank of each pair
//   pair_npts[n_valid]    points of each pair: depth ranks rd0 + k*H*W
//   cell_id[n_occ]        BEV rank of each occupied cell, ascending
//   cell_pair[n_occ + 1]  first pair of each occupied cell (+ end sentinel)
//   task_cell[tasks + 1]  first occupied cell owned by each task
//   item_info[items][4]   first cell, end cell, first pair, end pair of the
//                         task each work item belongs to, in task order
//   item_chunk[items]     channel chunk of the item | (chunks of its task << 16)
//   xcd_begin[kXcds + 1]  first item of each XCD: contiguous item ranges of
//                         about equal work, so an XCD's L2 holds the feature
//                         rows of one region of the BEV grid
// A pair is a maximal run of kept points with the same BEV rank, the same
// pixel and consecutive depth bins.
constexpr int kSchedTaskPairs = 2048;  // nominal pairs per task
constexpr int kHdrPairs = 0, kHdrTasks = 1, kHdrItems = 2, kHdrValid = 3, kHdrOcc = 4,
              kHdrOccFound = 5, kHdrWork = 6;
// gfx950 (MI355X) has 8 accelerator complex dies; workgroup i of a launch is
// dispatched to die i % 8, each die with its own L2.
constexpr int kXcds = 8;

struct ScheduleLayout {
  size_t header, pair_rd0, pair_cell, pair_npts, cell_id, cell_pair, task_cell, item_info,
      item_chunk, xcd_begin, total;
  int64_t n_valid, n_occ, tasks_cap, items_cap;
  // build workspace
  size_t ws_keys_a, ws_vals_a, ws_keys_b, ws_vals_b, ws_head, ws_tiles, ws_hist, ws_sums, ws_total;
  int64_t ntiles, nscan;
  int rf_bits, rb_bits;
};
ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals);
int schedule_max_chunks(const Dims& d);
hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream);
hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                   const void* depth, const void* feat, const void* schedule,
                                   int32_t n_valid, int32_t n_intervals, void* out,
                                   hipStream_t stream);

// ---- forward ---------------------------------------------------------------
size_t forward_workspace_bytes(const Dims& d);
hipError_t launch_forward(const Dims& d, int in_dtype, int out_dtype, const void* depth,
                          const void* feat, const int32_t* rd, const int32_t* rf,
                          const int32_t* rb, const int32_t* starts, const int32_t* lengths,
                          int32_t n_valid, int32_t n_intervals, void* out, void* workspace,
                          hipStream_t stream);

// ---- backward --------------------------------------------------------------
size_t backward_workspace_bytes(const Dims& d);
hipError_t launch_backward(const Dims& d, int in_dtype, int out_dtype, const void* grad_out,
                           const void* depth, const void* feat, const int32_t* rd,
                           const int32_t* rb, int32_t n_valid, void* grad_depth,
                           void* grad_feat, void* workspace, hipStream_t stream);

}  // namespace bevpool
