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
