// Internal interface between the C ABI (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

constexpr int kWaveLanes = 64;

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
// The block schedule regroups the kept points of a plan for the scheduled
// forward (and lists them pixel by pixel for the scheduled backward).
// Terms, every count over kept points:
//   strip  kSchedSW adjacent feature-map columns of one (sample, camera)
//          image, all H rows; strips are numbered (b*N + n) * nsw + w / SW,
//          nsw = ceil(W / SW); a pixel's column in its strip is w % SW
//   pair   a maximal run of one pixel's kept points in one cell over
//          consecutive depth bins (first bin d0, n points); pairs are ordered
//          by (strip, cell, h * SW + column, d0)
//   TC     (strip, cell) with pairs; within a strip TCs are ranked by (least
//          d0, cell)
//   piece  a run of consecutive TCs of one strip; a piece starts at a strip's
//          first TC, at every tcmax-th TC of the strip (tcmax = kSchedK *
//          min(4, kSchedEntries / (SW * K * H))) and where the strip's pair
//          count before the TC crosses a multiple of kSchedPairs.  One piece
//          is one workgroup of the scheduled forward.
//   CC     (TC, column) with pairs; within a piece, ordered by (column, least
//          d0, cell)
//   block  kSchedK consecutive CCs of one column of a piece (fewer at the end
//          of the column's run): the dense weight matrix of its CCs over the
//          column's rows [hlo, hlo + nu), entries ebase + u * K + k of the
//          piece's weight array
//   slot   a float32 row of the forward's workspace: the partial sum of a TC
//          whose cell is also reached from other strips; slots are numbered
//          in (cell, strip) order
// Device layout (int32 words, 256-byte aligned arrays; capacities from
// n_valid, see schedule_layout):
//   header[16]              counts, kSHdr*
//   piece[n_pieces][16]     strip, plo, nh, dlo, nd, blk0, nblk, rec0, nrec,
//                           tc0, ntc, cc0, ncc, nent, pix0, ncol (columns of
//                           the strip inside the image)
//   block[n_blocks][4]      column | ncells << 8, hlo, nu, ebase
//   cc[n_ccs]               ebase + k | hlo << 16 (piece CC table)
//   tc[n_tcs][2]            destination (BEV rank, or ~slot), and the partial
//                           row (block-in-piece * K + k) of each column, one
//                           byte each (0xff: no pair in that column)
//   pixrec[n_pixrec]        per piece, per local pixel (h - plo) * SW +
//                           column, its first record (relative to rec0), and
//                           nrec after the last pixel
//   rec[n_pairs]            per piece, pairs in (local pixel, d0) order:
//                           d0 - dlo | (n - 1) << 11 | CC of the piece << 24
//   comb_cell[n_comb], comb_slot0[n_comb + 1]   cells with several TCs
//   empty[n_empty]          cells no kept point reaches, ascending
//   bp_cell[n_pairs], bp_dn[n_pairs], pix_pair0[rows + 1]
//                           the pairs in feature-row order (stable): BEV
//                           rank, d0 | n << 16; first pair of every row
constexpr int kSchedSW = 4;          // strip width in columns
constexpr int kSchedK = 12;          // CCs per block
constexpr int kSchedPairs = 3000;    // pairs per piece
constexpr int kSchedEntries = 8192;  // most weight entries of a piece
constexpr int kSchedMaxCC = 256;     // most CCs of a piece (8-bit index)
constexpr int kSchedMaxD = 2048;     // depth bins a record can address
constexpr int kPieceWords = 16;
constexpr int kSHdrPairs = 0, kSHdrPieces = 1, kSHdrBlocks = 2, kSHdrValid = 3, kSHdrOcc = 4,
              kSHdrOccFound = 5, kSHdrEmpty = 6, kSHdrSlots = 7, kSHdrComb = 8, kSHdrTCs = 9,
              kSHdrCCs = 10, kSHdrMaxEnt = 11, kSHdrMaxBlk = 12, kSHdrMaxPix = 13,
              kSHdrPixrec = 14, kSHdrMaxRec = 15;
constexpr int kSchedHdrChecked = 16;  // header words a forward checks against its launch
static_assert(kSHdrPairs == BEVPOOL_SCHEDULE_PAIRS && kSHdrPieces == BEVPOOL_SCHEDULE_PIECES &&
                  kSHdrBlocks == BEVPOOL_SCHEDULE_BLOCKS && kSHdrValid == BEVPOOL_SCHEDULE_KEPT &&
                  kSHdrOcc == BEVPOOL_SCHEDULE_CELLS &&
                  kSHdrOccFound == BEVPOOL_SCHEDULE_CELLS_FOUND &&
                  kSHdrEmpty == BEVPOOL_SCHEDULE_EMPTY && kSHdrSlots == BEVPOOL_SCHEDULE_SLOTS,
              "header indices are part of the C interface");
// gfx950 (MI355X) has 8 accelerator complex dies; workgroup i of a launch is
// dispatched to die i % 8, each die with its own L2.
constexpr int kXcds = 8;

// Compute units of the current device (cached per device).
int device_cus();
// TCs per piece for a feature-map height H (0: H too large for a schedule).
int64_t sched_tc_max(int64_t H);

struct ScheduleLayout {
  size_t header, piece, block, cc, tc, pixrec, rec, comb_cell, comb_slot0, empty, bp_cell, bp_dn,
      pix_pair0, total;  // byte offsets of the schedule's arrays, and its size
  size_t ws_total;       // bytes of build workspace
  int64_t n_valid, n_occ, n_empty, piece_cap, pixrec_cap, nsw, strips;
};
ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals);
hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream);
// Float32 workspace rows of the scheduled forward: one per slot.
size_t forward_scheduled_workspace_bytes(const Dims& d, int64_t n_slots);
// `hdr` is the host copy of the schedule's header.
hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                    const void* depth, const void* feat, const void* schedule,
                                    const int32_t* hdr, void* out, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream);

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
hipError_t launch_backward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                     const void* grad_out, const void* depth, const void* feat,
                                     const void* schedule, int32_t n_valid, int32_t n_intervals,
                                     void* grad_depth, void* grad_feat, hipStream_t stream);

}  // namespace bevpool
