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
// A forward schedule regroups the kept points of a plan for the tiled forward
// kernel.  Definitions:
//   pair   maximal run of kept points with the same cell, the same pixel and
//          consecutive depth bins (their depth scores multiply one feature row)
//   cell   occupied BEV cell; cells are ordered by (b, z, Morton(y, x)) so that
//          consecutive cells are close in the grid (falls back to the BEV rank
//          when that key would not fit 31 bits)
//   tile   consecutive cells, cut where the first pair of a cell crosses a
//          multiple of kTilePairs / 2, where the cell index crosses a
//          multiple of tile_max_cells(), and around any cell with more than
//          kTilePairs / 2 pairs; so a tile of several cells has at most
//          kTilePairs pairs and at most tile_max_cells() cells
//   rows   the distinct feature rows of a tile, ascending: the rows the
//          forward stages in LDS
//   item   channel slice k of K of a tile; K grows with the tile's staged
//          bytes (counted at 4 bytes per element, so one schedule serves
//          both element types)
// Device layout (int32 / uint32, 256-byte aligned arrays):
//   header[16]               counts, see kHdr*
//   pair_rl[n_valid]         index of the pair's feature row in its tile's rows
//   pair_dn[n_valid]         first depth bin | (points << 16)
//   cell_out[n_occ + 1]      BEV rank of each cell in tile order
//   cell_pair[n_occ + 1]     first pair of each cell (+ end sentinel)
//   tile_cell[n_occ + 1]     first cell of each tile (+ end sentinel)
//   tile_row0[n_occ + 1]     first row entry of each tile (+ end sentinel)
//   rows[n_valid]            feature rank of each row entry
//   row_dbase[n_valid]       depth rank of each row entry's pixel at depth bin 0
//   empty[cells - n_occ + 1] BEV rank of each empty cell, ascending
//   bp_cell[n_valid]         pixel-major pairs (the same pairs sorted by feature
//   bp_dn[n_valid]             rank, then cell key): BEV rank, and d0 | points << 16
//   pix_pair0[rows + 1]      first pixel-major pair of each feature row
//   item_tile[items_cap]     tile of each item, in tile order
//   item_slice[items_cap]    k | (K << 16)
//   xcd_begin[kXcds + 1]     first item of each XCD: contiguous item ranges of
//                            about equal work, so one die's L2 holds the
//                            feature rows of one region of the grid
constexpr int kTilePairs = 4096;              // pairs a workgroup holds in LDS at once
constexpr int kTileThreads = 1024;            // forward workgroup
constexpr int kTileWindowBytes = 48 * 1024;   // LDS per buffer of staged feature rows (two)
constexpr int kTileMaxCells = 512;            // cap of tile_max_cells()
constexpr int kTileItemBytes = 192 * 1024;    // staged feature bytes per item (target)
constexpr int kHdrPairs = 0, kHdrTiles = 1, kHdrItems = 2, kHdrValid = 3, kHdrOcc = 4,
              kHdrOccFound = 5, kHdrEmpty = 6, kHdrRowEntries = 7, kHdrWork = 8;
// gfx950 (MI355X) has 8 accelerator complex dies; workgroup i of a launch is
// dispatched to die i % 8, each die with its own L2.
constexpr int kXcds = 8;

// Lane groups of the forward kernel.  A slice of `cs` channels is processed
// in sub-slices of at most 64 vectors of `vec` elements; a lane group has one
// lane per vector of a sub-slice and as many groups as fit in a wave share it.
// Each group holds the accumulators of at most tile_max_units(vec) (cell,
// chunk) units.
inline int tile_group_lanes(int64_t cs, int vec) {
  const int64_t g = (cs + vec - 1) / vec;
  return (int)(g > kWaveLanes ? kWaveLanes : g);
}
inline int tile_groups(int64_t cs, int vec) {
  return (kTileThreads / kWaveLanes) * (kWaveLanes / tile_group_lanes(cs, vec));
}
constexpr int tile_max_units(int vec) { return vec == 1 ? 8 : 16 / vec; }
// Most cells a tile may hold: the (cell, chunk) units of any item, at most
// one per cell plus one per chunk of a balanced split, must fit the groups'
// accumulators for every vector width the forward may use (1, 4, 8).
int tile_max_cells(const Dims& d);

struct ScheduleLayout {
  size_t header, pair_rl, pair_dn, cell_out, cell_pair, tile_cell, tile_row0, rows, row_dbase, empty,
      bp_cell, bp_dn, pix_pair0, item_tile, item_slice, xcd_begin, total;
  int64_t n_valid, n_occ, n_empty, items_cap;
  // build workspace
  size_t ws_ka, ws_va, ws_kb, ws_vb, ws_head, ws_pair_rb, ws_pair_row, ws_flags, ws_tiles,
      ws_hist, ws_sums, ws_total;
  int64_t ntiles, nscan;
  int row_bits, key_bits, tile_bits;
  int morton_level;  // cells keyed by (b*Z + z) << 2L | Morton(y, x); -1: by BEV rank
};
ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals);
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
hipError_t launch_backward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                     const void* grad_out, const void* depth, const void* feat,
                                     const void* schedule, int32_t n_valid, int32_t n_intervals,
                                     void* grad_depth, void* grad_feat, hipStream_t stream);

}  // namespace bevpool
