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
  size_t hist;                 // int32[256 * ntiles]: digit-major tile counts
  size_t digit_totals;         // int32[256]
  size_t cell_counts;          // int32[cells]
  size_t chunk_totals;         // int2[nchunks]: points and occupied cells per chunk
  size_t total;                // bytes
  int64_t ntiles0;             // first-pass tiles (1536 frustum points)
  int64_t ntiles;              // later-pass tiles (1024 points; the hist's row length)
  int key_bits, passes, digit_bits;
  int chunk_shift;               // log2 of the cells per chunk
  int64_t nchunks;
};
PrepareLayout prepare_layout(const Dims& d);

hipError_t launch_prepare(const Dims& d, const int32_t* coor, int32_t* ranks_depth,
                          int32_t* ranks_feat, int32_t* ranks_bev, int32_t* starts,
                          int32_t* lengths, int32_t* counts, void* workspace,
                          hipStream_t stream);

// ---- schedule ----------------------------------------------------------------
// A schedule regroups the kept points of a plan by image strips, for the
// scheduled forward and backward.  Definitions:
//   strip    a block of bh x bw feature pixels of one (sample, camera) image;
//            bh = min(H, R), bw = min(W, max(1, R / bh)) with R =
//            strip_pixels(C) (strips of the last block row and column are cut
//            at the image edge).  Strips are numbered (b, n, h / bh, w / bw)
//            row-major; a pixel's local index in its strip is row-major over
//            the strip's own width.  A column of pixels views one azimuth, so
//            a strip's points fall into few BEV cells.
//   pair     maximal run of kept points of one strip, one cell and one pixel
//            over consecutive depth bins; pairs are ordered by (strip, BEV
//            rank, local pixel, depth bin)
//   share    pairs [c_w, c_(w+1)) of all P pairs, w < S: one share per
//            workgroup of the scheduled forward (S = shares in the header), so
//            that every workgroup sums about the same number of pairs;
//            c_w = floor(P * w / S), moved to the start (end) of the strip it
//            falls in when less than kMinPiece pairs from it
//   item     a run of one strip's pairs inside one share: a strip is cut at
//            the share boundaries inside it, and each piece of L pairs into
//            K = ceil(L / I) items, I the schedule's item size
//            (schedule_item_pairs, in the header), item j starting at pair
//            floor(j * L / K) of the piece
//   segment  maximal run of pairs of one cell inside one item
//   slot     a float32 row of the forward workspace holding one segment's
//            partial sum; only cells covered by several segments have slots,
//            numbered by (cell, segment)
// Device layout (int32 / uint32, 256-byte aligned arrays):
//   header[16]                  counts, see kHdr*
//   pair_rd0[n_valid]           depth rank of the pair's first point
//   pair_ln[n_valid]            local pixel | segment head << 15 | points << 16
//   pair_seg[n_valid] (uint16)  the pair's segment within its item
//   item_strip[items_cap]       strip of each item
//   item_pair0[items_cap + 1]   first pair of each item (+ end sentinel)
//   item_seg0[items_cap + 1]    first segment of each item (+ end sentinel)
//   seg_dest[n_valid]           BEV rank of a segment alone in its cell, or
//                               ~slot (negative) for a cell with several
//   comb_cell[n_occ + 1]        cells with several segments, ascending
//   comb_slot0[n_occ + 1]       first slot of each (+ end sentinel: slots)
//   empty[cells - n_occ + 1]    BEV rank of each empty cell, ascending
//   bp_cell[n_valid]            pixel-major pairs (the pairs stably sorted by
//   bp_dn[n_valid]                feature rank): BEV rank, d0 | points << 16
//   pix_pair0[rows + 1]         first pixel-major pair of each feature row
//   share_item0[kMaxShares + 1] first item of each share (+ end sentinel:
//                               items), for the shares in the header
constexpr int kItemPairs = 2048;          // most pairs of one forward item
constexpr int kItemPairsBig = 3072;       //   of a schedule whose shares hold many items
constexpr int64_t kBigItemPoints = 16384 * 256;  // kept points from which items are big
constexpr int kStripBytes = 32 * 1024;    // staged feature bytes of a strip (4-byte elements)
constexpr uint32_t kPairHead = 1u << 15;  // pair_ln: first pair of a segment
constexpr uint32_t kPairPixel = kPairHead - 1;
constexpr int kHdrPairs = 0, kHdrItems = 1, kHdrSegs = 2, kHdrValid = 3, kHdrOcc = 4,
              kHdrOccFound = 5, kHdrEmpty = 6, kHdrSlots = 7, kHdrComb = 8, kHdrStrips = 9,
              kHdrShares = 10,     // S, the shares the items are cut at
              kHdrSharesOk = 11,   // 1 if no share has more than kShareItems items
              kHdrItemPairs = 12;  // the item size the pieces were cut at
constexpr int kMaxShares = 1024;   // most shares (workgroups of the scheduled forward)
// Item size of a schedule of n_valid kept points: big items where the
// shares of a whole GPU hold many (16,384 kept points each over 256
// workgroups: a workgroup then walks a dozen or more items, and each item
// stages its strip's rows once), else kItemPairs.  It depends on n_valid
// alone, so that a schedule built on one device runs on any other.
inline int schedule_item_pairs(int64_t n_valid) {
  return n_valid >= kBigItemPoints ? kItemPairsBig : kItemPairs;
}
constexpr int kShareItems = 128;   // most items of a share the forward takes as one
constexpr int kMinPiece = 512;     // share boundaries closer to a strip end move to it
static_assert(kHdrPairs == BEVPOOL_SCHEDULE_PAIRS && kHdrItems == BEVPOOL_SCHEDULE_ITEMS &&
                  kHdrSegs == BEVPOOL_SCHEDULE_SEGMENTS && kHdrValid == BEVPOOL_SCHEDULE_KEPT &&
                  kHdrOcc == BEVPOOL_SCHEDULE_CELLS && kHdrOccFound == BEVPOOL_SCHEDULE_CELLS_FOUND &&
                  kHdrEmpty == BEVPOOL_SCHEDULE_EMPTY && kHdrSlots == BEVPOOL_SCHEDULE_SLOTS,
              "header indices are part of the C interface");
// gfx950 (MI355X) has 8 accelerator complex dies; workgroup i of a launch is
// dispatched to die i % 8, each die with its own L2.
constexpr int kXcds = 8;

struct StripDims {
  int64_t bh, bw;    // strip height and width in pixels
  int64_t nhb, nwb;  // strips per image column and row
  int64_t strips;    // B * N * nhb * nwb
  int64_t pixels;    // bh * bw: most pixels of a strip
};
// Most pixels per strip: the staged feature rows of a 64-vector channel
// chunk (at most 256 four-byte elements per row) fit kStripBytes.
int64_t strip_pixels(int64_t C);
StripDims strip_dims(const Dims& d);

struct ScheduleLayout {
  size_t header, pair_rd0, pair_ln, pair_seg, item_strip, item_pair0, item_seg0, seg_dest, comb_cell,
      comb_slot0, empty, bp_cell, bp_dn, pix_pair0, share_item0, total;
  int64_t n_valid, n_occ, n_empty, items_cap;
  StripDims sd;
  // build workspace
  size_t ws_ka, ws_va, ws_kb, ws_vb, ws_head, ws_pair_rb, ws_pair_row, ws_pair_dn, ws_flags,
      ws_strip, ws_tiles, ws_hist, ws_sums, ws_total;
  int64_t ntiles, nscan;
  int row_bits, cell_bits, pixel_bits, strip_bits;
  // workspace of the build by strips in LDS (schedule_local.hip)
  size_t wl_map, wl_rkey, wl_rnpts, wl_strip_np, wl_strip_p0, wl_strip_it0, wl_pix_count,
      wl_item_nseg, wl_cell_nseg, wl_fill, wl_slot0, wl_head_cell, wl_head_item, wl_slot_seg,
      wl_cell_tot, wl_total;
  int wl_cell_shift;        // log2 of the cells per chunk of the cell scans
  int64_t wl_cell_chunks;
};
ScheduleLayout schedule_layout(const Dims& d, int64_t n_valid, int64_t n_intervals);

// Build by strips in LDS: usable when a strip's frustum points fit one
// workgroup's LDS sort (pixels * D <= kLocalPoints, pixels <= 256) and the
// sort key (cell within the sample, local pixel, depth bin) fits 32 bits.
constexpr int kLocalPoints = 12288;
bool schedule_local_ok(const Dims& d, int64_t n_valid);
void local_schedule_ws(const Dims& d, ScheduleLayout& L);
hipError_t launch_schedule_local(const Dims& d, const int32_t* rd, const int32_t* rb,
                                 int32_t n_valid, int32_t n_intervals, void* schedule,
                                 void* workspace, hipStream_t stream);
// Compute units of the current device (cached per device).
int device_cus();
// Workgroups of the scheduled forward on the current device: one per CU,
// a whole number per die; the shares a schedule is cut at.
int forward_workgroups();
hipError_t launch_schedule(const Dims& d, const int32_t* rd, const int32_t* rb, int32_t n_valid,
                           int32_t n_intervals, void* schedule, void* workspace,
                           hipStream_t stream);
// Float32 workspace rows of the scheduled forward: one per slot.
size_t forward_scheduled_workspace_bytes(const Dims& d, int64_t n_slots);
// bevpool_forward_scheduled_noalloc: the slots in a static device array of
// this many bytes; its device address on the current device (looked up on
// the first call per device)
constexpr size_t kNoAllocScratchBytes = BEVPOOL_NOALLOC_SCRATCH_BYTES;
hipError_t forward_noalloc_scratch(void** addr);
hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                    const void* depth, const void* feat, const void* schedule,
                                    int32_t n_valid, int32_t n_intervals, int32_t n_slots,
                                    void* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, const double* lse = nullptr);
// voxel index of every frustum point from per-camera parameters (float64,
// kCameraWords per camera of each (b, n))
constexpr int kCameraWords = BEVPOOL_CAMERA_WORDS;
hipError_t launch_geometry(const Dims& d, const bevpool_frustum& f, const double* cams,
                           int32_t* coor, hipStream_t stream);
// per-pixel log-sum-exp over the depth bins of depth logits (B, N, D, H, W)
hipError_t launch_depth_lse(const Dims& d, int in_dtype, const void* logits, double* lse,
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
