// Scheduled BEVPoolv2 pooling: the same sum as bevpool_forward (section 2.1),
// driven by a schedule built once from the plan (prepare.hip, internal.h).
//
// A pair (one cell, one pixel, consecutive depth bins) multiplies one feature
// row by the sum of its points' depth scores.  A tile is a run of nearby cells
// whose pairs share many feature rows; the schedule lists each tile's
// distinct rows (mostly runs of consecutive pixels, so contiguous memory).
// One workgroup per item (a channel slice of a tile):
//
//   1. stages the tile's row list in LDS and computes every pair's weight,
//      the sum of its depth scores, into LDS (one thread per pair);
//   2. cuts each cell's pairs into chunks of about (pairs / groups) and gives
//      each lane group up to tile_max_units() such (cell, chunk) units, with
//      one fp32 accumulator vector per unit in registers;
//   3. walks the row list in windows: the window's rows (this item's channel
//      slice) are copied from HBM/L2 into LDS, loads of the next window being
//      issued before the current one is consumed, and every group advances
//      each of its units over the pairs whose row lies in the window (a
//      cell's pairs are sorted by row, so that is a contiguous run);
//   4. stores each cell once: a cell held by one unit directly, a cell split
//      over several units after adding, in unit order, the partial sums the
//      other units left in LDS.
// Items of one die form a contiguous, work-balanced range in spatial order,
// walked by a persistent grid, so a die's L2 serves one region of the grid.
// Tiles with a single cell may hold more pairs than fit in LDS; they are
// processed in batches of kTilePairs pairs with the same accumulators.
//
// Every element of `out` is written exactly once, without atomics; the
// summation order depends only on the schedule, so results are bitwise
// reproducible.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

constexpr int kNT = kTileThreads;
constexpr int kWaves = kNT / kWave;
constexpr int kPairsPerThread = kTilePairs / kNT;  // pairs (and rows) of a batch per thread
constexpr int kDepthBurst = 4;  // depth scores per pair loaded before any is summed

struct TileArgs {
  const int32_t* hdr;
  const uint32_t* pair_rl;
  const uint32_t* pair_dn;
  const int32_t* cell_out;
  const int32_t* cell_pair;
  const int32_t* tile_cell;
  const int32_t* tile_row0;
  const int32_t* rows;
  const int32_t* row_dbase;
  const int32_t* empty;
  const int32_t* item_tile;
  const int32_t* item_slice;
  const int32_t* xcd_begin;
  int32_t n_occ;
  int32_t n_valid;
  int32_t items_cap;
  int32_t max_cells;
  int32_t C;
  int32_t D;
  int32_t hw32;  // H*W (depth ranks are below 2^31)
  int64_t n_rows, cells, n_empty;
};

struct PairW {
  float w;     // summed depth score
  int32_t rl;  // row index relative to the batch's first row
};

// Raw element vector moved between HBM and LDS without conversion.
template <typename T, int VEC>
struct Raw {
  typedef T type;
};
template <>
struct Raw<float, 4> {
  typedef float4_t type;
};
template <>
struct Raw<half_t, 8> {
  typedef float4_t type;
};

template <typename TIn, typename TOut, int VEC>
__global__ __launch_bounds__(kNT) void k_fwd_tiles(const TIn* __restrict__ depth,
                                                   const TIn* __restrict__ feat,
                                                   TOut* __restrict__ out, TileArgs a) {
  constexpr int MAXU = tile_max_units(VEC);
  typedef typename Raw<TIn, VEC>::type RawT;
  constexpr int kVecBytes = (int)sizeof(RawT);
  // vectors of one window each thread holds in registers while it is in flight
  constexpr int kWinRegsFull = (kTileWindowBytes / kVecBytes + kNT - 1) / kNT;
  constexpr int kWinRegs = kWinRegsFull < 6 ? kWinRegsFull : 6;
  constexpr int kChunk = VEC >= 8 ? 2 : 4;

  __shared__ PairW s_pair[kTilePairs];
  __shared__ int32_t s_rid[kTilePairs];   // feature rank of each row of the batch
  __shared__ int32_t s_cp[kTileMaxCells + 1];  // first pair of each cell, batch-relative
  __shared__ int32_t s_co[kTileMaxCells];      // BEV rank of each cell
  __shared__ int32_t s_u0[kTileMaxCells + 1];  // first unit of each cell
  __shared__ __attribute__((aligned(16))) char s_win0[kTileWindowBytes];
  __shared__ __attribute__((aligned(16))) char s_win1[kTileWindowBytes];
  // depth rank at depth bin 0 of each row's pixel: needed only while the pair
  // weights are computed, before the second window buffer is first filled
  int32_t* const s_rdb = reinterpret_cast<int32_t*>(s_win1);
  static_assert(kTileWindowBytes >= kTilePairs * (int)sizeof(int32_t), "s_rdb fits s_win1");

  const int32_t* hdr = a.hdr;
  if (hdr[kHdrOccFound] != a.n_occ || hdr[kHdrOcc] != a.n_occ) return;  // uniform
  const int32_t n_tiles = min(hdr[kHdrTiles], a.n_occ);
  const int32_t n_items = min(hdr[kHdrItems], a.items_cap);
  const int64_t C = a.C;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int xcd = blockIdx.x % kXcds;
  const int slot = blockIdx.x / kXcds;
  const int nslots = gridDim.x / kXcds;
  const int32_t i_end = min(a.xcd_begin[xcd + 1], n_items);

  for (int32_t it = max(a.xcd_begin[xcd], 0) + slot; it < i_end; it += nslots) {
    const int32_t t = a.item_tile[it];
    const int32_t ks = a.item_slice[it];
    const int32_t K = ks >> 16, k = ks & 0xffff;
    if (t < 0 || t >= n_tiles || K < 1 || k >= K || C % K != 0 || (C / K) % VEC != 0)
      continue;  // uniform
    const int32_t cb = a.tile_cell[t], ce = a.tile_cell[t + 1];
    const int32_t nc = ce - cb;
    if (cb < 0 || nc < 1 || ce > a.n_occ) continue;
    const int32_t pb = a.cell_pair[cb], pe = a.cell_pair[ce];
    const int32_t np = pe - pb;
    const int32_t r0 = a.tile_row0[t];
    const int32_t nrows = a.tile_row0[t + 1] - r0;
    const bool single = nc == 1;
    if (np < 1 || nrows < 1 || pb < 0 || pe > a.n_valid || r0 < 0 || r0 + nrows > a.n_valid) continue;
    if (!single && (np > kTilePairs || nc > a.max_cells || nrows > np)) continue;

    // zero-fill this tile's share of the empty cells (first slice only)
    if (k == 0 && a.n_empty > 0) {
      const int64_t e0 = a.n_empty * t / n_tiles, e1 = a.n_empty * (t + 1) / n_tiles;
      const int64_t per = C / VEC;
      for (int64_t i = tid; i < (e1 - e0) * per; i += kNT) {
        const int64_t cell = a.empty[e0 + i / per];
        if (cell >= 0 && cell < a.cells) store_zero<TOut, VEC>(out + cell * C + (i % per) * VEC);
      }
    }

    const int64_t c_lo = k * (C / K), c_hi = c_lo + C / K;
    const int32_t n_batch = single ? (np + kTilePairs - 1) / kTilePairs : 1;
    for (int64_t s0 = c_lo; s0 < c_hi; s0 += 64 * VEC) {
      // ---- lane groups of this sub-slice
      const int64_t sw = (c_hi - s0) < 64 * VEC ? (c_hi - s0) : 64 * VEC;  // channels
      const int G = (int)((sw + VEC - 1) / VEC);
      const int GPW = kWave / G;
      const int NG = kWaves * GPW;
      const int gi = lane / G, lg = lane % G;
      const bool active = gi < GPW;
      const int g = wave * GPW + gi;
      const int RS = G * kVecBytes;                  // bytes of one staged row slice
      const int R = min(kTileWindowBytes / RS, kWinRegs * kNT / G);  // rows per window
      const bool lane_on = active && (int64_t)lg * VEC < sw;

      float acc[MAXU][VEC];
#pragma unroll
      for (int u = 0; u < MAXU; ++u)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[u][e] = 0.f;
      int32_t n_units = 0;

      for (int32_t bi = 0; bi < n_batch; ++bi) {
        const int32_t bp0 = pb + bi * kTilePairs;
        const int32_t nb = min(kTilePairs, pe - bp0);
        int32_t r_lo = 0, r_hi = nrows;
        if (single) {
          r_lo = (int32_t)a.pair_rl[bp0];
          r_hi = (int32_t)a.pair_rl[bp0 + nb - 1] + 1;
          if (r_lo < 0 || r_hi > nrows || r_hi <= r_lo) r_lo = 0, r_hi = 0;
        }
        const int32_t nr = min(r_hi - r_lo, (int32_t)kTilePairs);

        // ---- 1. rows, cells and pair weights (kept across sub-slices when
        //         the tile is one batch).  Every global load of this phase is
        //         issued before any is consumed: row ids and pair records
        //         together, then the first window of rows together with the
        //         depth scores of every pair.
        const int32_t n_win = (nr + R - 1) / R;
        // Window w's rows (this sub-slice) are fetched into registers with
        // ordinary vector loads -- coalesced: a wave reads whole runs of
        // consecutive rows -- and written to an LDS buffer once the buffer is
        // free.  Vector v of the window lands at buf + v * kVecBytes, i.e.
        // row r at r * RS, column col at col * kVecBytes.
        RawT pf[kWinRegs];
        // row and column of window vector v (v < 2^24): a float reciprocal
        // estimate corrected by one step either way
        const float inv_g = 1.f / (float)G;
        auto split = [&](int32_t v, int32_t& r, int32_t& col) {
          r = (int32_t)((float)v * inv_g);
          col = v - r * G;
          if (col < 0) { --r; col += G; }
          if (col >= G) { ++r; col -= G; }
        };
        auto fetch = [&](int32_t w) {
          const int32_t w0 = w * R;
          const int32_t nvec = min(R, nr - w0) * G;
#pragma unroll
          for (int q = 0; q < kWinRegs; ++q) {
            const int32_t v = tid + q * kNT;
            int32_t r, col;
            split(v, r, col);
            if (v < nvec)
              pf[q] = *reinterpret_cast<const RawT*>(feat + (int64_t)s_rid[w0 + r] * C + s0 +
                                                      col * VEC);
          }
        };
        // (G * VEC equals the sub-slice width, so every column is a channel
        // of the slice)
        auto commit = [&](int32_t w, char* buf) {
          const int32_t nvec = min(R, nr - w * R) * G;
#pragma unroll
          for (int q = 0; q < kWinRegs; ++q) {
            const int32_t v = tid + q * kNT;
            if (v < nvec) *reinterpret_cast<RawT*>(buf + v * kVecBytes) = pf[q];
          }
        };
        bool first_window_issued = false;
        if (s0 == c_lo || n_batch > 1) {
          lds_barrier();  // previous item / batch is done with the LDS tables
          int32_t rid[kPairsPerThread], rdb[kPairsPerThread];
          uint32_t prl[kPairsPerThread], pdn[kPairsPerThread];
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i) {
            const int32_t x = tid + i * kNT;
            rid[i] = x < nr ? a.rows[r0 + r_lo + x] : 0;
            rdb[i] = x < nr ? a.row_dbase[r0 + r_lo + x] : 0;
            prl[i] = x < nb ? a.pair_rl[bp0 + x] : 0xffffffffu;
            pdn[i] = x < nb ? a.pair_dn[bp0 + x] : 0u;
          }
          if (!single) {
            for (int32_t c = tid; c <= nc; c += kNT) {
              s_cp[c] = min(max(a.cell_pair[cb + c] - pb, 0), np);
              if (c < nc) s_co[c] = a.cell_out[cb + c];
            }
          }
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i) {
            const int32_t x = tid + i * kNT;
            if (x < nr) {
              const bool ok = rid[i] >= 0 && rid[i] < a.n_rows;
              s_rid[x] = ok ? rid[i] : 0;
              s_rdb[x] = ok ? rdb[i] : 0;
            }
          }
          lds_barrier();
          // depth-score addresses first, so that no pair record is still in
          // flight when the row copies are issued (a wait for it would also
          // wait for the copies)
          // depth rank of each pair's first point: its row's base plus d0 bins
          int32_t base[kPairsPerThread], npt[kPairsPerThread], rlr[kPairsPerThread];
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i) {
            const int32_t x = tid + i * kNT;
            const int32_t rl = (int32_t)prl[i] - r_lo;
            const int32_t d0 = (int32_t)(pdn[i] & 0xffffu), n = (int32_t)(pdn[i] >> 16);
            const bool ok = x < nb && rl >= 0 && rl < nr && d0 + n <= a.D;
            base[i] = ok ? s_rdb[rl] + d0 * a.hw32 : 0;
            npt[i] = ok ? n : 0;
            rlr[i] = ok ? rl : 0x7fffffff;  // never inside a window: the pair is skipped
          }
          if (n_win > 0) {
            fetch(0);
            first_window_issued = true;
          }
          // the first kDepthBurst scores of every pair, all loads in flight at
          // once (lanes past a pair's points load nothing)
          TIn dv[kPairsPerThread][kDepthBurst];
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i)
#pragma unroll
            for (int q = 0; q < kDepthBurst; ++q) {
              dv[i][q] = TIn(0);
              if (q < npt[i]) dv[i][q] = depth[base[i] + q * a.hw32];
            }
          // keep the scheduler from interleaving the sums with the loads
          __builtin_amdgcn_sched_barrier(0);
          float wsum[kPairsPerThread];
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i) {
            wsum[i] = 0.f;
#pragma unroll
            for (int q = 0; q < kDepthBurst; ++q) wsum[i] += to_float(dv[i][q]);
          }
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i)  // longer runs (rare)
            for (int32_t q = kDepthBurst; q < npt[i]; ++q)
              wsum[i] += to_float(depth[base[i] + q * a.hw32]);
#pragma unroll
          for (int i = 0; i < kPairsPerThread; ++i) {
            const int32_t x = tid + i * kNT;
            if (x < nb) {
              PairW pw;
              pw.w = wsum[i];
              pw.rl = rlr[i];
              s_pair[x] = pw;
            }
          }
        }

        // ---- 2. units: (cell, chunk) of at most L pairs
        const int32_t L = (nb + NG - 1) / NG;
        lds_barrier();  // weights visible; s_u0 free
        if (single) {
          n_units = NG;
        } else {
          if (wave == 0) {
            int32_t carry = 0;
            for (int32_t c0 = 0; c0 < nc; c0 += kWave) {
              const int32_t c = c0 + lane;
              const int32_t u = c < nc ? (s_cp[c + 1] - s_cp[c] + L - 1) / L : 0;
              const int32_t inc = wave_inclusive_scan(u);
              if (c < nc) s_u0[c] = carry + inc - u;
              carry += __shfl(inc, kWave - 1, kWave);
            }
            if (lane == 0) s_u0[nc] = carry;
          }
          lds_barrier();
          n_units = s_u0[nc];
          if (n_units > NG * MAXU) n_units = NG * MAXU;  // cannot happen for a built schedule
        }
        int32_t cur[MAXU], end[MAXU];
#pragma unroll
        for (int u = 0; u < MAXU; ++u) {
          const int32_t j = g + u * NG;
          cur[u] = 0;
          end[u] = 0;
          if (!active || j >= n_units) continue;
          if (single) {
            if (u == 0) {
              cur[u] = min(j * L, nb);
              end[u] = min(cur[u] + L, nb);
            }
          } else {
            int32_t lo = 0, hi = nc - 1;  // cell of unit j
            while (lo < hi) {
              const int32_t mid = (lo + hi + 1) >> 1;
              if (s_u0[mid] <= j) lo = mid; else hi = mid - 1;
            }
            const int32_t c = lo;
            cur[u] = min(s_cp[c] + (j - s_u0[c]) * L, s_cp[c + 1]);
            end[u] = min(cur[u] + L, s_cp[c + 1]);
          }
        }

        // ---- 3. row windows, double-buffered: window w + 1 is in flight
        //         while window w is consumed
        if (!first_window_issued && n_win > 0) fetch(0);
        // Advances every unit over its pairs whose row lies in window w.  A
        // unit's pairs are sorted by row, so they form a run; full chunks of
        // pairs take one window test (on the last) and independent LDS
        // reads.  Rows are clamped into the window, which only matters for a
        // schedule that breaks the ordering.  Chunks hold kChunk pairs (four,
        // two for 8-wide vectors, whose rows take more registers).
        auto consume = [&](int32_t w, const char* buf) {
          const int32_t w0 = w * R, w1 = w0 + R;
          if (!lane_on) return;
          const char* lane_buf = buf + lg * kVecBytes;
          auto row_at = [&](int32_t rl) {
            const int32_t r = min(max(rl, w0), w1 - 1) - w0;
            return reinterpret_cast<const TIn*>(lane_buf + (uint32_t)r * (uint32_t)RS);
          };
#pragma unroll
          for (int u = 0; u < MAXU; ++u) {
            int32_t c = cur[u];
            const int32_t e = end[u];
            while (c + kChunk <= e) {
              const PairW pl = s_pair[c + kChunk - 1];
              if (pl.rl >= w1) break;
              PairW pp[kChunk];
              float x[kChunk][VEC];
#pragma unroll
              for (int k = 0; k < kChunk - 1; ++k) pp[k] = s_pair[c + k];
              pp[kChunk - 1] = pl;
#pragma unroll
              for (int k = 0; k < kChunk; ++k) Vec<TIn, VEC>::load(row_at(pp[k].rl), x[k]);
#pragma unroll
              for (int e2 = 0; e2 < VEC; ++e2) {
                float t = acc[u][e2];
#pragma unroll
                for (int k = 0; k < kChunk; ++k) t = fmaf(pp[k].w, x[k][e2], t);
                acc[u][e2] = t;
              }
              c += kChunk;
            }
            while (c < e) {
              const PairW p = s_pair[c];
              if (p.rl >= w1) break;
              float x[VEC];
              Vec<TIn, VEC>::load(row_at(p.rl), x);
#pragma unroll
              for (int k = 0; k < VEC; ++k) acc[u][k] = fmaf(p.w, x[k], acc[u][k]);
              ++c;
            }
            cur[u] = c;
          }
        };
        // Window w + 1 is in flight (registers) while window w is consumed;
        // the buffer a window is written to was last read two windows
        // earlier, which every wave finished before the previous barrier.
        for (int32_t w = 0; w < n_win; w += 2) {
          commit(w, s_win0);
          lds_barrier();
          if (w + 1 < n_win) fetch(w + 1);
          consume(w, s_win0);
          if (w + 1 < n_win) {
            commit(w + 1, s_win1);
            lds_barrier();
            if (w + 2 < n_win) fetch(w + 2);
            consume(w + 1, s_win1);
          }
        }
        // pairs a corrupt schedule placed outside every window are skipped
#pragma unroll
        for (int u = 0; u < MAXU; ++u) cur[u] = end[u];
      }  // batches

      // ---- 4. store each cell once
      lds_barrier();  // windows consumed: s_win0 holds the partial sums now
      float* slots = reinterpret_cast<float*>(s_win0);
      const int64_t ch = s0 + (int64_t)lg * VEC;
      // sum[e] += slot m's element for m in [first, first + count), in
      // order of m; loads are issued eight slots at a time
      auto add_slots = [&](float* sum, int32_t first, int32_t count) {
        const float* sp = slots + lg * VEC;
        int32_t m = 0;
        for (; m + 8 <= count; m += 8) {
          float v[8][VEC];
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[j][e] = sp[(int64_t)(first + m + j) * sw + e];
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int e = 0; e < VEC; ++e) sum[e] += v[j][e];
        }
        for (; m < count; ++m)
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] += sp[(int64_t)(first + m) * sw + e];
      };
      if (single) {
        if (lane_on) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) slots[(int64_t)g * sw + lg * VEC + e] = acc[0][e];
        }
        lds_barrier();
        if (lane_on && g == 0) {
          float sum[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] = 0.f;
          add_slots(sum, 0, NG);
          const int64_t cell = a.cell_out[cb];
          if (cell >= 0 && cell < a.cells) Vec<TOut, VEC>::store(out + cell * C + ch, sum);
        }
      } else {
        int32_t cell_of[MAXU];
#pragma unroll
        for (int u = 0; u < MAXU; ++u) {
          const int32_t j = g + u * NG;
          cell_of[u] = -1;
          if (!lane_on || j >= n_units) continue;
          int32_t lo = 0, hi = nc - 1;
          while (lo < hi) {
            const int32_t mid = (lo + hi + 1) >> 1;
            if (s_u0[mid] <= j) lo = mid; else hi = mid - 1;
          }
          cell_of[u] = lo;
          const int32_t c = lo;
          const int32_t uc = s_u0[c + 1] - s_u0[c];
          if (uc == 1) {
            const int64_t cell = s_co[c];
            if (cell >= 0 && cell < a.cells) Vec<TOut, VEC>::store(out + cell * C + ch, acc[u]);
          } else if (j > s_u0[c] && j - c - 1 < NG) {
            const int64_t sl = j - c - 1;  // slot of a non-first unit
#pragma unroll
            for (int e = 0; e < VEC; ++e) slots[sl * sw + lg * VEC + e] = acc[u][e];
          }
        }
        lds_barrier();
#pragma unroll
        for (int u = 0; u < MAXU; ++u) {
          const int32_t j = g + u * NG;
          const int32_t c = cell_of[u];
          if (c < 0 || j != s_u0[c]) continue;
          const int32_t uc = s_u0[c + 1] - s_u0[c];
          if (uc == 1) continue;
          float sum[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum[e] = acc[u][e];
          // the cell's other units left their sums in slots j - c .. j - c + uc - 2
          add_slots(sum, j - c, max(min(uc - 1, NG - (j - c)), 0));
          const int64_t cell = s_co[c];
          if (cell >= 0 && cell < a.cells) Vec<TOut, VEC>::store(out + cell * C + ch, sum);
        }
      }
      lds_barrier();  // slots and unit tables are reused by the next sub-slice
    }  // sub-slices
  }  // items
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero_all(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

// Workgroups that fit on the device at once, rounded to whole dies.
template <typename TIn, typename TOut, int VEC>
int resident_blocks() {
  static int cached[64];  // per device; 0 = not yet queried
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_fwd_tiles<TIn, TOut, VEC>, kNT, 0) !=
          hipSuccess ||
      per_cu <= 0)
    per_cu = 1;
  int blocks = cus * per_cu;
  blocks = ((blocks + kXcds - 1) / kXcds) * kXcds;
  cached[dev] = blocks;
  return blocks;
}

template <typename TIn, typename TOut, int VEC>
hipError_t run(const Dims& d, const void* depth, const void* feat, const TileArgs& a, void* out,
               int32_t n_valid, hipStream_t stream) {
  TOut* o = static_cast<TOut*>(out);
  if (a.n_occ == 0 || n_valid == 0) {
    const int64_t nvec = d.cells * (d.C / VEC);
    k_zero_all<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(o, nvec);
    return hipGetLastError();
  }
  const int blocks = resident_blocks<TIn, TOut, VEC>();
  k_fwd_tiles<TIn, TOut, VEC><<<dim3((unsigned)blocks), dim3(kNT), 0, stream>>>(
      static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), o, a);
  return hipGetLastError();
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                   const void* depth, const void* feat, const void* schedule,
                                   int32_t n_valid, int32_t n_intervals, void* out,
                                   hipStream_t stream) {
  const ScheduleLayout L = schedule_layout(d, n_valid, n_intervals);
  const char* sc = static_cast<const char*>(schedule);
  auto S = [&](size_t o) { return reinterpret_cast<const int32_t*>(sc + o); };
  TileArgs a;
  a.hdr = S(L.header);
  a.pair_rl = reinterpret_cast<const uint32_t*>(S(L.pair_rl));
  a.pair_dn = reinterpret_cast<const uint32_t*>(S(L.pair_dn));
  a.cell_out = S(L.cell_out);
  a.cell_pair = S(L.cell_pair);
  a.tile_cell = S(L.tile_cell);
  a.tile_row0 = S(L.tile_row0);
  a.rows = S(L.rows);
  a.row_dbase = S(L.row_dbase);
  a.empty = S(L.empty);
  a.item_tile = S(L.item_tile);
  a.item_slice = S(L.item_slice);
  a.xcd_begin = S(L.xcd_begin);
  a.n_occ = n_intervals;
  a.n_valid = n_valid;
  a.items_cap = (int32_t)L.items_cap;
  a.max_cells = tile_max_cells(d);
  a.C = (int32_t)d.C;
  a.D = (int32_t)d.D;
  a.hw32 = (int32_t)d.hw;
  a.n_rows = d.rows;
  a.cells = d.cells;
  a.n_empty = L.n_empty;
  const bool al = aligned16(feat) && aligned16(out);
  if (in_dtype == BEVPOOL_F32) {
    if (al && d.C % 4 == 0) return run<float, float, 4>(d, depth, feat, a, out, n_valid, stream);
    return run<float, float, 1>(d, depth, feat, a, out, n_valid, stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0) return run<half_t, half_t, 8>(d, depth, feat, a, out, n_valid, stream);
    return run<half_t, half_t, 1>(d, depth, feat, a, out, n_valid, stream);
  }
  if (al && d.C % 8 == 0) return run<half_t, float, 8>(d, depth, feat, a, out, n_valid, stream);
  return run<half_t, float, 1>(d, depth, feat, a, out, n_valid, stream);
}

}  // namespace bevpool
