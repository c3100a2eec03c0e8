// Scheduled BEVPoolv2 pooling: the same sum as bevpool_forward (section 2.1),
// organised by the block schedule built once from the plan (prepare.hip;
// layout and terms in internal.h).
//
// The image is cut into strips of kSchedSW feature columns.  Within one
// strip, a column's frustum points lie in one vertical plane, so the cells of
// a column follow each other along the ray as the depth grows and the
// pixel x cell weights of a run of consecutive cells form a nearly dense
// matrix.  Each workgroup takes one piece (a run of a strip's cells) and:
//   1. walks the piece's depth range once, every lane one pixel of the strip
//      and all lanes the same depth bin at a time, so the kSchedSW columns of
//      a row share each depth line; a lane sums the depth scores of each of
//      its pixel's runs into the run's weight entry (LDS);
//   2. every wave takes blocks (kSchedK cells of one column): lanes hold
//      KPL cells x VEC channels in registers, read each feature row once
//      from memory and the cells' weights for that row from LDS, and leave
//      the block's partial rows in LDS;
//   3. every cell of the piece adds its columns' partial rows in column
//      order and is stored: into `out` when no other strip reaches the cell,
//      else into its slot of the workspace.
// k_fwd_cross then adds the slots of each cell reached from several strips
// in strip order and writes the empty cells' zeros.
//
// Every element of `out` is written exactly once, no atomics are used, and
// the summation order depends only on the schedule: results are bitwise
// reproducible.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

#include <algorithm>

namespace bevpool {

namespace {

constexpr int kPT = 256;               // threads of a piece workgroup
constexpr int kPWaves = kPT / kWave;
constexpr int kWalkBatch = 16;         // depth bins in flight per lane (two batches overlap)
constexpr int kRowBatch = 8;           // feature rows in flight per lane (two batches overlap)
constexpr int kCrossThreads = 256;
constexpr size_t kLdsCap = 52 * 1024;  // three workgroups per compute unit

struct PieceArgs {
  const int32_t* hdr;
  const int32_t* piece;    // [n_pieces][kPieceWords]
  const int32_t* block;    // [n_blocks][4]
  const int32_t* cc;       // [n_ccs]
  const int32_t* tc;       // [n_tcs][2]
  const int32_t* pixrec;   // [n_pixrec]
  const uint32_t* rec;     // [n_pairs]
  const int32_t* comb_cell;
  const int32_t* comb_slot0;
  const int32_t* empty;
  float* slots;
  int64_t slot_cap;        // slots the workspace holds
  int32_t n_pieces, n_blocks, n_tcs, n_ccs, n_pairs, n_pixrec;
  int32_t max_ent, max_blk, max_pix, max_rec;
  int32_t n_comb, n_empty;
  int32_t hdr_expect[kSchedHdrChecked];  // header words the launch was sized from
  int32_t C, c_chunk, passes, D, H, W, nsw, strips, hw;  // passes: channel passes of a workgroup
  int64_t cells;
};

// The device header must hold the counts the launch was sized from.
__device__ __forceinline__ bool header_matches(const PieceArgs& a) {
  bool ok = true;
#pragma unroll
  for (int i = 0; i < kSchedHdrChecked; ++i) ok = ok && (a.hdr[i] == a.hdr_expect[i]);
  return ok;
}

template <int KPL>
__device__ __forceinline__ void load_weights(const float* p, float* w) {
  if constexpr (KPL == 4) {
    const float4_t t = *reinterpret_cast<const float4_t*>(p);
    w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
  } else if constexpr (KPL == 2) {
    typedef float float2_t __attribute__((ext_vector_type(2)));
    const float2_t t = *reinterpret_cast<const float2_t*>(p);
    w[0] = t.x; w[1] = t.y;
  } else {
#pragma unroll
    for (int k = 0; k < KPL; ++k) w[k] = p[k];
  }
}

// One workgroup per piece (die-major numbering: a die takes a contiguous run
// of pieces, so neighbouring strips, which share depth lines, meet in one
// L2), one channel chunk per blockIdx.y.
template <typename TIn, typename TOut, int VEC, int KPL>
__global__ __launch_bounds__(kPT) void k_fwd_pieces(const TIn* __restrict__ depth,
                                                    const TIn* __restrict__ feat,
                                                    TOut* __restrict__ out, PieceArgs a) {
  constexpr int G = kSchedK / KPL;  // cell groups of a wave
  extern __shared__ __attribute__((aligned(16))) char smem[];
  if (!header_matches(a)) return;  // (k_fwd_cross writes NaN everywhere)
  const int per_die = (a.n_pieces + kXcds - 1) / kXcds;
  const int pc = (int)(blockIdx.x % kXcds) * per_die + (int)(blockIdx.x / kXcds);
  if (pc >= a.n_pieces || (int)(blockIdx.x / kXcds) >= per_die) return;

  const int32_t* ph = a.piece + (int64_t)pc * kPieceWords;
  const int strip = ph[0], plo = ph[1], nh = ph[2], dlo = ph[3], nd = ph[4], blk0 = ph[5],
            nblk = ph[6], rec0 = ph[7], nrec = ph[8], tc0 = ph[9], ntc = ph[10], cc0 = ph[11],
            ncc = ph[12], nent = ph[13], pix0 = ph[14], ncol = ph[15];
  const int npix = nh * kSchedSW;
  // (a piece that breaks the schedule's invariants is skipped: nothing is
  // read or written outside the arrays; its cells keep unspecified values)
  const bool bad = strip < 0 || strip >= a.strips || plo < 0 || nh < 1 || plo + nh > a.H ||
                   dlo < 0 || nd < 1 || dlo + nd > a.D || blk0 < 0 || nblk < 1 ||
                   nblk > a.max_blk || blk0 + nblk > a.n_blocks || rec0 < 0 || nrec < 1 ||
                   nrec > a.max_rec || rec0 + nrec > a.n_pairs || tc0 < 0 || ntc < 1 ||
                   tc0 + ntc > a.n_tcs || cc0 < 0 || ncc < 1 || ncc > kSchedMaxCC ||
                   cc0 + ncc > a.n_ccs || nent < 1 || nent > a.max_ent || pix0 < 0 ||
                   npix > a.max_pix || pix0 + npix + 1 > a.n_pixrec || ncol < 1 ||
                   ncol > kSchedSW;
  if (bad) return;

  const int C = a.C;
  const int bn = strip / a.nsw;
  const int w0 = (strip - bn * a.nsw) * kSchedSW;
  const int ncols = min(ncol, a.W - w0);  // (columns inside the image, whatever the table says)
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;

  // LDS: weights | partial rows (one channel pass) | CC table | pixel table |
  // records | blocks
  float* s_w = reinterpret_cast<float*>(smem);
  float* s_part = s_w + a.max_ent;
  int32_t* s_cc = reinterpret_cast<int32_t*>(s_part + (int64_t)a.max_blk * kSchedK * a.c_chunk);
  int32_t* s_pix = s_cc + kSchedMaxCC;
  uint32_t* s_rec = reinterpret_cast<uint32_t*>(s_pix + a.max_pix + 1);
  int32_t* s_blk = reinterpret_cast<int32_t*>(s_rec + a.max_rec);

  for (int i = tid; i < nent; i += kPT) s_w[i] = 0.f;
  for (int i = tid; i < ncc; i += kPT) s_cc[i] = a.cc[cc0 + i];
  for (int i = tid; i <= npix; i += kPT) s_pix[i] = a.pixrec[pix0 + i];
  for (int i = tid; i < nrec; i += kPT) s_rec[i] = a.rec[rec0 + i];
  for (int i = tid; i < 4 * nblk; i += kPT) s_blk[i] = a.block[(int64_t)blk0 * 4 + i];
  __syncthreads();

  // ---- 1. depth walk: lane lp owns pixel (plo + lp / SW, w0 + lp % SW); all
  // lanes step through the piece's depth bins together, kWalkBatch bins per
  // batch, the next batch's loads issued before the current one is summed
  const int64_t hw = a.hw;
  for (int lp0 = 0; lp0 < npix; lp0 += kPT) {
    const int lp = lp0 + tid;
    const int hl = lp / kSchedSW;
    const int wl = lp - hl * kSchedSW;
    const int h = plo + hl;
    const bool valid = lp < npix && wl < ncols;
    int r = 0, r_end = 0;
    if (valid) {
      r = min(max(s_pix[lp], 0), nrec);
      r_end = min(max(s_pix[lp + 1], r), nrec);
    }
    // current run: depth bins [rs, re] (relative to dlo) into entry e
    int rs = INT32_MAX, re = -1, e = -1;
    auto fetch = [&]() {
      rs = INT32_MAX;
      if (r < r_end) {
        const uint32_t x = s_rec[r];
        const int cl = (int)(x >> 24);
        rs = (int)(x & 0x7FFu);
        re = rs + (int)((x >> 11) & 0x1FFFu);
        const int32_t ct = cl < ncc ? s_cc[cl] : -1;
        const int u = h - (int)((uint32_t)ct >> 16);
        e = (ct & 0xFFFF) + u * kSchedK;
        if (cl >= ncc || u < 0 || e < 0 || e >= nent) e = -1;
      }
    };
    fetch();
    // (a lane without runs loads nothing; its pointer is never dereferenced)
    const TIn* dp = depth + ((int64_t)(bn * a.D + dlo) * a.H + h) * a.W + w0 + wl;
    const bool any = valid && r < r_end;
    float acc = 0.f;
    float va[kWalkBatch], vb[kWalkBatch];
    auto load_batch = [&](float* v, int d0) {
#pragma unroll
      for (int u = 0; u < kWalkBatch; ++u)
        v[u] = (any && d0 + u < nd) ? to_float(dp[(int64_t)(d0 + u) * hw]) : 0.f;
    };
    auto sum_batch = [&](const float* v, int d0) {
#pragma unroll
      for (int u = 0; u < kWalkBatch; ++u) {
        const int dd = d0 + u;
        if (dd >= rs) {
          acc += v[u];
          if (dd >= re) {
            if (e >= 0) s_w[e] += acc;  // (this lane's pixel only: no other writer)
            acc = 0.f;
            ++r;
            fetch();
          }
        }
      }
    };
    load_batch(va, 0);
    for (int d0 = 0; d0 < nd; d0 += 2 * kWalkBatch) {
      if (d0 + kWalkBatch < nd) load_batch(vb, d0 + kWalkBatch);
      sum_batch(va, d0);
      if (d0 + kWalkBatch >= nd) break;
      if (d0 + 2 * kWalkBatch < nd) load_batch(va, d0 + 2 * kWalkBatch);
      sum_batch(vb, d0 + kWalkBatch);
    }
  }
  __syncthreads();

  // ---- 2 and 3, per channel pass of c_chunk channels
  const int64_t rowstride = (int64_t)a.W * C;
  for (int c0 = blockIdx.y * a.c_chunk * a.passes, pass = 0;
       pass < a.passes && c0 < C; ++pass, c0 += a.c_chunk) {
    const int cc_n = min(a.c_chunk, C - c0);  // channels of this pass
    const int cv = cc_n / VEC;                // vectors of this pass
    // 2. blocks: lanes (g, v) hold cells g*KPL .. of a block, vector v; each
    // lane reads a feature row once for its KPL cells
    const int g = lane / cv;
    const int v = lane - g * cv;
    const bool lane_on = g < G;
    for (int j = wave; j < nblk; j += kPWaves) {
      const int wl = s_blk[4 * j] & 0xFF;
      const int hlo = s_blk[4 * j + 1];
      const int nu = s_blk[4 * j + 2];
      const int eb = s_blk[4 * j + 3];
      float acc[KPL][VEC];
#pragma unroll
      for (int k = 0; k < KPL; ++k)
#pragma unroll
        for (int x = 0; x < VEC; ++x) acc[k][x] = 0.f;
      const bool ok = lane_on && wl < ncols && hlo >= 0 && nu >= 1 && hlo + nu <= a.H && eb >= 0 &&
                      eb + nu * kSchedK <= nent;
      if (ok) {
        const TIn* fp = feat + ((int64_t)(bn * a.H + hlo) * a.W + w0 + wl) * C + c0 + v * VEC;
        const float* wp = s_w + eb + g * KPL;
        float ra[kRowBatch][VEC], rb[kRowBatch][VEC];
        auto load_rows = [&](float (*row)[VEC], int u0) {
#pragma unroll
          for (int q = 0; q < kRowBatch; ++q)
            Vec<TIn, VEC>::load(fp + (int64_t)min(u0 + q, nu - 1) * rowstride, row[q]);
        };
        auto fma_rows = [&](const float (*row)[VEC], int u0) {
#pragma unroll
          for (int q = 0; q < kRowBatch; ++q) {
            if (u0 + q < nu) {
              float wt[KPL];
              load_weights<KPL>(wp + (u0 + q) * kSchedK, wt);
#pragma unroll
              for (int k = 0; k < KPL; ++k)
#pragma unroll
                for (int x = 0; x < VEC; ++x)
                  acc[k][x] = __builtin_fmaf(wt[k], row[q][x], acc[k][x]);
            }
          }
        };
        load_rows(ra, 0);
        for (int u0 = 0; u0 < nu; u0 += 2 * kRowBatch) {
          if (u0 + kRowBatch < nu) load_rows(rb, u0 + kRowBatch);
          fma_rows(ra, u0);
          if (u0 + kRowBatch >= nu) break;
          if (u0 + 2 * kRowBatch < nu) load_rows(ra, u0 + 2 * kRowBatch);
          fma_rows(rb, u0 + kRowBatch);
        }
      }
      if (lane_on) {
#pragma unroll
        for (int k = 0; k < KPL; ++k) {
          float* pp = s_part + ((int64_t)(j * kSchedK + g * KPL + k)) * a.c_chunk + v * VEC;
#pragma unroll
          for (int x = 0; x < VEC; ++x) pp[x] = acc[k][x];
        }
      }
    }
    __syncthreads();

    // 3. cells of the piece: column partials in column order
    const int gpw = kWave / cv;  // lane groups of a wave
    const int gg = lane / cv;
    const int vv = lane - gg * cv;
    const int64_t col = c0 + vv * VEC;
    if (gg < gpw) {
      for (int t = wave * gpw + gg; t < ntc; t += kPWaves * gpw) {
        const int32_t dest = a.tc[2 * (int64_t)(tc0 + t)];
        const uint32_t prs = (uint32_t)a.tc[2 * (int64_t)(tc0 + t) + 1];
        float sum[VEC];
#pragma unroll
        for (int x = 0; x < VEC; ++x) sum[x] = 0.f;
#pragma unroll
        for (int c = 0; c < kSchedSW; ++c) {
          const int pr = (int)((prs >> (8 * c)) & 0xFFu);
          if (pr != 0xFF && pr < nblk * kSchedK) {
            const float* pp = s_part + (int64_t)pr * a.c_chunk + vv * VEC;
#pragma unroll
            for (int x = 0; x < VEC; ++x) sum[x] += pp[x];
          }
        }
        if (dest >= 0) {
          if (dest < a.cells) Vec<TOut, VEC>::store(out + (int64_t)dest * C + col, sum);
        } else {
          const int64_t sl = ~(int64_t)dest;
          if (sl < a.slot_cap) Vec<float, VEC>::store(a.slots + sl * C + col, sum);
        }
      }
    }
    __syncthreads();  // (the next pass overwrites the partial rows)
  }
}

// Cells reached from several strips (sum of their slots in strip order) and
// empty cells (zeros); one lane group per cell.  If the schedule's header
// does not hold the counts the launch was sized from, every cell is NaN.
template <typename TOut, int VEC>
__global__ __launch_bounds__(kCrossThreads) void k_fwd_cross(TOut* __restrict__ out, PieceArgs a) {
  const int lane = lane_id();
  const int C = a.C;
  const int c0 = blockIdx.y * a.c_chunk;
  const int cv = min(a.c_chunk, C - c0) / VEC;
  const int gpw = kWave / cv;
  const int lg = lane / cv;
  const int vi = lane - lg * cv;
  if (lg >= gpw) return;
  const int64_t col = c0 + (int64_t)vi * VEC;
  const int64_t j0 = ((int64_t)blockIdx.x * (kCrossThreads / kWave) + threadIdx.x / kWave) * gpw + lg;
  const int64_t stride = (int64_t)gridDim.x * (kCrossThreads / kWave) * gpw;
  if (!header_matches(a)) {
    float nan[VEC];
#pragma unroll
    for (int x = 0; x < VEC; ++x) nan[x] = __builtin_nanf("");
    for (int64_t cell = j0; cell < a.cells; cell += stride)
      Vec<TOut, VEC>::store(out + cell * C + col, nan);
    return;
  }
  const int64_t n_comb = a.n_comb, n_empty = a.n_empty;
  for (int64_t j = j0; j < n_comb + n_empty; j += stride) {
    if (j < n_comb) {
      const int64_t cell = a.comb_cell[j];
      const int64_t s0 = a.comb_slot0[j], s1 = a.comb_slot0[j + 1];
      if (cell < 0 || cell >= a.cells) continue;
      float sum[VEC];
#pragma unroll
      for (int x = 0; x < VEC; ++x) sum[x] = 0.f;
      if (s0 < 0 || s1 <= s0 || s1 > a.slot_cap) {
#pragma unroll
        for (int x = 0; x < VEC; ++x) sum[x] = __builtin_nanf("");
      } else {
        int64_t s = s0;
        for (; s + 4 <= s1; s += 4) {
          float t[4][VEC];
#pragma unroll
          for (int k = 0; k < 4; ++k) Vec<float, VEC>::load(a.slots + (s + k) * C + col, t[k]);
#pragma unroll
          for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int x = 0; x < VEC; ++x) sum[x] += t[k][x];
        }
        for (; s < s1; ++s) {
          float t[VEC];
          Vec<float, VEC>::load(a.slots + s * C + col, t);
#pragma unroll
          for (int x = 0; x < VEC; ++x) sum[x] += t[x];
        }
      }
      Vec<TOut, VEC>::store(out + cell * C + col, sum);
    } else {
      const int64_t cell = a.empty[j - n_comb];
      if (cell >= 0 && cell < a.cells) store_zero<TOut, VEC>(out + cell * C + col);
    }
  }
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero_out(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

template <typename TOut, int VEC>
hipError_t zero_fill(const Dims& d, void* out, hipStream_t stream) {
  const int64_t nvec = d.cells * (d.C / VEC);
  k_zero_out<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(
      static_cast<TOut*>(out), nvec);
  return hipGetLastError();
}

// Channels per chunk: whole vectors, at most one wave of vectors, and the
// piece's LDS within kLdsCap.
// Channels per pass: the fewest passes whose partial rows keep the piece's
// LDS within kLdsCap, at most one wave of vectors each, split evenly (whole
// vectors).
int chunk_channels(const Dims& d, const PieceArgs& a, int vec) {
  const size_t fixed = 4 * ((size_t)a.max_ent + kSchedMaxCC + (size_t)a.max_pix + 1 +
                            (size_t)a.max_rec + 4 * (size_t)a.max_blk);
  const size_t per_ch = 4 * (size_t)a.max_blk * kSchedK;
  const int64_t by_lds = fixed < kLdsCap ? (int64_t)((kLdsCap - fixed) / per_ch) : 0;
  const int64_t limit = std::max<int64_t>(
      vec, std::min<int64_t>(std::min<int64_t>(d.C, (int64_t)kWave * vec), by_lds / vec * vec));
  int64_t passes = (d.C + limit - 1) / limit;
  int64_t cc = ((d.C + passes - 1) / passes + vec - 1) / vec * vec;
  while (cc > limit) {
    ++passes;
    cc = ((d.C + passes - 1) / passes + vec - 1) / vec * vec;
  }
  return (int)cc;
}

size_t piece_lds_bytes(const PieceArgs& a) {
  return 4 * ((size_t)a.max_ent + (size_t)a.max_blk * kSchedK * a.c_chunk + kSchedMaxCC +
              (size_t)a.max_pix + 1 + (size_t)a.max_rec + 4 * (size_t)a.max_blk);
}

template <typename TIn, typename TOut, int VEC, int KPL>
hipError_t launch_pieces(const void* depth, const void* feat, void* out, const PieceArgs& a,
                         unsigned chunks, hipStream_t stream) {
  const size_t lds = piece_lds_bytes(a);
  auto kern = k_fwd_pieces<TIn, TOut, VEC, KPL>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int per_die = (a.n_pieces + kXcds - 1) / kXcds;
  kern<<<dim3((unsigned)(per_die * kXcds), chunks), dim3(kPT), lds, stream>>>(
      static_cast<const TIn*>(depth), static_cast<const TIn*>(feat), static_cast<TOut*>(out), a);
  return hipGetLastError();
}

template <typename TIn, typename TOut, int VEC>
hipError_t run(const Dims& d, const void* depth, const void* feat, PieceArgs a, void* out,
               hipStream_t stream) {
  a.c_chunk = chunk_channels(d, a, VEC);
  // one workgroup per piece runs every channel pass (the depth walk is done
  // once); a workgroup takes at most one wave's worth of vectors per pass
  const int total_passes = (int)((d.C + a.c_chunk - 1) / a.c_chunk);
  a.passes = total_passes;
  const unsigned chunks = 1;
  const int cv = a.c_chunk / VEC;  // vectors of the widest chunk
  // the most cells per lane that keeps G = K / KPL groups of cv lanes in a wave
  hipError_t e;
  if (cv * 12 <= kWave) e = launch_pieces<TIn, TOut, VEC, 1>(depth, feat, out, a, chunks, stream);
  else if (cv * 6 <= kWave) e = launch_pieces<TIn, TOut, VEC, 2>(depth, feat, out, a, chunks, stream);
  else if (cv * 4 <= kWave) e = launch_pieces<TIn, TOut, VEC, 3>(depth, feat, out, a, chunks, stream);
  else if (cv * 3 <= kWave) e = launch_pieces<TIn, TOut, VEC, 4>(depth, feat, out, a, chunks, stream);
  else if (cv * 2 <= kWave) e = launch_pieces<TIn, TOut, VEC, 6>(depth, feat, out, a, chunks, stream);
  else e = launch_pieces<TIn, TOut, VEC, 12>(depth, feat, out, a, chunks, stream);
  if (e != hipSuccess) return e;
  const int64_t gpw = kWave / cv;
  const int64_t entries = std::max<int64_t>((int64_t)a.n_comb + a.n_empty, 1);
  const int64_t per_block = gpw * (kCrossThreads / kWave);
  const int64_t cblocks = std::min<int64_t>((entries + per_block - 1) / per_block, 65535);
  k_fwd_cross<TOut, VEC><<<dim3((unsigned)cblocks, (unsigned)total_passes), dim3(kCrossThreads), 0,
                            stream>>>(static_cast<TOut*>(out), a);
  return hipGetLastError();
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

int device_cus() {
  static int cached[64];  // per device; 0 = not yet queried
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  cached[dev] = cus;
  return cus;
}

size_t forward_scheduled_workspace_bytes(const Dims& d, int64_t n_slots) {
  return (size_t)(n_slots > 0 ? n_slots : 0) * (size_t)d.C * sizeof(float);
}

hipError_t launch_forward_scheduled(const Dims& d, int in_dtype, int out_dtype,
                                    const void* depth, const void* feat, const void* schedule,
                                    const int32_t* hdr, void* out, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  const bool al = aligned16(feat) && aligned16(out) && aligned16(workspace);
  const bool half_in = in_dtype == BEVPOOL_F16;
  const bool half_out = out_dtype == BEVPOOL_F16;
  const int vec = half_in ? ((al && d.C % 8 == 0) ? 8 : 1) : ((al && d.C % 4 == 0) ? 4 : 1);
  if (hdr[kSHdrValid] == 0 || hdr[kSHdrOcc] == 0 || hdr[kSHdrPieces] == 0) {
    if (half_out) return vec == 8 ? zero_fill<half_t, 8>(d, out, stream) : zero_fill<half_t, 1>(d, out, stream);
    if (vec == 4) return zero_fill<float, 4>(d, out, stream);
    if (vec == 8) return zero_fill<float, 8>(d, out, stream);
    return zero_fill<float, 1>(d, out, stream);
  }
  const ScheduleLayout L = schedule_layout(d, hdr[kSHdrValid], hdr[kSHdrOcc]);
  const char* sc = static_cast<const char*>(schedule);
  auto S = [&](size_t o) { return reinterpret_cast<const int32_t*>(sc + o); };
  PieceArgs a{};
  a.hdr = S(L.header);
  a.piece = S(L.piece);
  a.block = S(L.block);
  a.cc = S(L.cc);
  a.tc = S(L.tc);
  a.pixrec = S(L.pixrec);
  a.rec = reinterpret_cast<const uint32_t*>(S(L.rec));
  a.comb_cell = S(L.comb_cell);
  a.comb_slot0 = S(L.comb_slot0);
  a.empty = S(L.empty);
  a.slots = static_cast<float*>(workspace);
  a.slot_cap = workspace == nullptr ? 0 : (int64_t)(workspace_bytes / ((size_t)d.C * sizeof(float)));
  a.n_pieces = hdr[kSHdrPieces];
  a.n_blocks = hdr[kSHdrBlocks];
  a.n_tcs = hdr[kSHdrTCs];
  a.n_ccs = hdr[kSHdrCCs];
  a.n_pairs = hdr[kSHdrPairs];
  a.n_pixrec = hdr[kSHdrPixrec];
  a.max_ent = hdr[kSHdrMaxEnt];
  a.max_blk = hdr[kSHdrMaxBlk];
  a.max_pix = hdr[kSHdrMaxPix];
  a.max_rec = hdr[kSHdrMaxRec];
  a.n_comb = hdr[kSHdrComb];
  a.n_empty = hdr[kSHdrEmpty];
  for (int i = 0; i < kSchedHdrChecked; ++i) a.hdr_expect[i] = hdr[i];
  a.C = (int32_t)d.C;
  a.D = (int32_t)d.D;
  a.H = (int32_t)d.H;
  a.W = (int32_t)d.W;
  a.nsw = (int32_t)((d.W + kSchedSW - 1) / kSchedSW);
  a.strips = (int32_t)(d.B * d.N * a.nsw);
  a.hw = (int32_t)d.hw;
  a.cells = d.cells;
  if (!half_in) {
    if (vec == 4) return run<float, float, 4>(d, depth, feat, a, out, stream);
    return run<float, float, 1>(d, depth, feat, a, out, stream);
  }
  if (half_out) {
    if (vec == 8) return run<half_t, half_t, 8>(d, depth, feat, a, out, stream);
    return run<half_t, half_t, 1>(d, depth, feat, a, out, stream);
  }
  if (vec == 8) return run<half_t, float, 8>(d, depth, feat, a, out, stream);
  return run<half_t, float, 1>(d, depth, feat, a, out, stream);
}

}  // namespace bevpool
