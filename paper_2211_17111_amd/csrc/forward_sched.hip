// Scheduled BEVPoolv2 pooling: the same sum as bevpool_forward, driven by a
// schedule built once from the plan (see the schedule section of prepare.hip).
//
// The schedule groups kept points into pairs (one cell, one pixel,
// consecutive depth bins), so each pair reads its pixel's feature row once
// with the summed depth score of its points as the weight, and cuts the pairs
// into work items that own whole cells (a task larger than the nominal size
// is split by channel slices, which are independent).  Items are kept in
// spatial order and each of the 8 dies gets a contiguous run of items of
// about equal work, so a die's L2 holds the feature rows of one region of the
// grid; one persistent 1024-thread workgroup per CU walks its die's items.
// For each item:
//
//   1. zero-fill the empty cells just before each cell the task owns (and
//      after the last occupied cell);
//   2. split the item's pairs evenly over its lane groups (CV lanes per group,
//      one 16-byte vector of the channel slice per lane); each wave stages the
//      weight, feature rank and BEV rank of its groups' next pairs in LDS
//      (a pair's depth scores sit H*W apart and are gathered together), then
//      every group streams its feature rows, double-buffered, with up to 40/VEC
//      loads in flight, and
//      flushes a sum whenever the BEV rank changes;
//   3. a cell lying inside one group's range is stored directly; the parts of
//      a cell cut by group boundaries are kept in LDS and, after a barrier,
//      added in group order by the group holding the cell's first part.
//
// Every element of `out` is written exactly once, without atomics, and the
// summation order depends only on the schedule, so results are bitwise
// reproducible.

#include "device_utils.h"
#include "internal.h"
#include "vec.h"

namespace bevpool {

namespace {

constexpr int kItemThreads = 1024;
constexpr int kItemWaves = kItemThreads / kWave;
constexpr int kMetaEntries = 128;  // staged pairs per wave and round
constexpr int kRowRegs = 40;       // VGPRs per lane given to feature rows in flight
constexpr int kMaxGroups = kItemWaves * kWave;  // one lane per group at most

struct SchedArgs {
  const int32_t* hdr;
  const int32_t* pair_rd0;
  const int32_t* pair_cell;
  const int32_t* pair_npts;
  const int32_t* cell_id;
  const int32_t* item_info;
  const int32_t* item_chunk;
  const int32_t* xcd_begin;
  int32_t n_occ;
  int32_t n_valid;
  int32_t C;
  int32_t units;  // 16-channel units (C / 16), 0 when C is not a multiple of 16
  int64_t cells;
  int64_t P;
  int64_t rows;
  int64_t hw;        // H*W: distance between consecutive depth bins of a pixel
  int64_t per_view;  // D*H*W
};

struct PairMeta {
  float w;       // summed depth score of the pair's points
  int32_t row;   // feature rank
  int32_t cell;  // BEV rank
};

template <typename TIn, typename TOut, int VEC>
__global__ __launch_bounds__(kItemThreads) void k_fwd_items(const TIn* __restrict__ depth,
                                                            const TIn* __restrict__ feat,
                                                            TOut* __restrict__ out, SchedArgs a) {
  __shared__ PairMeta meta_all[kItemWaves][kMetaEntries];
  __shared__ float slot_a[kMaxGroups * VEC];  // first part of a cell continued from the previous group
  __shared__ float slot_b[kMaxGroups * VEC];  // last part of a cell continued in the next group
  __shared__ int32_t cell_a[kMaxGroups], cell_b[kMaxGroups], whole[kMaxGroups];

  // A schedule whose cell count does not match its plan is rejected (all
  // threads take the same branch).
  if (a.hdr[kHdrOccFound] != a.hdr[kHdrOcc]) return;
  // Workgroup b runs on die b % kXcds; it walks that die's item range.
  const int xcd = blockIdx.x % kXcds;
  const int slot = blockIdx.x / kXcds;
  const int slots = gridDim.x / kXcds;
  const int32_t item_end = min(a.xcd_begin[xcd + 1], a.hdr[kHdrItems]);
  for (int64_t item = a.xcd_begin[xcd] + slot; item < item_end; item += slots) {
  const int32_t n_pairs = a.hdr[kHdrPairs];
  const int32_t* info = a.item_info + 4 * item;
  const int32_t cb = max(0, min(info[0], a.n_occ));
  const int32_t ce = max(cb, min(info[1], a.n_occ));
  const int32_t pb = max(0, min(info[2], n_pairs));
  const int32_t pe = max(pb, min(info[3], n_pairs));
  const int32_t ic = a.item_chunk[item];
  const int chunk = ic & 0xffff, K = ic >> 16;

  const int C = a.C;
  int ch0 = 0, ch1 = C;
  if (K > 1 && a.units > 0) {
    ch0 = 16 * ((chunk * a.units) / K);
    ch1 = 16 * (((chunk + 1) * a.units) / K);
  }
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  PairMeta* meta = meta_all[wid];

  for (int sv = ch0 / VEC; sv < ch1 / VEC; sv += kWave) {
    const int cvc = min(kWave, ch1 / VEC - sv);
    const int G = kWave / cvc;
    const int g = lane / cvc;
    const int vi = lane - g * cvc;
    const bool in_group = g < G;
    const int q = wid * G + g;  // group index within the workgroup
    const int NG = kItemWaves * G;
    const int64_t col = (int64_t)(sv + vi) * VEC;

    // 1. zero-fill the gaps before the task's cells (and after the last cell)
    for (int32_t jb = cb + wid * kWave; jb < ce; jb += kItemWaves * kWave) {
      const int32_t j = jb + lane;
      int32_t c = -1, prev = -1;
      if (j < ce) {
        c = a.cell_id[j];
        prev = j > 0 ? a.cell_id[j - 1] : -1;
      }
      const bool last = (j == a.n_occ - 1);
      uint64_t todo = wave_ballot(j < ce && (prev + 1 < c || last));
      while (todo) {
        const int src = (int)__builtin_ctzll(todo);
        todo &= todo - 1;
        const int64_t kc = __shfl(c, src), kp = __shfl(prev, src);
        const int64_t r0 = max<int64_t>(kp + 1, 0), r1 = min<int64_t>(kc, a.cells);
        const int64_t gap = r1 > r0 ? (r1 - r0) * cvc : 0;
        for (int64_t idx = lane; idx < gap; idx += kWave)
          store_zero<TOut, VEC>(out + (r0 + idx / cvc) * C + (int64_t)(sv + idx % cvc) * VEC);
        if (jb + src == a.n_occ - 1) {
          const int64_t t0 = max<int64_t>(kc + 1, 0);
          const int64_t tail = a.cells > t0 ? (a.cells - t0) * cvc : 0;
          for (int64_t idx = lane; idx < tail; idx += kWave)
            store_zero<TOut, VEC>(out + (t0 + idx / cvc) * C + (int64_t)(sv + idx % cvc) * VEC);
        }
      }
    }

    // 2. stream the pairs
    const int32_t L = (pe - pb + NG - 1) / NG;  // pairs per group
    const int32_t gs = in_group ? min(pb + q * L, pe) : pe;
    const int32_t ge = in_group ? min(gs + L, pe) : pe;
    const int32_t prev_c = (gs > pb && gs < ge) ? a.pair_cell[gs - 1] : -1;
    const int32_t next_c = (ge < pe && gs < ge) ? a.pair_cell[ge] : -1;
    if (in_group && vi == 0) {
      cell_a[q] = -1;
      cell_b[q] = -1;
      whole[q] = (gs < ge && prev_c >= 0 && prev_c == next_c) ? 1 : 0;
    }

    float acc0[VEC], acc1[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc0[e] = acc1[e] = 0.f;
    int32_t cur = -2;
    auto flush = [&]() {
      float s[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        s[e] = acc0[e] + acc1[e];
        acc0[e] = acc1[e] = 0.f;
      }
      if (cur == prev_c) {
        Vec<float, VEC>::store(slot_a + (q * cvc + vi) * VEC, s);
        if (vi == 0) cell_a[q] = cur;
      } else if (cur == next_c) {
        Vec<float, VEC>::store(slot_b + (q * cvc + vi) * VEC, s);
        if (vi == 0) cell_b[q] = cur;
      } else if (cur >= 0 && cur < a.cells) {
        Vec<TOut, VEC>::store(out + (int64_t)cur * C + col, s);
      }
    };

    const int RM = kMetaEntries / G;  // staged pairs per group and round
    const int rounds = (L + RM - 1) / RM;
    const TIn* fbase = feat + col;
    for (int r = 0; r < rounds; ++r) {
      // stage (weight, row, cell) of every group's next RM pairs of this wave:
      // two entries per lane, records of both loaded before their depth scores
      static_assert(kMetaEntries == 2 * kWave, "two staged entries per lane");
      int64_t rd0[2];
      int32_t cellv[2], npts[2];
      bool live[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = lane + h * kWave;
        const int gg = e / RM;
        const int32_t gq = wid * G + gg;
        const int32_t gbeg = min(pb + gq * L, pe);
        const int32_t gend = min(gbeg + L, pe);
        const int32_t pr = gbeg + r * RM + (e - gg * RM);
        live[h] = e < G * RM && pr < gend;
        rd0[h] = -1;
        cellv[h] = -1;
        npts[h] = 0;
        if (live[h]) {
          rd0[h] = a.pair_rd0[pr];
          cellv[h] = a.pair_cell[pr];
          npts[h] = a.pair_npts[pr];
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = lane + h * kWave;
        PairMeta m;
        m.w = 0.f;
        m.row = 0;
        m.cell = cellv[h];
        const int64_t r0 = rd0[h];
        const int32_t n = npts[h];
        if (live[h] && r0 >= 0 && n > 0 && r0 + (int64_t)(n - 1) * a.hw < a.P) {
          float w = 0.f;
          for (int32_t t = 0; t < n; t += 4) {
            float dd[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
              dd[u] = (t + u < n) ? to_float(depth[r0 + (int64_t)(t + u) * a.hw]) : 0.f;
            w += (dd[0] + dd[1]) + (dd[2] + dd[3]);
          }
          m.w = w;
          m.row = (int32_t)((r0 / a.per_view) * a.hw + r0 % a.hw);
        }
        if (e < G * RM) meta[e] = m;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

      const int k_begin = g * RM;
      const int k_end = k_begin + (in_group ? max(0, min(RM, ge - (gs + r * RM))) : 0);
      if (k_end > k_begin) {
        // Double-buffered stream: the loads of the next half-batch are in
        // flight while the current one is consumed.  Entries past k_end read a
        // clamped, valid metadata slot and contribute weight 0.
        constexpr int UH = ((kRowRegs / VEC) < 16 ? (kRowRegs / VEC) : 16) / 2;
        float wa[UH], wb[UH];
        int32_t ca[UH], cb[UH];
        float va[UH][VEC], vb[UH][VEC];
        auto issue = [&](float* w, int32_t* c, float (*v)[VEC], int kk) {
#pragma unroll
          for (int u = 0; u < UH; ++u) {
            const int k = kk + u;
            const PairMeta m = meta[min(k, k_end - 1)];
            const bool ok = k < k_end;
            w[u] = ok ? m.w : 0.f;
            c[u] = ok ? m.cell : -1;
            Vec<TIn, VEC>::load(fbase + (int64_t)(ok ? m.row : 0) * C, v[u]);
          }
        };
        auto consume = [&](const float* w, const int32_t* c, const float (*v)[VEC], int kk) {
#pragma unroll
          for (int u = 0; u < UH; ++u) {
            if (kk + u < k_end && c[u] != cur) {
              if (cur != -2) flush();
              cur = c[u];
            }
            float* acc = (u & 1) ? acc1 : acc0;
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] = fmaf(w[u], v[u][e], acc[e]);
          }
        };
        issue(wa, ca, va, k_begin);
        for (int k0 = k_begin; k0 < k_end; k0 += 2 * UH) {
          issue(wb, cb, vb, k0 + UH);
          consume(wa, ca, va, k0);
          if (k0 + 2 * UH < k_end) issue(wa, ca, va, k0 + 2 * UH);
          consume(wb, cb, vb, k0 + UH);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (in_group && cur != -2) flush();
    __syncthreads();

    // 3. cells cut by group boundaries: the group holding the first part adds
    // the following groups' parts in order and stores the cell once.
    if (in_group && cell_b[q] >= 0) {
      const int32_t cell = cell_b[q];
      float s[VEC], t[VEC];
      Vec<float, VEC>::load(slot_b + (q * cvc + vi) * VEC, s);
      for (int rq = q + 1; rq < NG && cell_a[rq] == cell; ++rq) {
        Vec<float, VEC>::load(slot_a + (rq * cvc + vi) * VEC, t);
#pragma unroll
        for (int e = 0; e < VEC; ++e) s[e] += t[e];
        if (!whole[rq]) break;
      }
      if (cell < a.cells) Vec<TOut, VEC>::store(out + (int64_t)cell * C + col, s);
    }
    __syncthreads();
  }
  }  // item loop
}

template <typename TOut, int VEC>
__global__ __launch_bounds__(256) void k_zero_all(TOut* __restrict__ out, int64_t nvec) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nvec) store_zero<TOut, VEC>(out + i * VEC);
}

// Workgroups that fit on the device at once, rounded to whole dies.
template <typename TIn, typename TOut, int VEC>
int resident_items() {
  static int cached[64];  // per device; 0 = not yet queried
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_fwd_items<TIn, TOut, VEC>,
                                                    kItemThreads, 0) != hipSuccess ||
      per_cu <= 0)
    per_cu = 1;
  int blocks = cus * per_cu;
  blocks = ((blocks + kXcds - 1) / kXcds) * kXcds;
  cached[dev] = blocks;
  return blocks;
}

template <typename TIn, typename TOut, int VEC>
hipError_t run(const Dims& d, const void* depth, const void* feat, const SchedArgs& a,
               void* out, hipStream_t stream) {
  TOut* o = static_cast<TOut*>(out);
  if (a.n_occ == 0 || a.n_valid == 0) {
    const int64_t nvec = d.cells * (d.C / VEC);
    k_zero_all<TOut, VEC><<<dim3((unsigned)((nvec + 255) / 256)), dim3(256), 0, stream>>>(o, nvec);
    return hipGetLastError();
  }
  const int blocks = resident_items<TIn, TOut, VEC>();
  k_fwd_items<TIn, TOut, VEC><<<dim3((unsigned)blocks), dim3(kItemThreads), 0, stream>>>(
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
  SchedArgs a;
  a.hdr = S(L.header);
  a.pair_rd0 = S(L.pair_rd0);
  a.pair_cell = S(L.pair_cell);
  a.pair_npts = S(L.pair_npts);
  a.cell_id = S(L.cell_id);
  a.item_info = S(L.item_info);
  a.item_chunk = S(L.item_chunk);
  a.xcd_begin = S(L.xcd_begin);
  a.n_occ = n_intervals;
  a.n_valid = n_valid;
  a.C = (int32_t)d.C;
  a.units = (d.C % 16 == 0) ? (int32_t)(d.C / 16) : 0;
  a.cells = d.cells;
  a.P = d.P;
  a.rows = d.rows;
  a.hw = d.hw;
  a.per_view = d.per_view;
  const bool al = aligned16(feat) && aligned16(out);
  if (in_dtype == BEVPOOL_F32) {
    if (al && d.C % 4 == 0) return run<float, float, 4>(d, depth, feat, a, out, stream);
    return run<float, float, 1>(d, depth, feat, a, out, stream);
  }
  if (out_dtype == BEVPOOL_F16) {
    if (al && d.C % 8 == 0) return run<half_t, half_t, 8>(d, depth, feat, a, out, stream);
    return run<half_t, half_t, 1>(d, depth, feat, a, out, stream);
  }
  if (al && d.C % 8 == 0) return run<half_t, float, 8>(d, depth, feat, a, out, stream);
  return run<half_t, float, 1>(d, depth, feat, a, out, stream);
}

}  // namespace bevpool
