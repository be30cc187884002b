// Similarity-aware prefetch-set selection (Section 4.3, Eq. 6-8).
//
// One wavefront per (query, layer) row; lane j holds expert j (E <= 64).
//   1. Guiding probabilities: the matched map's row (float64 widening of the
//      stored value), or the similarity-weighted mean of the kept matches'
//      rows, summed in match order with explicit float64 roundings.
//   2. Threshold: fixed tau, or delta = Clip(1 - score, 0, 1).
//   3. Rank of lane j = experts ahead of it in (probability descending,
//      index ascending) order; NaN probabilities rank last.
//   4. The running sum over that order is taken sequentially in float64; k*
//      is the first prefix reaching the threshold (E if none), clamped to
//      [k_min, k_max]; the mask is the ballot of lanes with rank < k.
#include "fm_device.h"
#include "fm_guide.h"
#include "fm_internal.h"

namespace fm {

namespace {

struct SelArgs {
  const void* planes;
  int64_t plane_elems;
  int32_t n, L, E, row;
  fm_dtype dtype;
  const int32_t* idx;
  const float* score;
  int32_t B, k;
  const int32_t* lb;
  const int32_t* le;
  int32_t mode;
  float tau;
  int32_t k_min, k_max, blend;
  uint64_t* mask_out;
  uint8_t* count_out;
  uint32_t* flags;
};

// (p_i, i) is ahead of (p_j, j): larger probability, or equal and lower index;
// NaN is behind every number and NaNs keep index order.
__device__ __forceinline__ bool ahead(double pi, int i, double pj, int j) {
  const bool ni = pi != pi, nj = pj != pj;
  if (ni || nj) return (!ni && nj) || (ni && nj && i < j);
  return pi > pj || (pi == pj && i < j);
}

}  // namespace

// Ordered 64-bit key of a float64 probability: larger value -> larger key,
// -0 and +0 equal, NaN lowest (key 0).  Ranking by (key desc, index asc) is
// the (p desc, j asc, NaN last) order of ahead().
__device__ __forceinline__ uint64_t ord_f64(double p) {
  if (p != p) return 0ull;
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(p + 0.0));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// The selection of row (b, l) of the batch from the query's matches idx_b /
// score_b (k of them, best first) and its layer bounds lb[b] / le[b] (as
// given; clamped here); one wavefront, lane j = expert j.
__device__ __forceinline__ void select_row(const SelArgs& a, int b, int l, int lo, int hi, const int32_t* idx_b,
                                           const float* score_b, double* sorted, uint64_t* keys) {
  const int lane = threadIdx.x % kWave;
  const int64_t row = static_cast<int64_t>(b) * a.L + l;
  lo = lo < 0 ? 0 : (lo > a.L ? a.L : lo);
  hi = hi < 0 ? 0 : (hi > a.L ? a.L : hi);
  const int y0 = idx_b[0];

  // 1. guiding probability of expert `lane`: its loads need only the
  // matches, so they are issued before the row's bounds are looked at (a
  // row outside them discards the value)
  const GuideView gv{a.planes, a.plane_elems, a.n, a.row, a.dtype};
  double p = 0.0;
  if (lane < a.E && y0 >= 0 && y0 < a.n) p = guide_prob(gv, idx_b, score_b, a.k, a.blend, l, lane);

  bool live = l >= lo && l < hi && y0 >= 0;
  if (live && y0 >= a.n) {
    if (lane == 0) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_INDEX_RANGE));
    live = false;
  }
  if (!live) {
    if (lane == 0) {
      a.mask_out[row] = 0ull;
      a.count_out[row] = 0;
    }
    return;
  }

  // 2. threshold
  double tau;
  if (a.mode == FM_TAU_DYNAMIC) {
    const double s = static_cast<double>(score_b[0]);
    if (s != s) tau = 1.0;
    else {
      double t = 1.0 - s;
      tau = t < 0.0 ? 0.0 : (t > 1.0 ? 1.0 : t);
    }
  } else {
    tau = static_cast<double>(a.tau);
  }

  // 3. rank: every lane counts the experts ahead of its own, comparing
  // ordered integer keys read from LDS (broadcast reads, independent of
  // each other)
  const uint64_t key = ord_f64(p);
  if (lane < a.E) keys[lane] = key;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  int rank = 0;
#pragma unroll 8
  for (int i = 0; i < a.E; ++i) {
    const uint64_t ki = keys[i];
    rank += (ki > key || (ki == key && i < lane)) ? 1 : 0;
  }
  if (lane < a.E) sorted[rank] = p;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();

  // 4. sequential float64 prefix sum in rank order: k* is the first count
  // whose running sum reaches tau (E if none); values are read 8 at a time
  // ahead of the sequential adds
  int kstar = a.E;
  double run = 0.0;
  bool found = false;
  for (int k0 = 0; k0 < a.E && !found; k0 += 8) {
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = k0 + u < a.E ? sorted[k0 + u] : 0.0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (found || k0 + u >= a.E) break;
      if (run >= tau) {
        kstar = k0 + u;
        found = true;
        break;
      }
      run = __dadd_rn(run, v[u]);
    }
  }
  int kk = kstar < a.k_min ? a.k_min : kstar;
  kk = kk > a.k_max ? a.k_max : kk;
  const uint64_t mask = __ballot(lane < a.E && rank < kk);
  if (lane == 0) {
    a.mask_out[row] = mask;
    a.count_out[row] = static_cast<uint8_t>(kk);
  }
}

__global__ void __launch_bounds__(256) k_select(SelArgs a) {
  __shared__ double sorted[4][kMaxE];
  __shared__ uint64_t keys[4][kMaxE];
  const int wv = threadIdx.x / kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wv;
  if (row >= static_cast<int64_t>(a.B) * a.L) return;
  const int b = static_cast<int>(row / a.L);
  const int l = static_cast<int>(row - static_cast<int64_t>(b) * a.L);
  select_row(a, b, l, a.lb[b], a.le[b], a.idx + static_cast<int64_t>(b) * a.k, a.score + static_cast<int64_t>(b) * a.k,
             sorted[wv], keys[wv]);
}

// The cross-workgroup merge of a match call with the selection after it:
// one wavefront per (sorted position, layer) row merges the position's
// partial top-k lists (each of the row's L wavefronts on its own, so that no
// wave waits for another), the layer-0 one writes the query's matches, and
// every one selects its layer from the merged matches (staged in LDS).  The
// same merge as k_finalize and the same selection as k_select.
struct MergeArgs {
  const uint64_t* partial;   // [positions][R][KTOP]
  const int32_t* perm;       // query at each position (NULL: the position itself)
  int32_t R;                 // lists per position
  const int32_t* rgrp;       // lists per query group (NULL: R)
  int32_t qg;                // positions per query group
  int32_t* idx_out;          // [B][k]
  float* score_out;          // [B][k]
};

template <int KTOP>
__global__ void __launch_bounds__(256) k_merge_select(SelArgs a, MergeArgs m) {
  __shared__ double sorted[4][kMaxE];
  __shared__ uint64_t keys[4][kMaxE];
  __shared__ int32_t midx[4][kMaxK];
  __shared__ float mscore[4][kMaxK];
  const int lane = threadIdx.x % kWave;
  const int wv = threadIdx.x / kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wv;
  if (row >= static_cast<int64_t>(a.B) * a.L) return;
  const int pos = static_cast<int>(row / a.L);
  const int l = static_cast<int>(row - static_cast<int64_t>(pos) * a.L);
  // The loads that do not depend on the merge go first, side by side: the
  // group's list count, the query index (then its layer bounds) and, for
  // top-1 lists, the first kMaxPartials lists of the stride (those past the
  // group's count are read but not merged).
  const int nr = m.rgrp != nullptr ? m.rgrp[pos / m.qg] : m.R;
  const int b = m.perm != nullptr ? m.perm[pos] : pos;
  const uint64_t* plist = m.partial + static_cast<int64_t>(pos) * m.R * KTOP;
  TopK<KTOP> t;
  t.clear();
  int r0 = lane;
  if constexpr (KTOP == 1) {
    constexpr int kPre = kMaxPartials / kWave;
    uint64_t pk[kPre];
#pragma unroll
    for (int it = 0; it < kPre; ++it) pk[it] = lane + it * kWave < m.R ? plist[lane + it * kWave] : 0ull;
#pragma unroll
    for (int it = 0; it < kPre; ++it)
      if (lane + it * kWave < nr) t.merge(&pk[it]);
    r0 = lane + kMaxPartials;
  }
  const int lo = a.lb[b], hi = a.le[b];
  for (int r = r0; r < nr; r += kWave) t.merge(plist + static_cast<int64_t>(r) * KTOP);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint64_t o[KTOP];
#pragma unroll
    for (int jj = 0; jj < KTOP; ++jj) o[jj] = shfl_xor_u64(t.v[jj], off);
    t.merge(o);
  }
  if (lane == 0) {
#pragma unroll
    for (int jj = 0; jj < kMaxK; ++jj) {
      if (jj >= a.k) break;
      const uint64_t key = jj < KTOP ? t.v[jj < KTOP ? jj : 0] : 0ull;
      midx[wv][jj] = key_index(key);
      mscore[wv][jj] = key_score(key);
      if (l == 0) {
        m.idx_out[static_cast<int64_t>(b) * a.k + jj] = key_index(key);
        m.score_out[static_cast<int64_t>(b) * a.k + jj] = key_score(key);
      }
    }
  }
  // (LDS only: the bounds' loads stay in flight)
  wait_lgkm0();
  __builtin_amdgcn_wave_barrier();
  select_row(a, b, l, lo, hi, midx[wv], mscore[wv], sorted[wv], keys[wv]);
}

// Misses of the prefetch sets (Section 3): one wavefront per (query, layer)
// row; lane j ranks expert j of the query's own gate probabilities among the
// row (the same order as the selection), the K best are the activated
// experts, and the count of those outside the set is written.
struct MissArgs {
  const void* q;           // [B][L][E] of the map dtype
  fm_dtype dtype;
  int32_t B, L, E, K;
  const uint64_t* masks;   // [B][L]
  const int32_t* lb;
  const int32_t* le;
  uint8_t* miss_out;       // [B][L]
};

__global__ void __launch_bounds__(256) k_miss(MissArgs a) {
  __shared__ float vals[4][kMaxE];
  const int lane = threadIdx.x % kWave;
  const int wv = threadIdx.x / kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wv;
  if (row >= static_cast<int64_t>(a.B) * a.L) return;
  const int b = static_cast<int>(row / a.L);
  const int l = static_cast<int>(row - static_cast<int64_t>(b) * a.L);
  int lo = a.lb[b], hi = a.le[b];
  lo = lo < 0 ? 0 : (lo > a.L ? a.L : lo);
  hi = hi < 0 ? 0 : (hi > a.L ? a.L : hi);
  if (l < lo || l >= hi) {
    if (lane == 0) a.miss_out[row] = 0;
    return;
  }
  float p = 0.0f;
  if (lane < a.E) {
    const int64_t i = row * a.E + lane;
    p = a.dtype == FM_F32 ? static_cast<const float*>(a.q)[i] : bf16_to_f32(static_cast<const uint16_t*>(a.q)[i]);
    vals[wv][lane] = p;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  int rank = 0;
  for (int i = 0; i < a.E; ++i) {
    const float pi = vals[wv][i];
    if (i != lane && ahead(pi, i, p, lane)) ++rank;
  }
  const uint64_t act = __ballot(lane < a.E && rank < a.K);
  if (lane == 0) a.miss_out[row] = static_cast<uint8_t>(__popcll(act & ~a.masks[row]));
}

hipError_t launch_miss(const StoreView& s, const void* q, int32_t B, int32_t K, const uint64_t* masks,
                       const int32_t* lb, const int32_t* le, uint8_t* miss_out, hipStream_t st) {
  MissArgs a;
  a.q = q;
  a.dtype = s.map_dtype;
  a.B = B;
  a.L = s.L;
  a.E = s.E;
  a.K = K;
  a.masks = masks;
  a.lb = lb;
  a.le = le;
  a.miss_out = miss_out;
  const int64_t rows = static_cast<int64_t>(B) * s.L;
  hipLaunchKernelGGL(k_miss, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, st, a);
  return hipGetLastError();
}

namespace {

SelArgs select_args(const StoreView& s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                    const int32_t* lb, const int32_t* le, const fm_select_params& p, uint64_t* mask_out,
                    uint8_t* count_out) {
  SelArgs a;
  a.planes = s.planes;
  a.plane_elems = s.plane_elems;
  a.n = s.n;
  a.L = s.L;
  a.E = s.E;
  a.row = s.row;
  a.dtype = s.map_dtype;
  a.idx = idx;
  a.score = score;
  a.B = B;
  a.k = k;
  a.lb = lb;
  a.le = le;
  a.mode = p.mode;
  a.tau = p.tau;
  a.k_min = p.k_min;
  a.k_max = p.k_max;
  a.blend = p.blend;
  a.mask_out = mask_out;
  a.count_out = count_out;
  a.flags = s.flags;
  return a;
}

}  // namespace

hipError_t launch_select(const StoreView& s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                         const int32_t* lb, const int32_t* le, const fm_select_params& p, uint64_t* mask_out,
                         uint8_t* count_out, hipStream_t st) {
  const SelArgs a = select_args(s, idx, score, B, k, lb, le, p, mask_out, count_out);
  const int64_t rows = static_cast<int64_t>(B) * s.L;
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL(k_select, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_merge_select(const StoreView& s, const uint64_t* partial, const int32_t* perm, int32_t B, int32_t R,
                               int32_t k, int KTOP, const int32_t* rgrp, int32_t qg, int32_t* idx_out,
                               float* score_out, const SelectFuse& f, hipStream_t st) {
  const SelArgs a = select_args(s, nullptr, nullptr, B, k, f.lb, f.le, f.p, f.mask_out, f.count_out);
  MergeArgs m;
  m.partial = partial;
  m.perm = perm;
  m.R = R;
  m.rgrp = rgrp;
  m.qg = qg > 0 ? qg : 1;
  m.idx_out = idx_out;
  m.score_out = score_out;
  const int64_t rows = static_cast<int64_t>(B) * s.L;
  const dim3 grid(static_cast<unsigned>((rows + 3) / 4));
  if (KTOP == 1) hipLaunchKernelGGL(k_merge_select<1>, grid, dim3(256), 0, st, a, m);
  else if (KTOP == 4) hipLaunchKernelGGL(k_merge_select<4>, grid, dim3(256), 0, st, a, m);
  else hipLaunchKernelGGL(k_merge_select<8>, grid, dim3(256), 0, st, a, m);
  return hipGetLastError();
}

}  // namespace fm
