// Prefetch and eviction priorities (Section 4.5).
//
//   PRI^prefetch_{l,j} = p_{l,j} / (l - l_now)   experts of the query's
//                                                 prefetch set, layers l > l_now
//   PRI^evict_{l,j}    = 1 / (p_{l,j} freq_{l,j}) cached experts
//
// with p the query's guiding probabilities (as for the selection).  One
// workgroup per query: the candidates' priorities are computed in float64,
// rounded to float32 and packed with their expert index into 64-bit keys
// (priority order, then the lower l * E + j; NaN last), collected in LDS and
// placed by counting the keys above each one (up to 1024 candidates) or by a
// bitonic sort, then written out in that order.
#include "fm_device.h"
#include "fm_guide.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kPriThreads = 256;
constexpr int kPriMax = kMaxL * kMaxE;   // candidates per query at most
constexpr int kCountMax = 1024;          // up to this many candidates are ranked by counting

struct PriArgs {
  GuideView gv;
  int32_t L, E;
  const int32_t* idx;
  const float* score;
  int32_t B, k, blend, kind;
  const uint64_t* masks;   // PREFETCH: [B][L]; EVICT: [L]
  const int32_t* l_now;    // [B] (PREFETCH)
  const float* freq;       // [L][E] (EVICT)
  int32_t cap;
  int32_t* order_out;      // [B][cap]
  float* pri_out;          // [B][cap]
  int32_t* count_out;      // [B]
  uint32_t* flags;
};

// Order-preserving map of a float32 to uint32 (NaN -> 0, below every number;
// -0 and +0 equal).
__device__ __forceinline__ uint32_t ord_value(float s) {
  if (s != s) return 0u;
  s = s + 0.0f;
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace

__global__ void __launch_bounds__(kPriThreads) k_priority(PriArgs a) {
  constexpr int kPer = kPriMax / kPriThreads;   // (layer, expert) slots per thread
  __shared__ uint64_t keys[kPriMax];
  __shared__ uint64_t sets[kMaxL];
  __shared__ int n_cand;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int32_t* idx_b = a.idx + static_cast<int64_t>(b) * a.k;
  const float* score_b = a.score + static_cast<int64_t>(b) * a.k;
  // the match, the current layer and the layer's set load together
  const int y0 = idx_b[0];
  const int lnow = a.kind == FM_PRI_PREFETCH ? a.l_now[b] : 0;
  uint64_t bits = 0ull;
  if (tid < a.L) bits = a.kind == FM_PRI_PREFETCH ? a.masks[static_cast<int64_t>(b) * a.L + tid] : a.masks[tid];
  bool live = y0 >= 0;
  if (live && y0 >= a.gv.n) {
    if (tid == 0) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_INDEX_RANGE));
    live = false;
  }
  if (tid == 0) n_cand = 0;
  // the candidate sets of every layer (none after a missing match)
  if (tid < a.L) sets[tid] = live && (a.kind != FM_PRI_PREFETCH || tid > lnow) ? bits : 0ull;
  __syncthreads();
  // slot i = l * 64 + j: every probability load of this thread goes out
  // before any priority is ranked
  bool is[kPer];
  double pv[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + u * kPriThreads;
    const int l = i / kMaxE;
    const int j = i % kMaxE;
    is[u] = l < a.L && j < a.E && ((sets[l] >> j) & 1ull) != 0;
    pv[u] = is[u] ? guide_prob(a.gv, idx_b, score_b, a.k, a.blend, l, j) : 0.0;
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    if (!is[u]) continue;
    const int i = tid + u * kPriThreads;
    const int l = i / kMaxE;
    const int j = i % kMaxE;
    double v;
    if (a.kind == FM_PRI_PREFETCH) {
      v = __ddiv_rn(pv[u], static_cast<double>(l - lnow));
    } else {
      const double prod = __dmul_rn(pv[u], static_cast<double>(a.freq[l * a.E + j]));
      v = __ddiv_rn(1.0, prod);
    }
    const uint32_t e = static_cast<uint32_t>(l * a.E + j);
    const uint64_t key = (static_cast<uint64_t>(ord_value(static_cast<float>(v))) << 32) | static_cast<uint32_t>(~e);
    keys[atomicAdd(&n_cand, 1)] = key;
  }
  __syncthreads();
  const int N = n_cand;
  if (N <= kCountMax) {
    // rank by counting: a candidate's place is the number of keys above its
    // own (keys are distinct), read from LDS as broadcasts
    constexpr int kOwn = kCountMax / kPriThreads;
    uint64_t mine[kOwn];
    int rank[kOwn];
#pragma unroll
    for (int u = 0; u < kOwn; ++u) {
      mine[u] = tid + u * kPriThreads < N ? keys[tid + u * kPriThreads] : 0ull;
      rank[u] = 0;
    }
    for (int i = 0; i < N; ++i) {
      const uint64_t x = keys[i];
#pragma unroll
      for (int u = 0; u < kOwn; ++u) rank[u] += x > mine[u] ? 1 : 0;
    }
#pragma unroll
    for (int u = 0; u < kOwn; ++u) {
      if (tid + u * kPriThreads >= N || rank[u] >= a.cap) continue;
      const int64_t o = static_cast<int64_t>(b) * a.cap + rank[u];
      a.order_out[o] = static_cast<int32_t>(~static_cast<uint32_t>(mine[u]));
      a.pri_out[o] = unord_score(static_cast<uint32_t>(mine[u] >> 32));
    }
    for (int i = N + tid; i < a.cap; i += kPriThreads) {
      const int64_t o = static_cast<int64_t>(b) * a.cap + i;
      a.order_out[o] = -1;
      a.pri_out[o] = -__builtin_inff();
    }
    if (tid == 0) a.count_out[b] = N;
    return;
  }
  int P = 1;
  while (P < N) P <<= 1;
  for (int i = N + tid; i < P; i += kPriThreads) keys[i] = 0ull;   // padding ranks below everything
  __syncthreads();
  // bitonic sort, descending
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size / 2; stride > 0; stride >>= 1) {
      for (int i = tid; i < P / 2; i += kPriThreads) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const uint64_t x = keys[lo], y = keys[hi];
        const bool desc = (lo & size) == 0;
        if (desc ? (x < y) : (x > y)) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      __syncthreads();
    }
  }
  for (int i = tid; i < a.cap; i += kPriThreads) {
    const int64_t o = static_cast<int64_t>(b) * a.cap + i;
    if (i < N) {
      const uint64_t key = keys[i];
      a.order_out[o] = static_cast<int32_t>(~static_cast<uint32_t>(key));
      a.pri_out[o] = unord_score(static_cast<uint32_t>(key >> 32));
    } else {
      a.order_out[o] = -1;
      a.pri_out[o] = -__builtin_inff();
    }
  }
  if (tid == 0) a.count_out[b] = N;
}

hipError_t launch_priority(const StoreView& s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                           int32_t blend, int32_t kind, const uint64_t* masks, const int32_t* l_now,
                           const float* freq, int32_t cap, int32_t* order_out, float* pri_out, int32_t* count_out,
                           hipStream_t st) {
  PriArgs a;
  a.gv = GuideView{s.planes, s.plane_elems, s.n, s.row, s.map_dtype};
  a.L = s.L;
  a.E = s.E;
  a.idx = idx;
  a.score = score;
  a.B = B;
  a.k = k;
  a.blend = blend;
  a.kind = kind;
  a.masks = masks;
  a.l_now = l_now;
  a.freq = freq;
  a.cap = cap;
  a.order_out = order_out;
  a.pri_out = pri_out;
  a.count_out = count_out;
  a.flags = s.flags;
  hipLaunchKernelGGL(k_priority, dim3(B), dim3(kPriThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace fm
