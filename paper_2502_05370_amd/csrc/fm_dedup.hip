// Expert Map Store deduplication (Section 4.4).
//
// Once the store is full, every new iteration x replaces the stored
// iteration y it is most redundant with,
//     RDY[x][y] = (d/L) score_sem[x][y] + ((L-d)/L) score_traj[x][y],
// with score_sem the Eq. 4 cosine of the embeddings and score_traj the Eq. 5
// cosine over all L layers.  The two score matrices come from the semantic
// and trajectory scan kernels in their dense-output form (same arithmetic
// as the match calls).  Then
//   k_rdy_partial   RDY of each (x, y), weighted in float64 and rounded once
//                   to float32, and the 8 best y of each chunk of a row as
//                   packed keys (RDY descending, y ascending, NaN last);
//   k_finalize      (shared with the scans) merges the chunks of a row into
//                   its 8 best candidates;
//   k_dedup_assign  one workgroup takes the new iterations in batch order:
//                   each takes its first candidate not yet taken by an
//                   earlier one (the highest remaining RDY); if all 8 are
//                   taken it rescans its whole row, skipping taken entries;
//   k_insert_*      (store kernels) write every new iteration to its slot.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kCand = 8;         // candidates kept per new iteration
constexpr int kHashSlots = 4096;  // taken-set table (at most kChunkB entries)

// RDY of one pair from the float32 scores; a term with weight 0 is not read.
__device__ __forceinline__ float rdy_value(const float* S, const float* T, int64_t off, double w_sem,
                                           double w_traj) {
  double r = 0.0;
  if (w_sem > 0.0) r = r + w_sem * static_cast<double>(S[off]);
  if (w_traj > 0.0) r = r + w_traj * static_cast<double>(T[off]);
  return static_cast<float>(r);
}

struct RdyArgs {
  const float* S;      // [m][ld] semantic scores (unused when w_sem == 0)
  const float* T;      // [m][ld] trajectory scores (unused when w_traj == 0)
  int64_t ld;          // row stride = number of stored iterations scored
  int32_t size;        // stored iterations y in [0, size)
  int32_t m;           // new iterations (rows)
  int32_t R;           // chunks per row
  int32_t per;         // y per chunk
  double w_sem, w_traj;
  uint64_t* partial;   // [m][R][kCand] packed keys
};

__global__ void __launch_bounds__(256) k_rdy_partial(RdyArgs a) {
  __shared__ uint64_t lists[256 / kWave][kCand];
  const int r = blockIdx.y;
  const int rr = blockIdx.x;
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int lo = rr * a.per;
  const int hi = lo + a.per < a.size ? lo + a.per : a.size;
  const int64_t row = static_cast<int64_t>(r) * a.ld;
  TopK<kCand> t;
  t.clear();
  for (int y = lo + static_cast<int>(threadIdx.x); y < hi; y += 256)
    t.push(make_key(rdy_value(a.S, a.T, row + y, a.w_sem, a.w_traj), y));
  // lanes l and l ^ m hold lists of disjoint lane groups before each merge
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    uint64_t o[kCand];
#pragma unroll
    for (int j = 0; j < kCand; ++j) o[j] = shfl_xor_u64(t.v[j], m);
    t.merge(o);
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < kCand; ++j) lists[w][j] = t.v[j];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    TopK<kCand> b;
    b.clear();
#pragma unroll
    for (int ww = 0; ww < 256 / kWave; ++ww) b.merge(lists[ww]);
    uint64_t* out = a.partial + (static_cast<int64_t>(r) * a.R + rr) * kCand;
#pragma unroll
    for (int j = 0; j < kCand; ++j) out[j] = b.v[j];
  }
}

// Open-addressing set of taken store indices in LDS.
__device__ __forceinline__ int hash_slot(int32_t y) {
  return static_cast<int>((static_cast<uint32_t>(y) * 2654435761u) >> 20) & (kHashSlots - 1);
}
__device__ __forceinline__ bool taken_has(const int32_t* set, int32_t y) {
  for (int h = hash_slot(y);; h = (h + 1) & (kHashSlots - 1)) {
    const int32_t v = set[h];
    if (v == y) return true;
    if (v < 0) return false;
  }
}
__device__ __forceinline__ void taken_add(int32_t* set, int32_t y) {
  int h = hash_slot(y);
  while (set[h] >= 0) h = (h + 1) & (kHashSlots - 1);
  set[h] = y;
}

struct AssignArgs {
  const int32_t* cand;   // [m][kCand] candidates in ranking order (-1: none)
  const float* S;
  const float* T;
  int64_t ld;
  double w_sem, w_traj;
  int32_t size;          // stored iterations before the batch
  int32_t n_app;         // new iterations appended at size, size + 1, ...
  int32_t m;             // new iterations that replace a stored one
  int32_t* slots;        // [n_app + m]
  int32_t* slots_out;    // caller's copy, or null
};

__global__ void __launch_bounds__(256) k_dedup_assign(AssignArgs a) {
  __shared__ int32_t taken[kHashSlots];
  __shared__ uint64_t red[256 / kWave];
  __shared__ int32_t pick;
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int w = tid / kWave;
  for (int i = tid; i < kHashSlots; i += 256) taken[i] = -1;
  for (int i = tid; i < a.n_app; i += 256) {
    a.slots[i] = a.size + i;
    if (a.slots_out != nullptr) a.slots_out[i] = a.size + i;
  }
  __syncthreads();
  for (int r = 0; r < a.m; ++r) {
    if (w == 0) {
      int32_t y = -1;
      bool ok = false;
      if (lane < kCand && a.size > 0) {
        y = a.cand[static_cast<int64_t>(r) * kCand + lane];
        ok = y >= 0 && !taken_has(taken, y);
      }
      const uint64_t bal = __ballot(ok);
      const int first = bal != 0 ? __builtin_ctzll(bal) : 0;
      const int32_t yf = __shfl(y, first, kWave);
      // -2: every candidate is taken, the row must be rescanned
      if (lane == 0) pick = bal != 0 ? yf : (a.size > 0 ? -2 : -1);
    }
    __syncthreads();
    if (pick == -2) {
      uint64_t best = 0;
      const int64_t row = static_cast<int64_t>(r) * a.ld;
      for (int y = tid; y < a.size; y += 256) {
        if (taken_has(taken, y)) continue;
        const uint64_t key = make_key(rdy_value(a.S, a.T, row + y, a.w_sem, a.w_traj), y);
        best = key > best ? key : best;
      }
#pragma unroll
      for (int m = 1; m < kWave; m <<= 1) {
        const uint64_t o = shfl_xor_u64(best, m);
        best = o > best ? o : best;
      }
      if (lane == 0) red[w] = best;
      __syncthreads();
      if (tid == 0) {
        uint64_t b = 0;
#pragma unroll
        for (int ww = 0; ww < 256 / kWave; ++ww) b = red[ww] > b ? red[ww] : b;
        pick = key_index(b);
      }
    }
    if (tid == 0) {
      const int32_t y = pick;
      if (y >= 0) taken_add(taken, y);
      a.slots[a.n_app + r] = y;
      if (a.slots_out != nullptr) a.slots_out[a.n_app + r] = y;
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(256) k_fill_i32(int32_t* p, int32_t n, int32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

DedupScratch carve_dedup_scratch(void* base, int32_t cap, int32_t n_max) {
  char* p = static_cast<char*>(base);
  DedupScratch d;
  d.depth = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * kChunkB, kAlign);
  d.slots = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * kChunkB, kAlign);
  d.cand = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * kChunkB * kCand, kAlign);
  d.cand_score = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * kChunkB * kCand, kAlign);
  const size_t dense = align_up(sizeof(float) * static_cast<size_t>(n_max) * static_cast<size_t>(cap), kAlign);
  d.sem = reinterpret_cast<float*>(p);
  p += dense;
  d.traj = reinterpret_cast<float*>(p);
  return d;
}

size_t dedup_scratch_bytes(int32_t cap, int32_t n_max) {
  size_t b = 2 * align_up(sizeof(int32_t) * kChunkB, kAlign);
  b += align_up(sizeof(int32_t) * kChunkB * kCand, kAlign) + align_up(sizeof(float) * kChunkB * kCand, kAlign);
  b += 2 * align_up(sizeof(float) * static_cast<size_t>(n_max) * static_cast<size_t>(cap), kAlign);
  return b;
}

hipError_t launch_insert_dedup(const StoreView& s, const void* maps, const void* embs, int32_t n, int32_t d,
                               int32_t* slots_out, const Workspace& ws, const DedupScratch& sc, hipStream_t st) {
  const int32_t size = s.n;
  const int32_t free_slots = s.cap - size;
  const int32_t n_app = n < free_slots ? n : free_slots;
  const int32_t m = n - n_app;
  const double w_sem = static_cast<double>(d) / static_cast<double>(s.L);
  const double w_traj = static_cast<double>(s.L - d) / static_cast<double>(s.L);
  hipError_t err = hipSuccess;

  if (m > 0 && size > 0) {
    const int esz = s.map_dtype == FM_BF16 ? 2 : 4;
    if (w_traj > 0.0) {
      hipLaunchKernelGGL(k_fill_i32, dim3((m + 255) / 256), dim3(256), 0, st, sc.depth, m, s.L);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
      const char* q = static_cast<const char*>(maps) + static_cast<int64_t>(n_app) * s.L * s.E * esz;
      err = launch_match_trajectory(s, q, sc.depth, s.L, m, 1, nullptr, nullptr, sc.traj, ws, st);
      if (err != hipSuccess) return err;
    }
    if (w_sem > 0.0) {
      const uint16_t* q = static_cast<const uint16_t*>(embs) + static_cast<int64_t>(n_app) * s.d_emb;
      err = launch_match_semantic(s, q, m, 1, nullptr, nullptr, sc.sem, ws, st);
      if (err != hipSuccess) return err;
    }
    RdyArgs ra;
    ra.S = sc.sem;
    ra.T = sc.traj;
    ra.ld = size;
    ra.size = size;
    ra.m = m;
    // chunks of at least 4096 stored iterations, at most kMaxPartials per row
    int R = (size + 4095) / 4096;
    if (R > kMaxPartials) R = kMaxPartials;
    ra.R = R;
    ra.per = (size + R - 1) / R;
    ra.w_sem = w_sem;
    ra.w_traj = w_traj;
    ra.partial = ws.partial;
    hipLaunchKernelGGL(k_rdy_partial, dim3(R, m), dim3(256), 0, st, ra);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    err = launch_finalize(ws.partial, nullptr, m, R, kCand, kCand, sc.cand, sc.cand_score, st);
    if (err != hipSuccess) return err;
  }

  AssignArgs aa;
  aa.cand = sc.cand;
  aa.S = sc.sem;
  aa.T = sc.traj;
  aa.ld = size;
  aa.w_sem = w_sem;
  aa.w_traj = w_traj;
  aa.size = size;
  aa.n_app = n_app;
  aa.m = m;
  aa.slots = sc.slots;
  aa.slots_out = slots_out;
  hipLaunchKernelGGL(k_dedup_assign, dim3(1), dim3(256), 0, st, aa);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_insert(s, maps, embs, n, sc.slots, nullptr, st);
}

}  // namespace fm
