// Expert Map Store deduplication (Section 4.4).
//
// Once the store is full, every new iteration x replaces the stored
// iteration y it is most redundant with,
//     RDY[x][y] = (d/L) score_sem[x][y] + ((L-d)/L) score_traj[x][y],
// with score_sem the Eq. 4 cosine of the embeddings and score_traj the Eq. 5
// cosine over all L layers, both from the semantic and trajectory scan
// kernels in their dense-output form (same arithmetic as the match calls).
// The trajectory scan writes its scores, the semantic scan reads them in its
// epilogue and writes the dense RDY matrix (weighted in float64, rounded once
// to float32); with d = 0 or d = L only one scan runs and its scores are RDY.
// Then
//   k_rdy_partial   the 8 best y of each chunk of a row of RDY as packed
//                   keys (RDY descending, y ascending, NaN last);
//   k_finalize      (shared with the scans) merges the chunks of a row into
//                   its 8 best candidates;
//   k_dedup_assign  one wavefront takes the new iterations in batch order
//                   (64 at a time, one per lane): each takes its first
//                   candidate not yet taken by an earlier one (the highest
//                   remaining RDY); if all 8 are taken it rescans its whole
//                   row, skipping taken entries;
//   k_insert_*      (store kernels) write every new iteration to its slot.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kCand = 8;         // candidates kept per new iteration
constexpr int kHashSlots = 4096;  // taken-set table (at most kChunkB entries)

struct RdyArgs {
  const float* rdy;    // [m][size] dense RDY
  int32_t size;        // stored iterations y in [0, size)
  int32_t m;           // new iterations (rows)
  int32_t R;           // chunks per row
  int32_t per;         // y per chunk, a multiple of 256 * kUnroll
  uint64_t* partial;   // [m][R][kCand] packed keys
};

constexpr int kUnroll = 8;   // RDY values loaded per thread before they are ranked (sort8_desc)

__global__ void __launch_bounds__(256) k_rdy_partial(RdyArgs a) {
  __shared__ uint64_t lists[256 / kWave][kCand];
  const int r = blockIdx.y;
  const int rr = blockIdx.x;
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int lo = rr * a.per;
  const int hi = lo + a.per < a.size ? lo + a.per : a.size;
  const float* row = a.rdy + static_cast<int64_t>(r) * a.size;
  TopK<kCand> t;
  t.clear();
  // batches of 8 values per thread: loaded together, sorted by a network and
  // merged into the thread's list
  for (int y0 = lo + static_cast<int>(threadIdx.x); y0 < hi; y0 += 256 * kUnroll) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int y = y0 + 256 * u;
      v[u] = y < hi ? row[y] : 0.0f;
    }
    uint64_t keys[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int y = y0 + 256 * u;
      keys[u] = y < hi ? make_key(v[u], y) : 0ull;
    }
    sort8_desc(keys);
    t.merge(keys);
  }
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
  const float* rdy;      // [m][size] dense RDY
  int32_t size;          // stored iterations before the batch
  int32_t n_app;         // new iterations appended at size, size + 1, ...
  int32_t m;             // new iterations that replace a stored one
  int32_t* slots;        // [n_app + m]
  int32_t* slots_out;    // caller's copy, or null
};

// Insert y into the taken set by one lane among several inserting distinct
// values at once (compare-and-swap on the empty slot).
__device__ __forceinline__ void taken_add_concurrent(int32_t* set, int32_t y) {
  for (int h = hash_slot(y);; h = (h + 1) & (kHashSlots - 1))
    if (atomicCAS(&set[h], -1, y) == -1) return;
}

constexpr int kPropSlots = 2 * kWave;   // proposals of one round (at most kWave)

// The new iterations in batch order, 64 at a time (lane = iteration), one
// wavefront.  Each lane's choice is its first candidate not taken by an
// earlier iteration; a choice can only be changed by an earlier iteration of
// the same chunk taking that very candidate (its earlier candidates are
// taken already).  So a chunk is resolved in rounds: every unresolved lane
// proposes its first candidate left; the lanes before the first one whose
// proposal an earlier lane also made keep their proposals (distinct, and
// each still its first candidate left), their picks join the taken set, and
// the next round starts at that lane.  A lane with no candidate left, once
// every earlier lane is resolved, rescans its whole RDY row against the
// taken set.  The result is the greedy assignment in batch order.
__global__ void __launch_bounds__(kWave) k_dedup_assign(AssignArgs a) {
  __shared__ int32_t taken[kHashSlots];
  __shared__ int32_t pkey[kPropSlots];   // a round's proposals (open addressing)
  __shared__ int32_t pmin[kPropSlots];   // the lowest lane proposing each
  const int lane = threadIdx.x;
  for (int i = lane; i < kHashSlots; i += kWave) taken[i] = -1;
  for (int i = lane; i < a.n_app; i += kWave) {
    a.slots[i] = a.size + i;
    if (a.slots_out != nullptr) a.slots_out[i] = a.size + i;
  }
  __syncthreads();
  for (int c0 = 0; c0 < a.m; c0 += kWave) {
    const int r = c0 + lane;
    const int nl = a.m - c0 < kWave ? a.m - c0 : kWave;
    int32_t cd[kCand];
#pragma unroll
    for (int j = 0; j < kCand; ++j) cd[j] = (r < a.m && a.size > 0) ? a.cand[static_cast<int64_t>(r) * kCand + j] : -1;
    // candidates not taken by earlier chunks
    uint32_t avail = 0;
#pragma unroll
    for (int j = 0; j < kCand; ++j)
      if (cd[j] >= 0 && !taken_has(taken, cd[j])) avail |= 1u << j;
    int32_t pick = -1;
    int lo = 0;   // lanes below lo are resolved, their picks in the taken set
    while (a.size > 0 && lo < nl) {
      const bool live = lane >= lo && lane < nl;
      int32_t prop = -1;   // first candidate left
#pragma unroll
      for (int j = kCand - 1; j >= 0; --j) prop = ((avail >> j) & 1u) ? cd[j] : prop;
      const uint64_t none = __ballot(live && avail == 0);
      const int tr = none != 0 ? static_cast<int>(__builtin_ctzll(none)) : nl;
      // the lowest lane of [lo, tr) proposing each value
      pkey[lane] = -1;
      pkey[lane + kWave] = -1;
      pmin[lane] = kWave;
      pmin[lane + kWave] = kWave;
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_wave_barrier();
      const bool prop_here = lane >= lo && lane < tr;
      int h = 0;
      if (prop_here) {
        h = static_cast<int>((static_cast<uint32_t>(prop) * 2654435761u) >> 25) & (kPropSlots - 1);
        for (;;) {
          const int32_t old = atomicCAS(&pkey[h], -1, prop);
          if (old == -1 || old == prop) break;
          h = (h + 1) & (kPropSlots - 1);
        }
        atomicMin(&pmin[h], lane);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_wave_barrier();
      const uint64_t lose = __ballot(prop_here && pmin[h] != lane);
      const int T = lose != 0 ? static_cast<int>(__builtin_ctzll(lose)) : tr;
      if (lane >= lo && lane < T) {
        pick = prop;
        taken_add_concurrent(taken, prop);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_wave_barrier();
      if (T == tr && tr < nl) {
        // every candidate of iteration c0 + tr is taken: rescan its row
        uint64_t best = 0;
        const float* row = a.rdy + static_cast<int64_t>(c0 + tr) * a.size;
        for (int yy = lane; yy < a.size; yy += kWave) {
          if (taken_has(taken, yy)) continue;
          const uint64_t key = make_key(row[yy], yy);
          best = key > best ? key : best;
        }
#pragma unroll
        for (int m = 1; m < kWave; m <<= 1) {
          const uint64_t o = shfl_xor_u64(best, m);
          best = o > best ? o : best;
        }
        const int32_t choice = key_index(best);
        if (lane == tr) {
          pick = choice;
          if (choice >= 0) taken_add(taken, choice);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_wave_barrier();
        lo = tr + 1;
      } else {
        lo = T;
      }
      // the lanes still to resolve drop their candidates taken meanwhile
      if (lane >= lo && lane < nl) {
#pragma unroll
        for (int j = 0; j < kCand; ++j)
          if (((avail >> j) & 1u) && taken_has(taken, cd[j])) avail &= ~(1u << j);
      }
    }
    if (r < a.m) {
      a.slots[a.n_app + r] = pick;
      if (a.slots_out != nullptr) a.slots_out[a.n_app + r] = pick;
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
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
  d.rdy = reinterpret_cast<float*>(p);
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
      // trajectory scores alone are RDY when d = 0
      err = launch_match_trajectory(s, q, sc.depth, s.L, m, 1, nullptr, nullptr, w_sem > 0.0 ? sc.traj : sc.rdy,
                                    ws, st);
      if (err != hipSuccess) return err;
    }
    if (w_sem > 0.0) {
      const uint16_t* q = static_cast<const uint16_t*>(embs) + static_cast<int64_t>(n_app) * s.d_emb;
      err = w_traj > 0.0 ? launch_match_semantic(s, q, m, 1, nullptr, nullptr, sc.rdy, ws, st, sc.traj, w_sem, w_traj)
                         : launch_match_semantic(s, q, m, 1, nullptr, nullptr, sc.rdy, ws, st);
      if (err != hipSuccess) return err;
    }
    RdyArgs ra;
    ra.rdy = sc.rdy;
    ra.size = size;
    ra.m = m;
    // chunks of 16384 stored iterations (a multiple of 256 * kUnroll), at
    // most kMaxPartials per row
    constexpr int kStep = 256 * kUnroll;
    int per = 16384;
    int R = (size + per - 1) / per;
    if (R > kMaxPartials) {
      R = kMaxPartials;
      per = ((size + R - 1) / R + kStep - 1) / kStep * kStep;
      R = (size + per - 1) / per;
    }
    ra.R = R;
    ra.per = per;
    ra.partial = ws.partial;
    hipLaunchKernelGGL(k_rdy_partial, dim3(R, m), dim3(256), 0, st, ra);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    err = launch_finalize(ws.partial, nullptr, m, R, kCand, kCand, sc.cand, sc.cand_score, st);
    if (err != hipSuccess) return err;
  }

  AssignArgs aa;
  aa.cand = sc.cand;
  aa.rdy = sc.rdy;
  aa.size = size;
  aa.n_app = n_app;
  aa.m = m;
  aa.slots = sc.slots;
  aa.slots_out = slots_out;
  hipLaunchKernelGGL(k_dedup_assign, dim3(1), dim3(kWave), 0, st, aa);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_insert(s, maps, embs, n, sc.slots, nullptr, st);
}

}  // namespace fm
