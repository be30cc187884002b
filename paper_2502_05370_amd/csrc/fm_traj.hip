// Trajectory-based expert map search (Section 4.2.2, Eq. 5).
//
// Query b has observed the gate distributions of its first p_b layers; its
// score against stored iteration y is the cosine between the flattened
// prefixes q[b][0:p_b] and x[y][0:p_b].  All B queries of a batch are served
// by one pass over the store:
//
//   k_traj_prep  sorts the queries by depth (descending, stable), computes
//                1/|q[b][0:p_b]| in float64 and clears the result keys.
//   k_traj_scan  each workgroup takes a slice of 64*NB stored maps and a
//                group of 16*TQ depth-sorted queries.  Layer by layer it
//                stages the layer's query rows and map rows in LDS and
//                accumulates dot products with MFMA (A = 16 maps x K,
//                B = K x 16 queries); a query tile stops at its deepest
//                member, and rows beyond a query's depth are staged as zeros,
//                so every query gets exactly its own prefix.  Squared map-row
//                norms are summed per layer from the same operands, giving
//                every map's prefix norm at every depth.  The epilogue forms
//                the cosine, keeps a per-lane top-K in registers, merges it
//                across the workgroup and inserts it into the global top-k
//                list; the last workgroup to finish writes idx/score.
//
// float32 stores use v_mfma_f32_16x16x4_f32 (exact float32 products, float32
// accumulation); bf16 stores use v_mfma_f32_16x16x32_bf16 (exact products,
// float32 accumulation).
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

template <typename T> struct Traits;
template <> struct Traits<float> {
  static constexpr int kStep = 4;     // K per MFMA
  static constexpr int kPerLane = 1;  // K elements per lane per MFMA
};
template <> struct Traits<uint16_t> {
  static constexpr int kStep = 32;
  static constexpr int kPerLane = 8;
};

struct TrajArgs {
  const void* planes;
  int64_t plane_elems;
  const void* q;
  int32_t n, L, E;
  int32_t KS;       // MFMA k-steps per layer
  int32_t fill;     // K slots per layer (KS * kStep), elements >= E are zero
  int32_t es_s;     // LDS row stride of map rows (elements)
  int32_t es_q;     // LDS row stride of query rows (elements)
  int32_t B, k;
  int32_t n_qg;     // query groups
  int32_t n_units;  // (map slices) x (query groups)
  int32_t grid;
  int32_t dmax;     // bound on depths (max_depth)
  Workspace ws;
  int32_t* idx_out;
  float* score_out;
  float* dbg;       // optional dense scores [B][n]
};

__device__ __forceinline__ float load_val(const float* p) { return *p; }
__device__ __forceinline__ float load_val(const uint16_t* p) { return bf16_to_f32(*p); }

}  // namespace

// ----------------------------------------------------------------------------- prep

template <typename T>
__global__ void __launch_bounds__(256) k_traj_prep(const T* __restrict__ q, const int32_t* __restrict__ depth,
                                                   int32_t B, int32_t L, int32_t E, int32_t dmax, int32_t k,
                                                   Workspace ws, uint32_t* __restrict__ flags) {
  const int tid = threadIdx.x;
  if (blockIdx.x == 0) {
    // Stable counting sort by depth, deepest first: position of query b =
    // (queries deeper than b) + (queries of equal depth with a lower index).
    __shared__ unsigned long long bits[kMaxL][kChunkB / 64];
    __shared__ int32_t start[kMaxL + 1];
    for (int i = tid; i < kMaxL * (kChunkB / 64); i += 256) (&bits[0][0])[i] = 0ull;
    for (int i = tid; i < kChunkB * kMaxK; i += 256) ws.keys[i] = 0ull;
    if (tid == 0) ws.counter[0] = 0u;
    __syncthreads();
    for (int b = tid; b < B; b += 256) {
      int d = depth[b];
      int dc = d < 1 ? 1 : (d > dmax ? dmax : d);
      if (dc != d) atomicOr(flags, static_cast<uint32_t>(FM_FLAG_DEPTH_CLAMPED));
      atomicOr(&bits[dc - 1][b / 64], 1ull << (b % 64));
    }
    __syncthreads();
    if (tid == 0) {
      int run = 0;
      for (int d = dmax; d >= 1; --d) {
        start[d - 1] = run;
        int c = 0;
        for (int w = 0; w < kChunkB / 64; ++w) c += __popcll(bits[d - 1][w]);
        run += c;
      }
    }
    __syncthreads();
    for (int b = tid; b < B; b += 256) {
      int d = depth[b];
      int dc = d < 1 ? 1 : (d > dmax ? dmax : d);
      int w = b / 64;
      int r = 0;
      for (int i = 0; i < w; ++i) r += __popcll(bits[dc - 1][i]);
      r += __popcll(bits[dc - 1][w] & ((1ull << (b % 64)) - 1ull));
      int pos = start[dc - 1] + r;
      ws.perm[pos] = b;
      ws.sdepth[pos] = dc;
    }
    return;
  }
  // One wavefront per query: 1 / |q[b][0:p]| in float64.
  const int lane = tid % kWave;
  const int b = (blockIdx.x - 1) * kWaves + tid / kWave;
  if (b >= B) return;
  int d = depth[b];
  int p = d < 1 ? 1 : (d > dmax ? dmax : d);
  const T* row = q + static_cast<int64_t>(b) * L * E;
  double acc = 0.0;
  for (int j = lane; j < p * E; j += kWave) {
    double v = static_cast<double>(load_val(row + j));
    acc += v * v;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
  if (lane == 0) {
    float r;
    if (acc != acc) r = __uint_as_float(0x7fc00000u);
    else if (acc == 0.0) r = 0.0f;
    else r = static_cast<float>(1.0 / sqrt(acc));
    ws.rq[b] = r;
  }
}

// ----------------------------------------------------------------------------- scan

template <typename T, int TQ, int NB, int KTOP>
__global__ void __launch_bounds__(256) k_traj_scan(TrajArgs a) {
  constexpr int QG = 16 * TQ;          // queries per group
  constexpr int MW = 16 * NB;          // maps per wave per pass
  constexpr int kStep = Traits<T>::kStep;
  constexpr int kPerLane = Traits<T>::kPerLane;
  extern __shared__ __align__(16) unsigned char smem[];

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;

  // LDS carve-up.
  T* qs = reinterpret_cast<T*>(smem);                                         // [QG][es_q]
  T* ss = qs + QG * a.es_q;                                                   // [4][MW][es_s]
  float* cum = reinterpret_cast<float*>(ss + kWaves * MW * a.es_s);           // [4][dmax][MW]
  int32_t* gperm = reinterpret_cast<int32_t*>(cum + kWaves * a.dmax * MW);    // [QG]
  int32_t* gdep = gperm + QG;                                                 // [QG]
  float* grq = reinterpret_cast<float*>(gdep + QG);                           // [QG]
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(
      (reinterpret_cast<uintptr_t>(grq + QG) + 7) & ~static_cast<uintptr_t>(7));  // [4][QG][KTOP]
  __shared__ int32_t s_last;

  // Workgroup -> (map slice, query group), spread so that consecutive units
  // land on the same XCD (workgroups are dealt round-robin over 8 XCDs).
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  const bool active = u < a.n_units;
  const int slice = active ? u / a.n_qg : 0;
  const int qgrp = active ? u % a.n_qg : 0;
  const int g0 = qgrp * QG;

  for (int r = tid; r < QG; r += kThreads) {
    int pos = g0 + r;
    bool v = active && pos < a.B;
    int b = v ? a.ws.perm[pos] : 0;
    gperm[r] = b;
    gdep[r] = v ? a.ws.sdepth[pos] : 0;
    grq[r] = v ? a.ws.rq[b] : 0.0f;
  }
  __syncthreads();

  int tmd[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) tmd[t] = gdep[16 * t];
  const int D = tmd[0];

  TopK<KTOP> best[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) best[t].clear();

  const int y_pass = slice * (kWaves * MW);
  const int y_wave = y_pass + w * MW;
  const T* planes = static_cast<const T*>(a.planes);
  const T* qsrc = static_cast<const T*>(a.q);

  if (active && D > 0 && y_pass < a.n) {
    floatx4 acc[NB][TQ];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    float cumsq[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) cumsq[nb] = 0.0f;

    for (int l = 0; l < D; ++l) {
      // Stage query rows of layer l (zero beyond each query's depth and beyond E).
      for (int i = tid; i < QG * a.fill; i += kThreads) {
        int r = i / a.fill;
        int e = i - r * a.fill;
        T v = T(0);
        if (e < a.E && l < gdep[r]) v = qsrc[(static_cast<int64_t>(gperm[r]) * a.L + l) * a.E + e];
        qs[r * a.es_q + e] = v;
      }
      // Stage this wave's map rows of layer l (zero beyond the store and beyond E).
      {
        T* dst = ss + w * MW * a.es_s;
        const T* src = planes + static_cast<int64_t>(l) * a.plane_elems + static_cast<int64_t>(y_wave) * a.E;
        for (int i = lane; i < MW * a.fill; i += kWave) {
          int j = i / a.fill;
          int e = i - j * a.fill;
          T v = T(0);
          if (e < a.E && y_wave + j < a.n) v = src[j * a.E + e];
          dst[j * a.es_s + e] = v;
        }
      }
      __syncthreads();

      const T* sw = ss + w * MW * a.es_s;
      if constexpr (sizeof(T) == 4) {
        // float32: k-slot of lane group g in step ks is element KS*g + ks.
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const float* arow = reinterpret_cast<const float*>(sw) + (nb * 16 + c) * a.es_s + a.KS * g;
          float sq = 0.0f;
          for (int ks = 0; ks < a.KS; ++ks) {
            float av = arow[ks];
            sq = fmaf(av, av, sq);
#pragma unroll
            for (int t = 0; t < TQ; ++t) {
              if (tmd[t] > l) {
                float bv = reinterpret_cast<const float*>(qs)[(16 * t + c) * a.es_q + a.KS * g + ks];
                acc[nb][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[nb][t], 0, 0, 0);
              }
            }
          }
          sq += __shfl_xor(sq, 16, kWave);
          sq += __shfl_xor(sq, 32, kWave);
          cumsq[nb] += sq;
        }
      } else {
        // bf16: lane group g supplies elements 32*ks + 8*g .. +7 of step ks.
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const uint16_t* arow = reinterpret_cast<const uint16_t*>(sw) + (nb * 16 + c) * a.es_s + 8 * g;
          float sq = 0.0f;
          for (int ks = 0; ks < a.KS; ++ks) {
            u16x8 av = *reinterpret_cast<const u16x8*>(arow + 32 * ks);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              float f = bf16_to_f32(av[j]);
              sq = fmaf(f, f, sq);
            }
#pragma unroll
            for (int t = 0; t < TQ; ++t) {
              if (tmd[t] > l) {
                u16x8 bv = *reinterpret_cast<const u16x8*>(reinterpret_cast<const uint16_t*>(qs) +
                                                          (16 * t + c) * a.es_q + 32 * ks + 8 * g);
                acc[nb][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bv), acc[nb][t], 0, 0, 0);
              }
            }
          }
          sq += __shfl_xor(sq, 16, kWave);
          sq += __shfl_xor(sq, 32, kWave);
          cumsq[nb] += sq;
        }
      }
      if (g == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) cum[(w * a.dmax + l) * MW + nb * 16 + c] = cumsq[nb];
      }
      __syncthreads();
    }

    // 1/|x[y][0:p]| for every depth p <= D of this wave's maps.
    for (int i = lane; i < D * MW; i += kWave) {
      float v = cum[w * a.dmax * MW + i];
      cum[w * a.dmax * MW + i] = v > 0.0f ? 1.0f / sqrtf(v) : (v != v ? v : 0.0f);
    }
    __syncthreads();

    // Epilogue: cosine, optional dense output, per-lane top-K.
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
      const int r = 16 * t + c;
      const int p = gdep[r];
      if (p == 0) continue;
      const float rq = grq[r];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int jm = nb * 16 + 4 * g + i;
          const int y = y_wave + jm;
          if (y >= a.n) continue;
          const float rs = cum[(w * a.dmax + (p - 1)) * MW + jm];
          float s = acc[nb][t][i] * rq * rs;
          if (a.dbg != nullptr) a.dbg[static_cast<int64_t>(gperm[r]) * a.n + y] = s;
          best[t].push(make_key(s, y));
        }
      }
    }
  }

  // Merge the per-lane lists: across the 4 lane groups, then across waves.
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      uint64_t o[KTOP];
#pragma unroll
      for (int j = 0; j < KTOP; ++j) o[j] = shfl_xor_u64(best[t].v[j], m);
      best[t].merge(o);
    }
    if (g == 0) {
#pragma unroll
      for (int j = 0; j < KTOP; ++j) mbuf[(w * QG + 16 * t + c) * KTOP + j] = best[t].v[j];
    }
  }
  __syncthreads();
  for (int r = tid; r < QG; r += kThreads) {
    if (!active || g0 + r >= a.B || gdep[r] == 0) continue;
    TopK<KTOP> m;
    m.clear();
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) m.merge(mbuf + (ww * QG + r) * KTOP);
    global_topk_insert(a.ws.keys + static_cast<int64_t>(gperm[r]) * kMaxK, a.k, m.v, KTOP < a.k ? KTOP : a.k);
  }

  // The last workgroup to finish writes the results.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    uint32_t ticket = __hip_atomic_fetch_add(a.ws.counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (ticket == static_cast<uint32_t>(a.grid - 1)) ? 1 : 0;
  }
  __syncthreads();
  if (s_last && a.idx_out != nullptr) {
    __threadfence();
    for (int i = tid; i < a.B * a.k; i += kThreads) {
      int b = i / a.k;
      int j = i - b * a.k;
      uint64_t key = __hip_atomic_load(a.ws.keys + static_cast<int64_t>(b) * kMaxK + j, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
      a.idx_out[i] = key_index(key);
      a.score_out[i] = key_score(key);
    }
  }
}

// ----------------------------------------------------------------------------- launch

template <typename T, int TQ, int NB, int KTOP>
static hipError_t launch_on(const TrajArgs& a, size_t lds, hipStream_t st) {
  auto kern = k_traj_scan<T, TQ, NB, KTOP>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

static int traj_nb_for(int TQ) { return TQ <= 4 ? 2 : 1; }

hipError_t launch_match_trajectory(const StoreView& s, const void* q, const int32_t* depth, int32_t max_depth,
                                   int32_t B, int32_t k, int32_t* idx_out, float* score_out, float* dbg_scores,
                                   const Workspace& ws, hipStream_t st) {
  const bool bf = s.map_dtype == FM_BF16;
  const int esz = bf ? 2 : 4;
  const int kStep = bf ? 32 : 4;
  const int KS = (s.E + kStep - 1) / kStep;
  const int fill = KS * kStep;
  const int KTOP = k == 1 ? 1 : (k <= 4 ? 4 : 8);
  const int tq_max = KTOP == 1 ? (bf ? 16 : 32) : (KTOP == 4 ? 8 : 4);

  for (int b0 = 0; b0 < B; b0 += kChunkB) {
    const int Bc = (B - b0) < kChunkB ? (B - b0) : kChunkB;
    const char* qc = static_cast<const char*>(q) + static_cast<int64_t>(b0) * s.L * s.E * esz;
    // Prep: sort by depth, query norms, clear keys.
    const int prep_blocks = 1 + (Bc + kWaves - 1) / kWaves;
    if (bf) {
      hipLaunchKernelGGL(k_traj_prep<uint16_t>, dim3(prep_blocks), dim3(256), 0, st,
                         reinterpret_cast<const uint16_t*>(qc), depth + b0, Bc, s.L, s.E, max_depth, k, ws, s.flags);
    } else {
      hipLaunchKernelGGL(k_traj_prep<float>, dim3(prep_blocks), dim3(256), 0, st,
                         reinterpret_cast<const float*>(qc), depth + b0, Bc, s.L, s.E, max_depth, k, ws, s.flags);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    int TQ = 1;
    while (16 * TQ < Bc && TQ < tq_max) TQ *= 2;
    const int NB = traj_nb_for(TQ);
    const int n_qg = (Bc + 16 * TQ - 1) / (16 * TQ);
    const int maps_per_slice = kWaves * 16 * NB;
    const int slices = s.n > 0 ? (s.n + maps_per_slice - 1) / maps_per_slice : 0;
    TrajArgs a;
    a.planes = s.planes;
    a.plane_elems = s.plane_elems;
    a.q = qc;
    a.n = s.n;
    a.L = s.L;
    a.E = s.E;
    a.KS = KS;
    a.fill = fill;
    if (bf) {
      a.es_s = fill + 8;
      a.es_q = fill + 8;
    } else {
      a.es_s = fill + 1;
      a.es_q = fill + 1;
    }
    a.B = Bc;
    a.k = k;
    a.n_qg = n_qg;
    a.n_units = slices * n_qg;
    a.grid = ((a.n_units > 0 ? a.n_units : 1) + 7) / 8 * 8;
    a.dmax = max_depth;
    a.ws = ws;
    a.idx_out = idx_out != nullptr ? idx_out + static_cast<int64_t>(b0) * k : nullptr;
    a.score_out = score_out != nullptr ? score_out + static_cast<int64_t>(b0) * k : nullptr;
    a.dbg = dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr;

    const int es_s = a.es_s, es_q = a.es_q, dmax = a.dmax;
    auto lds_of = [=](int tq, int nb) -> size_t {
      size_t qg = 16 * tq, mw = 16 * nb;
      size_t bytes = qg * es_q * esz + kWaves * mw * es_s * esz;
      bytes = (bytes + 3) / 4 * 4;
      bytes += kWaves * static_cast<size_t>(dmax) * mw * 4 + 3 * qg * 4;
      bytes = (bytes + 7) / 8 * 8;
      bytes += kWaves * qg * static_cast<size_t>(KTOP) * 8;
      return bytes;
    };
    const size_t lds = lds_of(TQ, NB);
    if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
    if (bf) {
      if (KTOP == 1) err = (TQ == 1 ? launch_on<uint16_t, 1, 2, 1>(a, lds, st)
                           : TQ == 2 ? launch_on<uint16_t, 2, 2, 1>(a, lds, st)
                           : TQ == 4 ? launch_on<uint16_t, 4, 2, 1>(a, lds, st)
                           : TQ == 8 ? launch_on<uint16_t, 8, 1, 1>(a, lds, st)
                                     : launch_on<uint16_t, 16, 1, 1>(a, lds, st));
      else if (KTOP == 4) err = (TQ == 1 ? launch_on<uint16_t, 1, 2, 4>(a, lds, st)
                                : TQ == 2 ? launch_on<uint16_t, 2, 2, 4>(a, lds, st)
                                : TQ == 4 ? launch_on<uint16_t, 4, 2, 4>(a, lds, st)
                                          : launch_on<uint16_t, 8, 1, 4>(a, lds, st));
      else err = (TQ == 1 ? launch_on<uint16_t, 1, 2, 8>(a, lds, st)
                  : TQ == 2 ? launch_on<uint16_t, 2, 2, 8>(a, lds, st)
                            : launch_on<uint16_t, 4, 2, 8>(a, lds, st));
    } else {
      if (KTOP == 1) err = (TQ == 1 ? launch_on<float, 1, 2, 1>(a, lds, st)
                           : TQ == 2 ? launch_on<float, 2, 2, 1>(a, lds, st)
                           : TQ == 4 ? launch_on<float, 4, 2, 1>(a, lds, st)
                           : TQ == 8 ? launch_on<float, 8, 1, 1>(a, lds, st)
                           : TQ == 16 ? launch_on<float, 16, 1, 1>(a, lds, st)
                                      : launch_on<float, 32, 1, 1>(a, lds, st));
      else if (KTOP == 4) err = (TQ == 1 ? launch_on<float, 1, 2, 4>(a, lds, st)
                                : TQ == 2 ? launch_on<float, 2, 2, 4>(a, lds, st)
                                : TQ == 4 ? launch_on<float, 4, 2, 4>(a, lds, st)
                                          : launch_on<float, 8, 1, 4>(a, lds, st));
      else err = (TQ == 1 ? launch_on<float, 1, 2, 8>(a, lds, st)
                  : TQ == 2 ? launch_on<float, 2, 2, 8>(a, lds, st)
                            : launch_on<float, 4, 2, 8>(a, lds, st));
    }
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace fm
