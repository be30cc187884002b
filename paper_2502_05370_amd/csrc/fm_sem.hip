// Semantic-based expert map search (Section 4.2.1, Eq. 4).
//
// The score of query embedding q[b] against stored embedding x[y] is
// q[b].x[y] / (|q[b]| |x[y]|).  For a batch this is a dense B x n
// contraction over the hidden size, so it runs on bf16 MFMA
// (v_mfma_f32_16x16x32_bf16: exact bf16 products, float32 accumulation):
//
//   k_sem_scan  each workgroup owns a 128-map x (16*TQ)-query output tile
//               and walks the hidden dimension in chunks of 64, staging both
//               operands in LDS.  Four waves split the tile 2 x 2 (or 4 x 1
//               for a single query tile).  The epilogue scales by the stored
//               norms, keeps a per-lane top-K, merges it across the
//               workgroup and inserts it into the global top-k list; the last
//               workgroup to finish writes idx/score and clears the list.
//               Query norms are summed in float64 from the staged chunks.  The
//               B x n score matrix is never written (except into the optional
//               debug output).
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileMaps = 128;   // stored maps per workgroup tile
constexpr int kChunk = 64;       // hidden elements per LDS stage
constexpr int kRow = kChunk + 8; // LDS row stride (elements): 144 bytes, conflict-free 16-byte reads

struct SemArgs {
  const uint16_t* x;      // [cap][d]
  const float* xnorm;     // [cap]
  const uint16_t* q;      // [B][d]
  int32_t n, d, B, k;
  int32_t n_qg, n_units, grid;
  Workspace ws;
  int32_t* idx_out;
  float* score_out;
  float* dbg;
};

}  // namespace

template <int TQ, int WN, int KTOP>
__global__ void __launch_bounds__(256) k_sem_scan(SemArgs a) {
  constexpr int QT = 16 * TQ;              // queries per workgroup tile
  constexpr int WM = kWaves / WN;          // wave rows (maps)
  constexpr int MBW = kTileMaps / WM / 16; // 16-map blocks per wave
  constexpr int NBW = TQ / WN;             // 16-query blocks per wave
  constexpr int XU = kTileMaps * kChunk / 8 / kThreads;  // 16-byte units per thread (maps)
  constexpr int QU = (QT * kChunk / 8 + kThreads - 1) / kThreads;
  static_assert(NBW >= 1, "query tiles per wave");

  __shared__ __align__(16) uint16_t xs[kTileMaps * kRow];
  __shared__ __align__(16) uint16_t qs[QT * kRow];
  __shared__ uint64_t mbuf[WM][QT][KTOP];
  __shared__ float grq[QT];
  __shared__ int32_t s_last;

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;
  const int wm = w / WN;
  const int wn = w % WN;

  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  const bool active = u < a.n_units;
  const int tile = active ? u / a.n_qg : 0;
  const int qgrp = active ? u % a.n_qg : 0;
  const int y0 = tile * kTileMaps;
  const int b0 = qgrp * QT;

  for (int r = tid; r < QT; r += kThreads) grq[r] = 0.0f;

  TopK<KTOP> best[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) best[nb].clear();

  if (active) {
    floatx4 acc[MBW][NBW];
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] = floatx4{0.f, 0.f, 0.f, 0.f};

    // Register prefetch of one chunk of both operands.
    u16x8 xr[XU];
    u16x8 qr[QU];
    double qn2[QU];
#pragma unroll
    for (int i = 0; i < QU; ++i) qn2[i] = 0.0;
    auto load_chunk = [&](int kc) {
#pragma unroll
      for (int i = 0; i < XU; ++i) {
        int unit = tid + i * kThreads;
        int row = unit / (kChunk / 8);
        int part = unit % (kChunk / 8);
        int y = y0 + row;
        u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        if (y < a.n) v = *reinterpret_cast<const u16x8*>(a.x + static_cast<int64_t>(y) * a.d + kc + part * 8);
        xr[i] = v;
      }
#pragma unroll
      for (int i = 0; i < QU; ++i) {
        int unit = tid + i * kThreads;
        int row = unit / (kChunk / 8);
        int part = unit % (kChunk / 8);
        int b = b0 + row;
        u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        if (row < QT && b < a.B) v = *reinterpret_cast<const u16x8*>(a.q + static_cast<int64_t>(b) * a.d + kc + part * 8);
        qr[i] = v;
      }
    };
    auto store_chunk = [&]() {
#pragma unroll
      for (int i = 0; i < XU; ++i) {
        int unit = tid + i * kThreads;
        int row = unit / (kChunk / 8);
        int part = unit % (kChunk / 8);
        *reinterpret_cast<u16x8*>(xs + row * kRow + part * 8) = xr[i];
      }
#pragma unroll
      for (int i = 0; i < QU; ++i) {
        int unit = tid + i * kThreads;
        int row = unit / (kChunk / 8);
        int part = unit % (kChunk / 8);
        if (row < QT) *reinterpret_cast<u16x8*>(qs + row * kRow + part * 8) = qr[i];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const double f = static_cast<double>(bf16_to_f32(qr[i][j]));
          qn2[i] += f * f;
        }
      }
    };

    load_chunk(0);
    for (int kc = 0; kc < a.d; kc += kChunk) {
      store_chunk();
      __syncthreads();
      if (kc + kChunk < a.d) load_chunk(kc + kChunk);
#pragma unroll
      for (int kk = 0; kk < kChunk / 32; ++kk) {
        u16x8 af[MBW];
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
          af[mb] = *reinterpret_cast<const u16x8*>(xs + ((wm * MBW + mb) * 16 + c) * kRow + 32 * kk + 8 * g);
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
          u16x8 bf = *reinterpret_cast<const u16x8*>(qs + ((wn * NBW + nb) * 16 + c) * kRow + 32 * kk + 8 * g);
#pragma unroll
          for (int mb = 0; mb < MBW; ++mb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, af[mb]), __builtin_bit_cast(bf16x8, bf), acc[mb][nb], 0, 0, 0);
        }
      }
      __syncthreads();
    }

    // query norms: the 8 parts of a row sit in 8 consecutive lanes (fixed order)
#pragma unroll
    for (int i = 0; i < QU; ++i) {
      double v = qn2[i];
      v += __shfl_xor(v, 1, kWave);
      v += __shfl_xor(v, 2, kWave);
      v += __shfl_xor(v, 4, kWave);
      const int unit = tid + i * kThreads;
      const int row = unit / (kChunk / 8);
      if (row < QT && unit % (kChunk / 8) == 0) {
        float r;
        if (v != v) r = __uint_as_float(0x7fc00000u);
        else if (v == 0.0) r = 0.0f;
        else r = static_cast<float>(1.0 / sqrt(v));
        grq[row] = r;
      }
    }
    __syncthreads();

    // Epilogue: lane (g, c) holds maps 4g+i of each 16-map block for query c of each query block.
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int r = (wn * NBW + nb) * 16 + c;
      const int b = b0 + r;
      if (b >= a.B) continue;
      const float rq = grq[r];
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int y = y0 + (wm * MBW + mb) * 16 + 4 * g + i;
          if (y >= a.n) continue;
          const float xn = a.xnorm[y];
          const float rx = xn > 0.0f ? 1.0f / xn : (xn != xn ? xn : 0.0f);
          const float s = acc[mb][nb][i] * rq * rx;
          if (a.dbg != nullptr) a.dbg[static_cast<int64_t>(b) * a.n + y] = s;
          best[nb].push(make_key(s, y));
        }
      }
    }
  }

#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      uint64_t o[KTOP];
#pragma unroll
      for (int j = 0; j < KTOP; ++j) o[j] = shfl_xor_u64(best[nb].v[j], m);
      best[nb].merge(o);
    }
    if (g == 0) {
#pragma unroll
      for (int j = 0; j < KTOP; ++j) mbuf[wm][(wn * NBW + nb) * 16 + c][j] = best[nb].v[j];
    }
  }
  __syncthreads();
  for (int r = tid; r < QT; r += kThreads) {
    if (!active || b0 + r >= a.B) continue;
    TopK<KTOP> m;
    m.clear();
#pragma unroll
    for (int ww = 0; ww < WM; ++ww) m.merge(&mbuf[ww][r][0]);
    global_topk_insert<KTOP>(a.ws.keys + static_cast<int64_t>(b0 + r) * kMaxK, a.k, m.v);
  }

  __threadfence();
  __syncthreads();
  if (tid == 0) {
    uint32_t ticket = __hip_atomic_fetch_add(a.ws.counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (ticket == static_cast<uint32_t>(a.grid - 1)) ? 1 : 0;
  }
  __syncthreads();
  if (s_last) {
    __threadfence();
    for (int i = tid; i < a.B * a.k; i += kThreads) {
      const int b = i / a.k;
      const int j = i - b * a.k;
      uint64_t* slot = a.ws.keys + static_cast<int64_t>(b) * kMaxK + j;
      const uint64_t key = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a.idx_out != nullptr) {
        a.idx_out[i] = key_index(key);
        a.score_out[i] = key_score(key);
      }
      __hip_atomic_store(slot, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid == 0) __hip_atomic_store(a.ws.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int TQ, int WN, int KTOP>
static hipError_t sem_launch(const SemArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((k_sem_scan<TQ, WN, KTOP>), dim3(a.grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_match_semantic(const StoreView& s, const void* q, int32_t B, int32_t k, int32_t* idx_out,
                                 float* score_out, float* dbg_scores, const Workspace& ws, hipStream_t st) {
  const int KTOP = k == 1 ? 1 : (k <= 4 ? 4 : 8);
  const int tq_max = KTOP == 1 ? 16 : (KTOP == 4 ? 8 : 4);
  for (int b0 = 0; b0 < B; b0 += kChunkB) {
    const int Bc = (B - b0) < kChunkB ? (B - b0) : kChunkB;
    const uint16_t* qc = static_cast<const uint16_t*>(q) + static_cast<int64_t>(b0) * s.d_emb;
    hipError_t err = hipSuccess;
    int TQ = 1;
    while (16 * TQ < Bc && TQ < tq_max) TQ *= 2;
    const int n_qg = (Bc + 16 * TQ - 1) / (16 * TQ);
    const int tiles = s.n > 0 ? (s.n + kTileMaps - 1) / kTileMaps : 0;
    SemArgs a;
    a.x = s.embs;
    a.xnorm = s.emb_norm;
    a.q = qc;
    a.n = s.n;
    a.d = s.d_emb;
    a.B = Bc;
    a.k = k;
    a.n_qg = n_qg;
    a.n_units = tiles * n_qg;
    a.grid = ((a.n_units > 0 ? a.n_units : 1) + 7) / 8 * 8;
    a.ws = ws;
    a.idx_out = idx_out != nullptr ? idx_out + static_cast<int64_t>(b0) * k : nullptr;
    a.score_out = score_out != nullptr ? score_out + static_cast<int64_t>(b0) * k : nullptr;
    a.dbg = dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr;
    if (KTOP == 1) {
      switch (TQ) {
        case 1: err = sem_launch<1, 1, 1>(a, st); break;
        case 2: err = sem_launch<2, 2, 1>(a, st); break;
        case 4: err = sem_launch<4, 2, 1>(a, st); break;
        case 8: err = sem_launch<8, 2, 1>(a, st); break;
        default: err = sem_launch<16, 2, 1>(a, st); break;
      }
    } else if (KTOP == 4) {
      switch (TQ) {
        case 1: err = sem_launch<1, 1, 4>(a, st); break;
        case 2: err = sem_launch<2, 2, 4>(a, st); break;
        case 4: err = sem_launch<4, 2, 4>(a, st); break;
        default: err = sem_launch<8, 2, 4>(a, st); break;
      }
    } else {
      switch (TQ) {
        case 1: err = sem_launch<1, 1, 8>(a, st); break;
        case 2: err = sem_launch<2, 2, 8>(a, st); break;
        default: err = sem_launch<4, 2, 8>(a, st); break;
      }
    }
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace fm
