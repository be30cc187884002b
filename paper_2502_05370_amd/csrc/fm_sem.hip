// Semantic-based expert map search (Section 4.2.1, Eq. 4).
//
// The score of query embedding q[b] against stored embedding x[y] is
// q[b].x[y] / (|q[b]| |x[y]|).  For a batch this is a dense B x n
// contraction over the hidden size on bf16 MFMA
// (v_mfma_f32_16x16x32_bf16: exact bf16 products, float32 accumulation).
// Stored embeddings are kept as 1 KB MFMA operand tiles (emb_offset), so every
// operand load is one contiguous 1 KB read.  A batch of up to 1024 queries is
// served by three launches:
//
//  k_sem_prep   copies the queries into the same tile layout (zero rows pad
//               the last 16-query tile) and writes 1/|q| (float64 sum).
//  k_sem_scan   workgroup = a group of 16*TQ queries x an even share of the
//               store's 16-map blocks, walked as slices of 8 waves x NBA
//               blocks.  A stage is KS k-steps of one slice: the map tiles of
//               stage j+2 load into registers (raw buffer loads) and the query
//               tiles of stage j+2 into an LDS ring slot (direct global->LDS
//               loads) while stage j computes.  At the end of a slice the
//               epilogue scales by the stored norms and keeps a per-lane
//               top-K; the workgroup's merged list is stored as its partial
//               list per query.
//  k_finalize   (shared with the trajectory search) merges the partial lists.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

struct SemPrepArgs {
  const uint16_t* q;   // [B][d] bf16
  int32_t B, d, b_pad;
  uint16_t* qst;       // tiled [b_pad][d]
  float* rq;           // [b_pad]
};

struct SemArgs {
  const uint16_t* x;     // tiled embeddings
  int64_t x_bytes;       // bytes of the embedding region
  const float* xnorm;    // [cap] |x|
  int32_t n, d, B;
  int32_t n_qg;          // query groups
  int32_t R;             // workgroups per query group
  int32_t n_blocks;      // 16-map blocks of the store
  int32_t grid;
  Workspace ws;
  float* dbg;            // optional dense scores [B][n]
  // Optional second dense matrix [B][n]: when set, the dense output is the
  // weighted sum w_self * score + w_mix * mix (float64, rounded once).
  const float* mix;
  double w_self, w_mix;
};

// Position of stage j of the semantic scan: slice j / NKC, k-step pair
// j % NKC and query ring slot j % NS, stepped without divisions.
struct SemPos {
  int j, si, kc, slot;
};
__device__ __forceinline__ SemPos next_sem_pos(const SemPos& p, int nkc, int ns) {
  SemPos q;
  q.j = p.j + 1;
  const bool wrap = p.kc + 1 == nkc;
  q.kc = wrap ? 0 : p.kc + 1;
  q.si = wrap ? p.si + 1 : p.si;
  q.slot = p.slot + 1 == ns ? 0 : p.slot + 1;
  return q;
}

}  // namespace

// One wave per query position: the row is copied 8 dimensions (16 bytes) at a
// time into its tile slots; positions past B get zero rows.
__global__ void __launch_bounds__(256) k_sem_prep(SemPrepArgs a) {
  const int lane = threadIdx.x % kWave;
  const int pos = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (pos >= a.b_pad) return;
  double acc = 0.0;
  for (int j0 = 8 * lane; j0 < a.d; j0 += 8 * kWave) {
    u16x8 h = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
    if (pos < a.B) {
      h = *reinterpret_cast<const u16x8*>(a.q + static_cast<int64_t>(pos) * a.d + j0);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const double v = static_cast<double>(bf16_to_f32(h[t]));
        acc += v * v;
      }
    }
    *reinterpret_cast<u16x8*>(a.qst + emb_offset(pos, j0, a.d)) = h;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
  if (lane == 0) {
    float r;
    if (acc != acc) r = __uint_as_float(0x7fc00000u);
    else if (acc == 0.0) r = 0.0f;
    else r = static_cast<float>(1.0 / sqrt(acc));
    a.rq[pos] = pos < a.B ? r : 0.0f;
  }
}

// 8 waves; wave w owns NBA blocks of 16 maps of every slice.  Stage j =
// (slice j / NKC, k-steps KS * (j % NKC) ..).  During stage j every wave loads
// its share of the query tiles of stage j+3 into LDS slot (j+3) % 4 and, after
// its MFMAs, the map tiles of stage j+3 into the registers stage j used (three
// register sets rotate), so a load has two stages to land.  Every wave issues
// the same loads per stage (out-of-range offsets and a repeated query tile keep
// the count fixed), so "stage j+1 has landed" is vmcnt <= the loads of two
// stages at the end of stage j.  Slot (j+3) % 4 was last read in stage j-1,
// which every wave finished before the barrier of stage j.
template <int TQ, int KTOP, bool DBG>
__global__ void __launch_bounds__(512) k_sem_scan(SemArgs a) {
  constexpr int W = 8;                        // waves per workgroup
  constexpr int NBA = 2;                      // 16-map blocks per wave and slice
  constexpr int KS = 2;                       // k-steps (32 dimensions each) per stage
  constexpr int NS = 4;                       // query ring slots
  constexpr int QG = 16 * TQ;                 // queries per group
  constexpr int NQ = TQ * KS;                 // 1 KB query tiles per stage
  constexpr int NI_Q = (NQ + W - 1) / W;      // query tile loads per wave and stage
  constexpr int Q_STAGE = NQ * 1024;
  constexpr int NI_A = NBA * KS + 1;          // map tile loads and one map norm load per wave and stage
  constexpr int NI = NI_A + NI_Q;
  static_assert(NI < 64, "vmcnt field is 6 bits");

  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                      // [NS][Q_STAGE]
  float* grq = reinterpret_cast<float*>(smem + NS * Q_STAGE);      // [QG]
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(smem);              // after the loop: [W][QG][KTOP]

  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;

  // workgroup -> (query group, block range); the n_qg workgroups sharing a
  // block range are consecutive, hence on one XCD, and read the same map
  // tiles at about the same time (the later reads hit that XCD's L2)
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  const bool active = u < a.n_qg * a.R;
  const int qgrp = active ? u % a.n_qg : 0;
  const int rr = active ? u / a.n_qg : 0;
  const int b_begin = active ? static_cast<int>((static_cast<int64_t>(rr) * a.n_blocks) / a.R) : 0;
  const int b_end = active ? static_cast<int>((static_cast<int64_t>(rr + 1) * a.n_blocks) / a.R) : 0;
  const int n_slices = (b_end - b_begin + W * NBA - 1) / (W * NBA);
  const int g0 = qgrp * QG;
  const int ksteps = a.d / 32;
  const int NKC = ksteps / KS;
  const int nstages = n_slices * NKC;

  for (int r = tid; r < QG; r += W * kWave) grq[r] = a.ws.rq[g0 + r];
  __syncthreads();

  TopK<KTOP> best[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) best[t].clear();

  if (active && nstages > 0) {
    const char* xb = reinterpret_cast<const char*>(a.x);
    const char* qst = static_cast<const char*>(a.ws.qrows);
    const int64_t blk_bytes = static_cast<int64_t>(ksteps) * 1024;   // one 16-row block, all k-steps

    // Map tiles: descriptor based at the slice's first block; rows past the
    // store and blocks past the range read as zeros.  The first stage of a
    // slice also loads the slice's map norms (one per lane, shuffled to the
    // lanes that need them in the epilogue); the other stages issue the same
    // load out of range.
    const __amdgpu_buffer_rsrc_t rs_norm = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.xnorm), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(a.n) * 4u), kBufWord3);
    // The descriptor (based at the slice's first block) and a lane's offsets
    // are the same in every stage of a slice: they are set when a slice's
    // first stage loads (and for every load past the last stage, whose
    // offsets are all out of range), the offsets kept opaque so the loads
    // stay unconditional; a stage's k-step pair goes in as the loads' scalar
    // offset.  The descriptor's range ends with the slice's blocks, and lanes
    // with no row use an offset of 2^31 - 4 KB, which with any scalar offset
    // of the slice stays past that range without wrapping, so they read
    // zeros.
    constexpr uint32_t kNoRow = 0x7FFFF000u;
    uint32_t soff[NBA];
    __amdgpu_buffer_rsrc_t rs_slice = rs_norm;
    auto load_a = [&](const SemPos& p, u16x8 (&dst)[NBA][KS], float& dxn) {
      const bool real = p.j < nstages;
      const int si = real ? p.si : 0;
      const int kc = real ? p.kc : 0;
      const int blk0 = b_begin + si * (W * NBA);
      if (!real || kc == 0) {
        const int64_t base = static_cast<int64_t>(blk0) * blk_bytes;
        int64_t rem = a.x_bytes - base;
        if (rem > static_cast<int64_t>(W * NBA) * blk_bytes) rem = static_cast<int64_t>(W * NBA) * blk_bytes;
        if (rem < 0) rem = 0;
        rs_slice = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(xb + base), static_cast<short>(0),
                                                     static_cast<int>(static_cast<uint32_t>(rem)), kBufWord3);
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb) {
          const int blk = blk0 + w * NBA + nb;
          const bool ok = real && blk < b_end && 16 * blk + c < a.n;
          soff[nb] = ok ? static_cast<uint32_t>((w * NBA + nb) * ksteps * 1024 + lane * 16) : kNoRow;
          asm volatile("" : "+v"(soff[nb]));
        }
      }
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const uint32_t off = soff[nb] + static_cast<uint32_t>(ks * 1024);
          dst[nb][ks] = __builtin_bit_cast(
              u16x8, __builtin_amdgcn_raw_buffer_load_b128(rs_slice, static_cast<int>(off), kc * KS * 1024, 0));
        }
      }
      // lane l: the norm of map l % 16 of the wave's block (l / 16) % NBA
      const int nblk = blk0 + w * NBA + (lane / 16) % NBA;
      const uint32_t noff = (real && kc == 0 && nblk < b_end) ? static_cast<uint32_t>((16 * nblk + c) * 4) : kOutside;
      dxn = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs_norm, static_cast<int>(noff), 0, 0));
    };
    // Query tiles of stage j: tile (t, ks) is 1 KB at slot offset (t*KS+ks) KB;
    // wave w loads tiles w, w+8, ... (wrapping: a repeated tile rewrites
    // identical bytes).
    // this lane's source of each query tile it loads, at the first k-step pair
    const char* qsrc[NI_Q];
#pragma unroll
    for (int i = 0; i < NI_Q; ++i) {
      const int tile = (w + W * i) % NQ;
      const int t = tile / KS;
      const int ks = tile - t * KS;
      qsrc[i] = qst + ((static_cast<int64_t>(g0 / 16 + t) * ksteps + ks) * 1024) + lane * 16;
    }
    auto load_q = [&](const SemPos& p) {
      const bool real = p.j < nstages;
      const int kc = real ? p.kc : 0;
      unsigned char* st = ring + p.slot * Q_STAGE;
#pragma unroll
      for (int i = 0; i < NI_Q; ++i) dma16(qsrc[i] + kc * KS * 1024, st + ((w + W * i) % NQ) * 1024);
    };

    floatx4 acc[NBA][TQ];
#pragma unroll
    for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
      for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    // issue order: Q0 A0 Q1 A1 Q2 A2, then during stage j: Q(j+3) A(j+3)
    u16x8 ar0[NBA][KS], ar1[NBA][KS], ar2[NBA][KS];
    float xr0, xr1, xr2;
    // stage positions advance incrementally (no division per stage)
    SemPos p0{0, 0, 0, 0};
    SemPos p1 = next_sem_pos(p0, NKC, NS);
    SemPos p2 = next_sem_pos(p1, NKC, NS);
    SemPos p3 = next_sem_pos(p2, NKC, NS);
    load_q(p0);
    load_a(p0, ar0, xr0);
    load_q(p1);
    load_a(p1, ar1, xr1);
    load_q(p2);
    load_a(p2, ar2, xr2);

    // The map registers of a stage pass through an empty asm placed after
    // the wait for them, so no use of them is scheduled above it (the
    // compiler would then wait for every outstanding load itself, emptying
    // the prefetch).
    u16x8 cur[NBA][KS];
    float xn_slice = 0.0f;
    auto take = [&](const SemPos& p, u16x8 (&ring_regs)[NBA][KS], float& ring_xn) {
      wait_vmcnt<2 * NI>();
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          cur[nb][ks] = ring_regs[nb][ks];
          asm volatile("" : "+v"(cur[nb][ks]));
        }
      }
      if (p.kc == 0) {
        xn_slice = ring_xn;
        asm volatile("" : "+v"(xn_slice));
      }
    };

    auto stage = [&](const SemPos& q0, const SemPos& q1, const SemPos& q3, u16x8 (&ring_regs)[NBA][KS],
                     float& ring_xn, u16x8 (&next_regs)[NBA][KS], float& next_xn) {
      const int si = q0.si;
      const int kc = q0.kc;
      const int blk_wave = b_begin + si * (W * NBA) + w * NBA;
      const unsigned char* sq = ring + q0.slot * Q_STAGE;

      raw_barrier();
      load_q(q3);
      // The query tiles of a k-step land in registers of their own before
      // its MFMAs (the empty asm keeps the compiler from reusing one register
      // set per tile, which would serialise one LDS round trip per tile);
      // the next k-step's reads are issued before this k-step's MFMAs.
      u16x8 bq[KS][TQ];
      auto read_q = [&](int ks) {
#pragma unroll
        for (int t = 0; t < TQ; ++t) bq[ks][t] = *reinterpret_cast<const u16x8*>(sq + (t * KS + ks) * 1024 + lane * 16);
      };
      auto pin_q = [&](int ks) {
#pragma unroll
        for (int t = 0; t < TQ; ++t) asm volatile("" : "+v"(bq[ks][t]));
      };
      // A wave whose blocks all lie past the range (the short last slice of
      // a workgroup) skips the query reads and MFMAs; it still takes part in
      // the barriers and issues its share of the loads.
      if (blk_wave < b_end) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) read_q(ks);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) pin_q(ks);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int t = 0; t < TQ; ++t)
#pragma unroll
            for (int nb = 0; nb < NBA; ++nb) acc[nb][t] = mfma_bf16(cur[nb][ks], bq[ks][t], acc[nb][t]);
      }
      load_a(q3, ring_regs, ring_xn);

      if (kc == NKC - 1) {
        // End of a slice: cosine = dot * 1/|q| * 1/|x|; lane (g, c) holds maps
        // 16nb + 4g + i (i = 0..3) of query column c of each tile.
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb) {
          const bool blk_ok = blk_wave + nb < b_end;
          const int y0 = 16 * (blk_wave + nb) + 4 * g;
          floatx4 xn;
#pragma unroll
          for (int i = 0; i < 4; ++i) xn[i] = __shfl(xn_slice, nb * 16 + 4 * g + i, kWave);
          if (!blk_ok) continue;
#pragma unroll
          for (int t = 0; t < TQ; ++t) {
            const int r = 16 * t + c;
            const int b = g0 + r;
            if (b >= a.B) continue;
            const float rq = grq[r];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int y = y0 + i;
              if (y >= a.n) continue;
              const float rx = xn[i] > 0.0f ? 1.0f / xn[i] : (xn[i] != xn[i] ? xn[i] : 0.0f);
              const float s = acc[nb][t][i] * rq * rx;
              if constexpr (DBG) {
                const int64_t o = static_cast<int64_t>(b) * a.n + y;
                float v = s;
                if (a.mix != nullptr)
                  v = static_cast<float>(__dadd_rn(__dmul_rn(a.w_self, static_cast<double>(s)),
                                                   __dmul_rn(a.w_mix, static_cast<double>(a.mix[o]))));
                a.dbg[o] = v;
              }
              best[t].push(make_key(s, y));
            }
          }
        }
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
          for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      take(q1, next_regs, next_xn);
    };
    auto advance = [&]() {
      p0 = p1;
      p1 = p2;
      p2 = p3;
      p3 = next_sem_pos(p3, NKC, NS);
    };

    take(p0, ar0, xr0);
    while (p0.j + 3 <= nstages) {
      stage(p0, p1, p3, ar0, xr0, ar1, xr1);
      advance();
      stage(p0, p1, p3, ar1, xr1, ar2, xr2);
      advance();
      stage(p0, p1, p3, ar2, xr2, ar0, xr0);
      advance();
    }
    if (p0.j < nstages) {
      stage(p0, p1, p3, ar0, xr0, ar1, xr1);
      advance();
      if (p0.j < nstages) stage(p0, p1, p3, ar1, xr1, ar2, xr2);
    }
    wait_vmcnt<0>();   // drain the trailing loads
    __syncthreads();
  }

  // merge the per-lane lists across the 4 lane groups, then across waves
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      uint64_t o[KTOP];
#pragma unroll
      for (int jj = 0; jj < KTOP; ++jj) o[jj] = shfl_xor_u64(best[t].v[jj], m);
      best[t].merge(o);
    }
  }
  __syncthreads();
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
#pragma unroll
      for (int jj = 0; jj < KTOP; ++jj) mbuf[(w * QG + 16 * t + c) * KTOP + jj] = best[t].v[jj];
    }
  }
  __syncthreads();
  if (active) {
    for (int r = tid; r < QG; r += W * kWave) {
      TopK<KTOP> m;
      m.clear();
#pragma unroll
      for (int ww = 0; ww < W; ++ww) m.merge(mbuf + (ww * QG + r) * KTOP);
      uint64_t* out = a.ws.partial + (static_cast<int64_t>(g0 + r) * a.R + rr) * KTOP;
#pragma unroll
      for (int jj = 0; jj < KTOP; ++jj) out[jj] = m.v[jj];
    }
  }
}

namespace {

// Largest query-tile count per workgroup for each list size (registers).
constexpr int sem_tq_limit(int ktop) { return ktop == 1 ? 8 : 4; }

// LDS: four query ring slots and the query norms; the merge buffer reuses
// the ring.
size_t sem_lds(int TQ, int KTOP) {
  size_t ring = static_cast<size_t>(4) * TQ * 2 * 1024;
  const size_t merge = static_cast<size_t>(8) * 16 * TQ * KTOP * 8;
  if (merge > ring) ring = merge;
  return ring + static_cast<size_t>(16) * TQ * 4;
}

template <int TQ, int KTOP, bool DBG = false>
hipError_t sem_launch(const SemArgs& a, hipStream_t st) {
  const size_t lds = sem_lds(TQ, KTOP);
  auto kern = k_sem_scan<TQ, KTOP, DBG>;
  if (lds > 64 * 1024) {
    const hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (err != hipSuccess) return err;
  }
  const ScanEvents& ev = scan_events();
  if (ev.start != nullptr) {
    const hipError_t err = hipEventRecord(ev.start, st);
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(512), lds, st, a);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess || ev.stop == nullptr) return err;
  return hipEventRecord(ev.stop, st);
}

template <int KTOP, bool DBG = false>
hipError_t sem_tq(int TQ, const SemArgs& a, hipStream_t st) {
  switch (TQ) {
    case 1: return sem_launch<1, KTOP, DBG>(a, st);
    case 2: return sem_launch<2, KTOP, DBG>(a, st);
    case 4: return sem_launch<4, KTOP, DBG>(a, st);
    case 8:
      if constexpr (sem_tq_limit(KTOP) >= 8) return sem_launch<8, KTOP, DBG>(a, st);
      break;
    default: break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_match_semantic(const StoreView& s, const void* q, int32_t B, int32_t k, int32_t* idx_out,
                                 float* score_out, float* dbg_scores, const Workspace& ws, hipStream_t st,
                                 const float* mix, double w_self, double w_mix, const SelectFuse* fuse) {
  const int KTOP = k == 1 ? 1 : (k <= 4 ? 4 : 8);
  // the dense-output form keeps top-1 lists (k = 1)
  const int tq_max = sem_tq_limit(dbg_scores != nullptr ? 1 : KTOP);
  const int n_blocks = (s.n + 15) / 16;
  // top-1 searches and the dense form (which keeps no lists there) run on
  // the 128 x 128 wave-tile scan (fm_sem_mm.hip); lists of 4 or 8, and a
  // dense form that also returns matches, on the general scan
  const bool mm = dbg_scores != nullptr ? idx_out == nullptr : KTOP == 1 && mix == nullptr;
  for (int b0 = 0; b0 < B; b0 += kChunkB) {
    const int Bc = (B - b0) < kChunkB ? (B - b0) : kChunkB;
    int TQ = 1;
    while (16 * TQ < Bc && TQ < tq_max) TQ *= 2;
    if (mm) TQ = sem_mm_group(Bc) / 16;
    const int QG = 16 * TQ;
    const int n_qg = (Bc + QG - 1) / QG;
    const int b_pad = n_qg * QG;

    SemPrepArgs pa;
    pa.q = static_cast<const uint16_t*>(q) + static_cast<int64_t>(b0) * s.d_emb;
    pa.B = Bc;
    pa.d = s.d_emb;
    pa.b_pad = b_pad;
    pa.qst = static_cast<uint16_t*>(ws.qrows);
    pa.rq = ws.rq;
    hipLaunchKernelGGL(k_sem_prep, dim3((b_pad + 3) / 4), dim3(256), 0, st, pa);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    if (mm) {
      int R = 1;
      err = launch_sem_mm(s, Bc, b_pad, ws, dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr,
                          &R, st, mix != nullptr ? mix + static_cast<int64_t>(b0) * s.n : nullptr, w_self, w_mix);
      if (err != hipSuccess) return err;
      if (idx_out != nullptr) {
        err = fuse != nullptr
                  ? launch_merge_select(s, ws.partial, nullptr, Bc, R, k, 1, nullptr, 0,
                                        idx_out + static_cast<int64_t>(b0) * k,
                                        score_out + static_cast<int64_t>(b0) * k, fuse->at(b0, s.L), st)
                  : launch_finalize(ws.partial, nullptr, Bc, R, k, 1, idx_out + static_cast<int64_t>(b0) * k,
                                    score_out + static_cast<int64_t>(b0) * k, st);
        if (err != hipSuccess) return err;
      }
      continue;
    }

    // workgroups per query group: about one workgroup per CU in total, each
    // with an even share of the blocks (at least one)
    int R = 256 / n_qg;
    if (R < 1) R = 1;
    if (R > n_blocks) R = n_blocks > 0 ? n_blocks : 1;
    if (R > kMaxPartials) R = kMaxPartials;

    SemArgs a;
    a.x = s.embs;
    a.x_bytes = round16(s.cap) * static_cast<int64_t>(s.d_emb) * 2;
    a.xnorm = s.emb_norm;
    a.n = s.n;
    a.d = s.d_emb;
    a.B = Bc;
    a.n_qg = n_qg;
    a.R = R;
    a.n_blocks = n_blocks;
    a.grid = (n_qg * R + 7) / 8 * 8;
    a.ws = ws;
    a.dbg = dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr;
    a.mix = mix != nullptr ? mix + static_cast<int64_t>(b0) * s.n : nullptr;
    a.w_self = w_self;
    a.w_mix = w_mix;
    if (dbg_scores != nullptr) err = sem_tq<1, true>(TQ, a, st);
    else if (KTOP == 1) err = sem_tq<1>(TQ, a, st);
    else if (KTOP == 4) err = sem_tq<4>(TQ, a, st);
    else err = sem_tq<8>(TQ, a, st);
    if (err != hipSuccess) return err;
    if (idx_out != nullptr) {
      err = fuse != nullptr
                ? launch_merge_select(s, ws.partial, nullptr, Bc, R, k, KTOP, nullptr, 0,
                                      idx_out + static_cast<int64_t>(b0) * k, score_out + static_cast<int64_t>(b0) * k,
                                      fuse->at(b0, s.L), st)
                : launch_finalize(ws.partial, nullptr, Bc, R, k, KTOP, idx_out + static_cast<int64_t>(b0) * k,
                                  score_out + static_cast<int64_t>(b0) * k, st);
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

}  // namespace fm
