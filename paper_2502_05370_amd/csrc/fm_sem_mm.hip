// Semantic-based expert map search (Section 4.2.1, Eq. 4), top-1 form.
//
// The batched search is the contraction Q X^T of the query embeddings
// (B x d) with the stored embeddings (n x d), both bf16, on
// v_mfma_f32_16x16x32_bf16 (exact bf16 products, float32 accumulation),
// followed by the cosine scaling and the best stored index per query.  This
// kernel serves searches that keep one match per query; k_sem_scan
// (fm_sem.hip) serves top-4/8 lists and the dense forms of the deduplicating
// insert.  k_sem_prep stages the queries in the embedding tile layout and
// writes 1/|q| before it runs; k_finalize merges its partial lists after.
//
// Workgroup: 4 waves, one per SIMD, arranged GQ x GM over (queries, maps).
// Wave (wq, wm) holds 128 x 128 float32 accumulators: the group's query
// tiles 8 wq .. 8 wq + 7 (16 queries each) against the map blocks wm,
// wm + GM, ... of a slice (16 maps each, interleaved so that a short last
// slice still splits evenly over the waves).  Per k-step of 32 dimensions a
// wave reads 16 operand fragments (16 KB) from LDS for 64 MFMAs, i.e. 64
// bytes per clock per CU at the MFMA rate, half of what a 128 x 32 wave tile
// needs.
//
// Pipeline: a stage is one k-step of one slice (8 GM blocks of the
// workgroup's block range).  Its map tiles and the group's query tiles are
// 1 KB MFMA operand tiles in HBM (emb_offset), copied global -> LDS by
// buffer loads straight into ring slot j % NS.  At the start of stage j,
// once its own copies of stage j+1 have landed, each wave passes the one
// barrier of the stage; ring slot j % NS, whose fragments every wave already
// holds in registers, then receives the copies of stage j + NS, and the
// fragments of stage j+1 are read from LDS while the MFMAs of stage j run.
// Every stage issues the same number of copies per wave (copies past the
// last stage use offsets past every descriptor: zeros, no memory traffic),
// so "stage j+1 has landed" is a fixed vmcnt bound.  The map norms of a
// slice are copied with its first stage into one of two buffers.
//
// Epilogue of a slice: lane (g, c) holds, for block i and query tile t, the
// dots of maps 4g .. 4g+3 of the block with query c of the tile; the cosine
// is (dot * 1/|q|) * 1/|x| and the lane keeps the best (score, index) per
// query tile.  Maps are visited in increasing index order and only a
// strictly better score replaces the kept one, so equal scores keep the
// lower index; a NaN score is taken as -2 (below every cosine, above "no
// match").  The lists are merged over lane groups and waves and stored as
// the workgroup's partial list (one packed key per query).
#include <type_traits>

#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

struct SemMmArgs {
  const uint16_t* x;     // tiled embeddings
  const float* xnorm;    // [cap] |x|
  const uint16_t* qst;   // staged queries, tiled like the embeddings
  const float* rq;       // [b_pad] 1/|q|
  uint64_t* partial;     // [b_pad][R]: one packed key per (query, workgroup of its group)
  float* dbg;            // optional dense scores [B][n]
  int32_t n, ksteps, B;
  int32_t n_qg;          // query groups
  int32_t R;             // workgroups per query group
  int32_t n_blocks;      // 16-map blocks of the store
  int32_t grid;
};

// Position of stage j: slice si, k-step ks and ring slot, stepped without
// divisions.
struct MmPos {
  int j, si, ks, slot;
};

template <int NS>
__device__ __forceinline__ MmPos mm_next(const MmPos& p, int ksteps) {
  MmPos q;
  q.j = p.j + 1;
  const bool wrap = p.ks + 1 == ksteps;
  q.ks = wrap ? 0 : p.ks + 1;
  q.si = wrap ? p.si + 1 : p.si;
  q.slot = p.slot + 1 == NS ? 0 : p.slot + 1;
  return q;
}

template <int GQ>
struct MmShape {
  static constexpr int GM = 4 / GQ;
  static constexpr int NT = 8;                  // query tiles per wave
  static constexpr int NB = 6;                  // map blocks per wave and slice
  static constexpr int QG = 16 * NT * GQ;       // queries per group
  static constexpr int SB = NB * GM;            // map blocks per slice
  static constexpr int NS = 4;                  // ring slots
  static constexpr int TILES = SB + QG / 16;    // 1 KB tiles per stage
  static constexpr int MPW = SB / 4;            // map tile copies per wave and stage
  static constexpr int QPW = QG / 64;           // query tile copies per wave and stage
  static constexpr int NI = MPW + QPW;          // tile copies per wave and stage
  static constexpr int SLOT = TILES * 1024;
  static constexpr int NNORM = (SB * 16 * 4 + 1023) / 1024;   // 1 KB copies of one slice's map norms
  static constexpr int NSTRIDE = NNORM * 256;   // floats per norm buffer
  static constexpr int LDS = NS * SLOT + 2 * NNORM * 1024;
};

}  // namespace

template <int GQ, bool DBG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) k_sem_mm(SemMmArgs a) {
  using S = MmShape<GQ>;
  constexpr int GM = S::GM, NT = S::NT, NB = S::NB, QG = S::QG, SB = S::SB, NS = S::NS, NI = S::NI;
  constexpr int MPW = S::MPW, QPW = S::QPW;
  constexpr int SLOT = S::SLOT, NNORM = S::NNORM, NSTRIDE = S::NSTRIDE;
  static_assert(SB % 4 == 0 && QG % 64 == 0 && (NS - 1) * NI < 64, "tile copies per stage");
  static_assert(S::LDS <= 160 * 1024, "LDS");

  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                    // [NS][SLOT]
  float* xnb = reinterpret_cast<float*>(smem + NS * SLOT);       // [2][NSTRIDE] map norms
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(smem);            // after the loop: [GM][QG]

  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wq = w / GM;
  const int wm = w - wq * GM;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;

  // workgroup -> (query group, block range); the groups sharing a block
  // range are consecutive in u, hence on one XCD, and read the same map
  // tiles at about the same time (the later reads hit that XCD's L2)
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  const bool active = u < a.n_qg * a.R;
  const int qgrp = active ? u % a.n_qg : 0;
  const int rr = active ? u / a.n_qg : 0;
  const int b_begin = active ? static_cast<int>((static_cast<int64_t>(rr) * a.n_blocks) / a.R) : 0;
  const int b_end = active ? static_cast<int>((static_cast<int64_t>(rr + 1) * a.n_blocks) / a.R) : 0;
  const int n_slices = (b_end - b_begin + SB - 1) / SB;
  const int g0 = qgrp * QG;
  const int ksteps = a.ksteps;
  const int nstages = n_slices * ksteps;
  const int64_t blk_bytes = static_cast<int64_t>(ksteps) * 1024;

  float rqv[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) rqv[t] = a.rq[g0 + 16 * (NT * wq + t) + c];
  float best_s[NT];
  int best_i[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    best_s[t] = kEmptyScore;
    best_i[t] = -1;
  }

  if (nstages > 0) {
    const char* xb = reinterpret_cast<const char*>(a.x);
    const char* qbase = reinterpret_cast<const char*>(a.qst) + static_cast<int64_t>(g0 / 16) * blk_bytes;
    const __amdgpu_buffer_rsrc_t rs_q = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(qbase), static_cast<short>(0),
        static_cast<int>(static_cast<uint32_t>(QG / 16) * static_cast<uint32_t>(blk_bytes)), kBufWord3);
    const __amdgpu_buffer_rsrc_t rs_norm = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.xnorm), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(a.n) * 4u),
        kBufWord3);

    // Copies of the stage at position p into its ring slot.  Map tiles go
    // through a descriptor based at the slice's first block whose range ends
    // with the workgroup's blocks (rebuilt at each slice's first stage), so
    // blocks past the range read as zeros; positions past the last stage use
    // offsets past every descriptor.
    __amdgpu_buffer_rsrc_t rs_slice = rs_norm;
    auto load_stage = [&](const MmPos& p) __attribute__((always_inline)) {
      const bool real = p.j < nstages;
      if (!real || p.ks == 0) {
        const int blk0 = b_begin + (real ? p.si : 0) * SB;
        int64_t rem = real ? static_cast<int64_t>(b_end - blk0) * blk_bytes : 0;
        if (rem > static_cast<int64_t>(SB) * blk_bytes) rem = static_cast<int64_t>(SB) * blk_bytes;
        rs_slice = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(xb + static_cast<int64_t>(blk0) * blk_bytes),
                                                     static_cast<short>(0),
                                                     static_cast<int>(static_cast<uint32_t>(rem)), kBufWord3);
      }
      unsigned char* slot = ring + p.slot * SLOT;
      const uint32_t kofs = real ? static_cast<uint32_t>(p.ks * 1024 + lane * 16) : kOutside;
      // wave w copies map tiles w * MPW .. and query tiles w * QPW ..
#pragma unroll
      for (int i = 0; i < MPW; ++i) {
        const int tile = w * MPW + i;
        const uint32_t off = real ? static_cast<uint32_t>(tile) * static_cast<uint32_t>(blk_bytes) + kofs : kOutside;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_slice, (lds_vp)(slot + tile * 1024), 16, static_cast<int>(off), 0, 0,
                                                 0);
      }
#pragma unroll
      for (int i = 0; i < QPW; ++i) {
        const int tile = w * QPW + i;
        const uint32_t off = real ? static_cast<uint32_t>(tile) * static_cast<uint32_t>(blk_bytes) + kofs : kOutside;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_q, (lds_vp)(slot + (SB + tile) * 1024), 16, static_cast<int>(off), 0,
                                                 0, 0);
      }
      // the slice's map norms, with its first stage
      if (real && p.ks == 0 && w < NNORM) {
        const uint32_t off = static_cast<uint32_t>(((b_begin + p.si * SB) * 16 + w * 256 + lane * 4) * 4);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_norm, (lds_vp)(xnb + (p.si & 1) * NSTRIDE + w * 256), 16,
                                                 static_cast<int>(off), 0, 0, 0);
      }
    };

    floatx4 acc[NB][NT];
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto read_frags = [&](int slot, u16x8 (&fa)[NB], u16x8 (&fb)[NT]) __attribute__((always_inline)) {
      const unsigned char* sp = ring + slot * SLOT + lane * 16;
#pragma unroll
      for (int i = 0; i < NB; ++i) fa[i] = *reinterpret_cast<const u16x8*>(sp + (wm + GM * i) * 1024);
#pragma unroll
      for (int t = 0; t < NT; ++t) fb[t] = *reinterpret_cast<const u16x8*>(sp + (SB + NT * wq + t) * 1024);
    };

    // Slice epilogue: scores of this wave's blocks of slice si, best per query.
    auto epilogue = [&](int si) __attribute__((always_inline)) {
      const int blk_s = b_begin + si * SB;
      const float* xn_s = xnb + (si & 1) * NSTRIDE;
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int blk = blk_s + wm + GM * i;
        if (blk >= b_end) break;
        const floatx4 xn = *reinterpret_cast<const floatx4*>(xn_s + (wm + GM * i) * 16 + 4 * g);
        float rx[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) rx[r] = xn[r] > 0.0f ? 1.0f / xn[r] : (xn[r] != xn[r] ? xn[r] : 0.0f);
        const int y0 = 16 * blk + 4 * g;
        const bool full = 16 * blk + 16 <= a.n;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int y = y0 + r;
            const float s = acc[i][t][r] * rqv[t] * rx[r];
            if constexpr (DBG) {
              const int b = g0 + 16 * (NT * wq + t) + c;
              if (b < a.B && y < a.n) a.dbg[static_cast<int64_t>(b) * a.n + y] = s;
            }
            // NaN -> -2 (maximum of a NaN and a number is the number)
            const float sv = __builtin_fmaxf(s, kNanScore);
            if ((full || y < a.n) && sv > best_s[t]) {
              best_s[t] = sv;
              best_i[t] = y;
            }
          }
        }
        // one block's accumulators at a time
        __builtin_amdgcn_sched_barrier(0);
      }
      // the next slice accumulates from zero; the empty asm keeps the
      // compiler from treating the accumulators as known zeros (it would
      // then build the first MFMAs of a slice from a shared zero register)
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
    };

    // prologue: the copies of stages 0 .. NS-1, then stage 0's fragments
    MmPos pl{0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      load_stage(pl);
      pl = mm_next<NS>(pl, ksteps);
    }
    u16x8 fa0[NB], fb0[NT], fa1[NB], fb1[NT];
    wait_vmcnt<(NS - 1) * NI>();
    raw_barrier();
    read_frags(0, fa0, fb0);
    wait_lgkm0();

    // One stage: MFMAs of the first NBV blocks from fragments (fa, fb),
    // copies of stage j + NS, fragments of stage j+1 into (na, nb).  The
    // accumulators of blocks NBV.. are left alone (zero in a short slice).
    int slot_next = 1 % NS;
    int nbv_rt = NB;   // blocks of this wave in a short slice
    auto stage = [&](auto nbv_const, u16x8 (&fa)[NB], u16x8 (&fb)[NT], u16x8 (&na)[NB], u16x8 (&nb)[NT])
                     __attribute__((always_inline)) {
      constexpr int NBV = decltype(nbv_const)::value;
      // stage j+1's copies have landed (this wave's, then everyone's), and
      // every wave holds stage j's fragments: slot j % NS is free
      wait_vmcnt<(NS - 2) * NI>();
      raw_barrier();
      load_stage(pl);
      pl = mm_next<NS>(pl, ksteps);
      read_frags(slot_next, na, nb);
      slot_next = slot_next + 1 == NS ? 0 : slot_next + 1;
      if constexpr (NBV == NB) {
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[i][t] = mfma_bf16(fa[i], fb[t], acc[i][t]);
        // issue order: the copies and the fragment reads spread between the
        // stage's MFMAs, then the wait for the reads
        constexpr int NR = NB + NT;                    // fragment reads
        constexpr int NM = NB * NT;                    // MFMAs
        constexpr int PER = NM / (NI + NR) > 0 ? NM / (NI + NR) : 1;
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one copy
          __builtin_amdgcn_sched_group_barrier(0x008, PER, 0); // MFMAs
        }
#pragma unroll
        for (int k = 0; k < NR; ++k) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one fragment read
          __builtin_amdgcn_sched_group_barrier(0x008, PER, 0); // MFMAs
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);    // the remaining MFMAs
      } else {
        // the short last slice: only the blocks below b_end (nbv_rt of them)
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          if (i < nbv_rt) {
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[i][t] = mfma_bf16(fa[i], fb[t], acc[i][t]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      wait_lgkm0();
    };
    // all k-steps of one slice (ksteps is a multiple of 4)
    auto slice = [&](auto nbv_const) __attribute__((always_inline)) {
      for (int ks = 0; ks < ksteps; ks += 2) {
        stage(nbv_const, fa0, fb0, fa1, fb1);
        stage(nbv_const, fa1, fb1, fa0, fb0);
      }
    };
    const int n_full = (b_end - b_begin) / SB;
    for (int si = 0; si < n_full; ++si) {
      slice(std::integral_constant<int, NB>{});
      epilogue(si);
    }
    if (n_full < n_slices) {
      // the short last slice: this wave's blocks wm, wm + GM, ... below b_end
      const int rem = b_end - (b_begin + n_full * SB) - wm;
      nbv_rt = rem <= 0 ? 0 : (rem + GM - 1) / GM;
      slice(std::integral_constant<int, 0>{});
      epilogue(n_full);
    }
    wait_vmcnt<0>();   // the trailing copies
  }
  __syncthreads();

  // merge: the four lane groups of a query, then the GM waves of its tile row
  uint64_t key[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    key[t] = best_i[t] < 0 ? 0ull : make_key(best_s[t], best_i[t]);
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      const uint64_t o = shfl_xor_u64(key[t], m);
      key[t] = o > key[t] ? o : key[t];
    }
  }
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < NT; ++t) mbuf[wm * QG + 16 * (NT * wq + t) + c] = key[t];
  }
  __syncthreads();
  if (active) {
    for (int r = tid; r < QG; r += 4 * kWave) {
      uint64_t m = 0;
#pragma unroll
      for (int ww = 0; ww < GM; ++ww) m = mbuf[ww * QG + r] > m ? mbuf[ww * QG + r] : m;
      a.partial[static_cast<int64_t>(g0 + r) * a.R + rr] = m;
    }
  }
}

namespace {

template <int GQ, bool DBG>
hipError_t sem_mm_launch(const SemMmArgs& a, hipStream_t st) {
  constexpr size_t lds = MmShape<GQ>::LDS;
  auto kern = k_sem_mm<GQ, DBG>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       static_cast<int>(lds));
  if (err != hipSuccess) return err;
  const ScanEvents& ev = scan_events();
  if (ev.start != nullptr) {
    err = hipEventRecord(ev.start, st);
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(256), lds, st, a);
  err = hipGetLastError();
  if (err != hipSuccess || ev.stop == nullptr) return err;
  return hipEventRecord(ev.stop, st);
}

}  // namespace

int sem_mm_group(int32_t Bc) { return Bc > 128 ? 256 : 128; }

hipError_t launch_sem_mm(const StoreView& s, int32_t Bc, int32_t b_pad, const Workspace& ws, float* dbg, int32_t* R_out,
                         hipStream_t st) {
  const int QG = sem_mm_group(Bc);
  const int n_qg = b_pad / QG;
  const int n_blocks = (s.n + 15) / 16;
  // workgroups per query group: one per CU in total, each with an even share
  // of the blocks (at least one)
  int R = 256 / n_qg;
  if (R < 1) R = 1;
  if (R > n_blocks) R = n_blocks > 0 ? n_blocks : 1;
  if (R > kMaxPartials) R = kMaxPartials;
  SemMmArgs a;
  a.x = s.embs;
  a.xnorm = s.emb_norm;
  a.qst = static_cast<const uint16_t*>(ws.qrows);
  a.rq = ws.rq;
  a.partial = ws.partial;
  a.dbg = dbg;
  a.n = s.n;
  a.ksteps = s.d_emb / 32;
  a.B = Bc;
  a.n_qg = n_qg;
  a.R = R;
  a.n_blocks = n_blocks;
  a.grid = (n_qg * R + 7) / 8 * 8;
  *R_out = R;
  if (QG == 256) return dbg != nullptr ? sem_mm_launch<2, true>(a, st) : sem_mm_launch<2, false>(a, st);
  return dbg != nullptr ? sem_mm_launch<1, true>(a, st) : sem_mm_launch<1, false>(a, st);
}

}  // namespace fm
