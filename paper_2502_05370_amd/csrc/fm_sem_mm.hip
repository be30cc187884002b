// Semantic-based expert map search (Section 4.2.1, Eq. 4), top-1 form.
//
// The batched search is the contraction Q X^T of the query embeddings
// (B x d) with the stored embeddings (n x d), both bf16, on
// v_mfma_f32_16x16x32_bf16 (exact bf16 products, float32 accumulation),
// followed by the cosine scaling and the best stored index per query.  This
// kernel serves searches that keep one match per query and the dense form
// (every cosine, or its weighted sum with a second dense matrix: the
// deduplicating insert's RDY); k_sem_scan (fm_sem.hip) serves top-2..8
// lists.  k_sem_prep stages the queries in the embedding tile layout and
// writes 1/|q| before it runs; k_finalize (or k_merge_select, with the
// selection) merges its partial lists after.
//
// Workgroup: 8 waves, two per SIMD (two waves on a SIMD let one issue its
// LDS reads and copies while the other's MFMAs run), arranged GQ x GM over
// (queries, maps).  Wave (wq, wm) holds 128 x 64 float32 accumulators: the
// group's query tiles 8 wq .. 8 wq + 7 (16 queries each) against the map
// blocks wm, wm + GM, wm + 2 GM, wm + 3 GM of a slice (16 maps each).  Per
// k-step of 32 dimensions a wave reads 12 operand fragments (12 KB) from LDS
// for 32 MFMAs.
//
// Pipeline: a stage is one k-step of one slice (4 GM blocks of the
// workgroup's block range).  Its map tiles and the group's query tiles are
// 1 KB MFMA operand tiles in HBM (emb_offset), copied global -> LDS by
// buffer loads straight into ring slot j % NS.  At the start of stage j,
// once its own copies of stage j+1 have landed, each wave passes the one
// barrier of the stage; ring slot j % NS, whose fragments every wave already
// holds in registers, then receives the copies of stage j + NS, and the
// fragments of stage j+1 are read from LDS while the MFMAs of stage j run
// (the map fragments into a second register set, each query fragment into
// its register as soon as the MFMAs of its tile have read it).  Every stage
// issues the same copies per wave (copies past the last stage use offsets
// past every descriptor: zeros, no memory traffic), so "stage j+1 has
// landed" is a fixed vmcnt bound.  The map norms of a slice are copied into
// one of two buffers by one more copy of wave 0 at the slice's first stage
// (issued before that stage's tile copies, so the bound still holds).

// Epilogue of a slice: lane (g, c) holds, for block i and query tile t, the
// dots of maps 4g .. 4g+3 of the block with query c of the tile.  The top-1
// form ranks them by dot * 1/|x| (the query's factor 1/|q| is positive, or
// 0 for a zero query, and is applied once after the scan) and keeps the best
// (score, index) per query tile: maps are visited in increasing index order
// and only a strictly greater score replaces the kept one, so equal scores
// keep the lower index, and a NaN score ranks below every other.  The lists
// are merged over lane groups and waves and stored as the workgroup's
// partial list (one packed key per query).  The dense form writes the
// cosines (dot * 1/|q| * 1/|x|) instead, a lane's 4 maps of a row as one
// 16-byte store where the row allows it, and keeps no lists.
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
  // dense form only: the score written is w_self * cosine + w_mix * mix[b][y]
  // (float64, rounded once) when mix is set
  const float* mix;
  double w_self, w_mix;
  int32_t vec16;         // dense rows written (and mix read) 16 bytes at a time: n % 4 == 0, aligned buffers
  int32_t n, ksteps, B;
  int32_t n_qg;          // query groups
  int32_t R;             // workgroups per query group
  int32_t n_blocks;      // 16-map blocks of the store
  int32_t grid;
};

template <int GQ>
struct MmShape {
  static constexpr int W = 8;                   // waves per workgroup (two per SIMD)
  static constexpr int GM = W / GQ;
  static constexpr int NT = 8;                  // query tiles per wave
  static constexpr int NB = 4;                  // map blocks per wave and slice
  static constexpr int QG = 16 * NT * GQ;       // queries per group
  static constexpr int SB = NB * GM;            // map blocks per slice
  static constexpr int NS = GQ == 2 ? 4 : 3;    // ring slots
  static constexpr int TILES = SB + QG / 16;    // 1 KB tiles per stage
  static constexpr int MPW = SB / W;            // map tile copies per wave and stage
  static constexpr int QPW = QG / 16 / W;       // query tile copies per wave and stage
  static constexpr int NI = MPW + QPW;          // tile copies per wave and stage
  static constexpr int SLOT = TILES * 1024;
  static constexpr int NNORM = (SB * 16 * 4 + 1023) / 1024;   // 1 KB copies of one slice's map norms
  static constexpr int NSTRIDE = NNORM * 256;   // floats per norm buffer
  static constexpr int LDS = NS * SLOT + 2 * NNORM * 1024;
};

}  // namespace

template <int GQ, bool DBG>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) k_sem_mm(SemMmArgs a) {
  using S = MmShape<GQ>;
  constexpr int W = S::W, GM = S::GM, NT = S::NT, NB = S::NB, QG = S::QG, SB = S::SB, NS = S::NS, NI = S::NI;
  constexpr int MPW = S::MPW, QPW = S::QPW;
  constexpr int SLOT = S::SLOT, NNORM = S::NNORM, NSTRIDE = S::NSTRIDE;
  static_assert(SB % W == 0 && (QG / 16) % W == 0 && (NS - 1) * NI < 64 && NNORM <= W, "copies per stage");
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
  // (wave-uniform: stated, so that what is derived from them stays scalar)
  const int b_begin =
      __builtin_amdgcn_readfirstlane(active ? static_cast<int>((static_cast<int64_t>(rr) * a.n_blocks) / a.R) : 0);
  const int b_end =
      __builtin_amdgcn_readfirstlane(active ? static_cast<int>((static_cast<int64_t>(rr + 1) * a.n_blocks) / a.R) : 0);
  const int n_slices = (b_end - b_begin + SB - 1) / SB;
  const int g0 = qgrp * QG;
  const int ksteps = a.ksteps;
  const int nstages = n_slices * ksteps;
  const uint32_t blk32 = static_cast<uint32_t>(ksteps) * 1024u;   // bytes of one 16-row block (d < 2^21)

  // Best map per query tile, ranked by dot * 1/|x|: the query's factor 1/|q|
  // is positive (or 0 for a zero query, where every score is 0) and does not
  // change the order, so it is applied once at the end.  A NaN score ranks
  // below every other score: the list starts at the lane's first map with
  // the lowest finite float, which only a greater score replaces (a NaN
  // compares false).
  constexpr float kNanFloor = -3.40282347e38f;
  const int y_first = 16 * (b_begin + wm) + 4 * g;
  const bool first_ok = b_begin + wm < b_end && y_first < a.n;
  float best_s[NT];
  int best_i[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    best_s[t] = kNanFloor;
    best_i[t] = first_ok ? y_first : -1;
  }

  if (nstages > 0) {
    const char* qbase = reinterpret_cast<const char*>(a.qst) + static_cast<uint64_t>(g0 / 16) * blk32;
    const __amdgpu_buffer_rsrc_t rs_q = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(qbase), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(QG / 16) * blk32),
        kBufWord3);
    const __amdgpu_buffer_rsrc_t rs_norm = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.xnorm), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(a.n) * 4u),
        kBufWord3);

    // The copies run NS stages ahead of the MFMAs.  Their position (the
    // "copy position") is kept as running scalars stepped by one stage per
    // stage: its slice's first block and map descriptor, its k-step's byte
    // offset within a block (the loads' scalar offset), the stages left in
    // its slice, and the norm buffer its slice fills; the vector offsets of
    // this wave's tiles are fixed.  (Scalar instructions issue one per SIMD
    // every fourth cycle, shared by both waves of a SIMD.)
    int c_blk0 = b_begin;
    uint32_t c_kofs = 0;
    int c_left = ksteps;
    int c_nb = 0;          // norm buffer of the copy position's slice
    int c_slot = 0;        // ring slot of the current stage = slot of the copy position
    uint64_t c_xbase = reinterpret_cast<uint64_t>(a.x) + static_cast<uint64_t>(static_cast<uint32_t>(b_begin)) * blk32;
    uint32_t c_xrec;
    {
      int nbk = b_end - b_begin;
      nbk = nbk < 0 ? 0 : (nbk > SB ? SB : nbk);
      c_xrec = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(nbk) * blk32);
    }
    // this wave's map tiles w * MPW + i and query tiles w * QPW + i: the
    // tile's block offset plus the lane's 16 bytes
    uint32_t vmo[MPW], vqo[QPW];
#pragma unroll
    for (int i = 0; i < MPW; ++i) vmo[i] = static_cast<uint32_t>(w * MPW + i) * blk32 + static_cast<uint32_t>(lane * 16);
#pragma unroll
    for (int i = 0; i < QPW; ++i) vqo[i] = static_cast<uint32_t>(w * QPW + i) * blk32 + static_cast<uint32_t>(lane * 16);
    const uint32_t vno = static_cast<uint32_t>((w * 256 + lane * 4) * 4);

    // Copies of the copy position into the current stage's slot: at a
    // slice's first k-step the slice's map norms (waves below NNORM), then
    // the map tiles (blocks past the workgroup's range lie past the slice's
    // descriptor) and the query tiles.
    auto issue = [&]() __attribute__((always_inline)) {
      // (two uniform branches: the common path is one compare and branch)
      if (__builtin_expect(c_kofs == 0, 0)) {
        if (w < NNORM)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_norm, (lds_vp)(xnb + c_nb * NSTRIDE + w * 256), 16,
                                                   static_cast<int>(static_cast<uint32_t>(c_blk0) * 64u + vno), 0, 0,
                                                   0);
      }
      unsigned char* slot = ring + c_slot * SLOT;
      const __amdgpu_buffer_rsrc_t rs_slice = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<char*>(c_xbase), static_cast<short>(0), static_cast<int>(c_xrec), kBufWord3);
#pragma unroll
      for (int i = 0; i < MPW; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_slice, (lds_vp)(slot + (w * MPW + i) * 1024), 16,
                                                 static_cast<int>(vmo[i]), static_cast<int>(c_kofs), 0, 0);
#pragma unroll
      for (int i = 0; i < QPW; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_q, (lds_vp)(slot + (SB + w * QPW + i) * 1024), 16,
                                                 static_cast<int>(vqo[i]), static_cast<int>(c_kofs), 0, 0);
    };
    // the next ring slot (a mask when NS is a power of two)
    auto next_slot = [&](int sl) __attribute__((always_inline)) {
      if constexpr ((NS & (NS - 1)) == 0) return (sl + 1) & (NS - 1);
      else return sl == NS - 1 ? 0 : sl + 1;
    };
    auto step_copy = [&]() __attribute__((always_inline)) {
      c_slot = next_slot(c_slot);
      c_kofs += 1024u;
      if (__builtin_expect(--c_left == 0, 0)) {
        c_left = ksteps;
        c_kofs = 0;
        c_blk0 += SB;
        c_nb ^= 1;
        c_xbase += static_cast<uint64_t>(SB) * blk32;
        int nbk = b_end - c_blk0;
        nbk = nbk < 0 ? 0 : (nbk > SB ? SB : nbk);
        c_xrec = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(nbk) * blk32);
      }
    };

    floatx4 acc[NB][NT];
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto read_mfrag = [&](int slot, int i) __attribute__((always_inline)) {
      return *reinterpret_cast<const u16x8*>(ring + slot * SLOT + lane * 16 + (wm + GM * i) * 1024);
    };
    auto read_qfrag = [&](int slot, int t) __attribute__((always_inline)) {
      return *reinterpret_cast<const u16x8*>(ring + slot * SLOT + lane * 16 + (SB + NT * wq + t) * 1024);
    };

    // Slice epilogue: scores of this wave's blocks of slice si, best per query.
    auto epilogue = [&](int si) __attribute__((always_inline)) {
      const int blk_s = b_begin + si * SB;
      const float* xn_s = xnb + (si & 1) * NSTRIDE;
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int blk = blk_s + wm + GM * i;
        if (blk >= b_end) break;
        // The norms were copied into LDS with the slice's first stage, and
        // the stage waits have covered that copy; a plain LDS read here would
        // make the compiler wait for every copy still in flight, so the read
        // is written out, with its own wait that the value depends on.
        floatx4 xn;
        const uint32_t xaddr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(xn_s + (wm + GM * i) * 16 + 4 * g));
        asm volatile("ds_read_b128 %0, %1" : "=v"(xn) : "v"(xaddr));
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xn));
        // 1/|x| (within one unit in the last place; 0 for a zero norm, NaN for NaN)
        float rx[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) rx[r] = xn[r] > 0.0f ? __builtin_amdgcn_rcpf(xn[r]) : (xn[r] != xn[r] ? xn[r] : 0.0f);
        const int y0 = 16 * blk + 4 * g;
        // rows past the store (the last block) score NaN: never kept
#pragma unroll
        for (int r = 0; r < 4; ++r) rx[r] = y0 + r < a.n ? rx[r] : __builtin_nanf("");
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if constexpr (DBG) {
            // The dense form writes every cosine (or its weighted sum with
            // mix) and keeps no lists: the lane's 4 consecutive maps of its
            // query as one 16-byte store where the row allows it.
            const int b = g0 + 16 * (NT * wq + t) + c;
            if (b < a.B) {
              const int64_t o = static_cast<int64_t>(b) * a.n + y0;
              const bool whole = a.vec16 != 0 && y0 + 3 < a.n;
              const float rqb = a.rq[b];
              floatx4 v;
#pragma unroll
              for (int r = 0; r < 4; ++r) v[r] = acc[i][t][r] * rqb * rx[r];
              if (a.mix != nullptr) {
                floatx4 mv = floatx4{0.f, 0.f, 0.f, 0.f};
                if (whole) {
                  mv = *reinterpret_cast<const floatx4*>(a.mix + o);
                } else {
#pragma unroll
                  for (int r = 0; r < 4; ++r)
                    if (y0 + r < a.n) mv[r] = a.mix[o + r];
                }
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  v[r] = static_cast<float>(__dadd_rn(__dmul_rn(a.w_self, static_cast<double>(v[r])),
                                                      __dmul_rn(a.w_mix, static_cast<double>(mv[r]))));
              }
              if (whole) {
                *reinterpret_cast<floatx4*>(a.dbg + o) = v;
              } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (y0 + r < a.n) a.dbg[o + r] = v[r];
              }
            }
            continue;
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float sv = acc[i][t][r] * rx[r];
            if (sv > best_s[t]) {
              best_s[t] = sv;
              best_i[t] = y0 + r;
            }
          }
        }
        // one block's accumulators at a time
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    };

    // prologue: the copies of stages 0 .. NS-1, then stage 0's fragments
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      issue();
      step_copy();
    }
    u16x8 fa0[NB], fa1[NB], fb[NT];
    wait_vmcnt<(NS - 1) * NI>();
    raw_barrier();
#pragma unroll
    for (int i = 0; i < NB; ++i) fa0[i] = read_mfrag(0, i);
#pragma unroll
    for (int t = 0; t < NT; ++t) fb[t] = read_qfrag(0, t);
    wait_lgkm0();

    // One stage j: the copies of stage j + NS into slot j % NS (every wave
    // holds stage j's fragments, read during stage j-1, before this stage's
    // barrier); stage j+1's map fragments into na; per query tile the MFMAs
    // of stage j, then that tile's fragment of stage j+1 into the register
    // its MFMAs have just read. Blocks past the workgroup's range read as
    // zeros and their scores are never looked at, so a short last slice runs
    // the same code.
    auto stage = [&](u16x8 (&fa)[NB], u16x8 (&na)[NB]) __attribute__((always_inline)) {
      // stage j+1's copies have landed (this wave's, then everyone's)
      wait_vmcnt<(NS - 2) * NI>();
      raw_barrier();
      const int sn = next_slot(c_slot);
      issue();
      step_copy();
#pragma unroll
      for (int i = 0; i < NB; ++i) na[i] = read_mfrag(sn, i);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int i = 0; i < NB; ++i) acc[i][t] = mfma_bf16(fa[i], fb[t], acc[i][t]);
        fb[t] = read_qfrag(sn, t);
      }
      // issue order: the copies, the map fragment reads, then per query
      // tile its MFMAs and its next fragment
      __builtin_amdgcn_sched_group_barrier(0x020, NI, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, NB, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, NB, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
      wait_lgkm0();
    };
    for (int si = 0; si < n_slices; ++si) {
      // all k-steps of one slice (ksteps is even)
      for (int ks = 0; ks < ksteps; ks += 2) {
        stage(fa0, fa1);
        stage(fa1, fa0);
      }
      epilogue(si);
    }
    wait_vmcnt<0>();   // the trailing copies
  }
  // the dense form keeps no lists (it serves calls that return no matches)
  if constexpr (DBG) return;
  __syncthreads();

  // the cosine of each tile's best: its score times 1/|q|; a NaN score takes
  // the in-scan NaN value, and a NaN query (every cosine NaN) the lowest
  // index among this lane's maps
  {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float rq = a.rq[g0 + 16 * (NT * wq + t) + c];
      if (best_i[t] >= 0) {
        if (rq != rq) {
          best_s[t] = kNanScore;
          best_i[t] = first_ok ? y_first : -1;
        } else {
          best_s[t] = best_s[t] == kNanFloor ? kNanScore : best_s[t] * rq;
        }
      }
    }
  }

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
    for (int r = tid; r < QG; r += W * kWave) {
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
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(MmShape<GQ>::W * kWave), lds, st, a);
  err = hipGetLastError();
  if (err != hipSuccess || ev.stop == nullptr) return err;
  return hipEventRecord(ev.stop, st);
}

}  // namespace

int sem_mm_group(int32_t Bc) { return Bc > 128 ? 256 : 128; }

hipError_t launch_sem_mm(const StoreView& s, int32_t Bc, int32_t b_pad, const Workspace& ws, float* dbg, int32_t* R_out,
                         hipStream_t st, const float* mix, double w_self, double w_mix) {
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
  a.mix = mix;
  a.w_self = w_self;
  a.w_mix = w_mix;
  a.vec16 = s.n % 4 == 0 && reinterpret_cast<uintptr_t>(dbg) % 16 == 0 &&
            reinterpret_cast<uintptr_t>(mix) % 16 == 0;
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
