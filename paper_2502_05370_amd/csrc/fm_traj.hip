// Trajectory-based expert map search (Section 4.2.2, Eq. 5).
//
// Query b has observed the gate distributions of its first p_b layers; its
// score against stored iteration y is the cosine between the flattened
// prefixes q[b][0:p_b] and x[y][0:p_b].  One kernel launch serves a batch of
// up to 1024 queries with a single pass over the layer-major store planes:
//
//  * Every workgroup sorts the batch by depth (deepest first, stable, hence
//    the same order in every workgroup) and takes one group of 16*TQ queries
//    and one slice of 64*NBA stored maps (4 waves x NBA blocks of 16 maps).
//  * The contraction runs over "slots": each layer's E experts padded to a
//    multiple of 32, or LPG = 32/E layers per 32 slots when E divides 32.
//    A query tile (16 queries) stops at the layer group of its deepest
//    member, and rows beyond each query's own depth are staged as zeros, so
//    each query is scored on exactly its own prefix.
//  * Map rows go straight from HBM into registers (each wave owns its maps);
//    query rows are staged in LDS once per layer group for all four waves.
//    The next layer group's loads are in flight while the MFMAs of the
//    current one run.
//  * Products use v_mfma_f32_16x16x32_bf16.  A float32 value a is split into
//    three bf16 parts a = a1 + a2 + a3 + r, |r| <= 2^-27 |a| (round to
//    nearest at each step), and a.b is accumulated as the six terms
//    a1b1 + a1b2 + a2b1 + a1b3 + a2b2 + a3b1 (every dropped term is below
//    2^-25 |ab|) in float32 accumulators.  bf16 stores take one MFMA.
//  * Squared map-row norms come from the same loaded float32 values, giving
//    every map's prefix norm at every depth; query norms are summed in
//    float64 while staging.
//  * The epilogue forms the cosine, keeps a per-lane top-K of packed
//    (score, index) keys, merges it across the workgroup and inserts it into
//    the global top-k list (monotone atomic-max slots).  The last workgroup
//    to finish writes idx/score and clears the list and the counter.
#include <type_traits>

#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef uint32_t uint32x4 __attribute__((ext_vector_type(4)));

struct TrajArgs {
  const void* planes;
  int64_t plane_elems;
  const void* q;
  const int32_t* depth;
  int32_t n, L, E;
  int32_t spl;      // slots per layer: E when LPG > 1, else E rounded up to 32
  int32_t lpg;      // layers per layer group
  int32_t ksg;      // 32-slot k-steps per layer group
  int32_t B, k;
  int32_t n_qg;     // query groups
  int32_t n_units;  // (map slices) x (query groups)
  int32_t grid;
  int32_t dmax;     // bound on depths (max_depth)
  Workspace ws;
  uint32_t* flags;
  int32_t* idx_out;
  float* score_out;
  float* dbg;       // optional dense scores [B][n]
};

// float32 -> three bf16 parts (bit patterns), each rounded to nearest even.
// Pairs are converted with one packed conversion and read back as a whole
// 32-bit word (element-wise extraction of a bf16 vector lane is avoided).
__device__ __forceinline__ void split3(const floatx8& v, u16x8& h, u16x8& m, u16x8& l) {
  uint32x4 hw, mw, lw;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float2v x = {v[2 * j], v[2 * j + 1]};
    const bf16x2 hb = __builtin_convertvector(x, bf16x2);
    const float2v r1 = x - __builtin_convertvector(hb, float2v);
    const bf16x2 mb = __builtin_convertvector(r1, bf16x2);
    const float2v r2 = r1 - __builtin_convertvector(mb, float2v);
    const bf16x2 lb = __builtin_convertvector(r2, bf16x2);
    hw[j] = __builtin_bit_cast(uint32_t, hb);
    mw[j] = __builtin_bit_cast(uint32_t, mb);
    lw[j] = __builtin_bit_cast(uint32_t, lb);
  }
  h = __builtin_bit_cast(u16x8, hw);
  m = __builtin_bit_cast(u16x8, mw);
  l = __builtin_bit_cast(u16x8, lw);
}

__device__ __forceinline__ floatx4 mfma_bf16(const u16x8& a, const u16x8& b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

}  // namespace

template <bool BF, int TQ, int NBA, int KSG, int KTOP>
__global__ void __launch_bounds__(256) k_traj_scan(TrajArgs a) {
  constexpr int QG = 16 * TQ;                 // queries per group
  constexpr int MW = 16 * NBA;                // maps per wave
  constexpr int NP = BF ? 1 : 3;              // bf16 planes per operand
  constexpr int kMaxQU = (TQ * KSG + 3) / 4;  // staged 8-slot query units per thread
  constexpr int TC = TQ < 2 ? TQ : 2;         // query tiles whose operands are held at once
  using Raw = typename std::conditional<BF, u16x8, floatx8>::type;

  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int32_t s_last;
  __shared__ int32_t s_start[kMaxL];

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;
  const int qrow = 32 * KSG + 8;              // LDS row stride of staged queries (bf16 elements)

  // LDS carve-up
  uint16_t* qs = reinterpret_cast<uint16_t*>(smem);                        // [NP][QG][qrow]
  float* cum = reinterpret_cast<float*>(qs + NP * QG * qrow);              // [4][dmax][MW]
  int32_t* gperm = reinterpret_cast<int32_t*>(cum + kWaves * a.dmax * MW); // [QG]
  int32_t* gdep = gperm + QG;                                              // [QG]
  float* grq = reinterpret_cast<float*>(gdep + QG);                        // [QG]
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(
      (reinterpret_cast<uintptr_t>(grq + QG) + 7) & ~static_cast<uintptr_t>(7));  // [4][QG][KTOP]
  unsigned long long* bits = reinterpret_cast<unsigned long long*>(mbuf);  // prologue only: [kMaxL][16]

  // workgroup -> (map slice, query group); consecutive units share an XCD
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  const bool active = u < a.n_units;
  const int slice = active ? u / a.n_qg : 0;
  const int qgrp = active ? u % a.n_qg : 0;
  const int g0 = qgrp * QG;
  const int y_slice = slice * (kWaves * MW);
  const int y_wave = y_slice + w * MW;

  // ---- stable depth sort, deepest first: position of query b = queries
  // deeper than b + queries of equal depth with a lower index
  for (int i = tid; i < kMaxL * 16; i += kThreads) bits[i] = 0ull;
  for (int r = tid; r < QG; r += kThreads) {
    gdep[r] = 0;
    gperm[r] = 0;
    grq[r] = 0.0f;
  }
  __syncthreads();
  for (int b = tid; b < a.B; b += kThreads) {
    const int d = a.depth[b];
    const int dc = d < 1 ? 1 : (d > a.dmax ? a.dmax : d);
    if (dc != d && bid == 0) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_DEPTH_CLAMPED));
    atomicOr(&bits[(dc - 1) * 16 + b / 64], 1ull << (b % 64));
  }
  __syncthreads();
  if (w == 0) {
    int cnt = 0;
    if (lane < a.dmax) {
#pragma unroll
      for (int i = 0; i < 16; ++i) cnt += __popcll(bits[lane * 16 + i]);
    }
    int incl = cnt;  // inclusive suffix sum over buckets lane .. 63
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_down(incl, off, kWave);
      if (lane + off < 64) incl += o;
    }
    s_start[lane] = incl - cnt;
  }
  __syncthreads();
  for (int b = tid; b < a.B; b += kThreads) {
    const int d = a.depth[b];
    const int dc = d < 1 ? 1 : (d > a.dmax ? a.dmax : d);
    const unsigned long long* row = bits + (dc - 1) * 16;
    const int wd = b / 64;
    int r = 0;
    for (int i = 0; i < wd; ++i) r += __popcll(row[i]);
    r += __popcll(row[wd] & ((1ull << (b % 64)) - 1ull));
    const int pos = s_start[dc - 1] + r - g0;
    if (pos >= 0 && pos < QG) {
      gperm[pos] = b;
      gdep[pos] = dc;
    }
  }
  __syncthreads();

  int tmd[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) tmd[t] = active ? gdep[16 * t] : 0;
  const int D = tmd[0];
  const int NLG = (D + a.lpg - 1) / a.lpg;

  TopK<KTOP> best[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) best[t].clear();

  if (active && D > 0 && y_slice < a.n) {
    // ---- query staging units of this thread: unit = (row, 8-slot part).
    // What stays fixed from one layer group to the next is computed once:
    // the unit's element offset at layer group 0, its layer within the
    // group, how many of its 8 slots are real experts and its query's depth.
    constexpr int upr = 4 * KSG;              // units per row (4 or 8)
    const int nunits = QG * upr;
    const bool vec_ok = (a.E % 4) == 0;       // 8-slot runs start 16-byte (f32) / 8-byte (bf16) aligned
    int q_lds[kMaxQU], q_li[kMaxQU], q_nv[kMaxQU], q_p[kMaxQU];
    int64_t q_off[kMaxQU];
#pragma unroll
    for (int i = 0; i < kMaxQU; ++i) {
      const int id = tid + i * kThreads;
      q_lds[i] = -1;
      q_li[i] = 0;
      q_nv[i] = 0;
      q_p[i] = 0;
      q_off[i] = 0;
      if (id < nunits) {
        const int r = id / upr;
        const int s0 = 8 * (id % upr);
        const int li = s0 / a.spl;
        const int e0 = s0 - li * a.spl;
        const int nv = a.E - e0;
        q_lds[i] = r * qrow + s0;
        q_li[i] = li;
        q_nv[i] = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
        q_p[i] = (g0 + r < a.B) ? gdep[r] : 0;
        q_off[i] = static_cast<int64_t>(gperm[r]) * a.L * a.E + li * a.E + e0;
      }
    }
    const int64_t q_step = static_cast<int64_t>(a.lpg) * a.E;
    double qn2[kMaxQU];
#pragma unroll
    for (int i = 0; i < kMaxQU; ++i) qn2[i] = 0.0;

    Raw qraw[kMaxQU];
    auto load_q = [&](int lg) {
#pragma unroll
      for (int i = 0; i < kMaxQU; ++i) {
        Raw v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = 0;
        if (lg * a.lpg + q_li[i] < q_p[i]) {   // a real query that observed this layer
          const int64_t off = q_off[i] + lg * q_step;
          if constexpr (BF) {
            const uint16_t* p = static_cast<const uint16_t*>(a.q) + off;
            if (q_nv[i] == 8 && vec_ok) {
              const u16x4 lo = *reinterpret_cast<const u16x4*>(p);
              const u16x4 hi = *reinterpret_cast<const u16x4*>(p + 4);
              v = u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            } else {
#pragma unroll
              for (int j = 0; j < 8; ++j)
                if (j < q_nv[i]) v[j] = p[j];
            }
          } else {
            const float* p = static_cast<const float*>(a.q) + off;
            if (q_nv[i] == 8 && vec_ok) {
              const floatx4 lo = *reinterpret_cast<const floatx4*>(p);
              const floatx4 hi = *reinterpret_cast<const floatx4*>(p + 4);
              v = floatx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            } else {
#pragma unroll
              for (int j = 0; j < 8; ++j)
                if (j < q_nv[i]) v[j] = p[j];
            }
          }
        }
        qraw[i] = v;
      }
    };
    auto store_q = [&]() {
#pragma unroll
      for (int i = 0; i < kMaxQU; ++i) {
        if (q_lds[i] < 0) continue;
        uint16_t* dst = qs + q_lds[i];
        if constexpr (BF) {
          *reinterpret_cast<u16x8*>(dst) = qraw[i];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const double f = static_cast<double>(bf16_to_f32(qraw[i][j]));
            qn2[i] += f * f;
          }
        } else {
          u16x8 h, m, l;
          split3(qraw[i], h, m, l);
          *reinterpret_cast<u16x8*>(dst) = h;
          *reinterpret_cast<u16x8*>(dst + QG * qrow) = m;
          *reinterpret_cast<u16x8*>(dst + 2 * QG * qrow) = l;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const double f = static_cast<double>(qraw[i][j]);
            qn2[i] += f * f;
          }
        }
      }
    };

    // ---- this lane's map operand: rows y_wave + 16*nb + c, slots 32*ks + 8*g .. +7
    int a_li[KSG], a_nv[KSG];
    int64_t a_off[NBA][KSG];
    bool a_ok[NBA];
#pragma unroll
    for (int ks = 0; ks < KSG; ++ks) {
      const int s0 = 32 * ks + 8 * g;
      const int li = s0 / a.spl;
      const int e0 = s0 - li * a.spl;
      const int nv = a.E - e0;
      a_li[ks] = li;
      a_nv[ks] = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb)
        a_off[nb][ks] = li * a.plane_elems + static_cast<int64_t>(y_wave + 16 * nb + c) * a.E + e0;
    }
#pragma unroll
    for (int nb = 0; nb < NBA; ++nb) a_ok[nb] = y_wave + 16 * nb + c < a.n;
    const int64_t a_step = static_cast<int64_t>(a.lpg) * a.plane_elems;

    Raw araw[NBA][KSG];
    auto load_a = [&](int lg) {
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
        for (int ks = 0; ks < KSG; ++ks) {
          Raw v;
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = 0;
          if (a_ok[nb] && lg * a.lpg + a_li[ks] < a.L) {
            const int64_t off = a_off[nb][ks] + lg * a_step;
            const int nv = a_nv[ks];
            if constexpr (BF) {
              const uint16_t* p = static_cast<const uint16_t*>(a.planes) + off;
              if (vec_ok && nv >= 4) {
                const u16x4 lo = *reinterpret_cast<const u16x4*>(p);
                u16x4 hi = u16x4{0, 0, 0, 0};
                if (nv == 8) hi = *reinterpret_cast<const u16x4*>(p + 4);
                v = u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
              } else {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                  if (j < nv) v[j] = p[j];
              }
            } else {
              const float* p = static_cast<const float*>(a.planes) + off;
              if (vec_ok && nv >= 4) {
                const floatx4 lo = *reinterpret_cast<const floatx4*>(p);
                floatx4 hi = floatx4{0.f, 0.f, 0.f, 0.f};
                if (nv == 8) hi = *reinterpret_cast<const floatx4*>(p + 4);
                v = floatx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
              } else {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                  if (j < nv) v[j] = p[j];
              }
            }
          }
          araw[nb][ks] = v;
        }
      }
    };

    floatx4 acc[NBA][TQ];
#pragma unroll
    for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
      for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    float cumsq[NBA];
#pragma unroll
    for (int nb = 0; nb < NBA; ++nb) cumsq[nb] = 0.0f;

    // the padding columns of the staged rows are never written by staging
    for (int r = tid; r < NP * QG; r += kThreads) *reinterpret_cast<u16x8*>(qs + r * qrow + 32 * KSG) = u16x8{};

    load_q(0);
    load_a(0);
    for (int lg = 0; lg < NLG; ++lg) {
      store_q();
      // bf16 operand planes of this lane's map rows; squared norms per layer
      u16x8 ap[NP][NBA][KSG];
      float lsq[NBA];
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
        lsq[nb] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < KSG; ++ks) {
          if constexpr (BF) {
            ap[0][nb][ks] = araw[nb][ks];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const float f = bf16_to_f32(araw[nb][ks][j]);
              lsq[nb] = fmaf(f, f, lsq[nb]);
            }
          } else {
            split3(araw[nb][ks], ap[0][nb][ks], ap[1][nb][ks], ap[2][nb][ks]);
#pragma unroll
            for (int j = 0; j < 8; ++j) lsq[nb] = fmaf(araw[nb][ks][j], araw[nb][ks][j], lsq[nb]);
          }
        }
      }
      // Per-layer sums.  With LPG == 1 all four lane groups hold one layer;
      // with LPG > 1 layer li of the group occupies lane groups
      // [li*E/8, (li+1)*E/8).
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
        if (a.lpg == 1 || a.E == 32) {
          lsq[nb] += __shfl_xor(lsq[nb], 16, kWave);
          lsq[nb] += __shfl_xor(lsq[nb], 32, kWave);
        } else if (a.E == 16) {
          lsq[nb] += __shfl_xor(lsq[nb], 16, kWave);
        }
      }
      for (int li = 0; li < a.lpg; ++li) {
        const int l = lg * a.lpg + li;
        const int src = c + 16 * (a.lpg == 1 ? 0 : (li * a.E) / 8);
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb) {
          const float v = __shfl(lsq[nb], src, kWave);
          cumsq[nb] += v;
          if (g == 0 && l < a.dmax) cum[(w * a.dmax + l) * MW + 16 * nb + c] = cumsq[nb];
        }
      }
      __syncthreads();
      if (lg + 1 < NLG) {
        load_q(lg + 1);
        load_a(lg + 1);
      }
      // MFMAs of this layer group for the active query tiles
      const int l_first = lg * a.lpg;
#pragma unroll
      for (int ks = 0; ks < KSG; ++ks) {
#pragma unroll
        for (int tc = 0; tc < TQ; tc += TC) {
          if (tmd[tc] <= l_first) break;  // tiles are sorted by depth, deepest first
          u16x8 bq[NP][TC];
#pragma unroll
          for (int tt = 0; tt < TC; ++tt) {
#pragma unroll
            for (int pl = 0; pl < NP; ++pl)
              bq[pl][tt] = *reinterpret_cast<const u16x8*>(qs + (pl * QG + 16 * (tc + tt) + c) * qrow + 32 * ks + 8 * g);
          }
          if constexpr (BF) {
#pragma unroll
            for (int tt = 0; tt < TC; ++tt) {
              if (tmd[tc + tt] > l_first) {
#pragma unroll
                for (int nb = 0; nb < NBA; ++nb)
                  acc[nb][tc + tt] = mfma_bf16(ap[0][nb][ks], bq[0][tt], acc[nb][tc + tt]);
              }
            }
          } else {
            // the six cross terms, smallest first
            constexpr int TA[6] = {2, 1, 0, 1, 0, 0};
            constexpr int TB[6] = {0, 1, 2, 0, 1, 0};
#pragma unroll
            for (int term = 0; term < 6; ++term) {
#pragma unroll
              for (int tt = 0; tt < TC; ++tt) {
                if (tmd[tc + tt] > l_first) {
#pragma unroll
                  for (int nb = 0; nb < NBA; ++nb)
                    acc[nb][tc + tt] = mfma_bf16(ap[TA[term]][nb][ks], bq[TB[term]][tt], acc[nb][tc + tt]);
                }
              }
            }
          }
        }
      }
      __syncthreads();
    }

    // query norms: combine the partial sums of each row's units (fixed order)
#pragma unroll
    for (int i = 0; i < kMaxQU; ++i) {
      double v = qn2[i];
      for (int m = 1; m < upr; m <<= 1) v += __shfl_xor(v, m, kWave);
      const int id = tid + i * kThreads;
      if (id < nunits && id % upr == 0) {
        float r;
        if (v != v) r = __uint_as_float(0x7fc00000u);
        else if (v == 0.0) r = 0.0f;
        else r = static_cast<float>(1.0 / sqrt(v));
        grq[id / upr] = r;
      }
    }
    // 1/|x[y][0:p]| for every depth p <= D of this wave's maps
    for (int i = lane; i < D * MW; i += kWave) {
      const float v = cum[w * a.dmax * MW + i];
      cum[w * a.dmax * MW + i] = v > 0.0f ? 1.0f / sqrtf(v) : (v != v ? v : 0.0f);
    }
    __syncthreads();

    // epilogue: cosine, optional dense output, per-lane top-K
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
      const int r = 16 * t + c;
      const int p = gdep[r];
      if (p == 0) continue;
      const float rq = grq[r];
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int jm = 16 * nb + 4 * g + i;
          const int y = y_wave + jm;
          if (y >= a.n) continue;
          const float rs = cum[(w * a.dmax + (p - 1)) * MW + jm];
          const float s = acc[nb][t][i] * rq * rs;
          if (a.dbg != nullptr) a.dbg[static_cast<int64_t>(gperm[r]) * a.n + y] = s;
          best[t].push(make_key(s, y));
        }
      }
    }
  }

  // merge the per-lane lists across the 4 lane groups, then across waves
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      uint64_t o[KTOP];
#pragma unroll
      for (int j = 0; j < KTOP; ++j) o[j] = shfl_xor_u64(best[t].v[j], m);
      best[t].merge(o);
    }
  }
  __syncthreads();  // the sort bitmask (aliasing mbuf) is dead from here on
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
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
    global_topk_insert<KTOP>(a.ws.keys + static_cast<int64_t>(gperm[r]) * kMaxK, a.k, m.v);
  }

  // the last workgroup to finish writes the results and clears the workspace
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t ticket = __hip_atomic_fetch_add(a.ws.counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
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

// ----------------------------------------------------------------------------- launch

namespace {

template <bool BF, int TQ, int NBA, int KSG, int KTOP>
hipError_t launch_on(const TrajArgs& a, size_t lds, hipStream_t st) {
  auto kern = k_traj_scan<BF, TQ, NBA, KSG, KTOP>;
  if (lds > 64 * 1024) {
    const hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

template <bool BF, int KSG, int KTOP>
hipError_t launch_tq(int TQ, int NBA, const TrajArgs& a, size_t lds, hipStream_t st) {
  if (NBA == 2) {
    switch (TQ) {
      case 1: return launch_on<BF, 1, 2, KSG, KTOP>(a, lds, st);
      case 2: return launch_on<BF, 2, 2, KSG, KTOP>(a, lds, st);
      case 4: return launch_on<BF, 4, 2, KSG, KTOP>(a, lds, st);
      default: break;
    }
  } else {
    switch (TQ) {
      case 8:
        if constexpr (KTOP <= 4) return launch_on<BF, 8, 1, KSG, KTOP>(a, lds, st);
        break;
      case 16:
        if constexpr (KTOP == 1) return launch_on<BF, 16, 1, KSG, KTOP>(a, lds, st);
        break;
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

template <bool BF, int KTOP>
hipError_t launch_ksg(int KSG, int TQ, int NBA, const TrajArgs& a, size_t lds, hipStream_t st) {
  return KSG == 1 ? launch_tq<BF, 1, KTOP>(TQ, NBA, a, lds, st) : launch_tq<BF, 2, KTOP>(TQ, NBA, a, lds, st);
}

}  // namespace

size_t traj_lds_bytes(bool bf, int TQ, int NBA, int ksg, int max_depth, int KTOP) {
  const size_t np = bf ? 1 : 3;
  const size_t qg = 16 * TQ, mw = 16 * NBA;
  const size_t qrow = 32 * ksg + 8;
  size_t lds = np * qg * qrow * 2;
  lds += kWaves * static_cast<size_t>(max_depth) * mw * 4 + 3 * qg * 4;
  lds = (lds + 7) / 8 * 8;
  const size_t tail = kWaves * qg * static_cast<size_t>(KTOP) * 8;
  const size_t bits = kMaxL * 16 * 8;
  return lds + (tail > bits ? tail : bits);
}

hipError_t launch_match_trajectory(const StoreView& s, const void* q, const int32_t* depth, int32_t max_depth,
                                   int32_t B, int32_t k, int32_t* idx_out, float* score_out, float* dbg_scores,
                                   const Workspace& ws, hipStream_t st) {
  const bool bf = s.map_dtype == FM_BF16;
  const int esz = bf ? 2 : 4;
  TrajArgs a{};
  // slot geometry: E | 32 (E >= 8) packs 32/E layers per 32 slots, otherwise
  // each layer is padded to a multiple of 32 slots
  if (s.E >= 8 && 32 % s.E == 0) {
    a.spl = s.E;
    a.lpg = 32 / s.E;
    a.ksg = 1;
  } else {
    a.spl = (s.E + 31) / 32 * 32;
    a.lpg = 1;
    a.ksg = a.spl / 32;
  }
  const int KTOP = k == 1 ? 1 : (k <= 4 ? 4 : 8);
  const int tq_max = KTOP == 1 ? 16 : (KTOP == 4 ? 8 : 4);

  for (int b0 = 0; b0 < B; b0 += kChunkB) {
    const int Bc = (B - b0) < kChunkB ? (B - b0) : kChunkB;
    int TQ = 1;
    while (16 * TQ < Bc && TQ < tq_max) TQ *= 2;
    const int NBA = TQ <= 4 ? 2 : 1;
    const int n_qg = (Bc + 16 * TQ - 1) / (16 * TQ);
    const int maps_per_slice = kWaves * 16 * NBA;
    const int slices = s.n > 0 ? (s.n + maps_per_slice - 1) / maps_per_slice : 0;
    a.planes = s.planes;
    a.plane_elems = s.plane_elems;
    a.q = static_cast<const char*>(q) + static_cast<int64_t>(b0) * s.L * s.E * esz;
    a.depth = depth + b0;
    a.n = s.n;
    a.L = s.L;
    a.E = s.E;
    a.B = Bc;
    a.k = k;
    a.n_qg = n_qg;
    a.n_units = slices * n_qg;
    a.grid = ((a.n_units > 0 ? a.n_units : 1) + 7) / 8 * 8;
    a.dmax = max_depth;
    a.ws = ws;
    a.flags = s.flags;
    a.idx_out = idx_out != nullptr ? idx_out + static_cast<int64_t>(b0) * k : nullptr;
    a.score_out = score_out != nullptr ? score_out + static_cast<int64_t>(b0) * k : nullptr;
    a.dbg = dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr;

    const size_t lds = traj_lds_bytes(bf, TQ, NBA, a.ksg, max_depth, KTOP);
    if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
    hipError_t err;
    if (bf) {
      err = KTOP == 1 ? launch_ksg<true, 1>(a.ksg, TQ, NBA, a, lds, st)
          : KTOP == 4 ? launch_ksg<true, 4>(a.ksg, TQ, NBA, a, lds, st)
                      : launch_ksg<true, 8>(a.ksg, TQ, NBA, a, lds, st);
    } else {
      err = KTOP == 1 ? launch_ksg<false, 1>(a.ksg, TQ, NBA, a, lds, st)
          : KTOP == 4 ? launch_ksg<false, 4>(a.ksg, TQ, NBA, a, lds, st)
                      : launch_ksg<false, 8>(a.ksg, TQ, NBA, a, lds, st);
    }
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace fm
