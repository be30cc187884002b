// Trajectory-based expert map search (Section 4.2.2, Eq. 5).
//
// Query b has observed the gate distributions of its first p_b layers; its
// score against stored iteration y is the cosine between the flattened
// prefixes q[b][0:p_b] and x[y][0:p_b].  A batch of up to 1024 queries is
// served by three launches and one pass over the layer-major store planes:
//
//  k_traj_prep      sorts the batch by depth (deepest first, stable), writes
//                   1/|q[b][0:p_b]| (float64 sum) and, for every "layer
//                   group", the sorted query rows as MFMA-ready planes (two
//                   float16 parts of each float32 value, one bf16 plane for
//                   bf16 stores), zero beyond each query's depth, so the scan
//                   copies them verbatim; it also shares the scan's
//                   workgroups among the query groups by their cost.
//  k_traj_scan      workgroup = one group of 16*TQ sorted queries x an even
//                   share of the store (to the map) among the group's
//                   workgroups, walked as slices of 8 waves x NBA 16-map
//                   blocks.  The map quads of a stage two stages ahead load
//                   into registers (raw buffer loads), the query planes into
//                   a three-slot LDS ring (direct global->LDS loads); one
//                   barrier per stage.  A query tile (16 queries) stops at
//                   the layer group of its deepest member.  float32
//                   operands are scaled by 2^12 and split into two float16
//                   parts, A = 2^12 a = a1 + a2 + r with |r| <= 2^-22 |A|
//                   (absolute 2^-25 where a2 falls below the float16 normal
//                   range), and a.b = 2^-24 (a1b2 + a1b1 + a2b1) accumulates
//                   on v_mfma_f32_16x16x32_f16 (dropped a2b2 and residuals
//                   < 3 * 2^-22 |ab| + 2^-37 (|a| + |b|), for |a|, |b| <= 8);
//                   bf16 stores take one bf16 MFMA.  The slice epilogue
//                   divides by the query's and the store's prefix norms (the
//                   latter precomputed at insert and staged per slice in an
//                   LDS table), keeps a per-lane top-K of packed (score,
//                   index) keys, merges it across the workgroup and stores it
//                   (plain stores) as this workgroup's partial list per query.
//  k_finalize       merges each query's group's partial lists into idx/score.
//
// "Slots": each layer's E experts padded to a multiple of 32, or LPG = 32/E
// layers per 32 slots when E (>= 8) divides 32.  MFMA k position 8g + j of a
// 32-slot k-step holds slot 4g + j (j < 4) or 16 + 4g + j - 4 (j >= 4), so
// that the map operand of one k-step is two runs of whole expert quads.
#include <type_traits>

#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));


// Slot geometry of a store (host-computed).
struct Geo {
  int32_t spl;   // slots per layer: E when LPG > 1, else E rounded up to 32
  int32_t lpg;   // layers per layer group
  int32_t ksg;   // 32-slot k-steps per layer group
};

// Bytes of one staged query plane row: 32*ksg 16-bit slots, in 16-byte
// units.  With ksg > 1 unit u of row r is stored at unit u ^ (r & 7) of the
// row, so the 16 rows a wave reads at one logical unit spread over 8 distinct
// 16-byte bank groups (with ksg = 1 a wave's read of 16 rows is one
// contiguous 1 KB already).
__host__ __device__ __forceinline__ int qrow_bytes(int ksg) { return 64 * ksg; }
__host__ __device__ __forceinline__ int qrow_unit(int ksg, int row, int unit) {
  return ksg > 1 ? unit ^ (row & 7) : unit;
}

struct PrepArgs {
  const void* q;
  const int32_t* depth;
  int32_t B, L, E, dmax;
  Geo geo;
  int32_t nlg;        // layer groups staged (ceil(dmax / lpg))
  int32_t b_pad;      // positions per staged layer group (multiple of the group size)
  int32_t qg;         // queries per group (16 * TQ)
  int32_t n_qg;       // query groups
  int32_t G;          // scan workgroups to share among the groups
  int32_t epi16;      // a slice epilogue's cost in sixteenths of a stage's
  int32_t tiled;      // bf16 only: stage for k_traj_mm (MFMA operand tiles, groups interleaved)
  Workspace ws;
  uint32_t* flags;
};

struct ScanArgs {
  const void* planes;
  int64_t plane_bytes;
  const float* rnorm;   // [L][rn_stride] prefix inverse norms
  int64_t rn_stride;
  int32_t n, L, E, row;
  Geo geo;
  int32_t B, b_pad, dmax;
  int32_t n_qg;       // query groups
  int32_t R;          // partial lists per position (the workgroups of a group: ws.rgrp)
  int32_t n_blocks;   // 16-map blocks of the store (ceil(n / 16))
  int32_t grid;
  int32_t rt_bytes;   // LDS bytes of one inverse-norm table (whole 8 KB chunks)
  Workspace ws;
  float* dbg;         // optional dense scores [B][n]
};

// Stable sort of the batch by depth, deepest first.  A query's position is
// (queries deeper) + (queries of equal depth with a lower index): the same
// in every workgroup.  bits: LDS [kMaxL][16] words; start: LDS [kMaxL].
__device__ void depth_buckets(const int32_t* depth, int B, int dmax, unsigned long long* bits, int32_t* start) {
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  for (int i = tid; i < kMaxL * 16; i += blockDim.x) bits[i] = 0ull;
  __syncthreads();
  for (int b = tid; b < B; b += blockDim.x) {
    const int d = depth[b];
    const int dc = d < 1 ? 1 : (d > dmax ? dmax : d);
    atomicOr(&bits[(dc - 1) * 16 + b / 64], 1ull << (b % 64));
  }
  __syncthreads();
  if (tid < kWave) {
    int cnt = 0;
    if (lane < dmax) {
#pragma unroll
      for (int i = 0; i < 16; ++i) cnt += __popcll(bits[lane * 16 + i]);
    }
    int incl = cnt;  // inclusive suffix sum over buckets lane .. 63
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_down(incl, off, kWave);
      if (lane + off < 64) incl += o;
    }
    start[lane] = incl - cnt;
  }
  __syncthreads();
}

__device__ __forceinline__ int position_of(int b, int dc, const unsigned long long* bits, const int32_t* start) {
  const unsigned long long* row = bits + (dc - 1) * 16;
  const int wd = b / 64;
  int r = 0;
  for (int i = 0; i < wd; ++i) r += __popcll(row[i]);
  r += __popcll(row[wd] & ((1ull << (b % 64)) - 1ull));
  return start[dc - 1] + r;
}

// float32 -> two float16 parts (bit patterns) of A = 2^12 a: hi = RN16(A),
// lo = RN16(A - hi).  A - hi is exact in float32 (one fused multiply-add of
// the widened hi); hi is finite for |a| < 16 (values above 8 are flagged
// where they enter).  Pairs convert with one packed conversion each.
constexpr float kSplitScale = 4096.0f;                        // 2^12
constexpr float kDotUnscale = 1.0f / (4096.0f * 4096.0f);     // 2^-24
constexpr float kRangeLimit = 8.0f;
__device__ __forceinline__ void split2(const floatx8& v, u16x8& h, u16x8& l) {
  uint32x4 hw, lw;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float2v x = {v[2 * j] * kSplitScale, v[2 * j + 1] * kSplitScale};
    const half2v hb = __builtin_convertvector(x, half2v);
    float2v r;
    r[0] = __builtin_fmaf(static_cast<float>(hb[0]), -1.0f, x[0]);
    r[1] = __builtin_fmaf(static_cast<float>(hb[1]), -1.0f, x[1]);
    const half2v lb = __builtin_convertvector(r, half2v);
    hw[j] = __builtin_bit_cast(uint32_t, hb);
    lw[j] = __builtin_bit_cast(uint32_t, lb);
  }
  h = __builtin_bit_cast(u16x8, hw);
  l = __builtin_bit_cast(u16x8, lw);
}



// Position of stage j of the scan: slice j / NLG, layer group j % NLG and
// query ring slot j % NS, stepped from stage to stage without divisions.
struct StagePos {
  int j, si, lg, slot;
};
__device__ __forceinline__ StagePos next_pos(const StagePos& p, int nlg, int ns) {
  StagePos q;
  q.j = p.j + 1;
  const bool wrap = p.lg + 1 == nlg;
  q.lg = wrap ? 0 : p.lg + 1;
  q.si = wrap ? p.si + 1 : p.si;
  q.slot = p.slot + 1 == ns ? 0 : p.slot + 1;
  return q;
}

}  // namespace

// ----------------------------------------------------------------------------- prep

// grid = (b_pad / 16, nlg + 4).  Block (x, y < nlg) stages layer group y of
// queries 16x .. 16x+15 at their sorted positions; blocks (x, nlg .. nlg+3)
// write those queries' perm, depth and 1/|q| entries; block (0, nlg) also
// shares the scan's workgroups among the query groups.
template <bool BF>
__global__ void __launch_bounds__(256) k_traj_prep(PrepArgs a) {
  using T = typename std::conditional<BF, uint16_t, float>::type;
  constexpr int esz = sizeof(T);
  __shared__ unsigned long long bits[kMaxL * 16];
  __shared__ int32_t start[kMaxL];
  const int tid = threadIdx.x;
  const T* q = static_cast<const T*>(a.q);
  // Blocks are indexed by query (16 per block), not by sorted position, so
  // each thread's loads of its query's values are issued before, and land
  // during, the depth sort that tells where the staged row goes.
  if (static_cast<int>(blockIdx.y) < a.nlg) {
    // one thread per (query row, 8-slot unit)
    const int lg = blockIdx.y;
    const int upr = 4 * a.geo.ksg;
    const int rb = qrow_bytes(a.geo.ksg);
    constexpr int NP = BF ? 1 : 2;
    const int64_t plane_pitch = static_cast<int64_t>(a.qg) * rb;              // one plane of a group slab
    const int i = tid;
    const bool staged = i < 16 * upr;
    const int r = staged ? i / upr : 0;
    const int unit = i - r * upr;
    const int b = blockIdx.x * 16 + r;
    const bool real = staged && b < a.B;
    const int d = real ? a.depth[b] : 0;
    // k positions 8*unit .. 8*unit+7 hold the slot runs 32ks + 4g .. +3 and
    // 32ks + 16 + 4g .. +3 (unit = 4ks + g), the order in which the scan
    // loads the map quads; layers past the query's depth are zeroed below
    floatx8 v = floatx8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    u16x8 h = u16x8{}, l = u16x8{};
    int layer_of[2] = {a.L, a.L};
    if (real && unit < 4 * a.geo.ksg) {
      const int ks = unit / 4;
      const int gg = unit - 4 * ks;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int s0 = 32 * ks + 16 * half + 4 * gg;
        const int li = s0 / a.geo.spl;
        const int e0 = s0 - li * a.geo.spl;
        const int layer = lg * a.geo.lpg + li;
        layer_of[half] = layer;
        if (layer < a.dmax && e0 < a.E) {
          const T* src = q + (static_cast<int64_t>(b) * a.L + layer) * a.E + e0;
          const int nv = a.E - e0 < 4 ? a.E - e0 : 4;
          for (int k = 0; k < nv; ++k) {
            if constexpr (BF) h[4 * half + k] = src[k];
            else v[4 * half + k] = src[k];
          }
        }
      }
    }
    depth_buckets(a.depth, a.B, a.dmax, bits, start);
    if (!staged) return;
    const int dc = d < 1 ? 1 : (d > a.dmax ? a.dmax : d);
    // padding positions B .. b_pad-1 are the padding queries' own indices
    const int pos = real ? position_of(b, dc, bits, start) : b;
    bool big = false;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (layer_of[half] >= dc || !real) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if constexpr (BF) h[4 * half + k] = 0;
          else v[4 * half + k] = 0.f;
        }
      }
    }
    if constexpr (!BF) {
#pragma unroll
      for (int k = 0; k < 8; ++k) big = big || __builtin_fabsf(v[k]) > kRangeLimit;
      split2(v, h, l);
    }
    if (BF && a.tiled) {
      // k_traj_mm layout: sorted tile T = pos / 16 is local tile T % 16 of
      // band T / 16; the 1 KB operand tile of (layer group, k-step, band,
      // local tile) holds this unit at lane slot 16 g + c
      const int T = pos / 16;
      const int tg = T / 16;
      const int tl = T % 16;
      const int ks = unit / 4;
      const int gg = unit - 4 * ks;
      char* dst = static_cast<char*>(a.ws.qrows) +
                  ((((static_cast<int64_t>(lg) * a.geo.ksg + ks) * a.n_qg + tg) * 16 + tl) * 1024) +
                  (gg * 16 + pos % 16) * 16;
      *reinterpret_cast<u16x8*>(dst) = h;
      if (blockIdx.y == 0 && real && unit == 0 && dc != d) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_DEPTH_CLAMPED));
      return;
    }
    const int grp = pos / a.qg;
    char* slab = static_cast<char*>(a.ws.qrows) + (static_cast<int64_t>(lg) * a.b_pad + grp * a.qg) * NP * rb;
    const int row_in_grp = pos - grp * a.qg;
    char* dst = slab + static_cast<int64_t>(row_in_grp) * rb + 16 * qrow_unit(a.geo.ksg, row_in_grp, unit);
    *reinterpret_cast<u16x8*>(dst) = h;
    if constexpr (!BF) {
      *reinterpret_cast<u16x8*>(dst + plane_pitch) = l;
      if (big) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_VALUE_RANGE));
    }
    if (blockIdx.y == 0 && real && unit == 0 && dc != d) atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_DEPTH_CLAMPED));
    return;
  }
  depth_buckets(a.depth, a.B, a.dmax, bits, start);
  const int lane = tid % kWave;
  // Scan workgroups per query group.  Per slice of maps a group's scan takes
  // one stage per layer group its deepest query reaches (position g * qg,
  // the groups being depth-sorted) plus the slice epilogue (ranking every
  // score), so the G workgroups are shared in proportion to
  // 16 * stages + epi16, at least one each; the scan reads its group, share
  // and stage count back.
  if (blockIdx.x == 0 && static_cast<int>(blockIdx.y) == a.nlg && tid < kWave) {
    int dg = 0;
    if (lane < a.n_qg) {
      const int P = lane * a.qg;
      for (int l = 0; l < a.dmax; ++l) {
        const int hi = l == 0 ? a.B : start[l - 1];
        if (start[l] <= P && P < hi) dg = l + 1;
      }
    }
    const int nlg_g = (dg + a.geo.lpg - 1) / a.geo.lpg;
    const int wgt = lane < a.n_qg ? 16 * nlg_g + a.epi16 : 0;
    int tot = wgt;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) tot += __shfl_xor(tot, m, kWave);
    const int rg = lane < a.n_qg ? 1 + static_cast<int>(static_cast<int64_t>(a.G - a.n_qg) * wgt / (tot > 0 ? tot : 1)) : 0;
    int incl = rg;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off, kWave);
      if (lane >= off) incl += o;
    }
    if (lane < a.n_qg) {
      a.ws.rgrp[lane] = rg;
      a.ws.pgrp[lane] = incl - rg;
      a.ws.ngrp[lane] = nlg_g;
    }
  }
  // perm, depth and 1/|q[b][0:p]| of queries 16x .. 16x+15: blocks y = nlg ..
  // nlg+3 take four each, one wave per query, written at the query's sorted
  // position (padding queries b >= B fill positions b)
  const int b = blockIdx.x * 16 + (static_cast<int>(blockIdx.y) - a.nlg) * 4 + tid / kWave;
  const bool real = b < a.B;
  const int d = real ? a.depth[b] : 0;
  const int dc = d < 1 ? 1 : (d > a.dmax ? a.dmax : d);
  const int pos = real ? position_of(b, dc, bits, start) : b;
  double acc = 0.0;
  if (real) {
    // sixteen independent loads in flight per lane
    constexpr int U = 16;
    const int cnt = dc * a.E;
    const T* row = q + static_cast<int64_t>(b) * a.L * a.E;
    double part[U];
#pragma unroll
    for (int u = 0; u < U; ++u) part[u] = 0.0;
    for (int j0 = lane; j0 < cnt; j0 += U * kWave) {
      double f[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * kWave;
        f[u] = 0.0;
        if (j < cnt) {
          if constexpr (BF) f[u] = static_cast<double>(bf16_to_f32(row[j]));
          else f[u] = static_cast<double>(row[j]);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) part[u] += f[u] * f[u];
    }
#pragma unroll
    for (int u = 1; u < U; ++u) part[0] += part[u];
    acc = part[0];
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
  if (lane == 0) {
    float rqv;
    if (acc != acc) rqv = __uint_as_float(0x7fc00000u);
    else if (acc == 0.0) rqv = 0.0f;
    else rqv = static_cast<float>(1.0 / sqrt(acc));
    a.ws.rq[pos] = real ? rqv : 0.0f;
    a.ws.perm[pos] = real ? b : -1;
    a.ws.sdep[pos] = real ? dc : 0;
  }
}

// ----------------------------------------------------------------------------- scan

// 8 waves; wave w owns NBA blocks of 16 maps of every slice (W * NBA blocks
// of the workgroup's range).  Stage j = (slice j / NLG, layer group j % NLG).
// During stage j every wave loads its share of the query planes of stage j+2
// into LDS ring slot (j+2) % 3 (direct global->LDS loads) and, once stage
// j's map rows are split into bf16 parts, the map rows of stage j+2 into the
// freed registers (raw buffer loads), so both overlap the MFMAs.  Every wave
// issues the same loads per stage (out-of-range offsets keep the count fixed),
// so "stage j has landed" is vmcnt <= the loads of one stage.  Slot (j+2) % 3
// was last read in stage j-1, which every wave finished before the barrier of
// stage j, so one barrier per stage suffices.
template <bool BF, int TQ, int NBA, int KSG, int KTOP, bool DBG>
__global__ void __launch_bounds__(512) k_traj_scan(ScanArgs a) {
  using Raw = typename std::conditional<BF, u16x8, floatx8>::type;
  constexpr int W = 8;                        // waves per workgroup
  constexpr int NS = 3;                       // query-plane ring slots (two stages in flight)
  constexpr int esz = BF ? 2 : 4;
  constexpr int QG = 16 * TQ;                 // queries per group
  constexpr int MW = 16 * NBA;                // maps per wave and slice
  constexpr int NP = BF ? 1 : 2;              // MFMA parts per operand (bf16, or two float16)
  constexpr int RB = 64 * KSG;                // staged query plane row bytes (qrow_bytes)
  constexpr int NI_Q = (NP * QG * RB + W * 1024 - 1) / (W * 1024);  // 1 KB query loads per wave and stage
  constexpr int Q_STAGE = W * NI_Q * 1024;
  constexpr int NI_A = NBA * KSG * 2;         // map loads per wave and stage (two halves per unit)
  constexpr int NI = NI_A + NI_Q;
  static_assert(NI < 64, "vmcnt field is 6 bits");

  constexpr int SW = W * NBA * 16;            // maps per slice

  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                                              // [NS][Q_STAGE]
  unsigned char* rtab = smem + NS * Q_STAGE;                               // [2][rt_bytes]
  int32_t* gperm = reinterpret_cast<int32_t*>(rtab + 2 * a.rt_bytes);      // [QG]
  int32_t* gdep = gperm + QG;                                              // [QG]
  float* grq = reinterpret_cast<float*>(gdep + QG);                        // [QG]
  int32_t* gdi = reinterpret_cast<int32_t*>(grq + QG);                     // [QG] distinct-depth index
  int32_t* dval = gdi + QG;                                                // [QG] distinct depths
  uint64_t* dmask = reinterpret_cast<uint64_t*>(dval + QG);                // [QG / 64]
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(smem);                      // after the loop: [W][QG][KTOP]

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;

  // workgroup -> (query group, share of the store): group g owns the
  // workgroups [pgrp[g], pgrp[g] + rgrp[g]) of the XCD-aware numbering u
  // (consecutive u run on one XCD).
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  // A single group owns every workgroup and walks ceil(dmax / lpg) layer
  // groups (a bound on its deepest query; deeper staged rows are zero), so
  // it needs no read of the allocation.
  int pg_l = 0x7fffffff, rg_l = 0, ng_l = 0;
  if (a.n_qg == 1) {
    pg_l = 0;
    rg_l = a.R;
    ng_l = (a.dmax + a.geo.lpg - 1) / a.geo.lpg;
  } else if (lane < a.n_qg) {
    pg_l = a.ws.pgrp[lane];
    rg_l = a.ws.rgrp[lane];
    ng_l = a.ws.ngrp[lane];
  }
  const uint64_t gbal = __ballot(lane < a.n_qg && pg_l <= u);
  const int qg_u = gbal != 0 ? __popcll(gbal) - 1 : 0;
  // (read back as wave-uniform values, so everything derived from them stays
  // in scalar registers and uniform branches)
  const int Rg = __builtin_amdgcn_readfirstlane(__shfl(rg_l, qg_u, kWave));
  const int Pg = __builtin_amdgcn_readfirstlane(__shfl(pg_l, qg_u, kWave));
  const bool active = gbal != 0 && u - Pg < Rg;
  const int qgrp = active ? qg_u : 0;
  const int rr = active ? u - Pg : 0;
  // this workgroup's maps: [y_lo, y_hi), an even share of the store to the
  // map (so every workgroup streams the same bytes), covered by the 16-map
  // blocks [b_begin, b_end); a block shared with a neighbour loads only this
  // workgroup's rows.  The blocks are walked as slices of W * NBA blocks (the
  // last one partial).
  const int y_lo = active ? static_cast<int>((static_cast<int64_t>(rr) * a.n) / Rg) : 0;
  const int y_hi = active ? static_cast<int>((static_cast<int64_t>(rr + 1) * a.n) / Rg) : 0;
  const int b_begin = y_lo / 16;
  const int b_end = y_hi > y_lo ? (y_hi + 15) / 16 : b_begin;
  const int n_slices = (b_end - b_begin + W * NBA - 1) / (W * NBA);
  const int g0 = qgrp * QG;

  // Stages 0 and 1 load before the prologue fills LDS with the group's
  // sorted query info, so the latencies overlap.
  const bool has_work = active && n_slices > 0;
  TopK<KTOP> best[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) best[t].clear();
  const int ng_u = __builtin_amdgcn_readfirstlane(__shfl(ng_l, qg_u, kWave));
  const int NLG = ng_u > 0 ? ng_u : 1;
  const int nstages = has_work ? n_slices * NLG : 0;
  {
    // Lane constants.  Register element j of lane (g, c) in k-step ks holds
    // slot 32ks + 4g + j (j < 4) or 32ks + 16 + 4g + j - 4 (j >= 4) of map
    // row c of the block; each run of 4 slots is one quad of a layer of the
    // group, so the two loads of a lane read one quad each and the 64 lanes
    // of a load read 4 consecutive quads of a tile.
    uint32_t lane_off[KSG][2];
    bool quad_ok[KSG][2];
#pragma unroll
    for (int ks = 0; ks < KSG; ++ks) {
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int s0 = 32 * ks + 16 * half + 4 * g;
        const int li = s0 / a.geo.spl;
        const int e0 = s0 - li * a.geo.spl;
        quad_ok[ks][half] = e0 < a.row;
        lane_off[ks][half] = static_cast<uint32_t>(li) * static_cast<uint32_t>(a.plane_bytes) +
                             static_cast<uint32_t>(((e0 / 4) * 64 + c * 4) * esz);
      }
    }
    const char* planes = static_cast<const char*>(a.planes);
    const uint32_t tile_bytes = static_cast<uint32_t>(16 * a.row * esz);
    const char* qrows = static_cast<const char*>(a.ws.qrows);

    // Map quads are read with raw buffer loads over the planes of one layer
    // group.  Rows past the store, padding quads and layers at or past L use
    // offsets beyond the descriptor's range and read as zeros without
    // touching memory (the row padding itself is stored as zeros).
    // The quad offsets of a slice's map rows are the same in all its layer
    // groups (only the descriptor's base moves), so they are computed when a
    // slice's first layer group loads (and for every load past the last
    // stage, whose offsets are all out of range).  The empty asm makes them
    // opaque: the loads stay unconditional (the compiler would otherwise
    // branch around them, and a branch over in-flight loads costs a wait for
    // every outstanding load).
    uint32_t offs[NBA][KSG][2];
    auto set_offsets = [&](bool real, int si) {
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
        const int blk = b_begin + si * (W * NBA) + w * NBA + nb;
        const int y_blk = 16 * blk;
        const bool row_ok = real && blk < b_end && y_blk + c >= y_lo && y_blk + c < y_hi;
        const uint32_t blk_off = static_cast<uint32_t>(blk) * tile_bytes;
#pragma unroll
        for (int ks = 0; ks < KSG; ++ks) {
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            offs[nb][ks][half] = row_ok && quad_ok[ks][half] ? lane_off[ks][half] + blk_off : kOutside;
            asm volatile("" : "+v"(offs[nb][ks][half]));
          }
        }
      }
    };
    auto load_a = [&](const StagePos& p, Raw (&dst)[NBA][KSG]) {
      const bool real = p.j < nstages;
      const int lg = real ? p.lg : 0;
      const int l0 = lg * a.geo.lpg;
      const int nl = a.L - l0 < a.geo.lpg ? a.L - l0 : a.geo.lpg;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>(planes + l0 * a.plane_bytes), static_cast<short>(0),
          static_cast<int>(static_cast<uint32_t>(nl) * static_cast<uint32_t>(a.plane_bytes)), kBufWord3);
      if (!real || p.lg == 0) set_offsets(real, p.si);
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
        for (int ks = 0; ks < KSG; ++ks) {
          const uint32_t lo = offs[nb][ks][0];
          const uint32_t hi = offs[nb][ks][1];
          if constexpr (BF) {
            const uint32x2 vl = __builtin_amdgcn_raw_buffer_load_b64(rs, static_cast<int>(lo), 0, 0);
            const uint32x2 vh = __builtin_amdgcn_raw_buffer_load_b64(rs, static_cast<int>(hi), 0, 0);
            dst[nb][ks] = __builtin_bit_cast(u16x8, uint32x4{vl[0], vl[1], vh[0], vh[1]});
          } else {
            const uint32x4 vl = __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(lo), 0, 0);
            const uint32x4 vh = __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(hi), 0, 0);
            dst[nb][ks] = floatx8{__uint_as_float(vl[0]), __uint_as_float(vl[1]), __uint_as_float(vl[2]),
                                  __uint_as_float(vl[3]), __uint_as_float(vh[0]), __uint_as_float(vh[1]),
                                  __uint_as_float(vh[2]), __uint_as_float(vh[3])};
          }
        }
      }
    };
    auto load_q = [&](const StagePos& p) {
      const bool real = p.j < nstages;
      const int lg = real ? p.lg : 0;
      unsigned char* st = ring + p.slot * Q_STAGE;
      const char* qsl = qrows + (static_cast<int64_t>(lg) * a.b_pad + g0) * NP * RB;
#pragma unroll
      for (int i = 0; i < NI_Q; ++i) dma16(qsl + (w * NI_Q + i) * 1024 + lane * 16, st + (w * NI_Q + i) * 1024);
    };

    floatx4 acc[NBA][TQ];
#pragma unroll
    for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
      for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    // issue order: Q0 A0 Q1 A1, the prologue's loads, [RT0], then during
    // stage j: [RT] Q(j+2) A(j+2)
    Raw ar0[NBA][KSG], ar1[NBA][KSG];
    // Stage positions advance incrementally (no division per stage).
    const StagePos p_first{0, 0, 0, 0};
    if (has_work) {
      load_q(p_first);
      load_a(p_first, ar0);
      const StagePos p_second = next_pos(p_first, NLG, NS);
      load_q(p_second);
      load_a(p_second, ar1);
    }
    for (int r = tid; r < QG; r += W * kWave) {
      const int pos = g0 + r;
      gperm[r] = a.ws.perm[pos];
      gdep[r] = a.ws.sdep[pos];
      grq[r] = a.ws.rq[pos];
    }
    __syncthreads();
    // Distinct depths of the group (the positions are sorted by depth, deepest
    // first; padding has depth 0): dval[k] is the k-th one, gdi[r] the index of
    // gdep[r].  The epilogue of a slice reads the store's prefix inverse norms
    // 1/|x[y][0:p]| of the slice's maps from an LDS table with one row per
    // distinct depth.
    {
      const bool is_new = tid < QG && gdep[tid] > 0 && (tid == 0 || gdep[tid - 1] != gdep[tid]);
      const uint64_t bal = __ballot(is_new);
      if (lane == 0 && w < QG / 64 + (QG % 64 ? 1 : 0)) dmask[w] = bal;
      __syncthreads();
      if (tid < QG) {
        int before = 0;
        for (int ww = 0; ww < w; ++ww) before += __popcll(dmask[ww]);
        const int incl = before + __popcll(bal & ((2ull << lane) - 1ull));
        gdi[tid] = incl > 0 ? incl - 1 : 0;
        if (is_new) dval[incl - 1] = gdep[tid];
      }
      __syncthreads();
    }
    int nd = 0;
    for (int ww = 0; ww < QG / 64 + (QG % 64 ? 1 : 0); ++ww) nd += __popcll(dmask[ww]);
    int tmd[TQ];
#pragma unroll
    for (int t = 0; t < TQ; ++t) tmd[t] = gdep[16 * t];

    // Inverse-norm table of slice si into LDS buffer si % 2: row k holds
    // rnorm[dval[k] - 1][y_s .. y_s + SW) (y_s = the slice's first map), read
    // with raw buffer loads straight into LDS (offsets past the norms read as
    // zeros).  Issued one stage ahead of the slice's last stage and before
    // that stage's ring loads, so the counted ring waits also cover it and the
    // next barrier publishes it.
    const __amdgpu_buffer_rsrc_t rs_rn = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.rnorm), static_cast<short>(0),
        static_cast<int>(static_cast<uint32_t>(a.L) * static_cast<uint32_t>(a.rn_stride) * 4u), kBufWord3);
    const int rt_chunks = (nd * SW * 4 + W * 1024 - 1) / (W * 1024);   // 1 KB loads per wave
    auto load_rt = [&](int si) {
      unsigned char* dst = rtab + (si & 1) * a.rt_bytes;
      const int y_s = 16 * (b_begin + si * (W * NBA));
      for (int i = 0; i < rt_chunks; ++i) {
        const int byte = (w + W * i) * 1024 + lane * 16;
        const int k = byte / (SW * 4);
        const int col = (byte - k * SW * 4) / 4;
        const uint32_t off = k < nd ? static_cast<uint32_t>(((dval[k] - 1) * a.rn_stride + y_s + col) * 4) : kOutside;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_rn, (lds_vp)(dst + (w + W * i) * 1024), 16, static_cast<int>(off), 0,
                                                 0, 0);
      }
    };

    // With one layer group per slice, stage 0 is slice 0's last stage: its
    // inverse-norm table loads now and lands before the loop starts.
    if (has_work && NLG == 1) {
      load_rt(0);
      wait_vmcnt<0>();
    }

    // MFMAs of one k-step for the first NT (active) query tiles, term-major so
    // that consecutive MFMAs update different accumulators.
    auto mfma_tiles = [&](auto nt_const, int ks, const unsigned char* sq, const u16x8 (&ap)[NP][NBA][KSG]) {
      constexpr int NT = decltype(nt_const)::value;
      u16x8 bq[NP][NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int pl = 0; pl < NP; ++pl)
          bq[pl][t] = *reinterpret_cast<const u16x8*>(sq + (pl * QG + 16 * t + c) * RB +
                                                      16 * (KSG > 1 ? (4 * ks + g) ^ (c & 7) : 4 * ks + g));
      if constexpr (BF) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int nb = 0; nb < NBA; ++nb) acc[nb][t] = mfma_bf16(ap[0][nb][ks], bq[0][t], acc[nb][t]);
      } else {
        // hi x lo, hi x hi, lo x hi, term-major so that consecutive MFMAs
        // update different accumulators
        constexpr int TA[3] = {0, 0, 1};
        constexpr int TB[3] = {1, 0, 0};
#pragma unroll
        for (int term = 0; term < 3; ++term)
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int nb = 0; nb < NBA; ++nb)
              acc[nb][t] = mfma_f16(ap[TA[term]][nb][ks], bq[TB[term]][t], acc[nb][t]);
      }
    };

    // MFMA parts of the map operand of one stage.  k-step 0 is converted at
    // the end of the previous stage, once this wave's loads of the stage have
    // landed; further k-steps during the stage, between MFMAs.  The ring
    // registers pass through an empty asm placed after the wait, so no use of
    // them is scheduled above it (the compiler would then wait for every
    // outstanding load itself, emptying the prefetch).
    u16x8 ap[NP][NBA][KSG];
    auto convert_ks = [&](Raw (&src)[NBA][KSG], int ks) {
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb) {
        if constexpr (BF) ap[0][nb][ks] = src[nb][ks];
        else split2(src[nb][ks], ap[0][nb][ks], ap[1][nb][ks]);
      }
    };
    // (callers wait for the registers' loads first: wait_vmcnt<NI>)
    auto convert = [&](Raw (&ring_regs)[NBA][KSG]) {
#pragma unroll
      for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
        for (int ks = 0; ks < KSG; ++ks) asm volatile("" : "+v"(ring_regs[nb][ks]));
      convert_ks(ring_regs, 0);
    };

    // Stage j: the map operand was converted at the end of stage j-1 (by a
    // wave that may then wait at the barrier while the other wave of its SIMD
    // finishes its MFMAs); after the barrier every wave's query planes of
    // stage j are in LDS.
    auto stage = [&](const StagePos& p0, const StagePos& p1, const StagePos& p2, Raw (&ring_regs)[NBA][KSG],
                     Raw (&next_regs)[NBA][KSG]) {
      const int si = p0.si;
      const int lg = p0.lg;
      const int blk_wave = b_begin + si * (W * NBA) + w * NBA;
      const unsigned char* sq = ring + p0.slot * Q_STAGE;

      raw_barrier();
      // the inverse-norm table of the slice whose last stage is j+1
      if (p1.j < nstages && p1.lg == NLG - 1) load_rt(p1.si);
      // The query planes of stage j+2 go to slot (j+2) % 3 = (j-1) % 3,
      // which every wave finished reading before this barrier; the map rows
      // of stage j+2 go to the registers of stage j once all of its k-steps
      // are converted.
      load_q(p2);

      const bool last = lg == NLG - 1;

      // Query tiles are sorted by depth (deepest first): the first na tiles
      // are those whose deepest query still has layers in this group (the
      // first tile always does); shallower queries inside an active tile
      // only add zeros (their staged rows are zero).
      const int l_first = lg * a.geo.lpg;
      int na = 1;
#pragma unroll
      for (int t = 1; t < TQ; ++t) na += tmd[t] > l_first ? 1 : 0;
#pragma unroll
      for (int ks = 0; ks < KSG; ++ks) {
        if (ks > 0) convert_ks(ring_regs, ks);
        if (ks == KSG - 1) load_a(p2, ring_regs);
        if constexpr (TQ == 1) {
          mfma_tiles(std::integral_constant<int, 1>{}, ks, sq, ap);
        } else if constexpr (TQ == 2) {
          if (na == 1) mfma_tiles(std::integral_constant<int, 1>{}, ks, sq, ap);
          else mfma_tiles(std::integral_constant<int, 2>{}, ks, sq, ap);
        } else if constexpr (TQ == 4) {
          if (na == 1) mfma_tiles(std::integral_constant<int, 1>{}, ks, sq, ap);
          else if (na == 2) mfma_tiles(std::integral_constant<int, 2>{}, ks, sq, ap);
          else if (na == 3) mfma_tiles(std::integral_constant<int, 3>{}, ks, sq, ap);
          else mfma_tiles(std::integral_constant<int, 4>{}, ks, sq, ap);
        } else {
          // larger groups: chunks of 4 tiles, each run while its first tile
          // is active
#pragma unroll
          for (int tc = 0; tc < TQ; tc += 4) {
            if (tc > 0 && tc >= na) break;
            u16x8 bq[NP][4];
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
              for (int pl = 0; pl < NP; ++pl)
                bq[pl][tt] = *reinterpret_cast<const u16x8*>(sq + (pl * QG + 16 * (tc + tt) + c) * RB +
                                                             16 * (KSG > 1 ? (4 * ks + g) ^ (c & 7) : 4 * ks + g));
            if constexpr (BF) {
#pragma unroll
              for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int nb = 0; nb < NBA; ++nb) acc[nb][tc + tt] = mfma_bf16(ap[0][nb][ks], bq[0][tt], acc[nb][tc + tt]);
            } else {
              constexpr int TA[3] = {0, 0, 1};
              constexpr int TB[3] = {1, 0, 0};
#pragma unroll
              for (int term = 0; term < 3; ++term)
#pragma unroll
                for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                  for (int nb = 0; nb < NBA; ++nb)
                    acc[nb][tc + tt] = mfma_f16(ap[TA[term]][nb][ks], bq[TB[term]][tt], acc[nb][tc + tt]);
            }
          }
        }
      }

      // Stage j+1's loads (issued during stage j-1) have landed once at most
      // this stage's NI ring loads are outstanding.  Waiting here, before the
      // epilogue branch, also settles the registers the compiler may move
      // where the branch joins (a move of a register whose load is still in
      // flight would otherwise wait for every outstanding load).
      wait_vmcnt<NI>();
      if (last) {
        // End of a slice: cosine = dot * 1/|q[0:p]| * 1/|x[y][0:p]| with the
        // store's prefix inverse norm at the query's depth p; lane (g, c)
        // holds maps 16nb + 4g + i (i = 0..3) of query column c of each tile.
#pragma unroll
        for (int t = 0; t < TQ; ++t) {
          const int r = 16 * t + c;
          const int p = gdep[r];
          const float rq = grq[r];
          if (p == 0) continue;
          const float* rrow = reinterpret_cast<const float*>(rtab + (si & 1) * a.rt_bytes) + gdi[r] * SW;
#pragma unroll
          for (int nb = 0; nb < NBA; ++nb) {
            const int y0 = 16 * (blk_wave + nb) + 4 * g;
            const floatx4 rs = *reinterpret_cast<const floatx4*>(rrow + (w * NBA + nb) * 16 + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int y = y0 + i;
              // maps outside [y_lo, y_hi) belong to a neighbouring workgroup
              if (y < y_lo || y >= y_hi) continue;
              const float dot = BF ? acc[nb][t][i] : acc[nb][t][i] * kDotUnscale;
              const float s = dot * rq * rs[i];
              if constexpr (DBG) a.dbg[static_cast<int64_t>(gperm[r]) * a.n + y] = s;
              best[t].push(make_key(s, y));
            }
          }
        }
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb)
#pragma unroll
          for (int t = 0; t < TQ; ++t) acc[nb][t] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      // map operand of stage j+1 (loads issued during stage j-1)
      convert(next_regs);
    };

    // Two-stage register rotation: stage j computes from the parts of
    // ar[j % 2], reloads it with the map rows of stage j + 2, and converts
    // ar[(j + 1) % 2] for stage j + 1.
    if (has_work) {
      wait_vmcnt<NI>();
      convert(ar0);
      StagePos p0 = p_first;
      StagePos p1 = next_pos(p0, NLG, NS);
      StagePos p2 = next_pos(p1, NLG, NS);
      for (; p0.j + 2 <= nstages;) {
        stage(p0, p1, p2, ar0, ar1);
        p0 = p1;
        p1 = p2;
        p2 = next_pos(p2, NLG, NS);
        stage(p0, p1, p2, ar1, ar0);
        p0 = p1;
        p1 = p2;
        p2 = next_pos(p2, NLG, NS);
      }
      if (p0.j < nstages) stage(p0, p1, p2, ar0, ar1);
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

// ----------------------------------------------------------------------------- finalize

// One wave per position: merge its R partial lists into the k best and write
// them for query perm[pos] (or pos itself when perm is NULL).
template <int KTOP>
__global__ void __launch_bounds__(256) k_finalize(const uint64_t* __restrict__ partial, const int32_t* __restrict__ perm,
                                                  int32_t B, int32_t R, int32_t k, int32_t* __restrict__ idx_out,
                                                  float* __restrict__ score_out, const int32_t* __restrict__ rgrp,
                                                  int32_t qg) {
  const int lane = threadIdx.x % kWave;
  const int pos = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (pos >= B) return;
  const int nr = rgrp != nullptr ? rgrp[pos / qg] : R;
  TopK<KTOP> m;
  m.clear();
  for (int r = lane; r < nr; r += kWave) m.merge(partial + (static_cast<int64_t>(pos) * R + r) * KTOP);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint64_t o[KTOP];
#pragma unroll
    for (int jj = 0; jj < KTOP; ++jj) o[jj] = shfl_xor_u64(m.v[jj], off);
    m.merge(o);
  }
  if (lane == 0) {
    const int b = perm != nullptr ? perm[pos] : pos;
#pragma unroll
    for (int jj = 0; jj < kMaxK; ++jj) {
      if (jj >= k) break;
      const uint64_t key = jj < KTOP ? m.v[jj < KTOP ? jj : 0] : 0ull;
      idx_out[static_cast<int64_t>(b) * k + jj] = key_index(key);
      score_out[static_cast<int64_t>(b) * k + jj] = key_score(key);
    }
  }
}

hipError_t launch_finalize(const uint64_t* partial, const int32_t* perm, int32_t B, int32_t R, int32_t k, int KTOP,
                           int32_t* idx_out, float* score_out, hipStream_t st, const int32_t* rgrp, int32_t qg) {
  const dim3 grid((B + kWaves - 1) / kWaves);
  if (KTOP == 1)
    hipLaunchKernelGGL(k_finalize<1>, grid, dim3(kThreads), 0, st, partial, perm, B, R, k, idx_out, score_out, rgrp, qg);
  else if (KTOP == 4)
    hipLaunchKernelGGL(k_finalize<4>, grid, dim3(kThreads), 0, st, partial, perm, B, R, k, idx_out, score_out, rgrp, qg);
  else
    hipLaunchKernelGGL(k_finalize<8>, grid, dim3(kThreads), 0, st, partial, perm, B, R, k, idx_out, score_out, rgrp, qg);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------- launch

namespace {

Geo geometry(int E) {
  Geo g;
  if (E >= 8 && 32 % E == 0) {
    g.spl = E;
    g.lpg = 32 / E;
    g.ksg = 1;
  } else {
    g.spl = (E + 31) / 32 * 32;
    g.lpg = 1;
    g.ksg = g.spl / 32;
  }
  return g;
}

// 16-map blocks per wave (NBA): two, unless the query group is large; groups
// of 8 query tiles keep two when one k-step covers a layer group or the store
// is bf16 (their accumulators and operands still fit the registers).  Two
// blocks per wave halve the LDS reads of query fragments per MFMA.
constexpr int scan_nba(int TQ, int KSG, bool BF) { return (TQ <= 4 || (TQ == 8 && (KSG == 1 || BF))) ? 2 : 1; }

// One inverse-norm table: a row of the slice's 8 * NBA * 16 maps per distinct
// depth (at most min(QG, dmax) of them), in whole 8 KB chunks (one 1 KB load
// per wave).
int scan_rt_bytes(int TQ, int KSG, int dmax, bool bf) {
  const int QG = 16 * TQ;
  const int nba = scan_nba(TQ, KSG, bf);
  const int rows = QG < dmax ? QG : dmax;
  return (rows * 8 * nba * 16 * 4 + 8 * 1024 - 1) / (8 * 1024) * (8 * 1024);
}

// LDS of the scan: 3 ring slots of query planes (8 waves x NI_Q x 1 KB each),
// two inverse-norm tables, and the group's sorted query info (permutation,
// depth, 1/|q|, distinct-depth index and values, distinct-depth masks); the
// top-K merge buffer reuses the ring.
size_t scan_lds(bool bf, int TQ, int KSG, int KTOP, int dmax) {
  const int NP = bf ? 1 : 2;
  const int QG = 16 * TQ;
  const int ni_q = (NP * QG * qrow_bytes(KSG) + 8 * 1024 - 1) / (8 * 1024);
  size_t ring = static_cast<size_t>(3) * 8 * ni_q * 1024;
  const size_t merge = static_cast<size_t>(8) * QG * KTOP * 8;
  if (merge > ring) ring = merge;
  return ring + 2 * static_cast<size_t>(scan_rt_bytes(TQ, KSG, dmax, bf)) + static_cast<size_t>(5) * QG * 4 +
         static_cast<size_t>(8) * ((QG + 63) / 64);
}

template <bool BF, int TQ, int NBA, int KSG, int KTOP, bool DBG = false>
hipError_t scan_launch(const ScanArgs& a, size_t lds, hipStream_t st) {
  auto kern = k_traj_scan<BF, TQ, NBA, KSG, KTOP, DBG>;
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

// Largest query-tile count per workgroup whose registers fit without spills
// (512 threads leave 256 registers per lane); for top-1 lists 8 tiles with
// two blocks per wave beat 16 tiles with one (half the LDS fragment reads
// per MFMA).
constexpr int tq_limit(bool bf, int ksg, int ktop) {
  return ktop == 1 ? 8 : ktop == 4 ? ((bf || ksg == 1) ? 8 : 2) : (bf ? 4 : 2);
}

// NBA (16-map blocks per wave) follows from TQ and KSG (scan_nba).
template <bool BF, int KSG, int KTOP, int TQ, bool DBG>
hipError_t scan_tq1(const ScanArgs& a, size_t lds, hipStream_t st) {
  if constexpr (TQ <= tq_limit(BF, KSG, KTOP))
    return scan_launch<BF, TQ, scan_nba(TQ, KSG, BF), KSG, KTOP, DBG>(a, lds, st);
  return hipErrorInvalidValue;
}

template <bool BF, int KSG, int KTOP, bool DBG>
hipError_t scan_tq(int TQ, const ScanArgs& a, size_t lds, hipStream_t st) {
  switch (TQ) {
    case 1: return scan_tq1<BF, KSG, KTOP, 1, DBG>(a, lds, st);
    case 2: return scan_tq1<BF, KSG, KTOP, 2, DBG>(a, lds, st);
    case 4: return scan_tq1<BF, KSG, KTOP, 4, DBG>(a, lds, st);
    case 8: return scan_tq1<BF, KSG, KTOP, 8, DBG>(a, lds, st);
    case 16: return scan_tq1<BF, KSG, KTOP, 16, DBG>(a, lds, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool BF, int KTOP, bool DBG = false>
hipError_t scan_ksg(int KSG, int TQ, const ScanArgs& a, size_t lds, hipStream_t st) {
  return KSG == 1 ? scan_tq<BF, 1, KTOP, DBG>(TQ, a, lds, st) : scan_tq<BF, 2, KTOP, DBG>(TQ, a, lds, st);
}

}  // namespace

size_t traj_qrows_bytes(int L, int E, fm_dtype dt, int b_pad) {
  const Geo g = geometry(E);
  const int np = dt == FM_BF16 ? 1 : 2;
  const int nlg = (L + g.lpg - 1) / g.lpg;
  // + slack: a stage's loads round the last group slab up to whole 4 KB
  return static_cast<size_t>(nlg) * b_pad * np * qrow_bytes(g.ksg) + 16384;
}

hipError_t launch_match_trajectory(const StoreView& s, const void* q, const int32_t* depth, int32_t max_depth,
                                   int32_t B, int32_t k, int32_t* idx_out, float* score_out, float* dbg_scores,
                                   const Workspace& ws, hipStream_t st, const SelectFuse* fuse) {
  const bool bf = s.map_dtype == FM_BF16;
  const int esz = bf ? 2 : 4;
  const Geo geo = geometry(s.E);
  // the dense-output form keeps top-1 lists (k = 1)
  const int KTOP = (k == 1 || dbg_scores != nullptr) ? 1 : (k <= 4 ? 4 : 8);
  const int tq_max = tq_limit(bf, geo.ksg, KTOP);
  constexpr size_t kLds = 160 * 1024;

  const int nlg = (max_depth + geo.lpg - 1) / geo.lpg;
  for (int b0 = 0; b0 < B; b0 += kChunkB) {
    const int Bc = (B - b0) < kChunkB ? (B - b0) : kChunkB;
    if (traj_mm_fits(bf, KTOP, Bc, max_depth, nlg, geo.ksg)) {
      // bf16 top-1 (or dense) batches of more than 128 queries: k_traj_mm
      const int QG = traj_mm_group();
      const int n_qg = (Bc + QG - 1) / QG;
      const int b_pad = n_qg * QG;
      PrepArgs pa{};
      pa.q = static_cast<const char*>(q) + static_cast<int64_t>(b0) * s.L * s.E * esz;
      pa.depth = depth + b0;
      pa.B = Bc;
      pa.L = s.L;
      pa.E = s.E;
      pa.dmax = max_depth;
      pa.geo = geo;
      pa.nlg = nlg;
      pa.b_pad = b_pad;
      pa.qg = QG;
      pa.n_qg = n_qg;
      // the bands share the scan's workgroups by the layer groups they walk
      // (a stage costs about the same however many of its tiles are active)
      pa.G = traj_mm_workgroups();
      pa.epi16 = 0;
      pa.tiled = 1;
      pa.ws = ws;
      pa.flags = s.flags;
      hipLaunchKernelGGL(k_traj_prep<true>, dim3(b_pad / 16, nlg + 4), dim3(kThreads), 0, st, pa);
      hipError_t err = hipGetLastError();
      if (err != hipSuccess) return err;
      int32_t R = 0;
      err = launch_traj_mm(s, geo.spl, geo.lpg, geo.ksg, nlg, max_depth, b_pad, ws,
                           dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr, &R, st);
      if (err != hipSuccess) return err;
      if (idx_out != nullptr) {
        err = fuse != nullptr
                  ? launch_merge_select(s, ws.partial, ws.perm, Bc, R, k, 1, ws.rgrp, QG,
                                        idx_out + static_cast<int64_t>(b0) * k,
                                        score_out + static_cast<int64_t>(b0) * k, fuse->at(b0, s.L), st)
                  : launch_finalize(ws.partial, ws.perm, Bc, R, k, 1, idx_out + static_cast<int64_t>(b0) * k,
                                    score_out + static_cast<int64_t>(b0) * k, st, ws.rgrp, QG);
        if (err != hipSuccess) return err;
      }
      continue;
    }
    int TQ = 1;
    while (16 * TQ < Bc && TQ < tq_max) TQ *= 2;
    // smaller query groups when the staged planes of one would not fit the ring
    while (TQ > 1 && scan_lds(bf, TQ, geo.ksg, KTOP, max_depth) > kLds) TQ /= 2;
    const int QG = 16 * TQ;
    const int n_qg = (Bc + QG - 1) / QG;
    const int b_pad = n_qg * QG;

    PrepArgs pa{};
    pa.q = static_cast<const char*>(q) + static_cast<int64_t>(b0) * s.L * s.E * esz;
    pa.depth = depth + b0;
    pa.B = Bc;
    pa.L = s.L;
    pa.E = s.E;
    pa.dmax = max_depth;
    pa.geo = geo;
    pa.nlg = nlg;
    pa.b_pad = b_pad;
    pa.qg = QG;
    pa.ws = ws;
    pa.flags = s.flags;
    // scan workgroups: about one per CU, no more than the store's 16-map
    // blocks per group, at least one per group
    const int n_blocks = (s.n + 15) / 16;
    int G = n_qg * n_blocks < 256 ? n_qg * n_blocks : 256;
    if (G < n_qg) G = n_qg;
    pa.n_qg = n_qg;
    pa.G = G;
    // slice epilogue vs stage cost, measured on the top-4 Phi-shaped batch:
    // about 0.16 stage per score kept in a top-4 list, a third of that for
    // top-1
    pa.epi16 = TQ * scan_nba(TQ, geo.ksg, bf) * 4 * (KTOP == 1 ? 1 : 3);
    const dim3 pgrid(b_pad / 16, nlg + 4);
    if (bf) hipLaunchKernelGGL(k_traj_prep<true>, pgrid, dim3(kThreads), 0, st, pa);
    else hipLaunchKernelGGL(k_traj_prep<false>, pgrid, dim3(kThreads), 0, st, pa);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    const size_t lds = scan_lds(bf, TQ, geo.ksg, KTOP, max_depth);
    if (lds > kLds) return hipErrorInvalidConfiguration;

    const int R = G;   // partial lists per position (a group's share is at most G)

    ScanArgs a{};
    a.planes = s.planes;
    a.plane_bytes = s.plane_elems * esz;
    a.rnorm = s.rnorm;
    a.rn_stride = s.rn_stride;
    a.row = s.row;
    a.n = s.n;
    a.L = s.L;
    a.E = s.E;
    a.geo = geo;
    a.B = Bc;
    a.b_pad = b_pad;
    a.dmax = max_depth;
    a.n_qg = n_qg;
    a.R = R;
    a.n_blocks = n_blocks;
    a.grid = (G + 7) / 8 * 8;
    a.rt_bytes = scan_rt_bytes(TQ, geo.ksg, max_depth, bf);
    a.ws = ws;
    a.dbg = dbg_scores != nullptr ? dbg_scores + static_cast<int64_t>(b0) * s.n : nullptr;
    if (dbg_scores != nullptr) {
      // same arithmetic as the match kernels, plus the dense score stores
      err = bf ? scan_ksg<true, 1, true>(geo.ksg, TQ, a, lds, st) : scan_ksg<false, 1, true>(geo.ksg, TQ, a, lds, st);
    } else if (bf) {
      err = KTOP == 1 ? scan_ksg<true, 1>(geo.ksg, TQ, a, lds, st)
          : KTOP == 4 ? scan_ksg<true, 4>(geo.ksg, TQ, a, lds, st)
                      : scan_ksg<true, 8>(geo.ksg, TQ, a, lds, st);
    } else {
      err = KTOP == 1 ? scan_ksg<false, 1>(geo.ksg, TQ, a, lds, st)
          : KTOP == 4 ? scan_ksg<false, 4>(geo.ksg, TQ, a, lds, st)
                      : scan_ksg<false, 8>(geo.ksg, TQ, a, lds, st);
    }
    if (err != hipSuccess) return err;
    if (idx_out != nullptr) {
      err = fuse != nullptr
                ? launch_merge_select(s, ws.partial, ws.perm, Bc, R, k, KTOP, ws.rgrp, QG,
                                      idx_out + static_cast<int64_t>(b0) * k, score_out + static_cast<int64_t>(b0) * k,
                                      fuse->at(b0, s.L), st)
                : launch_finalize(ws.partial, ws.perm, Bc, R, k, KTOP, idx_out + static_cast<int64_t>(b0) * k,
                                  score_out + static_cast<int64_t>(b0) * k, st, ws.rgrp, QG);
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

}  // namespace fm
