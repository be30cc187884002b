// Trajectory-based expert map search (Section 4.2.2, Eq. 5), top-1 form for
// bfloat16 stores and batches of more than 128 queries.
//
// The batch is the contraction of the depth-sorted query prefixes with the
// stored maps' prefixes, layer group by layer group, on
// v_mfma_f32_16x16x32_bf16, followed by the division by the query's and the
// stored map's prefix norms (the latter precomputed at insert) and the best
// stored index per query.  k_traj_prep (fm_traj.hip) sorts and stages the
// queries before it runs; k_finalize merges its partial lists after.
//
// Query bands.  The sorted queries form tiles of 16 (deepest first); tiles
// 16 b .. 16 b + 15 form band b, which walks only the layer groups its
// deepest query reaches, and within a band a query tile takes part in the
// layer groups its own deepest query reaches (shallower queries of the tile
// contribute their staged zeros).  The scan's 256 workgroups are shared
// among the bands in proportion to the layer groups they walk (k_traj_prep
// writes the shares): with depths spread over the layers, the deep band's
// stages keep most of their tiles active and the shallow band runs half as
// many stages per map, whereas bands of mixed depths would each walk every
// layer with half of their tiles idle.  A band's workgroups take the
// store's 16-block slices round-robin, so every band sweeps the store from
// front to back at about the same pace; each band streams the planes of its
// own layers, and the shallow band's reads of the first layers come close
// enough in time to the deep band's to find them in the memory-side cache.
//
// Workgroup: 8 waves, two per SIMD, arranged 2 x 4 over (queries, maps).
// Wave (wq, wm) holds 128 x 64 float32 accumulators: the band's local query
// tiles wq, wq + 2, ..., wq + 14 (so the two query rows of waves stay
// equally deep) against the map blocks wm, wm + 4, wm + 8, wm + 12 of a
// slice (16 blocks of 16 maps).
//
// Pipeline: a stage is one k-step of one layer group of one slice.  Its map
// tiles (1 KB of a plane tile: 8 expert quads of 16 maps) and the band's
// query tiles (1 KB MFMA operand tiles staged by the prep) are copied
// global -> LDS by buffer loads straight into ring slot j % 3; tiles of
// queries that are all shallower than the layer group read as zeros without
// memory traffic.  At the start of stage j, once its own copies of stage
// j+1 have landed, each wave passes the one barrier of the stage; slot j % 3
// then receives the copies of stage j + 3 and the fragments of stage j+1
// are read while the MFMAs of stage j run.  The copies of a slice's last
// stage also bring the slice's prefix inverse norms: one 1 KB row per depth
// (rnorm[p-1] of the slice's 256 maps) into one of two tables.
//
// Epilogue of a slice: lane (g, c) holds, for block i and query tile t, the
// dots of maps 4g .. 4g+3 of the block with query c of the tile; the cosine
// at the query's depth p is (dot * 1/|q[0:p]|) * 1/|x[y][0:p]|.  The lane
// ranks by dot * 1/|x[y][0:p]| (1/|q[0:p]| is positive, or 0, and is applied
// once after the scan) and keeps the best (score, index) per query tile: a
// lane visits its maps in increasing index order (its slices in order, the
// blocks of a slice in order) and only a strictly greater score replaces the
// kept one, so equal scores keep the lower index, and a NaN score ranks
// below every other.  The lists are merged over lane groups and waves and
// stored as the workgroup's partial list.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

struct TrajMmArgs {
  const char* planes;     // [L] tiled bf16 planes
  uint32_t plane_bytes;   // bytes per plane
  uint32_t tile_bytes;    // bytes of one 16-map tile of a plane (32 * row)
  const float* rnorm;     // [L][rn_stride] prefix inverse norms
  int32_t rn_stride;
  const char* qst;        // staged queries: [lg][ks][band][local tile][1 KB]
  uint32_t qst_bytes;
  const float* rq;        // [b_pad] 1/|q[0:p]| at each sorted position
  const int32_t* sdep;    // [b_pad] depth at each sorted position (0: padding)
  const int32_t* perm;    // [b_pad] query index at each sorted position
  uint64_t* partial;      // [b_pad][R] one packed key per (position, workgroup of its band)
  const int32_t* pgrp;    // per band: its first workgroup (XCD-aware numbering)
  const int32_t* rgrp;    // per band: its workgroups
  const int32_t* ngrp;    // per band: the layer groups its deepest query reaches
  float* dbg;             // optional dense scores [B][n]
  int32_t n, L, row, spl, lpg, ksg, nlg, dmax;
  int32_t n_qg;           // query bands (256 queries each)
  int32_t R;              // stride of the partial lists per position (the grid's workgroups)
  int32_t n_blocks;       // 16-map blocks of the store
  int32_t grid;
};

constexpr int kW = 8;          // waves per workgroup (two per SIMD)
constexpr int kGM = 4;         // wave columns over the maps
constexpr int kNT = 8;         // query tiles per wave
constexpr int kNB = 4;         // map blocks per wave and slice
constexpr int kQG = 256;       // queries per band
constexpr int kSB = 16;        // map blocks per slice
constexpr int kNS = 3;         // ring slots
constexpr int kMPW = 2;        // map tile copies per wave and stage
constexpr int kQPW = 2;        // query tile copies per wave and stage
constexpr int kNI = kMPW + kQPW;
constexpr int kNTAB = 4;       // inverse-norm rows per wave (slice-last stages only)
constexpr int kRows = kW * kNTAB;   // table rows: depths 1 .. 32
constexpr int kSlot = (kSB + kQG / 16) * 1024;
constexpr int kTab = kRows * 1024;
constexpr int kLds = kNS * kSlot + 2 * kTab;
static_assert(kSB == kW * kMPW && kQG / 16 == kW * kQPW, "copies per stage");
static_assert(kLds <= 160 * 1024, "LDS");

}  // namespace

template <bool DBG, int KSG>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) k_traj_mm(TrajMmArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ring = smem;                    // [kNS][kSlot]
  unsigned char* tab = smem + kNS * kSlot;       // [2][kRows][256] float
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(smem);   // after the loop: [kGM][kQG]

  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wq = w / kGM;
  const int wm = w - wq * kGM;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;

  // workgroup -> (query band, share of the store): band b owns the
  // workgroups [pgrp[b], pgrp[b] + rgrp[b]) of the XCD-aware numbering u
  // (shared in proportion to the layer groups the bands walk); values read
  // back wave-uniform
  const int bid = blockIdx.x;
  const int u = (bid % 8) * (a.grid / 8) + bid / 8;
  int pg_l = 0x7fffffff, rg_l = 0, ng_l = 0;
  if (lane < a.n_qg) {
    pg_l = a.pgrp[lane];
    rg_l = a.rgrp[lane];
    ng_l = a.ngrp[lane];
  }
  const uint64_t gbal = __ballot(lane < a.n_qg && pg_l <= u);
  const int qg_u = gbal != 0 ? __popcll(gbal) - 1 : 0;
  const int Rg = __builtin_amdgcn_readfirstlane(__shfl(rg_l, qg_u, kWave));
  const int Pg = __builtin_amdgcn_readfirstlane(__shfl(pg_l, qg_u, kWave));
  const int Ng = __builtin_amdgcn_readfirstlane(__shfl(ng_l, qg_u, kWave));
  const bool active = gbal != 0 && u - Pg < Rg;
  const int grp = active ? qg_u : 0;
  const int rr = active ? u - Pg : 0;
  // The band's workgroups take the store's slices (kSB blocks from block 0)
  // round-robin: workgroup rr the slices rr, rr + Rg, rr + 2 Rg, ...  So
  // every band sweeps the store from front to back at the pace of its
  // layer share, and the bands read the planes they have in common at
  // about the same time (the later read finds them in the memory-side
  // cache).
  const int n_sl_all = (a.n_blocks + kSB - 1) / kSB;
  const int n_slices = active && rr < n_sl_all ? (n_sl_all - rr + Rg - 1) / Rg : 0;
  const int b_begin = rr * kSB;              // first block of the first slice
  const int b_end = a.n_blocks;
  const int sstep = Rg * kSB;                // blocks from one of its slices to the next
  // the band's layer groups, at least two stages per slice (the staged rows
  // of layer groups past every query of the band are zeros)
  int nlg = Ng < 1 ? 1 : Ng;
  if (nlg * KSG < 2) nlg = 2;
  if (nlg > a.nlg) nlg = a.nlg;
  // stages per slice, an even count: with one k-step per layer group an odd
  // count gets one more group, past every query of the band (its tiles take
  // no MFMAs; past the store's groups its copies read as zeros)
  if (KSG == 1) nlg += nlg & 1;
  const int nst = nlg * KSG;
  const int nstages = n_slices * nst;

  // sorted position of query c of this wave's tile t (local tile wq + 2t of the band)
  auto pos_of = [&](int t) __attribute__((always_inline)) { return (grp * 16 + wq + 2 * t) * 16 + c; };
  uint32_t rows4[kNT / 4];   // the query's inverse-norm table row (depth - 1), a byte per tile
  int tmd[kNT];              // depth of the tile's deepest query (wave-uniform)
#pragma unroll
  for (int t = 0; t < kNT / 4; ++t) rows4[t] = 0;
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    const int p = pos_of(t);
    const int d = a.sdep[p];
    rows4[t / 4] |= static_cast<uint32_t>(d > 0 ? d - 1 : 0) << (8 * (t % 4));
    tmd[t] = __builtin_amdgcn_readfirstlane(d);   // lane 0 holds row 0 of the tile, its deepest query
  }
  // Best map per query tile, ranked by dot * 1/|x[0:p]|: the query's own
  // factor 1/|q[0:p]| is positive (or 0 for a zero query, where every score
  // is 0) and does not change the order, so it is applied once at the end.
  // A NaN score ranks below every other score: the list starts at the
  // lane's first map with the lowest finite float, which only a greater
  // score replaces (a NaN compares false).
  constexpr float kNanFloor = -3.40282347e38f;
  const int y_first = 16 * (b_begin + wm) + 4 * g;
  const bool first_ok = n_slices > 0 && b_begin + wm < b_end && y_first < a.n;
  float best_s[kNT];
  int best_i[kNT];
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    best_s[t] = kNanFloor;
    best_i[t] = first_ok ? y_first : -1;
  }

  if (nstages > 0) {
    // Lane L of a map tile copy takes 16 bytes of quad L / 8 (maps 2m, 2m+1,
    // m = L % 8) of k-step ks: slots 32 ks + 4 (L / 8) .. +3 lie in layer li
    // of the layer group at expert e0; quads past the row read as zeros.
    uint32_t loff[KSG];
    bool qv[KSG];
#pragma unroll
    for (int ks = 0; ks < KSG; ++ks) {
      const int s0 = 32 * ks + 4 * (lane / 8);
      const int li = s0 / a.spl;
      const int e0 = s0 - li * a.spl;
      qv[ks] = e0 < a.row;
      loff[ks] = static_cast<uint32_t>(li) * a.plane_bytes + static_cast<uint32_t>((e0 / 4) * 128 + (lane % 8) * 16);
    }

    const __amdgpu_buffer_rsrc_t rs_q = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.qst), static_cast<short>(0), static_cast<int>(a.qst_bytes), kBufWord3);
    const __amdgpu_buffer_rsrc_t rs_rn = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.rnorm), static_cast<short>(0),
        static_cast<int>(static_cast<uint32_t>(a.L) * static_cast<uint32_t>(a.rn_stride) * 4u), kBufWord3);

    // The copies run kNS stages ahead of the MFMAs.  Their position (the
    // "copy position") is kept as running scalars, stepped by one stage per
    // stage: its layer group's first plane and byte count (the map
    // descriptor), the byte offset of its staged query tiles, and its slice;
    // the vector offsets of this wave's tiles depend on the slice only.
    // (Scalar instructions are issued one per SIMD every fourth cycle and
    // both waves of a SIMD need theirs: per-stage scalar work is kept small.)
    const uint64_t lpgb = static_cast<uint64_t>(a.lpg) * a.plane_bytes;   // bytes of a layer group
    const int last_lg = (a.L + a.lpg - 1) / a.lpg - 1;                     // the store's last group
    const uint32_t full_rec = static_cast<uint32_t>(lpgb);
    const uint32_t last_rec = static_cast<uint32_t>(a.L - last_lg * a.lpg) * a.plane_bytes;
    const uint32_t qstep = static_cast<uint32_t>(a.n_qg) * 16384u;
    auto rec_of = [&](int lg) __attribute__((always_inline)) {
      return lg < last_lg ? full_rec : (lg == last_lg ? last_rec : 0u);
    };
    uint64_t c_base = reinterpret_cast<uint64_t>(a.planes);
    uint32_t c_rec = rec_of(0);
    int c_lg = 0;
    uint32_t c_qoff = static_cast<uint32_t>(grp) * 16384u;
    int c_blk0 = b_begin;
    int c_tab = 0;          // which inverse-norm table the copy position's slice fills
    int c_slot = 0;         // ring slot of the current stage = slot of the copy position
    bool tab_prev = false;  // the copies issued last included table rows
    // this wave's map tiles of the copy position's slice: byte offset in a
    // plane and whether the block lies in the workgroup's range (copies of
    // blocks past it, and of quads past the row, are outside every descriptor)
    uint32_t c_moff[kMPW];
    bool c_mok[kMPW];
    auto set_slice = [&](int blk0) __attribute__((always_inline)) {
#pragma unroll
      for (int m = 0; m < kMPW; ++m) {
        const int blk = blk0 + w * kMPW + m;
        c_moff[m] = static_cast<uint32_t>(blk) * a.tile_bytes;
        c_mok[m] = blk < b_end;
      }
    };
    set_slice(b_begin);
    const uint32_t vqo = static_cast<uint32_t>(w * kQPW * 1024 + lane * 16);

    // Part `part` of the copies of the copy position (k-step KSC of its layer
    // group) into the current stage's slot: parts 0 and 1 a map tile each, 2
    // and 3 a query tile each, 4 the table rows when the position is its
    // slice's last stage.
    auto issue_part = [&](auto ksc_c, int part, bool with_tab) __attribute__((always_inline)) {
      constexpr int KSC = decltype(ksc_c)::value;
      unsigned char* slot = ring + c_slot * kSlot;
      if (part < kMPW) {
        const __amdgpu_buffer_rsrc_t rs_map = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<char*>(c_base), static_cast<short>(0), static_cast<int>(c_rec), kBufWord3);
        const int tile = w * kMPW + part;
        const uint32_t off = (qv[KSC] && c_mok[part]) ? loff[KSC] + c_moff[part] : kOutside;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_map, (lds_vp)(slot + tile * 1024), 16, static_cast<int>(off), 0,
                                                 0, 0);
      } else if (part < kNI) {
        const int i = part - kMPW;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_q, (lds_vp)(slot + (kSB + w * kQPW + i) * 1024), 16,
                                                 static_cast<int>(c_qoff + vqo + static_cast<uint32_t>(i * 1024)), 0,
                                                 0, 0);
      } else if (with_tab) {
        unsigned char* tb = tab + c_tab * kTab;
#pragma unroll
        for (int i = 0; i < kNTAB; ++i) {
          const int r = w * kNTAB + i;
          const uint32_t off = r < a.dmax ? (static_cast<uint32_t>(r) * static_cast<uint32_t>(a.rn_stride) +
                                             static_cast<uint32_t>(16 * c_blk0)) * 4u + static_cast<uint32_t>(lane * 16)
                                          : kOutside;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_rn, (lds_vp)(tb + r * 1024), 16, static_cast<int>(off), 0, 0, 0);
        }
      }
    };
    // Step the copy position past a stage: k-step KSC of its layer group,
    // the group's last k-step when KSC == KSG - 1 (then the next group, or
    // the next slice after the slice's last group).
    auto step_copy = [&](auto ksc_c, bool with_tab) __attribute__((always_inline)) {
      constexpr int KSC = decltype(ksc_c)::value;
      c_slot = c_slot == kNS - 1 ? 0 : c_slot + 1;
      c_qoff += qstep;
      tab_prev = with_tab;
      if constexpr (KSC == KSG - 1) {
        if (with_tab) {
          c_lg = 0;
          c_base = reinterpret_cast<uint64_t>(a.planes);
          c_rec = rec_of(0);
          c_qoff = static_cast<uint32_t>(grp) * 16384u;
          c_blk0 += sstep;
          c_tab ^= 1;
          set_slice(c_blk0);
        } else {
          ++c_lg;
          c_base += lpgb;
          c_rec = rec_of(c_lg);
        }
      }
    };
    auto copy_last = [&](auto ksc_c) __attribute__((always_inline)) {
      constexpr int KSC = decltype(ksc_c)::value;
      return KSC == KSG - 1 && c_lg == nlg - 1;
    };

    floatx4 acc[kNB][kNT];
#pragma unroll
    for (int i = 0; i < kNB; ++i)
#pragma unroll
      for (int t = 0; t < kNT; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    // map fragment of block i: quads g and 4 + g of map c (two 8-byte reads
    // 512 bytes apart); query fragment of local tile wq + 2t
    auto read_mfrag = [&](int slot, int i) __attribute__((always_inline)) {
      const unsigned char* p = ring + slot * kSlot + (wm + kGM * i) * 1024 + g * 128 + c * 8;
      const uint32x2 lo = *reinterpret_cast<const uint32x2*>(p);
      const uint32x2 hi = *reinterpret_cast<const uint32x2*>(p + 512);
      return __builtin_bit_cast(u16x8, uint32x4{lo[0], lo[1], hi[0], hi[1]});
    };
    auto read_qfrag = [&](int slot, int t) __attribute__((always_inline)) {
      return *reinterpret_cast<const u16x8*>(ring + slot * kSlot + (kSB + wq + 2 * t) * 1024 + lane * 16);
    };

    // Slice epilogue: scores of this wave's blocks of slice si, best per
    // query, in 8 groups (block i, tiles 4h .. 4h+3).  Each group needs the
    // inverse norms of its 4 tiles' rows (one 16-byte LDS read per tile); the
    // reads of the next group are issued before the current group is scored,
    // so that their latency hides behind its arithmetic.  The table was copied
    // with the slice's last stage and the stage waits have covered it; the
    // reads are written out (with waits the values depend on) so that the
    // compiler does not wait for every copy still in flight.
    auto epilogue = [&](int si) __attribute__((always_inline)) {
      const int blk_s = b_begin + si * sstep;
      const unsigned char* tb = tab + (si & 1) * kTab;
      auto read_rows = [&](floatx4 (&xr)[4], int grp) __attribute__((always_inline)) {
        const int i = grp / 2;
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const int row = (rows4[grp % 2] >> (8 * h)) & 0xFF;
          const uint32_t addr =
              static_cast<uint32_t>(reinterpret_cast<uintptr_t>(tb + row * 1024 + (wm + kGM * i) * 64 + 16 * g));
          asm volatile("ds_read_b128 %0, %1" : "=v"(xr[h]) : "v"(addr));
        }
      };
      // (the last block of the store checks its rows against n; the others
      // take a copy of the loop without the check)
      auto score_group = [&](const floatx4 (&xr)[4], int grp, auto full_c) __attribute__((always_inline)) {
        constexpr bool FULL = decltype(full_c)::value;
        const int i = grp / 2;
        const int y0 = 16 * (blk_s + wm + kGM * i) + 4 * g;
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
          const int t = 4 * (grp % 2) + tt;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int y = y0 + r;
            if constexpr (DBG) {
              // the dense form writes every cosine and keeps no lists
              const int p = pos_of(t);
              const int b = a.perm[p];
              if (b >= 0 && y < a.n) a.dbg[static_cast<int64_t>(b) * a.n + y] = acc[i][t][r] * a.rq[p] * xr[tt][r];
            } else {
              const float sv = acc[i][t][r] * xr[tt][r];
              if ((FULL || y < a.n) && sv > best_s[t]) {
                best_s[t] = sv;
                best_i[t] = y;
              }
            }
          }
        }
      };
      floatx4 xa[4], xb[4];
      read_rows(xa, 0);
#pragma unroll
      for (int grp = 0; grp < 2 * kNB; ++grp) {
        floatx4 (&cur)[4] = grp % 2 == 0 ? xa : xb;
        floatx4 (&nxt)[4] = grp % 2 == 0 ? xb : xa;
        // blocks past the store (the store's last slice) are read but not
        // scored: the table row stays within its kilobyte
        if (grp + 1 < 2 * kNB) {
          read_rows(nxt, grp + 1);
          asm volatile("s_waitcnt lgkmcnt(4)" : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]));
        } else {
          asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]));
        }
        const int blk = blk_s + wm + kGM * (grp / 2);
        if (blk < b_end) {
          if (16 * blk + 16 <= a.n) score_group(cur, grp, std::true_type{});
          else score_group(cur, grp, std::false_type{});
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // (the zeros are hidden from the compiler: known-zero accumulators
      // would otherwise be folded into the next MFMAs and no longer share
      // registers with the other paths)
#pragma unroll
      for (int i = 0; i < kNB; ++i)
#pragma unroll
        for (int t = 0; t < kNT; ++t) {
          acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};
          asm volatile("" : "+v"(acc[i][t]));
        }
    };

    // depth of each of this wave's tiles' deepest query, tile t at lane t:
    // the tiles active in a layer group are those reaching its first layer
    const int vtmd = lane < kNT ? a.sdep[(grp * 16 + wq + 2 * lane) * 16] : 0;

    // prologue: the copies of stages 0 .. kNS-1, then stage 0's fragments
#pragma unroll
    for (int s = 0; s < kNS; ++s) {
      if constexpr (KSG == 2) {
        if (s % 2 == 0) {
#pragma unroll
          for (int part = 0; part <= kNI; ++part) issue_part(std::integral_constant<int, 0>{}, part, false);
          step_copy(std::integral_constant<int, 0>{}, false);
        } else {
          const bool tl = copy_last(std::integral_constant<int, 1>{});
#pragma unroll
          for (int part = 0; part <= kNI; ++part) issue_part(std::integral_constant<int, 1>{}, part, tl);
          step_copy(std::integral_constant<int, 1>{}, tl);
        }
      } else {
        const bool tl = copy_last(std::integral_constant<int, 0>{});
#pragma unroll
        for (int part = 0; part <= kNI; ++part) issue_part(std::integral_constant<int, 0>{}, part, tl);
        step_copy(std::integral_constant<int, 0>{}, tl);
      }
    }
    u16x8 fa0[kNB], fa1[kNB], fb[kNT];
    wait_vmcnt<0>();
    raw_barrier();
#pragma unroll
    for (int i = 0; i < kNB; ++i) fa0[i] = read_mfrag(0, i);
#pragma unroll
    for (int t = 0; t < kNT; ++t) fb[t] = read_qfrag(0, t);
    wait_lgkm0();

    // One stage: its MFMAs (tiles whose deepest query reaches first layer
    // l_first), the next stage's fragments, and the copy position's copies
    // (k-step KSC of its group) into the current slot.  A slice's LAST stage
    // reads no fragments: the next slice's are read after the epilogue, so
    // that none of them is held through it.
    auto stage = [&](auto ksc_c, auto last_c, int l_first, u16x8 (&fa)[kNB], u16x8 (&na)[kNB])
                     __attribute__((always_inline)) {
      constexpr bool LAST = decltype(last_c)::value;
      // stage j+1's copies have landed once only the latest ones (those of
      // stage j+2) are outstanding
      if (tab_prev) wait_vmcnt<kNI + kNTAB>();
      else wait_vmcnt<kNI>();
      raw_barrier();
      const bool tl = copy_last(ksc_c);
      const int sn = c_slot == kNS - 1 ? 0 : c_slot + 1;
      if constexpr (!LAST) {
#pragma unroll
        for (int i = 0; i < kNB; ++i) na[i] = read_mfrag(sn, i);
      }
      // (tiles at lanes 0..7: the low half of the ballot)
      const int nact = __builtin_popcount(static_cast<uint32_t>(__ballot(vtmd > l_first)));   // the depths fall with t
      __builtin_amdgcn_s_setprio(1);
      // per tile a uniform branch: its MFMAs, then its fragment of the next
      // stage into the register they have just read; copy part t after tile t
      // (the fragment address is computed once, not in every tile's branch)
      uint32_t qa = static_cast<uint32_t>(sn * kSlot + (kSB + wq) * 1024 + lane * 16);
      asm volatile("" : "+v"(qa));
#pragma unroll
      for (int t = 0; t < kNT; ++t) {
        if (t < nact) {
#pragma unroll
          for (int i = 0; i < kNB; ++i) acc[i][t] = mfma_bf16(fa[i], fb[t], acc[i][t]);
          if constexpr (!LAST) fb[t] = *reinterpret_cast<const u16x8*>(ring + qa + t * 2048);
        }
        if (t <= kNI) issue_part(ksc_c, t, tl);
      }
      __builtin_amdgcn_s_setprio(0);
      step_copy(ksc_c, tl);
      if constexpr (!LAST) wait_lgkm0();
    };
    using C0 = std::integral_constant<int, 0>;
    using CA = std::integral_constant<int, KSG - 1>;
    using F = std::false_type;
    using T = std::true_type;
    // Per slice its stages in pairs, the epilogue, then the next slice's
    // first fragments (into fa0 and fb).  The copy position is kNS = 3
    // stages ahead: with two k-steps per layer group the first stage of a
    // pair (k-step 0) copies k-step 1 and the second k-step 0.
    for (int si = 0; si < n_slices; ++si) {
      int l0 = 0;
      for (int s2 = 0; s2 + 2 < nst; s2 += 2) {
        stage(CA{}, F{}, l0, fa0, fa1);
        if constexpr (KSG == 1) l0 += a.lpg;
        stage(C0{}, F{}, l0, fa1, fa0);
        l0 += a.lpg;
      }
      stage(CA{}, F{}, l0, fa0, fa1);
      if constexpr (KSG == 1) l0 += a.lpg;
      stage(C0{}, T{}, l0, fa1, fa0);
      epilogue(si);
      // the next stage's slot (its copies have landed: waited for at the
      // start of the last stage)
#pragma unroll
      for (int i = 0; i < kNB; ++i) fa0[i] = read_mfrag(c_slot, i);
#pragma unroll
      for (int t = 0; t < kNT; ++t) fb[t] = read_qfrag(c_slot, t);
      wait_lgkm0();
    }
    wait_vmcnt<0>();   // the trailing copies
  }
  __syncthreads();

  // the cosine of each tile's best: its score times 1/|q[0:p]|; a NaN score
  // takes the in-scan NaN value, and a NaN query (every cosine NaN) the
  // lowest index among this lane's maps
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    const float rq = a.rq[pos_of(t)];
    if (best_i[t] >= 0) {
      if (rq != rq) {
        best_s[t] = kNanScore;
        best_i[t] = first_ok ? y_first : -1;
      } else {
        best_s[t] = best_s[t] == kNanFloor ? kNanScore : best_s[t] * rq;
      }
    }
  }

  // merge: the four lane groups of a query, then the kGM waves of its tile row
  uint64_t key[kNT];
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    key[t] = best_i[t] < 0 ? 0ull : make_key(best_s[t], best_i[t]);
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      const uint64_t o = shfl_xor_u64(key[t], m);
      key[t] = o > key[t] ? o : key[t];
    }
  }
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < kNT; ++t) mbuf[wm * kQG + (wq + 2 * t) * 16 + c] = key[t];
  }
  __syncthreads();
  if (active) {
    for (int r = tid; r < kQG; r += kW * kWave) {
      uint64_t m = 0;
#pragma unroll
      for (int ww = 0; ww < kGM; ++ww) m = mbuf[ww * kQG + r] > m ? mbuf[ww * kQG + r] : m;
      const int p = grp * kQG + r;
      a.partial[static_cast<int64_t>(p) * a.R + rr] = m;
    }
  }
}

namespace {

template <bool DBG, int KSG>
hipError_t traj_mm_launch(const TrajMmArgs& a, hipStream_t st) {
  auto kern = k_traj_mm<DBG, KSG>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       kLds);
  if (err != hipSuccess) return err;
  const ScanEvents& ev = scan_events();
  if (ev.start != nullptr) {
    err = hipEventRecord(ev.start, st);
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(kern, dim3(a.grid), dim3(kW * kWave), kLds, st, a);
  err = hipGetLastError();
  if (err != hipSuccess || ev.stop == nullptr) return err;
  return hipEventRecord(ev.stop, st);
}

}  // namespace

bool traj_mm_fits(bool bf, int KTOP, int32_t Bc, int32_t max_depth, int nlg, int ksg) {
  return bf && KTOP == 1 && Bc > 128 && max_depth <= kRows && nlg * ksg >= 2 && (ksg == 1 || ksg == 2);
}

int traj_mm_group() { return kQG; }

int traj_mm_workgroups() { return 256; }

hipError_t launch_traj_mm(const StoreView& s, int spl, int lpg, int ksg, int nlg, int32_t max_depth, int32_t b_pad,
                          const Workspace& ws, float* dbg, int32_t* R_out, hipStream_t st) {
  const int n_qg = b_pad / kQG;
  const int n_blocks = (s.n + 15) / 16;
  const int R = traj_mm_workgroups();   // the prep shared them among the bands
  TrajMmArgs a;
  a.planes = static_cast<const char*>(s.planes);
  a.plane_bytes = static_cast<uint32_t>(s.plane_elems * 2);
  a.tile_bytes = static_cast<uint32_t>(16 * s.row * 2);
  a.rnorm = s.rnorm;
  a.rn_stride = static_cast<int32_t>(s.rn_stride);
  a.qst = static_cast<const char*>(ws.qrows);
  a.qst_bytes = static_cast<uint32_t>(static_cast<int64_t>(nlg) * ksg * b_pad * 64);
  a.rq = ws.rq;
  a.sdep = ws.sdep;
  a.perm = ws.perm;
  a.partial = ws.partial;
  a.pgrp = ws.pgrp;
  a.rgrp = ws.rgrp;
  a.ngrp = ws.ngrp;
  a.dbg = dbg;
  a.n = s.n;
  a.L = s.L;
  a.row = s.row;
  a.spl = spl;
  a.lpg = lpg;
  a.ksg = ksg;
  a.nlg = nlg;
  a.dmax = max_depth;
  a.n_qg = n_qg;
  a.R = R;
  a.n_blocks = n_blocks;
  a.grid = R;
  *R_out = R;
  if (ksg == 2) return dbg != nullptr ? traj_mm_launch<true, 2>(a, st) : traj_mm_launch<false, 2>(a, st);
  return dbg != nullptr ? traj_mm_launch<true, 1>(a, st) : traj_mm_launch<false, 1>(a, st);
}

}  // namespace fm
