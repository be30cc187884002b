// Incremental trajectory re-search (Section 4.2.2): within one pass the
// trajectory search is repeated after every newly observed layer, each time
// with the prefix grown by one layer.  The Eq. 5 cosine over the first p
// layers is dot_p / (|q[0:p]| |x[y][0:p]|) with dot_p = dot_{p-1} + the new
// layer's dot product, so a step keeps the running dot of every (query,
// stored map) pair in a caller-owned state buffer and reads one map plane
// instead of p.
//
//   k_traj_step   one 16-map tile of the store per wave: the layer's dot
//                 products by float32 MFMA (16 maps x 16 queries x 4 experts
//                 per instruction, exact float32 products), added onto the
//                 running dots, scored with the stored prefix inverse norm at
//                 depth p and the query's running float64 norm, per-lane
//                 top-K, merged per workgroup into partial lists; workgroup 0
//                 also advances the query norms and checks the state header
//                 (same store size as at layer 0, layers in order);
//   k_finalize    (shared with the scans) merges the partial lists.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

namespace {

constexpr int kStepQ = 64;        // queries per launch (4 query tiles)
constexpr int kStepW = 4;         // waves per workgroup
constexpr int kStepThreads = kStepW * kWave;
// workgroups per launch at most: the partial lists of kStepQ queries fill
// the match workspace's kChunkB x kMaxPartials lists
constexpr int kStepMaxR = kChunkB * kMaxPartials / kStepQ;

struct StepHeader {
  int32_t n_begin;     // store size at layer 0
  int32_t last_layer;  // last layer added
};

// State of one chunk of kStepQ queries: [header, 256 B][query sums of squares
// after even layers: kStepQ float64][after odd layers: kStepQ float64]
// [dots: n_tiles x 4 query tiles x 64 lanes x 4 float32].  A step reads the
// sums in the previous layer's slot and workgroup 0 writes the other slot, so
// no workgroup reads a slot while it is written.
constexpr size_t kStepHead = 256 + 2 * kStepQ * 8;

struct StepArgs {
  const void* planes;
  int64_t plane_elems;
  const float* rnorm;
  int64_t rn_stride;
  int32_t n, E, row, layer, Bc;
  int32_t R, n_tiles;
  const void* q;        // [Bc][E]
  char* state;          // chunk state
  uint64_t* partial;    // [kStepQ][R][KTOP]
  uint32_t* flags;
};

}  // namespace

// Lane (g, c) = (lane / 16, lane % 16).  For 4 quads of experts at a time,
// lane (g, c) loads quad 4s+g of map c of the tile (one 16-byte load: 4
// consecutive experts) and holds the same 4 experts of query c of its query
// tile; the j-th MFMA of the group takes the j-th of those experts, so the 4
// MFMAs together cover experts 16s .. 16s+15 (the k index of a product does
// not matter to the dot product).  The accumulator of lane (g, c) holds maps
// 4g .. 4g+3 of the tile for query c.
//
// A workgroup takes a contiguous range of tiles; its 4 waves split into TQ
// query tiles x (4 / TQ) phases: wave w serves query tile w % TQ and the
// tiles of the range with index = w / TQ modulo 4 / TQ.  Each wave keeps the
// loads of its next two tiles in flight.
template <bool BF, int TQ, int KTOP>
__global__ void __launch_bounds__(kStepThreads) k_traj_step(StepArgs a) {
  constexpr int NPH = kStepW / TQ;   // phases
  constexpr int P = 3;               // register buffers: current + 2 ahead
  __shared__ uint64_t mbuf[kStepW][16][KTOP];
  using T = typename std::conditional<BF, uint16_t, float>::type;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int g = lane / 16;
  const int c = lane % 16;
  const int qt = w % TQ;
  const int ph = w / TQ;
  const int nq4 = a.row / 16 + (a.row % 16 != 0 ? 1 : 0);   // groups of 4 quads
  const int nquads = a.row / 4;
  const T* plane = static_cast<const T*>(a.planes) + static_cast<int64_t>(a.layer) * a.plane_elems;
  const float* rn = a.rnorm + static_cast<int64_t>(a.layer) * a.rn_stride;
  float* dots = reinterpret_cast<float*>(a.state + kStepHead);
  const int t_begin = static_cast<int>((static_cast<int64_t>(blockIdx.x) * a.n_tiles) / a.R);
  const int t_end = static_cast<int>((static_cast<int64_t>(blockIdx.x + 1) * a.n_tiles) / a.R);

  auto load_tile = [&](int tl, floatx4 (&av)[4], floatx4& prev, floatx4& rs) {
    const T* tb = plane + static_cast<int64_t>(tl) * 16 * a.row;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int quad = 4 * s + g;
      floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
      if (s < nq4 && quad < nquads) {
        const T* p = tb + quad * 64 + c * 4;
        if constexpr (BF) {
          const uint32x2 h = *reinterpret_cast<const uint32x2*>(p);
          v[0] = __uint_as_float(h[0] << 16);
          v[1] = __uint_as_float(h[0] & 0xffff0000u);
          v[2] = __uint_as_float(h[1] << 16);
          v[3] = __uint_as_float(h[1] & 0xffff0000u);
        } else {
          v = *reinterpret_cast<const floatx4*>(p);
        }
      }
      av[s] = v;
    }
    const float* dp = dots + (static_cast<int64_t>(tl) * 4 + qt) * 256 + lane * 4;
    prev = a.layer == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : *reinterpret_cast<const floatx4*>(dp);
    rs = *reinterpret_cast<const floatx4*>(rn + 16 * tl + 4 * g);
  };

  // the first tiles' loads go out before anything else
  floatx4 av[P][4], acc[P], rs[P];
#pragma unroll
  for (int i = 0; i < P - 1; ++i) {
    const int tl = t_begin + ph + i * NPH;
    if (tl < t_end) load_tile(tl, av[i], acc[i], rs[i]);
  }

  // query operands of query tile qt: experts 16s + 4g .. +3 of query 16qt + c
  const int b = 16 * qt + c;
  floatx4 bq[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
    const int e0 = 16 * s + 4 * g;
    if (s < nq4 && b < a.Bc) {
      const int64_t k = static_cast<int64_t>(b) * a.E + e0;
      if (!BF && a.E % 4 == 0 && e0 < a.E) {
        v = *reinterpret_cast<const floatx4*>(static_cast<const float*>(a.q) + k);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (e0 + j < a.E)
            v[j] = BF ? bf16_to_f32(static_cast<const uint16_t*>(a.q)[k + j]) : static_cast<const float*>(a.q)[k + j];
        }
      }
    }
    bq[s] = v;
  }
  // 1/|q[0:p]|: the previous layers' float64 sum of squares plus this
  // layer's (lane partials, then across the 4 lane groups of a query)
  double* qsq = reinterpret_cast<double*>(a.state + 256);
  double sq = 0.0;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < 4; ++j) sq += static_cast<double>(bq[s][j]) * static_cast<double>(bq[s][j]);
  sq += __shfl_xor(sq, 16, kWave);
  sq += __shfl_xor(sq, 32, kWave);
  const double tot = (a.layer == 0 ? 0.0 : qsq[((a.layer - 1) & 1) * kStepQ + b]) + sq;
  if (blockIdx.x == 0 && ph == 0 && g == 0) qsq[(a.layer & 1) * kStepQ + b] = tot;
  float rq;
  if (tot != tot) rq = __uint_as_float(0x7fc00000u);
  else if (tot == 0.0) rq = 0.0f;
  else rq = static_cast<float>(1.0 / sqrt(tot));
  if (blockIdx.x == 0 && tid == 0) {
    StepHeader* h = reinterpret_cast<StepHeader*>(a.state);
    if (a.layer == 0) {
      h->n_begin = a.n;
    } else if (h->n_begin != a.n || h->last_layer != a.layer - 1) {
      atomicOr(a.flags, static_cast<uint32_t>(FM_FLAG_STATE_STALE));
    }
    h->last_layer = a.layer;
  }

  TopK<KTOP> best;
  best.clear();
  const bool live_q = b < a.Bc;
  int i = 0;
  for (int tl = t_begin + ph; tl < t_end; tl += NPH, ++i) {
    // buffer i % P holds tile tl; issue the loads of tile tl + (P-1) NPH
    const int nxt = tl + (P - 1) * NPH;
#pragma unroll
    for (int u = 0; u < P; ++u) {
      if (u != (i + P - 1) % P) continue;
      if (nxt < t_end) load_tile(nxt, av[u], acc[u], rs[u]);
    }
#pragma unroll
    for (int u = 0; u < P; ++u) {
      if (u != i % P) continue;
      floatx4 d = acc[u];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s >= nq4) break;
#pragma unroll
        for (int j = 0; j < 4; ++j) d = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u][s][j], bq[s][j], d, 0, 0, 0);
      }
      *reinterpret_cast<floatx4*>(dots + (static_cast<int64_t>(tl) * 4 + qt) * 256 + lane * 4) = d;
      if (live_q) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int y = 16 * tl + 4 * g + k;
          if (y < a.n) best.push(make_key(d[k] * rq * rs[u][k], y));
        }
      }
    }
  }

  // merge the 4 lane groups, then the phases of each query tile
#pragma unroll
  for (int m = 16; m <= 32; m <<= 1) {
    uint64_t o[KTOP];
#pragma unroll
    for (int jj = 0; jj < KTOP; ++jj) o[jj] = shfl_xor_u64(best.v[jj], m);
    best.merge(o);
  }
  if (g == 0) {
#pragma unroll
    for (int jj = 0; jj < KTOP; ++jj) mbuf[w][c][jj] = best.v[jj];
  }
  __syncthreads();
  if (tid < 16 * TQ) {
    const int r = tid;
    const int rqt = r / 16;
    if (r < a.Bc) {
      TopK<KTOP> m;
      m.clear();
#pragma unroll
      for (int p2 = 0; p2 < NPH; ++p2) m.merge(mbuf[p2 * TQ + rqt][r % 16]);
      uint64_t* out = a.partial + (static_cast<int64_t>(r) * a.R + blockIdx.x) * KTOP;
#pragma unroll
      for (int jj = 0; jj < KTOP; ++jj) out[jj] = m.v[jj];
    }
  }
}

namespace {

size_t chunk_state_bytes(int32_t cap) {
  return kStepHead + static_cast<size_t>(round16(cap) / 16) * 4 * 256 * sizeof(float);
}

template <bool BF, int KTOP>
void launch_step_tq(int TQ, const StepArgs& a, hipStream_t st) {
  if (TQ == 1) hipLaunchKernelGGL((k_traj_step<BF, 1, KTOP>), dim3(a.R), dim3(kStepThreads), 0, st, a);
  else if (TQ == 2) hipLaunchKernelGGL((k_traj_step<BF, 2, KTOP>), dim3(a.R), dim3(kStepThreads), 0, st, a);
  else hipLaunchKernelGGL((k_traj_step<BF, 4, KTOP>), dim3(a.R), dim3(kStepThreads), 0, st, a);
}

// The step kernel launch, bracketed by the caller's measurement events when
// set (fm_debug_scan_events).
template <bool BF>
hipError_t launch_step(int KTOP, int TQ, const StepArgs& a, hipStream_t st) {
  const ScanEvents& ev = scan_events();
  if (ev.start != nullptr) {
    const hipError_t err = hipEventRecord(ev.start, st);
    if (err != hipSuccess) return err;
  }
  if (KTOP == 1) launch_step_tq<BF, 1>(TQ, a, st);
  else if (KTOP == 4) launch_step_tq<BF, 4>(TQ, a, st);
  else launch_step_tq<BF, 8>(TQ, a, st);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess || ev.stop == nullptr) return err;
  return hipEventRecord(ev.stop, st);
}

}  // namespace

size_t traj_state_bytes(int32_t cap, int32_t B_max) {
  const size_t chunks = static_cast<size_t>((B_max + kStepQ - 1) / kStepQ);
  return chunks * align_up(chunk_state_bytes(cap), kAlign);
}

hipError_t launch_traj_step(const StoreView& s, void* state, const void* q, int32_t layer, int32_t B, int32_t k,
                            int32_t* idx_out, float* score_out, const Workspace& ws, hipStream_t st) {
  const bool bf = s.map_dtype == FM_BF16;
  const int esz = bf ? 2 : 4;
  const int KTOP = k == 1 ? 1 : (k <= 4 ? 4 : 8);
  const int n_tiles = static_cast<int>((s.n + 15) / 16);
  const size_t cbytes = align_up(chunk_state_bytes(s.cap), kAlign);
  for (int b0 = 0; b0 < B; b0 += kStepQ) {
    const int Bc = B - b0 < kStepQ ? B - b0 : kStepQ;
    char* cs = static_cast<char*>(state) + static_cast<size_t>(b0 / kStepQ) * cbytes;
    const void* qc = static_cast<const char*>(q) + static_cast<int64_t>(b0) * s.E * esz;
    StepArgs a;
    a.planes = s.planes;
    a.plane_elems = s.plane_elems;
    a.rnorm = s.rnorm;
    a.rn_stride = s.rn_stride;
    a.n = s.n;
    a.E = s.E;
    a.row = s.row;
    a.layer = layer;
    a.Bc = Bc;
    a.n_tiles = n_tiles;
    // about 8 tiles per workgroup (an empty store still launches one
    // workgroup: it advances the query norms and the header)
    int R = (n_tiles + 7) / 8;
    if (R > kStepMaxR) R = kStepMaxR;
    if (R < 1) R = 1;
    a.R = R;
    a.q = qc;
    a.state = cs;
    a.partial = ws.partial;
    a.flags = s.flags;
    const int TQ = Bc <= 16 ? 1 : (Bc <= 32 ? 2 : 4);
    hipError_t err = bf ? launch_step<true>(KTOP, TQ, a, st) : launch_step<false>(KTOP, TQ, a, st);
    if (err != hipSuccess) return err;
    err = launch_finalize(ws.partial, nullptr, Bc, a.R, k, KTOP, idx_out + static_cast<int64_t>(b0) * k,
                          score_out + static_cast<int64_t>(b0) * k, st);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace fm
