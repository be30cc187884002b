// Store residency: new iterations enter the Expert Map Store (Step 5 of
// Section 3.2).  Maps arrive map-major [n][L][E] and are transposed into
// layer-major planes of 16-map tiles (row = E rounded up to 4, zero padded;
// see tile_offset), so a scan over the first p layers reads p contiguous
// planes; the prefix inverse norms of every map at every depth are computed
// once here.  Embeddings are copied row by row and their norms are
// computed once here (float64 sum of squares, rounded to float32), so the
// semantic scan (Eq. 4) never recomputes them.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

// Slot of new iteration i: first_slot + i, or slot_of[i] when a slot array
// is given (deduplicating inserts; -1 means the iteration is dropped).
__device__ __forceinline__ int64_t slot_for(int32_t first_slot, const int32_t* slot_of, int i) {
  return slot_of != nullptr ? static_cast<int64_t>(slot_of[i]) : static_cast<int64_t>(first_slot) + i;
}

// One workgroup per new map; wave w handles layers w, w + 4, ... and lane e
// expert e of a layer row (row <= 64).  Every row is copied into its plane
// (with zeros in the row padding).  The float64 sum of squares of a layer is
// a fixed-order tree reduction across the wave; the running sum over layers
// 0..l, taken in layer order, gives the prefix inverse norm 1/|x[y][0:l+1]|
// that the trajectory scan (Eq. 5) divides by at depth l+1.
template <typename T>
__global__ void __launch_bounds__(256) k_insert_maps(const T* __restrict__ src, T* __restrict__ planes,
                                                     int64_t plane_elems, float* __restrict__ rnorm,
                                                     int64_t rn_stride, int32_t first_slot,
                                                     const int32_t* __restrict__ slot_of, int32_t n_new,
                                                     int32_t L, int32_t E, int32_t row,
                                                     int32_t* __restrict__ slots_out, uint32_t* __restrict__ flags) {
  constexpr int kLayersPerWave = kMaxL / 4;
  __shared__ double sq[kMaxL];
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int i = blockIdx.x;
  const int64_t y = slot_for(first_slot, slot_of, i);
  if (y < 0) return;
  // all loads first, then the stores and the per-layer reductions
  T v[kLayersPerWave];
#pragma unroll
  for (int j = 0; j < kLayersPerWave; ++j) {
    const int l = w + 4 * j;
    v[j] = T(0);
    if (l < L && lane < E) v[j] = src[(static_cast<int64_t>(i) * L + l) * E + lane];
  }
  // float32 maps: the trajectory scan's float16 split holds for magnitudes
  // up to 8; a larger (or infinite) value is flagged
  if constexpr (sizeof(T) == 4) {
    bool big = false;
#pragma unroll
    for (int j = 0; j < kLayersPerWave; ++j) big = big || __builtin_fabsf(v[j]) > 8.0f;
    if (__any(big) && lane == 0) atomicOr(flags, static_cast<uint32_t>(FM_FLAG_VALUE_RANGE));
  }
#pragma unroll
  for (int j = 0; j < kLayersPerWave; ++j) {
    const int l = w + 4 * j;
    if (l >= L) break;
    if (lane < row) planes[l * plane_elems + tile_offset(y, lane, row)] = v[j];
    double f;
    if constexpr (sizeof(T) == 2) f = static_cast<double>(bf16_to_f32(v[j]));
    else f = static_cast<double>(v[j]);
    double s2 = f * f;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s2 += __shfl_xor(s2, m, kWave);
    if (lane == 0) sq[l] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double cum = 0.0;
    for (int l = 0; l < L; ++l) {
      cum += sq[l];
      float r;
      if (cum != cum) r = __uint_as_float(0x7fc00000u);
      else if (cum == 0.0) r = 0.0f;
      else r = static_cast<float>(1.0 / sqrt(cum));
      rnorm[l * rn_stride + y] = r;
    }
    if (slots_out != nullptr) slots_out[i] = static_cast<int32_t>(y);
  }
}

// One workgroup per embedding row: copy it into the tiled layout
// (emb_offset, 8 consecutive dimensions per 16-byte store) and compute its
// norm (float64: each thread sums its chunks in order, then a fixed-order
// tree across the wave and the 4 waves in order).
__global__ void __launch_bounds__(256) k_insert_embs(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                                     float* __restrict__ norms, int32_t first_slot,
                                                     const int32_t* __restrict__ slot_of, int32_t n_new, int32_t d) {
  __shared__ double part[4];
  const int lane = threadIdx.x % kWave;
  const int w = threadIdx.x / kWave;
  const int row = blockIdx.x;
  const uint16_t* s = src + static_cast<int64_t>(row) * d;
  const int64_t y = slot_for(first_slot, slot_of, row);
  if (y < 0) return;
  double acc = 0.0;
  for (int j0 = 8 * static_cast<int>(threadIdx.x); j0 < d; j0 += 8 * 256) {
    const u16x8 h = *reinterpret_cast<const u16x8*>(s + j0);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const double v = static_cast<double>(bf16_to_f32(h[t]));
      acc += v * v;
    }
    *reinterpret_cast<u16x8*>(dst + emb_offset(y, j0, d)) = h;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
  if (lane == 0) part[w] = acc;
  __syncthreads();
  if (threadIdx.x == 0) norms[y] = static_cast<float>(sqrt(((part[0] + part[1]) + part[2]) + part[3]));
}

hipError_t launch_insert(const StoreView& s, const void* maps, const void* embs, int32_t n_new,
                         const int32_t* slot_of, int32_t* slots_out, hipStream_t st) {
  if (n_new <= 0) return hipSuccess;
  const dim3 grid(n_new);
  if (s.map_dtype == FM_F32) {
    hipLaunchKernelGGL(k_insert_maps<float>, grid, dim3(256), 0, st, static_cast<const float*>(maps),
                       static_cast<float*>(s.planes), s.plane_elems, s.rnorm, s.rn_stride, s.n, slot_of, n_new, s.L,
                       s.E, s.row, slots_out, s.flags);
  } else {
    hipLaunchKernelGGL(k_insert_maps<uint16_t>, grid, dim3(256), 0, st, static_cast<const uint16_t*>(maps),
                       static_cast<uint16_t*>(s.planes), s.plane_elems, s.rnorm, s.rn_stride, s.n, slot_of, n_new,
                       s.L, s.E, s.row, slots_out, s.flags);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (s.d_emb > 0) {
    hipLaunchKernelGGL(k_insert_embs, grid, dim3(256), 0, st, static_cast<const uint16_t*>(embs), s.embs,
                       s.emb_norm, s.n, slot_of, n_new, s.d_emb);
    err = hipGetLastError();
  }
  return err;
}

}  // namespace fm
