// Store residency: new iterations enter the Expert Map Store (Step 5 of
// Section 3.2).  Maps arrive map-major [n][L][E] and are transposed into
// layer-major planes [L][cap][E], so a scan over the first p layers reads p
// contiguous planes.  Embeddings are copied row by row and their norms are
// computed once here (float64 sum of squares, rounded to float32), so the
// semantic scan (Eq. 4) never recomputes them.
#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

template <typename T>
__global__ void __launch_bounds__(256) k_insert_maps(const T* __restrict__ src, T* __restrict__ planes,
                                                     int64_t plane_elems, int32_t first_slot, int32_t n_new,
                                                     int32_t L, int32_t E, int32_t* __restrict__ slots_out) {
  // One thread per element of the map-major input (coalesced reads).
  const int64_t total = static_cast<int64_t>(n_new) * L * E;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < total; t += stride) {
    const int64_t row = t / E;            // (i, l)
    const int32_t e = static_cast<int32_t>(t - row * E);
    const int32_t i = static_cast<int32_t>(row / L);
    const int32_t l = static_cast<int32_t>(row - static_cast<int64_t>(i) * L);
    planes[l * plane_elems + static_cast<int64_t>(first_slot + i) * E + e] = src[t];
    if (slots_out != nullptr && l == 0 && e == 0) slots_out[i] = first_slot + i;
  }
}

// One wavefront per embedding row: copy it and compute its norm.
__global__ void __launch_bounds__(256) k_insert_embs(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                                     float* __restrict__ norms, int32_t first_slot, int32_t n_new,
                                                     int32_t d) {
  const int lane = threadIdx.x % kWave;
  const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (row >= n_new) return;
  const uint16_t* s = src + static_cast<int64_t>(row) * d;
  uint16_t* o = dst + static_cast<int64_t>(first_slot + row) * d;
  double acc = 0.0;
  for (int j = lane; j < d; j += kWave) {
    uint16_t h = s[j];
    o[j] = h;
    double v = static_cast<double>(bf16_to_f32(h));
    acc += v * v;
  }
  // Fixed-order tree reduction across the wave.
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
  if (lane == 0) norms[first_slot + row] = static_cast<float>(sqrt(acc));
}

hipError_t launch_insert(const StoreView& s, const void* maps, const void* embs, int32_t n_new,
                         int32_t* slots_out, hipStream_t st) {
  if (n_new <= 0) return hipSuccess;
  const int64_t total = static_cast<int64_t>(n_new) * s.L * s.E;
  int64_t blocks64 = (total + 255) / 256;
  const int blocks = static_cast<int>(blocks64 > 65536 ? 65536 : blocks64);
  if (s.map_dtype == FM_F32) {
    hipLaunchKernelGGL(k_insert_maps<float>, dim3(blocks), dim3(256), 0, st, static_cast<const float*>(maps),
                       static_cast<float*>(s.planes), s.plane_elems, s.n, n_new, s.L, s.E, slots_out);
  } else {
    hipLaunchKernelGGL(k_insert_maps<uint16_t>, dim3(blocks), dim3(256), 0, st,
                       static_cast<const uint16_t*>(maps), static_cast<uint16_t*>(s.planes), s.plane_elems, s.n,
                       n_new, s.L, s.E, slots_out);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (s.d_emb > 0) {
    const int rows_per_block = 256 / kWave;
    hipLaunchKernelGGL(k_insert_embs, dim3((n_new + rows_per_block - 1) / rows_per_block), dim3(256), 0, st,
                       static_cast<const uint16_t*>(embs), s.embs, s.emb_norm, s.n, n_new, s.d_emb);
    err = hipGetLastError();
  }
  return err;
}

}  // namespace fm
