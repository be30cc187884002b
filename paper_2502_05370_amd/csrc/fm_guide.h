// Guiding probabilities of a query's matched map(s), shared by the
// selection (Section 4.3, Eq. 6-8) and the priority ordering (Section 4.5):
// the best match's stored row, or the similarity-weighted mean of the rows of
// the k matches (weights max(score, 0), the plain mean if all are 0), summed
// in match order with explicit float64 roundings.
#pragma once

#include "fm_device.h"
#include "fm_internal.h"

namespace fm {

struct GuideView {
  const void* planes;
  int64_t plane_elems;
  int32_t n, row;
  fm_dtype dtype;
};

__device__ __forceinline__ double stored_prob(const GuideView& v, int y, int l, int j) {
  const int64_t off = static_cast<int64_t>(l) * v.plane_elems + tile_offset(y, j, v.row);
  if (v.dtype == FM_F32) return static_cast<double>(static_cast<const float*>(v.planes)[off]);
  return static_cast<double>(bf16_to_f32(static_cast<const uint16_t*>(v.planes)[off]));
}

// p of expert j at layer l for one query: idx_b / score_b are its k matches
// in ranking order (idx_b[0] is a valid store index; -1 entries are skipped).
__device__ __forceinline__ double guide_prob(const GuideView& v, const int32_t* idx_b, const float* score_b, int k,
                                             int blend, int l, int j) {
  if (blend != FM_BLEND_SCORE) return stored_prob(v, idx_b[0], l, j);
  bool any_pos = false;
  for (int i = 0; i < k; ++i) {
    const int y = idx_b[i];
    if (y < 0 || y >= v.n) continue;
    if (static_cast<double>(score_b[i]) > 0.0) any_pos = true;
  }
  double num = 0.0, den = 0.0;
  for (int i = 0; i < k; ++i) {
    const int y = idx_b[i];
    if (y < 0 || y >= v.n) continue;
    const double s = static_cast<double>(score_b[i]);
    const double wgt = any_pos ? (s > 0.0 ? s : 0.0) : 1.0;
    num = __dadd_rn(num, __dmul_rn(wgt, stored_prob(v, y, l, j)));
    den = __dadd_rn(den, wgt);
  }
  return __ddiv_rn(num, den);
}

}  // namespace fm
