// Device helpers shared by the kernels of libfinemoe_map (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fm {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// Score used inside the scans for a NaN cosine: below every real cosine
// (which lies in [-1, 1] up to rounding) and above the empty sentinel.
constexpr float kNanScore = -2.0f;
constexpr float kEmptyScore = -3.0f;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Order-preserving map from float to uint32: larger float -> larger key.
// NaN (and the in-scan NaN sentinel) maps to 0, the lowest key.
__device__ __forceinline__ uint32_t ord_score(float s) {
  if (s != s || s == kNanScore) return 0u;
  s = s + 0.0f;  // -0 -> +0, so equal scores compare equal
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float unord_score(uint32_t o) {
  if (o == 0u) return __uint_as_float(0x7fc00000u);
  uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  return __uint_as_float(u);
}

// Packed ranking key: larger key = better match.  Score order first, then
// the lower store index.  Key 0 means "no match".
__device__ __forceinline__ uint64_t make_key(float s, int32_t idx) {
  return (static_cast<uint64_t>(ord_score(s)) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(idx));
}
__device__ __forceinline__ int32_t key_index(uint64_t key) {
  return key == 0 ? -1 : static_cast<int32_t>(~static_cast<uint32_t>(key));
}
__device__ __forceinline__ float key_score(uint64_t key) {
  return key == 0 ? -__builtin_inff() : unord_score(static_cast<uint32_t>(key >> 32));
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, kWave);
  uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, kWave);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Top-K list in registers, sorted descending, of packed keys.
template <int K>
struct TopK {
  uint64_t v[K];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int j = 0; j < K; ++j) v[j] = 0;
  }
  // Insert key x (keys are distinct).
  __device__ __forceinline__ void push(uint64_t x) {
    if (x <= v[K - 1]) return;
    uint64_t nv[K];
    nv[0] = x > v[0] ? x : v[0];
#pragma unroll
    for (int j = 1; j < K; ++j) nv[j] = x > v[j - 1] ? v[j - 1] : (x > v[j] ? x : v[j]);
#pragma unroll
    for (int j = 0; j < K; ++j) v[j] = nv[j];
  }
  // Merge another sorted list; keeps the K largest.
  __device__ __forceinline__ void merge(const uint64_t* o) {
#pragma unroll
    for (int j = 0; j < K; ++j) push(o[j]);
  }
};

// Insert a descending list of candidate keys into a global top-k list
// (k slots, descending, 0 = empty) shared by all workgroups.  Each slot only
// grows; a displaced key moves on to the next slot.  The final contents are
// the k largest keys ever offered, whatever the arrival order.
template <int KTOP>
__device__ __forceinline__ void global_topk_insert(uint64_t* slots, int k, const uint64_t (&cand)[KTOP]) {
#pragma unroll
  for (int c = 0; c < KTOP; ++c) {
    if (c >= k) return;
    uint64_t carry = cand[c];
    if (carry == 0) return;
    const uint64_t last = __hip_atomic_load(slots + (k - 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (carry <= last) return;  // the list is descending: later candidates are smaller still
    for (int j = 0; j < k && carry != 0; ++j) {
      const uint64_t old = __hip_atomic_fetch_max(slots + j, carry, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      carry = old < carry ? old : carry;
    }
  }
}

}  // namespace fm
