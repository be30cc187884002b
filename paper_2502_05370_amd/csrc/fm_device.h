// Device helpers shared by the kernels of libfinemoe_map (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fm {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));

typedef uint32_t uint32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t uint32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void* lds_vp;
typedef __attribute__((address_space(1))) void* gbl_vp;

constexpr int kWave = 64;

// Fourth word of a raw buffer descriptor (32-bit data format, no swizzle), and
// a byte offset beyond every descriptor's range: loads there return zeros
// without touching memory.
constexpr int kBufWord3 = 0x00020000;
constexpr uint32_t kOutside = 0xFFFFF000u;

// Raw s_waitcnt bounding only the vector-memory counter (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_lgkm0() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));
  asm volatile("" ::: "memory");
}
// Workgroup barrier without the implicit release/acquire fence (which would
// wait for every outstanding global->LDS load); callers wait explicitly.
__device__ __forceinline__ void raw_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16 bytes per lane from src into LDS at lds_base + 16 * lane.
__device__ __forceinline__ void dma16(const void* src, void* lds_base) {
  __builtin_amdgcn_global_load_lds((gbl_vp)(const_cast<void*>(src)), (lds_vp)(lds_base), 16, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_bf16(const u16x8& a, const u16x8& b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f16(const u16x8& a, const u16x8& b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a), __builtin_bit_cast(halfx8, b), c, 0, 0,
                                                0);
}

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
  // Merge another list sorted descending; keeps the K largest.  Bitonic:
  // the elementwise maximum of this list and the other one reversed holds
  // the K largest of both as a bitonic sequence, which a half-cleaner
  // network then sorts.
  __device__ __forceinline__ void merge(const uint64_t* o) {
    if constexpr (K == 1) {
      v[0] = o[0] > v[0] ? o[0] : v[0];
    } else {
#pragma unroll
      for (int j = 0; j < K; ++j) v[j] = o[K - 1 - j] > v[j] ? o[K - 1 - j] : v[j];
#pragma unroll
      for (int st = K / 2; st >= 1; st /= 2) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
          if ((j & st) == 0) {
            const uint64_t hi = v[j] > v[j + st] ? v[j] : v[j + st];
            const uint64_t lo = v[j] > v[j + st] ? v[j + st] : v[j];
            v[j] = hi;
            v[j + st] = lo;
          }
        }
      }
    }
  }
};

// Sort 8 keys descending in place (19-comparator network).
__device__ __forceinline__ void sort8_desc(uint64_t* x) {
  constexpr int kNet[19][2] = {{0, 2}, {1, 3}, {4, 6}, {5, 7}, {0, 4}, {1, 5}, {2, 6}, {3, 7}, {0, 1}, {2, 3},
                               {4, 5}, {6, 7}, {2, 4}, {3, 5}, {1, 4}, {3, 6}, {1, 2}, {3, 4}, {5, 6}};
#pragma unroll
  for (int c = 0; c < 19; ++c) {
    const int i = kNet[c][0], j = kNet[c][1];
    const uint64_t hi = x[i] > x[j] ? x[i] : x[j];
    const uint64_t lo = x[i] > x[j] ? x[j] : x[i];
    x[i] = hi;
    x[j] = lo;
  }
}


}  // namespace fm
