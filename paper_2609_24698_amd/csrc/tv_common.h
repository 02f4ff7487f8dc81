// Device helpers shared by the gfx950 kernels of the tree-verify library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tv.h"

namespace tv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// bfloat16 bits <-> float32.
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
__device__ __forceinline__ float bf2f_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf2f_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// float32 -> bfloat16 bits, round to nearest, ties to even (NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

// Row of the current launch may run: device-side validity shared by every
// kernel after the mask (status still OK and 0 <= len <= max_len).
__device__ __forceinline__ bool len_ok(int32_t L, int32_t max_len) { return L >= 0 && L <= max_len; }

// Position q's raw row in the ring of row b.
__device__ __forceinline__ const uint16_t *ring_row(const uint16_t *ring, int b, int ring_cap, int d_u, int64_t q) {
  return ring + ((int64_t)b * ring_cap + (q & (ring_cap - 1))) * d_u;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sortable key of a float score: larger score -> larger key; -0 and +0 equal.
__device__ __forceinline__ uint32_t score_key(float s) {
  if (s == 0.0f) s = 0.0f;
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace tv
