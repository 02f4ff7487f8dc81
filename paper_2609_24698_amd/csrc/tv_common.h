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

// FP8 E4M3 (OCP "fn": sign, 4 exponent bits with bias 7, 3 mantissa bits;
// largest finite 448) indexer keys.
//
// Code -> bfloat16 bits, exactly: a normal code (exponent field e > 0) is
// 2^(e-7) (1 + m/8), whose bfloat16 exponent field is e + 120 and mantissa
// m << 4; a subnormal code is m 2^-9, exactly representable in float32.  The
// NaN codes (0x7F, 0xFF) give a bfloat16 NaN.
__device__ __forceinline__ uint32_t e4m3_to_bf16(uint32_t c) {
  const uint32_t em = c & 0x7Fu;
  const uint32_t mag = em >= 8u ? (em == 0x7Fu ? 0x7FC0u : (em << 4) + 0x3C00u)
                                : (__float_as_uint((float)em * 0x1p-9f) >> 16);
  return mag | ((c & 0x80u) << 8);
}
// Eight codes (bytes of w, low byte first) -> eight bfloat16 values, by the
// hardware pair conversion (v_cvt_pk_f32_fp8, which on gfx950 decodes OCP
// E4M3 exactly, NaN codes to NaN: checked against every code) and an exact
// narrowing of the float32 pairs.
typedef __attribute__((ext_vector_type(2))) float tv_f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 tv_bf16x2;
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_to_bf16x2(uint32_t w) {
  const tv_f32x2 f = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, HI);
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, tv_bf16x2));
}
__device__ __forceinline__ uint4 e4m3x8_to_bf16x8(uint2 w) {
  uint4 r;
  r.x = e4m3x2_to_bf16x2<false>(w.x);
  r.y = e4m3x2_to_bf16x2<true>(w.x);
  r.z = e4m3x2_to_bf16x2<false>(w.y);
  r.w = e4m3x2_to_bf16x2<true>(w.y);
  return r;
}
// float32 -> E4M3 code, one rounding to nearest with ties to even; magnitudes
// of 464 (the tie between 448 and the unrepresentable 480) and beyond
// saturate to +-448.  Below 2^-6 the results are multiples of 2^-9 (scaling
// by 512 is exact, rint rounds half to even; 8 of them is 2^-6, code 0x08);
// above, the float32 significand keeps its top 3 bits, rounded half to even
// on the 20 discarded ones (a carry moves into the exponent).
__device__ __forceinline__ uint32_t f32_to_e4m3(float f) {
  const uint32_t sign = (__float_as_uint(f) >> 24) & 0x80u;
  const float a = fabsf(f);
  if (!(a < 464.0f)) return sign | 0x7Eu;
  if (a < 0x1p-6f) return sign | (uint32_t)__builtin_rintf(a * 512.0f);
  const uint32_t u = __float_as_uint(a);
  const uint32_t r = (u + 0x7FFFFu + ((u >> 20) & 1u)) & ~0xFFFFFu;
  return sign | ((((r >> 23) - 120u) << 3) | ((r >> 20) & 7u));
}
// A bfloat16 value that is an E4M3 value (an FP8 key held in scratch) -> its code.
__device__ __forceinline__ uint32_t bf16_to_e4m3(uint16_t b) { return f32_to_e4m3(bf2f(b)); }

// Row of the current launch may run: device-side validity shared by every
// kernel after the mask (status still OK and 0 <= len <= max_len).
__device__ __forceinline__ bool len_ok(int32_t L, int32_t max_len) { return L >= 0 && L <= max_len; }

// Position q's raw row in the ring of row b.
__device__ __forceinline__ const uint16_t *ring_row(const uint16_t *ring, int b, int ring_cap, int d_u, int64_t q) {
  return ring + ((int64_t)b * ring_cap + (q & (ring_cap - 1))) * d_u;
}

// Inclusive prefix sum over the 64 lanes of a wavefront (lane l gets the
// sum over lanes 0..l), from DPP row shifts (a Hillis-Steele scan inside
// each 16-lane row) and two row broadcasts: no LDS-crossbar shuffles.  Every
// lane of the wavefront must be active.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15 -> rows 1, 3
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31 -> rows 2, 3
  return x;
}
// Sum over the wavefront's 64 lanes, the same value in every lane.
__device__ __forceinline__ uint32_t wave_total(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_prefix_sum(x), 63);
}

// Maximum (minimum) over the wavefront's 64 lanes, the same value in every
// lane: a running maximum by the same DPP steps, where a lane without a
// source keeps its own value.  Every lane must be active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x111, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x112, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x114, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x118, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x142, 0xa, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x143, 0xc, 0xf, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}
__device__ __forceinline__ int wave_min_i32(int x) {
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x111, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x112, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x114, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x118, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x142, 0xa, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x143, 0xc, 0xf, false));
  return __builtin_amdgcn_readlane(x, 63);
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
