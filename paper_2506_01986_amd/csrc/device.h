// Device-side helpers for gfx950 (CDNA4): operand types for the bf16 matrix
// cores, bf16 <-> fp32 conversions, and the (value, id) order used by top-k and
// argmax.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specmemo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even; inputs are finite here.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair (round to nearest even; one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// Value of lane l combined with lane l^32 (the two halves of a wave hold the
// same rows).  v_permlane32_swap of x with itself leaves the low half of x in
// both halves of the first result and the high half in both halves of the
// second, so every lane combines (x of lane l mod 32, x of lane l mod 32 + 32)
// in that order.
__device__ __forceinline__ float max_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Maximum over the 64 lanes of a wave, in every lane, without LDS: DPP steps
// within each 16-lane row (swap adjacent lanes, then pairs, then the row's
// halves mirrored, then the row mirrored), then v_permlane16_swap (rows 0/1
// and 2/3) and v_permlane32_swap (the two halves).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));    // quad_perm [1, 0, 3, 2]
  v = fmaxf(v, dpp_f<0x4E>(v));    // quad_perm [2, 3, 0, 1]
  v = fmaxf(v, dpp_f<0x141>(v));   // row_half_mirror
  v = fmaxf(v, dpp_f<0x140>(v));   // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  return max_with_other_half(v);
}

// Unsigned maximum / minimum over the 64 lanes of a wave, in every lane (the
// same DPP / permlane steps as wave_max).
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v) {
  auto op = [](uint32_t x, uint32_t y) { return MAX ? (x > y ? x : y) : (x < y ? x : y); };
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));
  const auto r16 = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = op(r16[0], r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return op(r32[0], r32[1]);
}

// Larger value first; equal values by lower id.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib);

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xF, 0xF, false);
}

// Best (value, id) pair over the 64 lanes of a wave, in every lane: the same
// DPP / permlane steps as wave_max, moving both halves of the pair.
__device__ __forceinline__ void wave_argbest(float &v, int &id) {
  auto step = [&](float ov, int oi) {
    if (better(ov, oi, v, id)) {
      v = ov;
      id = oi;
    }
  };
  step(dpp_f<0xB1>(v), dpp_i<0xB1>(id));
  step(dpp_f<0x4E>(v), dpp_i<0x4E>(id));
  step(dpp_f<0x141>(v), dpp_i<0x141>(id));
  step(dpp_f<0x140>(v), dpp_i<0x140>(id));
  {
    const auto rv = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const auto ri = __builtin_amdgcn_permlane16_swap((uint32_t)id, (uint32_t)id, false, false);
    v = __uint_as_float(rv[0]);
    id = (int)ri[0];
    step(__uint_as_float(rv[1]), (int)ri[1]);
  }
  {
    const auto rv = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const auto ri = __builtin_amdgcn_permlane32_swap((uint32_t)id, (uint32_t)id, false, false);
    v = __uint_as_float(rv[0]);
    id = (int)ri[0];
    step(__uint_as_float(rv[1]), (int)ri[1]);
  }
}

// Larger value first; equal values by lower id.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// 16-byte load when `pred`, else zeros (a value select, never an address select).
__device__ __forceinline__ uint4 ld16_or_zero(bool pred, const void *p) {
  uint4 v = {0u, 0u, 0u, 0u};
  if (pred) v = *reinterpret_cast<const uint4 *>(p);
  return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace specmemo
