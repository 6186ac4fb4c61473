// Device-side helpers: bfloat16 conversion, storage access, wave reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asr_kernels.h"

namespace asr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }

// float32 -> bfloat16, round to nearest even (gfx950's v_cvt_pk_bf16_f32);
// NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
// Two values in one conversion: a in the low half, b in the high half.
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

template <typename T>
struct St;
template <>
struct St<float> {
  static __device__ __forceinline__ float ld(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void st(float* p, int64_t i, float v) { p[i] = v; }
  // four values at element i (i a multiple of 4, p 16-byte aligned)
  static __device__ __forceinline__ void st4(float* p, int64_t i, float4 v) {
    *(float4*)(p + i) = v;
  }
};
template <>
struct St<bf16_t> {
  static __device__ __forceinline__ float ld(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void st(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }
  // four values at element i (i a multiple of 4, p 8-byte aligned)
  static __device__ __forceinline__ void st4(bf16_t* p, int64_t i, float4 v) {
    *(uint2*)(p + i) = make_uint2(pack2_bf16(v.x, v.y), pack2_bf16(v.z, v.w));
  }
};

// GELU(x) = x Phi(x), Phi the standard normal CDF, with erf from
// Abramowitz & Stegun 7.1.26 (Hastings' rational approximation, |error| <=
// 1.5e-7 on the erf): for z = |x|/sqrt 2, 1 - erf(z) = t (a1 + t (a2 + ... +
// t a5)) e^{-z^2}, t = 1 / (1 + p z).  Its half is h = Phi(-|x|); GELU(x) is
// x - x h for x >= 0 and x h for x < 0, so the negative tail never subtracts
// nearly equal numbers.  The 1/sqrt 2 folds into p, the 1/2 into the a_i and
// e^{-z^2} = 2^(-x^2 log2(e) / 2): twelve VALU instructions and two
// transcendentals instead of a library erf; the error sits far below the
// bfloat16 rounding of the products that use it.
__device__ __forceinline__ float gelu_erf(float x) {
  const float t =
      __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, fabsf(x), 1.0f));
  float poly = fmaf(0.5f * 1.061405429f, t, 0.5f * -1.453152027f);
  poly = fmaf(poly, t, 0.5f * 1.421413741f);
  poly = fmaf(poly, t, 0.5f * -0.284496736f);
  poly = fmaf(poly, t, 0.5f * 0.254829592f);
  const float h = poly * t * __builtin_amdgcn_exp2f(x * x * (-0.5f * 1.4426950408889634f));
  const float xh = x * h;
  return x >= 0.0f ? x - xh : xh;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// The same sum without LDS round trips: DPP adds within each 16-lane row
// (quad swaps, half-row and row mirrors), then the gfx950 lane swaps
// v_permlane16_swap (rows 0<->1, 2<->3) and v_permlane32_swap (halves).
// Every lane ends with the total.
#define ASR_DPP_ADD(v, ctrl)                                                               \
  ((v) + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), (ctrl), 0xF, 0xF, \
                                                    true)))
__device__ __forceinline__ float wave_sum_lanes(float v) {
  v = ASR_DPP_ADD(v, 0xB1);    // quad_perm [1,0,3,2]
  v = ASR_DPP_ADD(v, 0x4E);    // quad_perm [2,3,0,1]
  v = ASR_DPP_ADD(v, 0x141);   // row_half_mirror
  v = ASR_DPP_ADD(v, 0x140);   // row_mirror
  const uint32_t u = __float_as_uint(v);
  const auto p16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __uint_as_float(p16[0]) + __uint_as_float(p16[1]);
  const uint32_t w = __float_as_uint(v);
  const auto p32 = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __uint_as_float(p32[0]) + __uint_as_float(p32[1]);
}
#undef ASR_DPP_ADD
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Total order on floats as unsigned integers (larger float -> larger key).
__device__ __forceinline__ uint32_t ordered_u32(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_ordered_u32(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

}  // namespace asr
