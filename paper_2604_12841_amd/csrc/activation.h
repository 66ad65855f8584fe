// activation.h -- the per-value epilogue arithmetic shared by the conv
// kernels: the activation (Sec. IV.B; the GELU in its tanh form, ReLU, or
// none), bf16 rounding (round to nearest even) and a dispatch that turns the
// runtime activation code into a compile-time one, so an epilogue is one
// straight-line body per activation instead of a branch per value; and the
// OCP E4M3 conversions of the fp8 path (round to nearest even, magnitudes
// above 448 saturated to 448 before the conversion instruction, which would
// give NaN past the format's rounding range).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pd {

// Activation codes of the C ABI: 0 none, 1 GELU (tanh form), 2 ReLU.
// GELU: 0.5 y (1 + tanh(u)) = y / (1 + exp(-2u)) with
// u = sqrt(2/pi) (y + 0.044715 y^3), evaluated as
// y / (1 + exp2(y (c1 + c3 y^2))), c1 = -2 log2(e) sqrt(2/pi),
// c3 = 0.044715 c1 (three multiply-adds, one exp2, one reciprocal).
template <int ACT>
__device__ __forceinline__ float act_fn(float y) {
  if constexpr (ACT == 1) {
    constexpr float c1 = -2.0 * 1.4426950408889634 * 0.7978845608028654;
    constexpr float c3 = -2.0 * 1.4426950408889634 * 0.7978845608028654 * 0.044715;
    const float e = __builtin_amdgcn_exp2f(y * __builtin_fmaf(c3, y * y, c1));
    return y * __builtin_amdgcn_rcpf(1.0f + e);
  } else if constexpr (ACT == 2) {
    return y > 0.0f ? y : 0.0f;
  } else {
    return y;
  }
}

// Calls f(std::integral_constant<int, ACT>) for the runtime code act.
template <typename F>
__host__ __device__ inline void with_activation(int act, F&& f) {
  if (act == 1)
    f(std::integral_constant<int, 1>());
  else if (act == 2)
    f(std::integral_constant<int, 2>());
  else
    f(std::integral_constant<int, 0>());
}

__device__ __forceinline__ uint32_t bf16_bits(float v) {
  __bf16 h = (__bf16)v;
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Two values rounded to bf16 and packed, lo in bits 0-15 (one conversion
// instruction on gfx950).
__device__ __forceinline__ uint32_t bf16_pack(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) float f32x2_t;
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ float bf16_round(float v) { return __uint_as_float(bf16_bits(v) << 16); }

__device__ __forceinline__ float e4m3_clamp(float v) { return __builtin_fminf(__builtin_fmaxf(v, -448.0f), 448.0f); }

// Four values as E4M3 codes, v0 in bits 0-7 (two conversion instructions).
__device__ __forceinline__ uint32_t e4m3_pack4(float v0, float v1, float v2, float v3) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(v0), e4m3_clamp(v1), 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(v2), e4m3_clamp(v3), lo, true);
}

// v rounded to E4M3 and back.
__device__ __forceinline__ float e4m3_round(float v) {
  const int c = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(v), 0.0f, 0, false);
  return __builtin_amdgcn_cvt_f32_fp8(c, 0);
}

}  // namespace pd
