// activation.h -- the per-value epilogue arithmetic shared by the conv
// kernels: the activation (Sec. IV.B; the GELU in its tanh form, ReLU, or
// none), bf16 rounding (round to nearest even) and a dispatch that turns the
// runtime activation code into a compile-time one, so an epilogue is one
// straight-line body per activation instead of a branch per value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pd {

// Activation codes of the C ABI: 0 none, 1 GELU (tanh form), 2 ReLU.
template <int ACT>
__device__ __forceinline__ float act_fn(float y) {
  if constexpr (ACT == 1) {  // 0.5 y (1 + tanh(u)) = y / (1 + exp(-2u)), u = sqrt(2/pi) (y + 0.044715 y^3)
    const float k0 = 0.7978845608028654f;          // sqrt(2 / pi)
    const float kl = -2.0f * 1.4426950408889634f;  // -2 log2(e)
    const float u = k0 * (y + 0.044715f * y * y * y);
    const float e = __builtin_amdgcn_exp2f(kl * u);
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

__device__ __forceinline__ float bf16_round(float v) { return __uint_as_float(bf16_bits(v) << 16); }

}  // namespace pd
