// peak.hip -- measurement aids: the ceilings the roofline fractions of the
// conv kernels and of the bit-moving stages are quoted against, measured on
// the device at hand next to the published ones.
//
//   predecoder_peak_mfma: back-to-back matrix instructions on register
//     operands read once from a small device buffer (all zero, or random,
//     which draws more power and lowers the sustained clock): the bf16
//     instruction of the conv kernels (v_mfma_f32_32x32x16_bf16) or the fp8
//     one (32x32x64, E4M3 operands), four independent accumulators per wave so
//     that the instruction's latency is covered, four waves per workgroup.
//   predecoder_peak_copy: a plain device copy, 16 bytes per lane, one lane
//     per granule (HBM read + write bandwidth).
#include <hip/hip_runtime.h>

#include "../../include/predecoder.h"
#include "internal.h"

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) int i32x8;

template <bool F8>
__global__ void __launch_bounds__(256) mfma_peak_kernel(const uint4* __restrict__ operands, float* __restrict__ out,
                                                        int iters) {
  const int lane = threadIdx.x & 63;
  // lane l: A operand bytes [64 l, 64 l + 32), B operand [64 l + 32, 64 l + 64)
  const uint4 a0 = operands[4 * lane], a1 = operands[4 * lane + 1];
  const uint4 b0 = operands[4 * lane + 2], b1 = operands[4 * lane + 3];
  f32x16 acc[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[k][e] = 0.0f;
  if constexpr (F8) {
    const i32x8 a = {(int)a0.x, (int)a0.y, (int)a0.z, (int)a0.w, (int)a1.x, (int)a1.y, (int)a1.z, (int)a1.w};
    const i32x8 b = {(int)b0.x, (int)b0.y, (int)b0.z, (int)b0.w, (int)b1.x, (int)b1.y, (int)b1.z, (int)b1.w};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        acc[k] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[k], 0, 0, 0, 0, 0, 0);
    }
  } else {
    const bf16x8 a = __builtin_bit_cast(bf16x8, a0);
    const bf16x8 b = __builtin_bit_cast(bf16x8, b0);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[k][e];
  out[(long long)blockIdx.x * blockDim.x + threadIdx.x] = s;  // keeps every instruction live
}

__global__ void __launch_bounds__(256) copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                   long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

}  // namespace

extern "C" {

pd_status predecoder_peak_mfma(void* hip_stream, int32_t dtype, const void* operands, int32_t iters,
                               int32_t n_workgroups, float* out) {
  if (!operands || !out || iters < 1 || n_workgroups < 1) return PD_ERR_INVALID_ARG;
  if (dtype != PD_DTYPE_BF16 && dtype != PD_DTYPE_FP8) return PD_ERR_INVALID_ARG;
  const hipStream_t st = (hipStream_t)hip_stream;
  if (dtype == PD_DTYPE_FP8)
    hipLaunchKernelGGL(mfma_peak_kernel<true>, dim3((unsigned)n_workgroups), dim3(256), 0, st,
                       (const uint4*)operands, out, iters);
  else
    hipLaunchKernelGGL(mfma_peak_kernel<false>, dim3((unsigned)n_workgroups), dim3(256), 0, st,
                       (const uint4*)operands, out, iters);
  if (hipGetLastError() != hipSuccess) return PD_ERR_DEVICE;
  return PD_OK;
}

pd_status predecoder_peak_copy(void* hip_stream, const void* src, void* dst, size_t bytes) {
  if (!src || !dst || bytes == 0 || bytes % 16 != 0) return PD_ERR_INVALID_ARG;
  const long long n = (long long)(bytes / 16);
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)hip_stream,
                     (const uint4*)src, (uint4*)dst, n);
  if (hipGetLastError() != hipSuccess) return PD_ERR_DEVICE;
  return PD_OK;
}

}  // extern "C"
