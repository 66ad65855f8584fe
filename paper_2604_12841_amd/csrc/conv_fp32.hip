// conv_fp32.hip -- one 3x3x3 conv3d layer in fp32 end to end (the fp32
// workload: d = 5, 32 hidden channels).  Same zero-halo NTHWC layout as the
// bf16 path, so every tap is an index shift.  Each thread computes 8 output
// channels of one voxel with fp32 FMAs; weights are [tap][c_in][c_out] fp32.
// The fp32 workload is ~2 GFLOP per batch, far below any roofline that
// matters here; this kernel exists for exact fp32 semantics, not speed.
#include "internal.h"

namespace pd {

__device__ __forceinline__ float activation_f32(float y, int act) {
  if (act == 1) {  // GELU, tanh form: y / (1 + exp(-2u)), u = sqrt(2/pi)(y + 0.044715 y^3)
    const float k0 = 0.7978845608028654f;
    const float kl = -2.0f * 1.4426950408889634f;
    float u = k0 * (y + 0.044715f * y * y * y);
    float e = __builtin_amdgcn_exp2f(kl * u);
    return y / (1.0f + e);
  }
  if (act == 2) return y > 0.0f ? y : 0.0f;
  return y;
}

__global__ void __launch_bounds__(256) conv_fp32_kernel(Geom g, int cin, int cout, int act,
                                                        const float* __restrict__ x,
                                                        float* __restrict__ y,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias, int batch) {
  const int ngroups = cout / 8;
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long total = (long long)batch * g.V * ngroups;
  if (gid >= total) return;
  const int grp = (int)(gid % ngroups);
  const long long vox = gid / ngroups;
  const int b = (int)(vox / g.V);
  const int v = (int)(vox - (long long)b * g.V);
  const int HH = g.H * g.H;
  const int t = v / HH, s = v - t * HH;
  const int i = s / g.H, j = s - i * g.H;
  const long long p = padded_index(g, b, t, i, j);
  const int co0 = grp * 8;
  float acc[8];
#pragma unroll
  for (int o = 0; o < 8; ++o) acc[o] = bias[co0 + o];
  for (int tap = 0; tap < 27; ++tap) {
    const int dt = tap / 9, di = (tap / 3) % 3, dj = tap % 3;
    const long long q = p + (long long)(dt - 1) * g.P + (long long)(di - 1) * g.Wp + (dj - 1);
    const float* xr = x + q * cin;
    const float* wr = w + (long long)tap * cin * cout + co0;
    for (int ci = 0; ci < cin; ++ci) {
      const float xv = xr[ci];
#pragma unroll
      for (int o = 0; o < 8; ++o) acc[o] = fmaf(xv, wr[(long long)ci * cout + o], acc[o]);
    }
  }
  float* yr = y + p * cout + co0;
#pragma unroll
  for (int o = 0; o < 8; ++o) yr[o] = activation_f32(acc[o], act);
}

hipError_t launch_conv_fp32(const Geom& g, int cin, int cout, int act, const float* x, float* y,
                            const float* w, const float* bias, int batch, hipStream_t stream) {
  long long total = (long long)batch * g.V * (cout / 8);
  unsigned grid = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(conv_fp32_kernel, dim3(grid), dim3(256), 0, stream, g, cin, cout, act, x, y, w,
                     bias, batch);
  return hipGetLastError();
}

}  // namespace pd
