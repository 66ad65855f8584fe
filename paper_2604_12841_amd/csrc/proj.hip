// proj.hip -- the 1x1x1 projection shortcut of a residual block (Model 6,
// Sec. VI, Fig. Model8Representation): y[p][co] = bf16(b[co] + sum_ci
// w[co][ci] x[p][ci]) for every interior voxel p of the zero-halo layout,
// an fp32 FMA chain in channel order (the same chain the second conv's
// epilogue runs when it projects a block input of a few channels itself).  HBM-bound and small next to the block's two
// convolutions: one thread per (voxel, 4 output channels), reading the
// voxel's c_in bf16 inputs (16 bytes at a time when c_in is a multiple of 8)
// and the (L1-resident) weights.
#include "activation.h"
#include "internal.h"

namespace pd {
namespace {

__global__ void __launch_bounds__(256) proj_kernel(Geom g, const uint16_t* __restrict__ x, int cin, int xstride,
                                                   const float* __restrict__ w, const float* __restrict__ b, int cout,
                                                   uint16_t* __restrict__ y, int ystride, int batch) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int groups = cout / 4;
  if (gid >= (long long)batch * g.V * groups) return;
  const long long vox = gid / groups;
  const int c0 = (int)(gid - vox * groups) * 4;
  const int bb = (int)(vox / g.V);
  const int v = (int)(vox - (long long)bb * g.V);
  const int HH = g.H * g.H;
  const int t = v / HH, s = v - t * HH;
  const int i = s / g.H, j = s - i * g.H;
  const long long p = padded_index(g, bb, t, i, j);
  const uint16_t* xr = x + p * xstride;
  float acc[4] = {b[c0], b[c0 + 1], b[c0 + 2], b[c0 + 3]};
  auto add = [&](int ci, float xv) {
#pragma unroll
    for (int o = 0; o < 4; ++o) acc[o] = __builtin_fmaf(w[(long long)(c0 + o) * cin + ci], xv, acc[o]);
  };
  if (cin % 8 == 0) {
    for (int ci = 0; ci < cin; ci += 8) {
      const uint4 q = *reinterpret_cast<const uint4*>(xr + ci);
      const uint32_t qw[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        add(ci + 2 * e, __uint_as_float(qw[e] << 16));
        add(ci + 2 * e + 1, __uint_as_float(qw[e] & 0xFFFF0000u));
      }
    }
  } else {
    for (int ci = 0; ci < cin; ++ci) add(ci, __uint_as_float((uint32_t)xr[ci] << 16));
  }
  uint2 out;
  out.x = bf16_pack(acc[0], acc[1]);
  out.y = bf16_pack(acc[2], acc[3]);
  *reinterpret_cast<uint2*>(y + p * ystride + c0) = out;
}

}  // namespace

hipError_t launch_proj(const Geom& g, const void* x, int cin, int xstride, const float* w, const float* b, int cout,
                       void* y, int ystride, int batch, hipStream_t stream) {
  if (cout % 4 != 0 || cin < 1 || (cin % 8 == 0 && xstride % 8 != 0) || (ystride % 4) != 0) return hipErrorInvalidValue;
  const long long total = (long long)batch * g.V * (cout / 4);
  hipLaunchKernelGGL(proj_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, g,
                     (const uint16_t*)x, cin, xstride, w, b, cout, (uint16_t*)y, ystride, batch);
  return hipGetLastError();
}

}  // namespace pd
