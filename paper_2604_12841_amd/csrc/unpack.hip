// unpack.hip -- K1: packed detector events -> 2-channel planes (Sec. IV.B.1:
// each detector event is placed at its stabilizer's grid site, X-type in
// channel 0 and Z-type in channel 1; every other grid location is 0).
//
// One thread per interior voxel (b, t, i, j); the thread reads the one bit it
// needs (the packed row of a sample is a few hundred bytes, so these reads hit
// L1/L2) and writes both channels with one 4-byte (bf16 pair) or 8-byte (fp32
// pair) store.  Consecutive threads write consecutive voxels of a grid row.
// HBM-bound: reads W_det * 8 bytes and writes 2 * V * sizeof(elem) bytes per
// sample.
#include "internal.h"

namespace pd {

template <bool FP32, bool PADDED>
__global__ void __launch_bounds__(256) unpack_kernel(Geom g, const int32_t* __restrict__ comp_of_site,
                                                     const uint64_t* __restrict__ det, int batch,
                                                     void* __restrict__ out) {
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long total = (long long)batch * g.V;
  if (gid >= total) return;
  int b = (int)(gid / g.V);
  int v = (int)(gid - (long long)b * g.V);
  int HH = g.H * g.H;
  int t = v / HH;
  int s = v - t * HH;
  int n = comp_of_site[s];
  unsigned bit = 0;
  if (n >= 0) {
    long long k = (long long)t * g.nstab + n;
    bit = (unsigned)((det[(long long)b * g.Wd + (k >> 6)] >> (k & 63)) & 1ull);
  }
  unsigned ch = (n >= g.K) ? 1u : 0u;  // X sites come first in the compact order
  long long o;
  if (PADDED) {
    int i = s / g.H, j = s - (s / g.H) * g.H;
    o = padded_index(g, b, t, i, j);
  } else {
    o = gid;
  }
  if (FP32) {
    float2 val;
    val.x = (bit && ch == 0) ? 1.0f : 0.0f;
    val.y = (bit && ch == 1) ? 1.0f : 0.0f;
    reinterpret_cast<float2*>(out)[o] = val;
  } else {
    uint32_t one = 0x3F80u;  // bf16 1.0
    uint32_t val = bit ? (one << (16 * ch)) : 0u;
    reinterpret_cast<uint32_t*>(out)[o] = val;
  }
}

hipError_t launch_unpack(const Geom& g, const int32_t* comp_of_site, const uint64_t* det, int batch,
                         void* out, int out_padded, int fp32, hipStream_t stream) {
  long long total = (long long)batch * g.V;
  unsigned grid = (unsigned)((total + 255) / 256);
  if (fp32) {
    if (out_padded)
      hipLaunchKernelGGL((unpack_kernel<true, true>), dim3(grid), dim3(256), 0, stream, g, comp_of_site, det, batch, out);
    else
      hipLaunchKernelGGL((unpack_kernel<true, false>), dim3(grid), dim3(256), 0, stream, g, comp_of_site, det, batch, out);
  } else {
    if (out_padded)
      hipLaunchKernelGGL((unpack_kernel<false, true>), dim3(grid), dim3(256), 0, stream, g, comp_of_site, det, batch, out);
    else
      hipLaunchKernelGGL((unpack_kernel<false, false>), dim3(grid), dim3(256), 0, stream, g, comp_of_site, det, batch, out);
  }
  return hipGetLastError();
}

}  // namespace pd
