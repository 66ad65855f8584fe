// unpack.hip -- K1: packed detector events -> input planes (Sec. IV.B.1).
//
// Plaquette layout: two channels on the (d+1) x (d+1) grid, each detector
// event at its stabilizer's site, X-type in channel 0 and Z-type in channel 1
// (every other grid location is 0).
// Paper layout (Eqs. encTrainX1-encTrainX4): four channels on the D x D grid
// of data qubits, every stabilizer drawn onto one qubit of its support:
// x_type / z_type carry the detector events of the X / Z stabilizer drawn at
// the qubit, x_present / z_present its weight / 4 (1 or 0.5), cleared in the
// first round for the basis the qubit is prepared in (Z clears x_present, X
// clears z_present) and in the last round for the basis it is measured in.
//
// One thread per interior voxel (t, i, j), looping over the samples; for each
// sample it reads the bits it needs (the packed row of a sample is a few
// hundred bytes, so these reads hit L1/L2) and writes all channels of the
// voxel with one store.  Consecutive threads write consecutive voxels of a
// grid row.  HBM-bound: reads W_det * 8
// bytes and writes c_in * V * sizeof(elem) bytes per sample.
#include <algorithm>

#include "internal.h"

namespace pd {

// Store voxel (t, s) of sample b given its two detector events.
template <bool FP32, bool PADDED, bool PAPER>
__device__ __forceinline__ void unpack_store(const Geom& g, int b, int v, int t, int s, unsigned ex, unsigned ez,
                                             float px, float pz, void* __restrict__ out, FastDiv by_h) {
  long long o;
  if (PADDED) {
    const int i = (int)fastdiv((uint32_t)s, by_h), j = s - i * g.H;
    o = padded_index(g, b, t, i, j);
  } else {
    o = (long long)b * g.V + v;
  }
  if constexpr (PAPER) {
    static_assert(!FP32, "the paper's layout runs in bf16");
    // bf16 patterns: 1.0 = 0x3F80, 0.5 = 0x3F00
    auto bf = [](float f) -> uint32_t { return f == 1.0f ? 0x3F80u : (f == 0.5f ? 0x3F00u : 0u); };
    uint2 val;
    val.x = (ex ? 0x3F80u : 0u) | ((ez ? 0x3F80u : 0u) << 16);
    val.y = bf(px) | (bf(pz) << 16);
    reinterpret_cast<uint2*>(out)[o] = val;
  } else if (FP32) {
    float2 val;
    val.x = ex ? 1.0f : 0.0f;
    val.y = ez ? 1.0f : 0.0f;
    reinterpret_cast<float2*>(out)[o] = val;
  } else {
    reinterpret_cast<uint32_t*>(out)[o] = (ex ? 0x3F80u : 0u) | ((ez ? 0x3F80u : 0u) << 16);
  }
}

// Grid: x covers one sample's V voxels (one thread each), y strides over the
// batch; the per-voxel tables are read once per thread, the voxel split uses
// 32-bit reciprocal divisions (by_hh: H H, by_h: H).  V < 2^31 for every
// supported grid.  The detector bit of compact stabilizer n in round t is bit
// k = t nstab + n of the sample's row; a site without a stabilizer of a type
// reads bit 0 and masks it.
template <bool FP32, bool PADDED, bool PAPER>
__global__ void __launch_bounds__(256) unpack_kernel(Geom g, const int32_t* __restrict__ tables,
                                                     const uint64_t* __restrict__ det, int batch,
                                                     void* __restrict__ out, FastDiv by_hh, FastDiv by_h) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= g.V) return;
  const int HH = g.H * g.H;
  const int t = (int)fastdiv((uint32_t)v, by_hh);
  const int s = v - t * HH;
  const int nx = tables[tables_comp_x(g) + s], nz = tables[tables_comp_z(g) + s];
  float px = 0.0f, pz = 0.0f;
  if constexpr (PAPER) {
    // weight / 4 of the stabilizer drawn here: 1 for four qubits, 0.5 for two
    auto present = [&](int n, int kind) -> float {
      if (n < 0) return 0.0f;
      if ((t == 0 && g.first == kind) || (t == g.T - 1 && g.last == kind)) return 0.0f;
      const int32_t* sp = tables + tables_supp(g) + n * 4;
      return (sp[2] >= 0) ? 1.0f : 0.5f;
    };
    px = present(nx, 1);
    pz = present(nz, 2);
  }
  const int kx = t * g.nstab + max(nx, 0), kz = t * g.nstab + max(nz, 0);
  const uint64_t mx = nx >= 0 ? 1ull << (kx & 63) : 0ull, mz = nz >= 0 ? 1ull << (kz & 63) : 0ull;
  // samples blockIdx.y + k gridDim.y, four per pass: their detector reads
  // are issued together before any store
  const int gy = gridDim.y;
  int b = blockIdx.y;
  for (; b + 3 * gy < batch; b += 4 * gy) {
    uint64_t wx[4], wz[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint64_t* row = det + (long long)(b + u * gy) * g.Wd;
      wx[u] = row[kx >> 6];
      wz[u] = row[kz >> 6];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      unpack_store<FP32, PADDED, PAPER>(g, b + u * gy, v, t, s, (wx[u] & mx) != 0, (wz[u] & mz) != 0, px, pz,
                                        out, by_h);
  }
  for (; b < batch; b += gy) {
    const uint64_t* row = det + (long long)b * g.Wd;
    unpack_store<FP32, PADDED, PAPER>(g, b, v, t, s, (row[kx >> 6] & mx) != 0, (row[kz >> 6] & mz) != 0, px,
                                      pz, out, by_h);
  }
}

hipError_t launch_unpack(const Geom& g, const int32_t* tables, const uint64_t* det, int batch, void* out,
                         int out_padded, int fp32, hipStream_t stream) {
  if (batch <= 0) return hipSuccess;
  // about 4096 workgroups in all (16 per CU): each thread then covers
  // several samples, which amortises its table reads and keeps workgroups
  // long enough that dispatch does not bound a large batch
  const long long gx = (g.V + 255) / 256;
  const long long gy = std::max(1ll, std::min<long long>(std::min(batch, 65535), 4096 / gx));
  const dim3 grid((unsigned)gx, (unsigned)gy);
  const FastDiv by_hh = make_fastdiv((uint32_t)(g.H * g.H)), by_h = make_fastdiv((uint32_t)g.H);
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, g, tables, det, batch, out, by_hh, by_h);
  };
  if (g.layout == 1) {
    if (fp32) return hipErrorInvalidValue;
    if (out_padded)
      go(unpack_kernel<false, true, true>);
    else
      go(unpack_kernel<false, false, true>);
  } else if (fp32) {
    if (out_padded)
      go(unpack_kernel<true, true, false>);
    else
      go(unpack_kernel<true, false, false>);
  } else {
    if (out_padded)
      go(unpack_kernel<false, true, false>);
    else
      go(unpack_kernel<false, false, false>);
  }
  return hipGetLastError();
}

}  // namespace pd

namespace pd {

// One thread per granule (16 or 8 bytes) of an interior voxel row:
// out[(b, t, i, j)] <- act[padded (b, t, i, j)].
template <typename G>
__global__ void __launch_bounds__(256) extract_kernel(Geom g, const G* __restrict__ act, int gran, int batch,
                                                      G* __restrict__ out) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long total = (long long)batch * g.V * gran;
  if (gid >= total) return;
  const long long vox = gid / gran;
  const int q = (int)(gid - vox * gran);
  const int b = (int)(vox / g.V);
  const int v = (int)(vox - (long long)b * g.V);
  const int HH = g.H * g.H;
  const int t = v / HH, s = v - t * HH;
  const int i = s / g.H, j = s - i * g.H;
  out[gid] = act[padded_index(g, b, t, i, j) * gran + q];
}

hipError_t launch_extract(const Geom& g, const void* act, int row_bytes, int batch, void* out, hipStream_t stream) {
  if (row_bytes <= 0 || row_bytes % 8 != 0) return hipErrorInvalidValue;
  if (row_bytes % 16 == 0) {
    const int gran = row_bytes / 16;
    const long long total = (long long)batch * g.V * gran;
    hipLaunchKernelGGL(extract_kernel<uint4>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, g,
                       (const uint4*)act, gran, batch, (uint4*)out);
  } else {  // rows of four bf16 channels (a projection to the 4 output channels)
    const int gran = row_bytes / 8;
    const long long total = (long long)batch * g.V * gran;
    hipLaunchKernelGGL(extract_kernel<uint2>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, g,
                       (const uint2*)act, gran, batch, (uint2*)out);
  }
  return hipGetLastError();
}

}  // namespace pd

namespace pd {

__global__ void __launch_bounds__(256) zero_kernel(uint4* __restrict__ p, long long n) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid < n) p[gid] = uint4{0u, 0u, 0u, 0u};
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream) {
  if (bytes % 16 != 0) return hipErrorInvalidValue;
  const long long n = (long long)(bytes / 16);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, (uint4*)p, n);
  return hipGetLastError();
}

}  // namespace pd
