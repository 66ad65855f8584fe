// head_residual.hip -- K4 and K5 of the pre-decoder path.
//
// K4 (head + threshold): the 1x1x1 output layer (c_in -> 4) at every grid
// voxel, the threshold logit > 0 (sigmoid > 1/2 of the BCE objective,
// Sec. IV.B.5), and the read-out of the four correction channels where they
// are defined (Eqs. ZcorreJK, XcorreJK, SynXCorrJK, SynZCorrJK): channels 0/1
// at data qubits (grid sites (r, c), r, c < d), channel 2 where an X
// stabilizer sits (or is drawn, in the paper's layout), channel 3 likewise
// for Z.  The four flip bits of a voxel are kept as one nibble per voxel in a
// small workspace; fp32 logits are written only when asked for.
//
// K5 (residual + repack): one wave64 per packed 64-bit output word.  Lane l
// computes bit 64 w + l of either the residual row (Eqs. Resk1X..ReskG1Z:
// detector ^ measurement flip of this round ^ of the previous round ^ parity
// of the data corrections on the plaquette, Eqs. SXJK/SZJK) or the flip row,
// and __ballot packs the 64 bits of the wave into the word, which lane 0
// stores.  Rows are whole words per sample, so no word is shared between
// waves and no atomics are needed; padding bits come out 0.
#include "internal.h"

namespace pd {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

template <bool FP32>
__global__ void __launch_bounds__(256) head_kernel(Geom g, int cin, const void* __restrict__ x,
                                                   const float* __restrict__ w_head,
                                                   const float* __restrict__ b_head,
                                                   const int32_t* __restrict__ tables,
                                                   uint8_t* __restrict__ nib, float* __restrict__ logits,
                                                   int batch) {
  __shared__ float w[4 * 128];
  for (int e = threadIdx.x; e < 4 * cin; e += blockDim.x) w[e] = w_head[e];
  __syncthreads();
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)batch * g.V) return;
  const int b = (int)(gid / g.V);
  const int v = (int)(gid - (long long)b * g.V);
  const int HH = g.H * g.H;
  const int t = v / HH, s = v - t * HH;
  const int i = s / g.H, j = s - i * g.H;
  const long long p = padded_index(g, b, t, i, j);
  float acc[4] = {b_head[0], b_head[1], b_head[2], b_head[3]};
  if (FP32) {
    const float* xr = reinterpret_cast<const float*>(x) + p * cin;
    for (int c = 0; c < cin; ++c) {
      float xv = xr[c];
#pragma unroll
      for (int o = 0; o < 4; ++o) acc[o] = fmaf(w[o * cin + c], xv, acc[o]);
    }
  } else {
    const u32x4* xr = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(x) + p * cin);
    for (int c8 = 0; c8 < cin / 8; ++c8) {
      u32x4 q = xr[c8];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        float lo = __uint_as_float(q[h] << 16);
        float hi = __uint_as_float(q[h] & 0xffff0000u);
        const int c = c8 * 8 + 2 * h;
#pragma unroll
        for (int o = 0; o < 4; ++o) {
          acc[o] = fmaf(w[o * cin + c], lo, acc[o]);
          acc[o] = fmaf(w[o * cin + c + 1], hi, acc[o]);
        }
      }
    }
  }
  nib[gid] = (uint8_t)flip_nibble(g, tables, i, j, acc);
  if (logits) {
#pragma unroll
    for (int o = 0; o < 4; ++o) logits[(((long long)b * 4 + o) * g.T + t) * HH + s] = acc[o];
  }
}

// Residual bit of (sample b, round t, compact stabilizer n) given a functor
// flip(ch, t, site) -> 0/1.
template <typename Flip>
__device__ __forceinline__ unsigned residual_bit(const Geom& g, const int32_t* __restrict__ site_of,
                                                 const int32_t* __restrict__ supp, int t, int n,
                                                 Flip flip) {
  const int s = site_of[n];
  const bool isx = n < g.K;
  const int mch = isx ? 2 : 3;  // measurement correction of this stabilizer type
  const int dch = isx ? 0 : 1;  // X checks see Z corrections, Z checks see X corrections
  unsigned r = flip(mch, t, s);
  if (t > 0) r ^= flip(mch, t - 1, s);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int qs = supp[n * 4 + q];
    if (qs >= 0) r ^= flip(dch, t, qs);
  }
  return r;
}

__global__ void __launch_bounds__(256) residual_pack_kernel(Geom g, const int32_t* __restrict__ tables,
                                                            const uint64_t* __restrict__ det,
                                                            const uint8_t* __restrict__ nib,
                                                            uint64_t* __restrict__ flips,
                                                            uint64_t* __restrict__ residual, int batch) {
  const int lane = threadIdx.x & 63;
  const long long wid = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const long long words = g.Wd + g.Wf;
  if (wid >= (long long)batch * words) return;  // whole wave exits together
  const int b = (int)(wid / words);
  const long long w = wid - (long long)b * words;
  const int32_t* site_of = tables + tables_site_of(g);
  const int32_t* supp = tables + tables_supp(g);
  const int HH = g.H * g.H;
  const uint8_t* nb = nib + (long long)b * g.V;
  auto flip = [&](int ch, int t, int s) -> unsigned { return (nb[t * HH + s] >> ch) & 1u; };
  unsigned bit = 0;
  if (w < g.Wd) {
    const long long k = w * 64 + lane;
    if (k < (long long)g.T * g.nstab) {
      const int t = (int)(k / g.nstab), n = (int)(k - (long long)t * g.nstab);
      bit = (unsigned)((det[(long long)b * g.Wd + w] >> lane) & 1ull);
      bit ^= residual_bit(g, site_of, supp, t, n, flip);
    }
    const unsigned long long m = __ballot(bit);
    if (lane == 0) residual[(long long)b * g.Wd + w] = m;
  } else {
    const long long wf = w - g.Wd;
    const long long k = wf * 64 + lane;
    if (k < (long long)g.T * g.nflip) {
      const int t = (int)(k / g.nflip), n = (int)(k - (long long)t * g.nflip);
      const int dd = g.d * g.d;
      int ch, s;
      if (n < dd) {
        ch = 0;
        s = (n / g.d) * g.H + n % g.d;
      } else if (n < 2 * dd) {
        ch = 1;
        s = ((n - dd) / g.d) * g.H + (n - dd) % g.d;
      } else {
        const int n2 = n - 2 * dd;
        ch = n2 < g.K ? 2 : 3;
        s = site_of[n2];
      }
      bit = flip(ch, t, s);
    }
    const unsigned long long m = __ballot(bit);
    if (lane == 0) flips[(long long)b * g.Wf + wf] = m;
  }
}

__global__ void __launch_bounds__(256) residual_from_flips_kernel(Geom g, const int32_t* __restrict__ tables,
                                                                  const uint64_t* __restrict__ det,
                                                                  const uint64_t* __restrict__ flips,
                                                                  uint64_t* __restrict__ residual,
                                                                  int batch) {
  const int lane = threadIdx.x & 63;
  const long long wid = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (wid >= (long long)batch * g.Wd) return;
  const int b = (int)(wid / g.Wd);
  const long long w = wid - (long long)b * g.Wd;
  const int32_t* site_of = tables + tables_site_of(g);
  const int32_t* comp_x = tables + tables_comp_x(g);
  const int32_t* comp_z = tables + tables_comp_z(g);
  const int32_t* supp = tables + tables_supp(g);
  const uint64_t* fr = flips + (long long)b * g.Wf;
  const int dd = g.d * g.d;
  auto flip = [&](int ch, int t, int s) -> unsigned {
    long long fk = (long long)t * g.nflip;
    if (ch < 2) {
      const int r = s / g.H, c = s - (s / g.H) * g.H;
      fk += ch * dd + r * g.d + c;
    } else {
      fk += 2 * dd + (ch == 2 ? comp_x[s] : comp_z[s]);
    }
    return (unsigned)((fr[fk >> 6] >> (fk & 63)) & 1ull);
  };
  unsigned bit = 0;
  const long long k = w * 64 + lane;
  if (k < (long long)g.T * g.nstab) {
    const int t = (int)(k / g.nstab), n = (int)(k - (long long)t * g.nstab);
    bit = (unsigned)((det[(long long)b * g.Wd + w] >> lane) & 1ull);
    bit ^= residual_bit(g, site_of, supp, t, n, flip);
  }
  const unsigned long long m = __ballot(bit);
  if (lane == 0) residual[(long long)b * g.Wd + w] = m;
}

hipError_t launch_head(const Geom& g, int cin, int fp32, const void* x, const float* w_head,
                              const float* b_head, const int32_t* tables, uint8_t* nib, float* logits,
                              int batch, hipStream_t stream) {
  long long total = (long long)batch * g.V;
  unsigned grid = (unsigned)((total + 255) / 256);
  if (fp32)
    hipLaunchKernelGGL(head_kernel<true>, dim3(grid), dim3(256), 0, stream, g, cin, x, w_head, b_head,
                       tables, nib, logits, batch);
  else
    hipLaunchKernelGGL(head_kernel<false>, dim3(grid), dim3(256), 0, stream, g, cin, x, w_head, b_head,
                       tables, nib, logits, batch);
  return hipGetLastError();
}

hipError_t launch_residual_pack(const Geom& g, const int32_t* tables, const uint64_t* det,
                                const uint8_t* nib, uint64_t* flips, uint64_t* residual, int batch,
                                hipStream_t stream) {
  long long waves = (long long)batch * (g.Wd + g.Wf);
  unsigned grid = (unsigned)((waves + 3) / 4);
  hipLaunchKernelGGL(residual_pack_kernel, dim3(grid), dim3(256), 0, stream, g, tables, det, nib, flips,
                     residual, batch);
  return hipGetLastError();
}

hipError_t launch_residual_from_flips(const Geom& g, const int32_t* tables, const uint64_t* det,
                                      const uint64_t* flips, uint64_t* residual, int batch,
                                      hipStream_t stream) {
  long long waves = (long long)batch * g.Wd;
  unsigned grid = (unsigned)((waves + 3) / 4);
  hipLaunchKernelGGL(residual_from_flips_kernel, dim3(grid), dim3(256), 0, stream, g, tables, det, flips,
                     residual, batch);
  return hipGetLastError();
}

}  // namespace pd
