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
// K5 (residual + repack): a wave64 builds one packed 64-bit output word at a
// time from nibble rows staged in LDS.  Lane l computes bit 64 w + l of
// either the residual row (Eqs. Resk1X..ReskG1Z: detector ^ measurement flip
// of this round ^ of the previous round ^ parity of the data corrections on
// the plaquette, Eqs. SXJK/SZJK) or the flip row, and __ballot packs the 64
// bits of the wave into the word, which lane 0 stores.  Rows are whole words per sample, so no word is shared between
// waves and no atomics are needed; padding bits come out 0.
#include <algorithm>

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

// K5 layout: a workgroup (four waves) takes a chunk of one sample's words --
// up to cd residual words or cf flip words -- stages the nibble rows of the
// rounds those words read (one more round before, for the previous-round
// measurement flip) from HBM into LDS with coalesced dword loads, then each
// wave builds words from LDS.  Every nibble byte of a sample is read from HBM
// about once per word kind instead of once per stencil term.  Bit indices
// within a sample fit 32 bits (T nflip < 2^31), so index splits are 32-bit
// reciprocal divisions.
struct ResidualPlan {
  FastDiv by_stab, by_flip, by_chunks;
  int cd, cf;  // words per residual / flip chunk
  int nd, nf;  // residual / flip chunks per sample
};

// LDS bytes a launch may stage (rounds of T x H x H nibble rows).
constexpr int kResidualLds = 32768;

// The words [w0, w1) of one row kind of sample b, from the staged nibble rows
// (rows[(t - ta) HH + s] = nibble of round t, site s) and the per-bit
// descriptors of the tables (sten for residual rows, fsite for flip rows).  A
// wave takes words w, w + 4, w + 8, w + 12 per pass: first every descriptor
// and detector read of the four words, then the LDS reads, so the reads go
// out together instead of one dependent chain per word.  Indices are clamped
// into range and bits past the row masked, so the body has no branches.
template <bool RES>
__device__ __forceinline__ void chunk_words_build(const Geom& g, const uint8_t* rows, int ta, int HH,
                                                  const int32_t* __restrict__ tables,
                                                  const uint64_t* __restrict__ det, uint64_t* __restrict__ out,
                                                  int b, int w0, int w1, int kend, FastDiv by_n, int nbits,
                                                  int lane) {
  constexpr int U = 4;
  const long long row_words = RES ? g.Wd : g.Wf;
  const u32x4* sten = reinterpret_cast<const u32x4*>(tables + tables_sten(g));
  const uint32_t* fsite = reinterpret_cast<const uint32_t*>(tables + tables_fsite(g));
  for (int w = w0 + (int)(threadIdx.x >> 6); w < w1; w += 4 * U) {  // uniform per wave
    int t[U];
    u32x4 ds[U];
    unsigned dw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ww = min(w + 4 * u, w1 - 1);
      const int k = min(ww * 64 + lane, kend - 1);
      t[u] = (int)fastdiv((uint32_t)k, by_n);
      const int n = k - t[u] * nbits;
      if constexpr (RES) {
        ds[u] = sten[n];
        dw[u] = (unsigned)(det[(long long)b * g.Wd + ww] >> lane);
      } else {
        ds[u][0] = fsite[n];
      }
    }
    unsigned bits[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint8_t* row = rows + (t[u] - ta) * HH;
      unsigned bit;
      if constexpr (RES) {
        // Eqs. Resk1X..ReskG1Z: detector ^ measurement flips of rounds t and
        // t - 1 at the stabilizer's site ^ data flips on its support (the
        // data channel is mch - 2: 0 for X checks, 1 for Z checks)
        const unsigned site = ds[u][0] & 0xffffu, mch = ds[u][0] >> 16;
        const unsigned m0 = row[site], m1 = row[(t[u] > ta ? -HH : 0) + (int)site];
        const unsigned dsum = row[ds[u][1] & 0xffffu] ^ row[ds[u][1] >> 16] ^ row[ds[u][2] & 0xffffu] ^
                              row[ds[u][2] >> 16];
        bit = dw[u] ^ ((m0 ^ (t[u] > 0 ? m1 : 0u)) >> mch) ^ (dsum >> (mch - 2u));
      } else {
        // flip row: data X / Z flips on the d x d data sites, then the
        // measurement flips at the stabilizer sites
        bit = (unsigned)row[ds[u][0] & 0xffffu] >> (ds[u][0] >> 16);
      }
      const bool real = w + 4 * u < w1 && (w + 4 * u) * 64 + lane < kend;
      bits[u] = real ? (bit & 1u) : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const unsigned long long m = __ballot(bits[u]);
      if (lane == 0 && w + 4 * u < w1) out[(long long)b * row_words + w + 4 * u] = m;
    }
  }
}

__global__ void __launch_bounds__(256) residual_pack_kernel(Geom g, const int32_t* __restrict__ tables,
                                                            const uint64_t* __restrict__ det,
                                                            const uint8_t* __restrict__ nib,
                                                            uint64_t* __restrict__ flips,
                                                            uint64_t* __restrict__ residual, ResidualPlan p) {
  extern __shared__ uint32_t lds_words[];
  uint8_t* lds = reinterpret_cast<uint8_t*>(lds_words);
  const int b = (int)fastdiv(blockIdx.x, p.by_chunks);
  const int c = (int)blockIdx.x - b * (p.nd + p.nf);
  const bool is_res = c < p.nd;
  const int nbits = is_res ? g.nstab : g.nflip;
  const FastDiv by_n = is_res ? p.by_stab : p.by_flip;
  const int w0 = is_res ? c * p.cd : (c - p.nd) * p.cf;
  const int wlim = is_res ? (int)g.Wd : (int)g.Wf;
  const int w1 = min(w0 + (is_res ? p.cd : p.cf), wlim);
  const int kend = min(w1 * 64, g.T * nbits);  // first bit past the chunk's real bits
  int ta = (int)fastdiv((uint32_t)(w0 * 64), by_n);
  if (is_res && ta > 0) --ta;  // previous round of the first word's round
  const int tb = (int)fastdiv((uint32_t)(max(kend, 1) - 1), by_n);
  const int HH = g.H * g.H;
  // stage bytes [ta HH, (tb + 1) HH) of the sample's nibbles: LDS byte
  // (src & 3) + i holds byte i, so the 4-aligned middle moves as dwords
  const uint8_t* src = nib + (long long)b * g.V + (long long)ta * HH;
  const int nbytes = (tb - ta + 1) * HH;
  const int mis = (int)((uintptr_t)src & 3);
  const int head = min((4 - mis) & 3, nbytes);
  const int nw = (nbytes - head) >> 2;
  const uint32_t* mid = reinterpret_cast<const uint32_t*>(src + head);
  for (int i = threadIdx.x; i < nw; i += 256) lds_words[(mis + head) / 4 + i] = mid[i];
  if (threadIdx.x < head) lds[mis + threadIdx.x] = src[threadIdx.x];
  const int tail0 = head + 4 * nw;
  if ((int)threadIdx.x < nbytes - tail0) lds[mis + tail0 + threadIdx.x] = src[tail0 + threadIdx.x];
  __syncthreads();
  const uint8_t* rows = lds + mis;  // byte (t - ta) HH + s = nibble of (t, s), ta <= t <= tb
  const int lane = threadIdx.x & 63;
  if (is_res)
    chunk_words_build<true>(g, rows, ta, HH, tables, det, residual, b, w0, w1, kend, by_n, nbits, lane);
  else
    chunk_words_build<false>(g, rows, ta, HH, tables, det, flips, b, w0, w1, kend, by_n, nbits, lane);
}

// Words per chunk for a word row of `nbits` bits per round: the most words
// whose rounds (plus one earlier round for residual rows) fit the LDS budget,
// at most `want`, at least 1.
static int chunk_words(const Geom& g, int nbits, int extra, int want) {
  const int HH = g.H * g.H;  // three rounds of the largest grid (H = 64) fit the budget
  int cw = want;
  // rounds touched by cw words: <= ceil(64 cw / nbits) + 1, plus `extra`
  while (cw > 1 && ((64 * cw + nbits - 1) / nbits + 1 + extra) * HH + 4 > kResidualLds) cw = cw * 3 / 4;
  return cw;
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
  if (batch <= 0) return hipSuccess;
  // chunks of words / 4096 words (at least one word per wave): about 4096
  // workgroups at large batch (a whole row per workgroup at d = 13), more
  // and shorter ones at small batch, so no wave runs a long serial chain
  const long long words = (long long)batch * (g.Wd + g.Wf);
  const int want = (int)std::max(4ll, std::min(words / 4096, (long long)INT32_MAX));
  ResidualPlan p;
  p.cd = chunk_words(g, g.nstab, 1, (int)std::min((long long)want, g.Wd));
  p.cf = chunk_words(g, g.nflip, 0, (int)std::min((long long)want, g.Wf));
  p.nd = (int)((g.Wd + p.cd - 1) / p.cd);
  p.nf = (int)((g.Wf + p.cf - 1) / p.cf);
  const long long blocks = (long long)batch * (p.nd + p.nf);
  if (blocks >= (1ll << 31)) return hipErrorInvalidValue;  // block ids are split with 32-bit divisions
  p.by_stab = make_fastdiv((uint32_t)g.nstab);
  p.by_flip = make_fastdiv((uint32_t)g.nflip);
  p.by_chunks = make_fastdiv((uint32_t)(p.nd + p.nf));
  // staged rounds of either chunk kind, +4 bytes of alignment slack
  const int HH = g.H * g.H;
  const int rd = (64 * p.cd + g.nstab - 1) / g.nstab + 2, rf = (64 * p.cf + g.nflip - 1) / g.nflip + 1;
  const size_t lds = (size_t)std::min(std::max(rd, rf), g.T) * HH + 4;
  if (lds > (size_t)kResidualLds + 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(residual_pack_kernel, dim3((unsigned)blocks), dim3(256), lds, stream, g, tables, det, nib,
                     flips, residual, p);
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
