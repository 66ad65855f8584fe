// conv_bf16.hip -- K2 + K3: one 3x3x3 conv3d layer (Sec. III.B, Fig.
// ConvArch; stride 1, zero padding, cross-correlation) as an implicit GEMM on
// the gfx950 matrix cores, with the bias + activation + bf16 rounding
// epilogue fused in.
//
//   out[m][co] = act(bias[co] + sum_{tap, ci} X[m + shift(tap)][ci] * W[tap][ci][co])
//
// GEMM view: M = output voxels, N = c_out, K = 27 * c_in.  Activations live in
// the zero-halo NTHWC layout of internal.h, so every tap is an index shift
// and no bounds checks are needed in the K loop.
//
// Work split (one workgroup = 256 threads = 4 wave64):
//   * a tile is 256 output voxels (see Tiling) x all c_out channels;
//   * wave w owns rows [128 * (w & 1), +128) and columns
//     [(c_out / 2) * (w >> 1), +c_out / 2): 4 x (c_out / 64) blocks of
//     v_mfma_f32_32x32x16_bf16, fp32 accumulators in registers;
//   * the input footprint of the tile is staged in LDS, 32 input channels
//     (64 bytes per voxel) at a time, double buffered; the next chunk is
//     copied with global_load_lds_dwordx4 (HBM/L2 -> LDS without registers)
//     while the current one feeds the MFMAs;
//   * each voxel's four 16-byte granules are XOR-swizzled by (voxel >> 1) & 3
//     so the 32 rows of an A fragment (consecutive voxels, 64-byte stride)
//     hit distinct LDS banks;
//   * weights are pre-arranged at create time in MFMA B-fragment order and
//     read straight from global memory (one coalesced 16-byte load per lane
//     per fragment; a layer is <= 0.9 MB and stays L2-resident);
//   * epilogue: acc + bias -> activation (fp32) -> bf16 (RNE, v_cvt_pk_bf16_f32)
//     -> LDS transpose -> 16-byte coalesced stores into the interior of the
//     output (the halo is never written).
// Layer 1 (c_in = 2) uses the same tile machinery with K = 27 taps x 2
// channels padded to 64: each lane gathers 4 taps x 2 channels per fragment.
#include "internal.h"

namespace pd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int KC = 32;              // input channels per LDS chunk
constexpr int kOutPad = 16;         // bytes of padding per row of the output tile
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ float activation(float y, int act) {
  if (act == 1) {  // GELU, tanh form: 0.5 y (1 + tanh(u)) = y / (1 + exp(-2u))
    const float k0 = 0.7978845608028654f;      // sqrt(2 / pi)
    const float kl = -2.0f * 1.4426950408889634f;  // -2 log2(e)
    float u = k0 * (y + 0.044715f * y * y * y);
    float e = __builtin_amdgcn_exp2f(kl * u);
    return y * __builtin_amdgcn_rcpf(1.0f + e);
  }
  if (act == 2) return y > 0.0f ? y : 0.0f;
  return y;
}

__device__ __forceinline__ uint16_t to_bf16_bits(float v) {
  __bf16 h = (__bf16)v;
  return __builtin_bit_cast(uint16_t, h);
}

// Decodes row r (0..255) of tile `tile`: returns false if the row is outside
// the volume; otherwise the padded index of the output voxel.
__host__ __device__ inline bool tile_row(const Geom& g, const Tiling& tl, long long tile, int r,
                                         int batch, long long* pidx, int* lds_base,
                                         long long* stage_origin) {
  if (tl.mode == 0) {
    long long seg = tile / tl.tiles_per_seg;
    long long k0 = (tile - seg * tl.tiles_per_seg) * (long long)kTileRows;
    long long u0 = seg * tl.seg_len + k0;
    int b0 = (int)(u0 / g.V);
    int v0 = (int)(u0 - (long long)b0 * g.V);
    int HH = g.H * g.H;
    int t0 = v0 / HH, s0 = v0 - t0 * HH;
    long long p0 = padded_index(g, b0, t0, s0 / g.H, s0 % g.H);
    *stage_origin = p0 - (g.P + g.Wp + 1);
    long long u = u0 + r;
    bool ok = (k0 + r < tl.seg_len) && (u < (long long)batch * g.V);
    if (!ok) {
      *lds_base = 0;
      return false;
    }
    int b = (int)(u / g.V);
    int v = (int)(u - (long long)b * g.V);
    int t = v / HH, s = v - t * HH;
    long long p = padded_index(g, b, t, s / g.H, s % g.H);
    *pidx = p;
    *lds_base = (int)(p - p0);
    return true;
  } else {
    long long per = (long long)tl.ntT * tl.ntI * tl.ntJ;
    int b = (int)(tile / per);
    int rem = (int)(tile - (long long)b * per);
    int tt = rem / (tl.ntI * tl.ntJ);
    int ti = (rem / tl.ntJ) % tl.ntI;
    int tj = rem % tl.ntJ;
    int t0 = tt * tl.BT, i0 = ti * tl.BI, j0 = tj * tl.BJ;
    *stage_origin = (long long)b * g.S + (long long)t0 * g.P + (long long)i0 * g.Wp + j0;
    int bij = tl.BI * tl.BJ;
    int a = r / bij, c = (r / tl.BJ) % tl.BI, e = r % tl.BJ;
    int t = t0 + a, i = i0 + c, j = j0 + e;
    bool ok = (r < tl.BT * bij) && t < g.T && i < g.H && j < g.H;
    *lds_base = ok ? (a * (tl.BI + 2) + c) * (tl.BJ + 2) + e : 0;
    if (!ok) return false;
    *pidx = padded_index(g, b, t, i, j);
    return true;
  }
}

// Padded box origin of a box-mode tile, in padded coordinates.
struct BoxOrigin {
  int t0, i0, j0;
};

// Global padded voxel of staged voxel vv (clamped to voxel 0, a zero halo
// voxel, when outside the batch or outside the sample's padded box).
__host__ __device__ inline long long staged_voxel(const Geom& g, const Tiling& tl, long long origin,
                                                  const BoxOrigin& bo, int vv, long long limit) {
  if (tl.mode == 0) {
    long long p = origin + vv;
    return (p < limit) ? p : 0;
  }
  const int bj2 = tl.BJ + 2, bij2 = (tl.BI + 2) * bj2;
  const int a = vv / bij2;
  const int rem = vv - a * bij2;
  const int c = rem / bj2;
  const int e = rem - c * bj2;
  if (bo.t0 + a >= g.T + 2 || bo.i0 + c >= g.Wp || bo.j0 + e >= g.Wp) return 0;
  return origin + (long long)a * g.P + (long long)c * g.Wp + e;
}

template <int CIN, int COUT>
__global__ void __launch_bounds__(256) conv_bf16_kernel(Geom g, Tiling tl, int act,
                                                        const uint16_t* __restrict__ x,
                                                        uint16_t* __restrict__ y,
                                                        const u32x4* __restrict__ wfrag,
                                                        const float* __restrict__ bias, int batch,
                                                        int abuf_bytes, int region_bytes) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int NB = COUT / 64;   // 32-wide column blocks per wave
  constexpr int NBT = COUT / 32;  // column blocks in total
  constexpr int MB = 4;           // 32-row blocks per wave
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;

  // Consecutive workgroups are dispatched round-robin over the 8 XCDs; give
  // each XCD a contiguous run of tiles so neighbouring tiles (which share
  // halo voxels) meet in the same L2.
  const unsigned per_xcd = gridDim.x >> 3;
  const long long tile = (long long)(blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (tile >= tl.ntiles) return;

  char* abuf0 = smem;
  char* abuf1 = smem + abuf_bytes;
  char* region_end = smem + region_bytes;
  long long* row_pidx = reinterpret_cast<long long*>(region_end);
  int* row_base = reinterpret_cast<int*>(region_end + 256 * sizeof(long long));

  long long origin = 0;
  {
    long long p = -1;
    int lb = 0;
    bool ok = tile_row(g, tl, tile, tid, batch, &p, &lb, &origin);
    row_pidx[tid] = ok ? p : -1;
    row_base[tid] = lb;
  }
  const long long limit = (long long)batch * g.S;
  BoxOrigin bo{0, 0, 0};
  if (tl.mode == 1) {
    long long rem = origin - (origin / g.S) * g.S;
    bo.t0 = (int)(rem / g.P);
    int r2 = (int)(rem - (long long)bo.t0 * g.P);
    bo.i0 = r2 / g.Wp;
    bo.j0 = r2 - bo.i0 * g.Wp;
  }
  __syncthreads();

  int rb[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) rb[mb] = row_base[wm * 128 + mb * 32 + (lane & 31)];

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][nb][v] = 0.0f;

  if constexpr (CIN == 2) {
    // ---- Layer 1: stage the 2-channel planes (4 bytes per voxel) once ----
    const int nvox = tl.span;
    for (int base = 0; base < nvox; base += 256) {
      int vv = base + tid;
      long long gv = staged_voxel(g, tl, origin, bo, vv < nvox ? vv : 0, limit);
      const uint32_t* src = reinterpret_cast<const uint32_t*>(x) + gv;
      __builtin_amdgcn_global_load_lds(src, (lds_void*)(abuf0 + (base + wave * 64) * 4), 4, 0, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const uint32_t* a32 = reinterpret_cast<const uint32_t*>(abuf0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      u32x4 bfr[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) bfr[nb] = wfrag[(ks * NBT + wn * NB + nb) * 64 + lane];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        u32x4 av;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          int tap = ks * 8 + (lane >> 5) * 4 + q;
          uint32_t val = 0;
          if (tap < 27) {
            int dt = tap / 9, di = (tap / 3) % 3, dj = tap % 3;
            val = a32[rb[mb] + dt * tl.sa + di * tl.sb + dj];
          }
          av[q] = val;
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bfr[nb]), acc[mb][nb], 0, 0, 0);
      }
    }
  } else {
    // ---- Hidden layers: chunks of 32 input channels, double buffered ----
    constexpr int NCHUNK = CIN / KC;
    const int ngran = tl.span * 4;  // 16-byte granules per chunk
    auto stage = [&](int chunk, char* buf) {
      for (int base = 0; base < ngran; base += 256) {
        int q = base + wave * 64 + lane;
        int vv = q >> 2;
        int ps = q & 3;
        int s = ps ^ ((vv >> 1) & 3);
        long long gv = staged_voxel(g, tl, origin, bo, q < ngran ? vv : 0, limit);
        const uint16_t* src = x + gv * CIN + chunk * KC + s * 8;
        __builtin_amdgcn_global_load_lds(src, (lds_void*)(buf + (base + wave * 64) * 16), 16, 0, 0);
      }
    };
    stage(0, abuf0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    for (int chunk = 0; chunk < NCHUNK; ++chunk) {
      char* cur = (chunk & 1) ? abuf1 : abuf0;
      if (chunk + 1 < NCHUNK) stage(chunk + 1, (chunk & 1) ? abuf0 : abuf1);
      const u32x4* wchunk = wfrag + (long long)chunk * 27 * 2 * NBT * 64 + (wn * NB) * 64 + lane;
      // weights of tap + 1 are fetched while tap runs (one tap = 2 k-steps)
      u32x4 bnext[2][NB];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bnext[ks][nb] = wchunk[(ks * NBT + nb) * 64];
#pragma unroll 1
      for (int tap = 0; tap < 27; ++tap) {
        const int dt = tap / 9, di = (tap / 3) % 3, dj = tap - (tap / 3) * 3;
        const int toff = dt * tl.sa + di * tl.sb + dj;
        u32x4 bcur[2][NB];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) bcur[ks][nb] = bnext[ks][nb];
        if (tap + 1 < 27) {
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bnext[ks][nb] = wchunk[(((tap + 1) * 2 + ks) * NBT + nb) * 64];
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int seg = ks * 2 + (lane >> 5);
          u32x4 av[MB];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            const int vox = rb[mb] + toff;
            const int off = vox * 64 + ((seg ^ ((vox >> 1) & 3)) << 4);
            av[mb] = *reinterpret_cast<const u32x4*>(cur + off);
          }
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  __builtin_bit_cast(bf16x8, av[mb]), __builtin_bit_cast(bf16x8, bcur[ks][nb]), acc[mb][nb],
                  0, 0, 0);
        }
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
  }

  // ---- Epilogue: bias + activation + bf16, transposed through LDS ----
  __syncthreads();
  constexpr int OSTRIDE = COUT * 2 + kOutPad;
  char* otile = smem;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = wn * (COUT / 2) + nb * 32 + (lane & 31);
    const float bcol = bias[col];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = wm * 128 + mb * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
        float val = activation(acc[mb][nb][v] + bcol, act);
        *reinterpret_cast<uint16_t*>(otile + row * OSTRIDE + col * 2) = to_bf16_bits(val);
      }
  }
  __syncthreads();
  constexpr int GPR = COUT / 8;  // 16-byte granules per row
  for (int q = tid; q < 256 * GPR; q += 256) {
    const int row = q / GPR, gc = q % GPR;
    const long long p = row_pidx[row];
    if (p >= 0) {
      u32x4 v = *reinterpret_cast<const u32x4*>(otile + row * OSTRIDE + gc * 16);
      *reinterpret_cast<u32x4*>(y + p * COUT + gc * 8) = v;
    }
  }
}

// LDS layout of one launch: [staging buffer 0][staging buffer 1] (the output
// tile reuses this region) followed by the per-row tables.
static void lds_layout(int cin, int cout, int span, size_t* abuf, size_t* region, size_t* total) {
  if (cin == 2)
    *abuf = ((size_t)span * 4 + 1023) / 1024 * 1024;  // whole 256-voxel staging rounds
  else
    *abuf = ((size_t)span * 64 + 4095) / 4096 * 4096;  // whole 256-granule staging rounds
  size_t out = 256 * (size_t)(cout * 2 + kOutPad);
  *region = 2 * *abuf > out ? 2 * *abuf : out;
  *total = *region + 256 * (sizeof(long long) + sizeof(int));
}

size_t conv_bf16_lds_bytes(int cin, int span) {
  size_t a, r, t;
  lds_layout(cin, 128, span, &a, &r, &t);
  return t;
}

template <int CIN, int COUT>
static hipError_t launch_one(const Geom& g, const Tiling& tl, int act, const void* x, void* y,
                             const void* wfrag, const float* bias, int batch, hipStream_t stream) {
  size_t abuf, region, lds;
  lds_layout(CIN, COUT, tl.span, &abuf, &region, &lds);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)conv_bf16_kernel<CIN, COUT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  long long nt = tl.ntiles;
  unsigned grid = (unsigned)(((nt + 7) / 8) * 8);
  hipLaunchKernelGGL((conv_bf16_kernel<CIN, COUT>), dim3(grid), dim3(256), lds, stream, g, tl, act,
                     (const uint16_t*)x, (uint16_t*)y, (const u32x4*)wfrag, bias, batch, (int)abuf,
                     (int)region);
  return hipGetLastError();
}

hipError_t launch_conv_bf16(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x,
                            void* y, const void* wfrag, const float* bias, int batch,
                            hipStream_t stream) {
  if (cin == 2 && cout == 64) return launch_one<2, 64>(g, tl, act, x, y, wfrag, bias, batch, stream);
  if (cin == 2 && cout == 128) return launch_one<2, 128>(g, tl, act, x, y, wfrag, bias, batch, stream);
  if (cin == 64 && cout == 64) return launch_one<64, 64>(g, tl, act, x, y, wfrag, bias, batch, stream);
  if (cin == 128 && cout == 128) return launch_one<128, 128>(g, tl, act, x, y, wfrag, bias, batch, stream);
  if (cin == 64 && cout == 128) return launch_one<64, 128>(g, tl, act, x, y, wfrag, bias, batch, stream);
  if (cin == 128 && cout == 64) return launch_one<128, 64>(g, tl, act, x, y, wfrag, bias, batch, stream);
  return hipErrorInvalidValue;
}

}  // namespace pd
