// conv_first.hip -- K2: the first 3x3x3 conv3d layer (Sec. IV.B, Fig.
// ConvArch; c_in = 2 detector-event channels on the plaquette grid, or the 4
// channels of the paper's layout, -> c_out = 64 or 128) with the bias +
// activation + bf16 epilogue fused in, when it is not also the last hidden
// layer.
//
// K = k^3 taps x c_in channels is small (27 taps: 4 or 7 MFMA k-steps of 16;
// 125 taps of a 5x5x5 layer with 4 channels: 32),
// so the layer is bound by its epilogue (one activation per output value)
// and its output write, not by the matrix cores.  It streams: each wave takes
// a few blocks of 32 consecutive interior voxels x all c_out channels.
//   * B operand (16 k x 32 voxels, k = c_in tap + channel): lane l gathers,
//     for voxel l % 32, the 8 / c_in taps of its half of the k-step, each as
//     one load of all c_in bf16 channels of a plane voxel, straight from the
//     zero-halo planes, which stay in L2; taps past the last contribute zero.
//   * A operand: the layer's weight fragments (k-steps x c_out/32 blocks,
//     16 bytes per lane each), staged in LDS once per workgroup.  A 5x5x5
//     layer's fragments are 32 k-steps deep (64 KB per 64 channels), so
//     each of its workgroups takes one 64-channel part of the output (and
//     stages only that part's fragments) and each wave several blocks,
//     which amortise the staging.
//   * Epilogue: + bias, activation, bf16 (or, on the fp8 path, E4M3: one
//     byte per value); the wave transposes its 32 x c_out tile through its
//     own LDS slice and writes whole voxel rows with 16-byte stores.
#include <algorithm>

#include "activation.h"
#include "internal.h"

namespace pd {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2_w;
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_w;
typedef __attribute__((address_space(3))) uint32_t lds_u32_w;

constexpr int BPW = 2;  // 32-voxel blocks per wave on large launches (1 on small ones)

// Waves per workgroup.
template <int KS, int COUT>
constexpr int waves() {
  return 4;
}

// Divisors of the interior-voxel decode u -> (b, t, i, j).
struct Decode {
  FastDiv by_v, by_hh, by_h;
};

// Padded index of interior voxel u (u < nvox < 2^31).
__device__ __forceinline__ long long voxel_padded(const Geom& g, const Decode& dc, int u) {
  const int HH = g.H * g.H;
  const int b = (int)fastdiv((uint32_t)u, dc.by_v);
  const int v = u - b * g.V;
  const int t = (int)fastdiv((uint32_t)v, dc.by_hh);
  const int s = v - t * HH;
  const int i = (int)fastdiv((uint32_t)s, dc.by_h);
  return padded_index(g, b, t, i, s - i * g.H);
}

// k-steps of 16 covering K = KS^3 c_in.
template <int CIN, int KS>
constexpr int ksteps() {
  return (KS * KS * KS * CIN + 15) / 16;
}

// B fragments for this lane's voxel (padded index p): k = 16 ks + 8 half + e,
// i.e. taps (16 ks + 8 half) / CIN + q, q < 8 / CIN, all CIN channels each;
// tap (dt, di, dj) reads the voxel (dt - h, di - h, dj - h) away, h =
// (KS - 1) / 2 (within the halo).
template <int CIN, int KS>
__device__ __forceinline__ void gather(const Geom& g, const void* __restrict__ planes, long long p, bool valid,
                                       int half, u32x4 (&bx)[ksteps<CIN, KS>()]) {
  constexpr int TPF = 8 / CIN;  // taps per lane per k-step
  constexpr int TAPS = KS * KS * KS, HW = (KS - 1) / 2;
#pragma unroll
  for (int ks = 0; ks < ksteps<CIN, KS>(); ++ks)
#pragma unroll
    for (int q = 0; q < TPF; ++q) {
      const int tap = (16 * ks + 8 * half) / CIN + q;  // >= TAPS only in the last k-step
      const int dt = tap / (KS * KS), di = (tap / KS) % KS, dj = tap % KS;
      const long long at = p + (long long)(dt - HW) * g.P + (long long)(di - HW) * g.Wp + (dj - HW);
      const bool in = valid && tap < TAPS;
      if constexpr (CIN == 2) {
        bx[ks][q] = in ? reinterpret_cast<const uint32_t*>(planes)[at] : 0u;
      } else {
        const u32x2 v = in ? reinterpret_cast<const u32x2*>(planes)[at] : u32x2{0u, 0u};
        bx[ks][2 * q] = v.x;
        bx[ks][2 * q + 1] = v.y;
      }
    }
}

// Each workgroup stages the weight fragments in LDS once; each of its waves
// then handles bpw consecutive work units: a unit is a 32-voxel block and,
// with hsplit = 2 (small launches, c_out = 128), one half of its channels.
// 5x5x5 layers (WGPART): the part is the workgroup's (blockIdx % hsplit)
// and the workgroup stages only the fragments of that part's channels.
// F8: y holds E4M3 codes.
template <int CIN, int COUT, int ACT, bool F8, int KSZ>
__global__ void __launch_bounds__((64 * waves<KSZ, COUT>())) conv_first_kernel(Geom g, const void* __restrict__ planes,
                                                                          void* __restrict__ y, int ystride,
                                                                          const u32x4* __restrict__ wfrag,
                                                                          const float* __restrict__ bias, Decode dc,
                                                                          int nvox, int bpw, int hsplit) {
  constexpr int WAVES = waves<KSZ, COUT>();
  constexpr int NB = COUT / 32;
  constexpr int ESZ = F8 ? 1 : 2;        // bytes per output value
  constexpr int OSTR = COUT * ESZ + 16;  // padded LDS row stride (bytes)
  constexpr int GPR = COUT * ESZ / 16;   // 16-byte granules per voxel row
  constexpr int KS = ksteps<CIN, KSZ>();
  constexpr bool WGPART = KSZ == 5;
  const int NBS = WGPART ? NB / hsplit : NB;  // 32-channel blocks staged in LDS
  const int WFR = KS * NBS * 64;              // weight fragments x lanes (16 bytes each)
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int wgpart = WGPART ? (int)(blockIdx.x % hsplit) : 0;
  const int wgblk = WGPART ? (int)(blockIdx.x / hsplit) : (int)blockIdx.x;
  const int sb0 = wgpart * NBS;  // first staged block
  lds_u32x4_w* const wl = (lds_u32x4_w*)smem;
  lds_char* const tile = (lds_char*)smem + WFR * 16 + wave * 32 * OSTR;
  int* const prow = (int*)((lds_char*)smem + WFR * 16 + WAVES * 32 * OSTR) + wave * 32;  // row -> padded index
  for (int e = tid; e < WFR; e += 64 * WAVES) {
    const int ks = e / (NBS * 64), r = e - ks * NBS * 64;
    wl[e] = wfrag[(ks * NB + sb0) * 64 + r];
  }
  __syncthreads();

#pragma unroll 1
  for (int j = 0; j < bpw; ++j) {
    const int unit = (wgblk * WAVES + wave) * bpw + j;
    const int blk = (WGPART || hsplit == 1) ? unit : unit >> 1;
    const int part = WGPART ? wgpart : unit - blk * hsplit;
    const int u0 = blk * 32;
    if (u0 >= nvox) break;
    const int hb = part * (NB / hsplit), he = hb + NB / hsplit;  // this unit's 32-channel blocks
    const bool valid = u0 + l32 < nvox;
    const long long p = valid ? voxel_padded(g, dc, u0 + l32) : -1;
    u32x4 bx[KS];
    gather<CIN, KSZ>(g, planes, p, valid, half, bx);
    if (half == 0) ((__attribute__((address_space(3))) int*)prow)[l32] = (int)p;
    // channel halves of 64 (NH blocks of 32) one after the other: fewer
    // live accumulators, more waves per SIMD to hide the gathers
    constexpr int NH = NB < 2 ? NB : 2;
#pragma unroll
    for (int h0 = 0; h0 < NB; h0 += NH) {
      if (h0 < hb || h0 >= he) continue;  // uniform per wave
      f32x16 acc[NH];
#pragma unroll
      for (int nb = 0; nb < NH; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[nb][v] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int nb = 0; nb < NH; ++nb) {
          const u32x4 wf = *(const lds_u32x4*)(smem + ((ks * NBS + h0 + nb - sb0) * 64 + lane) * 16);
          acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wf),
                                                            __builtin_bit_cast(bf16x8, bx[ks]), acc[nb], 0, 0, 0);
        }
      // epilogue of these channels: lane holds co .. co + 3 (co = 32 nb +
      // 8 q + 4 half) of voxel row l32
#pragma unroll
      for (int nb = 0; nb < NH; ++nb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int co = (h0 + nb) * 32 + q * 8 + half * 4;
          const float v0 = act_fn<ACT>(acc[nb][4 * q + 0] + bias[co + 0]);
          const float v1 = act_fn<ACT>(acc[nb][4 * q + 1] + bias[co + 1]);
          const float v2 = act_fn<ACT>(acc[nb][4 * q + 2] + bias[co + 2]);
          const float v3 = act_fn<ACT>(acc[nb][4 * q + 3] + bias[co + 3]);
          if constexpr (F8) {
            *(lds_u32_w*)(tile + l32 * OSTR + co) = e4m3_pack4(v0, v1, v2, v3);
          } else {
            u32x2 packed;
            packed.x = bf16_pack(v0, v1);
            packed.y = bf16_pack(v2, v3);
            *(lds_u32x2_w*)(tile + l32 * OSTR + co * 2) = packed;
          }
        }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's tile is in LDS
    __builtin_amdgcn_wave_barrier();
    // the unit's part of each row: 32 rows x gpp granules of 16 bytes, 64
    // lanes at a time
    const int gpp = GPR / hsplit, c0 = part * gpp;
#pragma unroll
    for (int k = 0; k < 32 * GPR / 64; ++k) {
      if (k * 64 >= 32 * gpp) break;  // uniform
      const int qq = k * 64 + lane;
      const int row = qq / gpp, c = c0 + qq % gpp;
      const int pr = ((__attribute__((address_space(3))) const int*)prow)[row];
      const u32x4 val = *(lds_u32x4*)(tile + row * OSTR + c * 16);
      if (pr >= 0) *reinterpret_cast<u32x4*>((char*)y + (long long)pr * ystride * ESZ + c * 16) = val;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // the tile's LDS reads are done before the next block writes it
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace

hipError_t launch_conv_first(const Geom& g, int cin, int cout, int act, const void* planes, void* y, int ystride,
                             const void* wfrag, const float* bias, int batch, int fp8, int ks, hipStream_t stream) {
  const long long nvox = (long long)batch * g.V;  // < 2^31 (host check)
  if ((cin != 2 && cin != 4) || (cout != 64 && cout != 128) || act < 0 || act > 2) return hipErrorInvalidValue;
  if ((ks != 3 && ks != 5) || (ks - 1) / 2 > g.pad || (ks == 5 && (cin != 4 || fp8))) return hipErrorInvalidValue;
  const int WAVES = 4;
  int bpw, hsplit;
  long long nblk;
  if (ks == 3) {
    // two blocks per wave amortise the weight staging once the launch has
    // 512 or more workgroups of them; below that (small batches) one block
    // per wave doubles the waves on a mostly idle chip
    bpw = nvox >= 512LL * 32 * WAVES * BPW ? BPW : 1;
    // ... and below 256 workgroups of single blocks, 128-channel layers
    // split each block's channels over two waves
    hsplit = (bpw == 1 && cout == 128 && nvox < 256LL * 32 * WAVES) ? 2 : 1;
    nblk = (nvox * hsplit + 32 * WAVES * bpw - 1) / (32 * WAVES * bpw);
  } else {
    // 5x5x5: workgroups of one 64-channel part; up to 8 blocks per wave while
    // the launch keeps 1024 or more workgroups
    hsplit = cout / 64;
    const long long blocks = (nvox + 31) / 32;
    bpw = (int)std::max(1LL, std::min(8LL, blocks * hsplit / (1024LL * WAVES)));
    nblk = (blocks + (long long)WAVES * bpw - 1) / ((long long)WAVES * bpw) * hsplit;
  }
  Decode dc;
  dc.by_v = make_fastdiv((uint32_t)g.V);
  dc.by_hh = make_fastdiv((uint32_t)(g.H * g.H));
  dc.by_h = make_fastdiv((uint32_t)g.H);
  auto launch = [&](auto CI, auto CO, auto A, auto K) {
    constexpr int C = decltype(CO)::value, I = decltype(CI)::value, KZ = decltype(K)::value;
    constexpr int W = waves<KZ, C>();
    constexpr int NBS = KZ == 5 ? 2 : C / 32;  // staged 32-channel blocks (5x5x5: one 64-channel part)
    const size_t lds = (size_t)ksteps<I, KZ>() * NBS * 64 * 16 + (size_t)W * 32 * (C * 2 + 16 + 4);
    static_assert(ksteps<I, KZ>() * NBS * 64 * 16 + W * 32 * (C * 2 + 16 + 4) <= 160 * 1024, "LDS");
    if constexpr (KZ == 5) {  // bf16 only; more than 64 KB of LDS
      if (hipFuncSetAttribute((const void*)conv_first_kernel<I, C, decltype(A)::value, false, KZ>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return;
      hipLaunchKernelGGL((conv_first_kernel<I, C, decltype(A)::value, false, KZ>), dim3((unsigned)nblk),
                         dim3(64 * W), lds, stream, g, planes, y, ystride, (const u32x4*)wfrag, bias, dc, (int)nvox,
                         bpw, hsplit);
    } else if (fp8) {
      hipLaunchKernelGGL((conv_first_kernel<I, C, decltype(A)::value, true, KZ>), dim3((unsigned)nblk), dim3(64 * W),
                         lds, stream, g, planes, y, ystride, (const u32x4*)wfrag, bias, dc, (int)nvox, bpw, hsplit);
    } else {
      hipLaunchKernelGGL((conv_first_kernel<I, C, decltype(A)::value, false, KZ>), dim3((unsigned)nblk),
                         dim3(64 * W), lds, stream, g, planes, y, ystride, (const u32x4*)wfrag, bias, dc, (int)nvox,
                         bpw, hsplit);
    }
  };
  with_activation(act, [&](auto A) {
    using I2 = std::integral_constant<int, 2>;
    using I4 = std::integral_constant<int, 4>;
    using C64 = std::integral_constant<int, 64>;
    using C128 = std::integral_constant<int, 128>;
    using K3 = std::integral_constant<int, 3>;
    using K5 = std::integral_constant<int, 5>;
    if (ks == 3) {
      if (cin == 2 && cout == 64) launch(I2(), C64(), A, K3());
      if (cin == 2 && cout == 128) launch(I2(), C128(), A, K3());
      if (cin == 4 && cout == 64) launch(I4(), C64(), A, K3());
      if (cin == 4 && cout == 128) launch(I4(), C128(), A, K3());
    } else {
      if (cout == 64) launch(I4(), C64(), A, K5());
      if (cout == 128) launch(I4(), C128(), A, K5());
    }
  });
  return hipGetLastError();
}

}  // namespace pd
