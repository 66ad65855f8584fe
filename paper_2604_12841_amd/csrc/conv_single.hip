// conv_single.hip -- K2 + K4 for a network with a single hidden layer: the
// first 3x3x3 conv3d layer (Sec. IV.B, Fig. ConvArch; c_in = 2 detector
// channels -> c_out = 64 or 128; stride 1, zero padding, cross-correlation)
// on the gfx950 matrix cores, whose epilogue applies bias + activation,
// rounds to bf16, then applies the 1x1x1 head and the threshold (logit > 0)
// and writes one flip nibble per voxel.  (With more hidden layers, layer 1
// is conv_first.hip and the others conv_hidden.hip.)
//
//   out[co][m] = act(bias[co] + sum_{tap, ci} W[co][ci][tap] * X[m + shift(tap)][ci])
//
// GEMM view (transposed so the epilogue holds 4 consecutive channels per
// lane): rows = c_out, columns = output voxels, K = 27 taps x 2 channels
// padded to 64 (4 k-steps of v_mfma_f32_32x32x16_bf16; taps past 26 are
// zero weights).
//
// Work split: persistent workgroups of 512 threads (8 wave64), one per CU.
// A tile is 256 output voxels x all c_out channels; wave w owns 32 channels
// (w / WM) of ROWS voxels.  The tile's input planes (both bf16 channels of a
// voxel in 4 bytes) are staged in LDS with the tilings of tiles.h, double
// buffered: the next tile's planes are loaded into registers while this tile
// computes.  Each lane gathers its B fragment (4 taps x 2 channels) from the
// staged planes; taps on a flat tile's halo columns read as zero.
#include "activation.h"
#include "internal.h"
#include "tiles.h"

namespace pd {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const uint32_t lds_u32;
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) uint32_t lds_u32_w;

constexpr int NT = 512;                 // threads per workgroup: 8 wave64
constexpr int PLANE_RMAX = 2;           // staging rounds of NT voxels x 4 bytes
constexpr int MAX_SPAN = PLANE_RMAX * NT;
constexpr int ABUF = MAX_SPAN * 4;      // bytes per staging buffer

// Wave split of the 256 x COUT output tile: WN waves across the channels (32
// each), WM across the voxels (ROWS each, MB blocks of 32).
template <int COUT>
struct Split {
  static constexpr int WN = COUT / 32;
  static constexpr int WM = (NT / 64) / WN;
  static constexpr int ROWS = kTileRows / WM;
  static constexpr int MB = ROWS / 32;
  static_assert(WM * WN * 64 == NT && WM * MB * 32 == kTileRows, "wave split");
};

// LDS layout of one workgroup (byte offsets): two staging buffers, the
// destination of the staging past the last tile, the bias [COUT], the head
// weights [4][COUT] and the head partial sums [WN][256][4].
template <int COUT>
struct Lds {
  static constexpr int trash = 2 * ABUF;
  static constexpr int bias = trash + NT * 4;
  static constexpr int headw = bias + COUT * 4;
  static constexpr int part = headw + 4 * COUT * 4;
  static constexpr int total = part + Split<COUT>::WN * kTileRows * 4 * 4;
  static_assert(total <= 64 * 1024, "LDS budget");
};

// Both channels (4 bytes) of staged voxel NT k + tid (voxel 0, a zero halo
// voxel, past the footprint).
__device__ __forceinline__ uint32_t plane_load(const Geom& g, const Tiling& tl, const uint32_t* __restrict__ planes,
                                               const StageSrc& src, long long limit, int k, int tid) {
  const int vv = k * NT + tid;
  return planes[staged_voxel(g, tl, src.origin, src.bo, vv < tl.span ? vv : 0, limit)];
}

template <int COUT, int MODE>
__global__ void __launch_bounds__(NT) conv_single_kernel(Geom g, Tiling tl, int act,
                                                         const uint32_t* __restrict__ planes,
                                                         const u32x4* __restrict__ wfrag,
                                                         const float* __restrict__ bias,
                                                         const float* __restrict__ head_w,
                                                         const float* __restrict__ head_b,
                                                         const int32_t* __restrict__ tables,
                                                         uint8_t* __restrict__ nib, float* __restrict__ logits,
                                                         int batch) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  using W = Split<COUT>;
  using L = Lds<COUT>;
  constexpr int MB = W::MB;
  constexpr int NBT = COUT / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % W::WM, wn = wave / W::WM;
  const int half = lane >> 5, l32 = lane & 31;
  const int ntiles = (int)tl.ntiles;
  const long long limit = (long long)batch * g.S;

  lds_char* const lds = (lds_char*)smem;
  lds_float* const bias_s = (lds_float*)(lds + L::bias);
  lds_float* const headw_s = (lds_float*)(lds + L::headw);
  lds_float* const head_part = (lds_float*)(lds + L::part);
  for (int e = tid; e < COUT; e += NT) bias_s[e] = bias[e];
  for (int e = tid; e < 4 * COUT; e += NT) headw_s[e] = head_w[e];

  int tile = tile_of(blockIdx.x, gridDim.x, 0, ntiles);
  if (tile < 0) return;

  auto source_of = [&](int t) { return tile_source(g, tl, t, batch); };

  // First tile: stage its planes synchronously.
  {
    const StageSrc src = source_of(tile);
#pragma unroll
    for (int k = 0; k < PLANE_RMAX; ++k)
      *(lds_u32_w*)(lds + (k * NT + tid) * 4) = plane_load(g, tl, planes, src, limit, k, tid);
  }
  // This wave's weight fragments (4 k-steps of its 32 channels): the same
  // for every tile.
  u32x4 wf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) wf[ks] = wfrag[(ks * NBT + wn) * 64 + lane];
  __syncthreads();  // staged planes, bias and head weights visible

  int gbuf = 0;  // staging buffer of the current tile
  for (int it = 0; tile >= 0; ++it) {
    const int next = tile_of(blockIdx.x, gridDim.x, it + 1, ntiles);
    const StageSrc next_src = source_of(next >= 0 ? next : tile);
    // rows of this lane: voxel wm ROWS + 32 mb + l32 of the tile
    int rb[MB];
    bool zl[MB], zr[MB];  // flat tiles: the row is in the first / last column
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      long long p = -1, o;
      int lb = 0, col = -1;
      tile_row(g, tl, tile, wm * W::ROWS + mb * 32 + l32, batch, &p, &lb, &o, &col);
      rb[mb] = lb;
      zl[mb] = MODE == 0 && col == 0;
      zr[mb] = MODE == 0 && col == g.H - 1;
    }
    // next tile's planes into registers while this tile computes
    uint32_t nxt[PLANE_RMAX];
#pragma unroll
    for (int k = 0; k < PLANE_RMAX; ++k) nxt[k] = plane_load(g, tl, planes, next_src, limit, k, tid);

    lds_u32* const a32 = (lds_u32*)(lds + gbuf * ABUF);
    f32x16 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][v] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        u32x4 av;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int tap = ks * 8 + half * 4 + q;  // k = 2 tap + channel
          uint32_t val = 0;
          if (tap < 27) {
            const int dt = tap / 9, di = (tap / 3) % 3, dj = tap % 3;
            val = a32[rb[mb] + dt * tl.sa + di * tl.sb + dj];
            if ((dj == 0 && zl[mb]) || (dj == 2 && zr[mb])) val = 0;
          }
          av[q] = val;
        }
        acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wf[ks]),
                                                          __builtin_bit_cast(bf16x8, av), acc[mb], 0, 0, 0);
      }
    // the other buffer (the scratch round past the last tile); every wave
    // finished reading it before the previous tile's epilogue barriers
    lds_char* const oth = next >= 0 ? lds + (gbuf ^ 1) * ABUF : lds + L::trash;
#pragma unroll
    for (int k = 0; k < PLANE_RMAX; ++k) *(lds_u32_w*)(oth + ((next >= 0 ? k * NT : 0) + tid) * 4) = nxt[k];

    // ---- epilogue: lane holds channels co .. co + 3 (co = 32 wn + 8 q +
    // 4 half) of voxel row wm ROWS + 32 mb + l32.  1x1x1 head on the
    // bf16-rounded activations: partial sums over this lane's channels, then
    // over the half-waves, then over the channel waves through LDS ----
    float part[MB][4];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int o = 0; o < 4; ++o) part[mb][o] = 0.0f;
    with_activation(act, [&](auto A) {
      constexpr int ACT = decltype(A)::value;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int co = wn * 32 + q * 8 + half * 4;
        const float4 bv = {bias_s[co], bias_s[co + 1], bias_s[co + 2], bias_s[co + 3]};
        float4 hw[4];
#pragma unroll
        for (int o = 0; o < 4; ++o)
          hw[o] = {headw_s[o * COUT + co], headw_s[o * COUT + co + 1], headw_s[o * COUT + co + 2],
                   headw_s[o * COUT + co + 3]};
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const float a0 = bf16_round(act_fn<ACT>(acc[mb][4 * q + 0] + bv.x));
          const float a1 = bf16_round(act_fn<ACT>(acc[mb][4 * q + 1] + bv.y));
          const float a2 = bf16_round(act_fn<ACT>(acc[mb][4 * q + 2] + bv.z));
          const float a3 = bf16_round(act_fn<ACT>(acc[mb][4 * q + 3] + bv.w));
#pragma unroll
          for (int o = 0; o < 4; ++o) part[mb][o] += hw[o].x * a0 + hw[o].y * a1 + hw[o].z * a2 + hw[o].w * a3;
        }
      }
    });
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int o = 0; o < 4; ++o) part[mb][o] += __shfl_xor(part[mb][o], 32);
    if (half == 0) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        lds_float* hp = head_part + (wn * kTileRows + wm * W::ROWS + mb * 32 + l32) * 4;
        hp[0] = part[mb][0];
        hp[1] = part[mb][1];
        hp[2] = part[mb][2];
        hp[3] = part[mb][3];
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): partials and next planes written
    __builtin_amdgcn_s_barrier();
    // one thread per voxel row: logits, threshold, flip nibble
    if (tid < kTileRows) {
      const int r = tid;
      int b, t, i, j;
      if (tile_row_coords(g, tl, tile, r, batch, &b, &t, &i, &j)) {
        float lg[4] = {head_b[0], head_b[1], head_b[2], head_b[3]};
#pragma unroll
        for (int w2 = 0; w2 < W::WN; ++w2) {
          const lds_float* hp = head_part + (w2 * kTileRows + r) * 4;
          lg[0] += hp[0];
          lg[1] += hp[1];
          lg[2] += hp[2];
          lg[3] += hp[3];
        }
        const int HH = g.H * g.H;
        const int s = i * g.H + j;
        nib[(long long)b * g.V + (long long)t * HH + s] = (uint8_t)flip_nibble(g, tables, i, j, lg);
        if (logits) {
#pragma unroll
          for (int o = 0; o < 4; ++o) logits[(((long long)b * 4 + o) * g.T + t) * HH + s] = lg[o];
        }
      }
    }
    // partials read before the next tile writes them
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
    tile = next;
    gbuf ^= 1;
  }
}

template <int COUT, int MODE>
hipError_t launch_one(const Geom& g, const Tiling& tl, int act, const void* planes, const void* wfrag,
                      const float* bias, const float* head_w, const float* head_b, const int32_t* tables,
                      uint8_t* nib, float* logits, int batch, int n_workgroups, hipStream_t stream) {
  const long long nwg = conv_workgroups(tl.ntiles, n_workgroups);
  hipLaunchKernelGGL((conv_single_kernel<COUT, MODE>), dim3((unsigned)nwg), dim3(NT), (size_t)Lds<COUT>::total,
                     stream, g, tl, act, (const uint32_t*)planes, (const u32x4*)wfrag, bias, head_w, head_b,
                     tables, nib, logits, batch);
  return hipGetLastError();
}

}  // namespace

int conv_single_max_span() { return MAX_SPAN; }

hipError_t launch_conv_single(const Geom& g, const Tiling& tl, int cout, int act, const void* planes,
                              const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                              const int32_t* tables, uint8_t* nib, float* logits, int batch,
                              int n_workgroups, hipStream_t stream) {
  if (tl.span <= 0 || tl.span > MAX_SPAN) return hipErrorInvalidValue;
  if (cout == 64)
    return tl.mode == 0 ? launch_one<64, 0>(g, tl, act, planes, wfrag, bias, head_w, head_b, tables, nib,
                                            logits, batch, n_workgroups, stream)
                        : launch_one<64, 1>(g, tl, act, planes, wfrag, bias, head_w, head_b, tables, nib,
                                            logits, batch, n_workgroups, stream);
  if (cout == 128)
    return tl.mode == 0 ? launch_one<128, 0>(g, tl, act, planes, wfrag, bias, head_w, head_b, tables, nib,
                                             logits, batch, n_workgroups, stream)
                        : launch_one<128, 1>(g, tl, act, planes, wfrag, bias, head_w, head_b, tables, nib,
                                             logits, batch, n_workgroups, stream);
  return hipErrorInvalidValue;
}

}  // namespace pd
