// conv_hidden.hip -- K3 (+ K4 for the last layer): a hidden 3x3x3 conv3d
// layer, c_in = 64 or 128 -> c_out = 64 or 128 (Sec. IV.B, Fig. ConvArch;
// stride 1, zero padding, cross-correlation) as an implicit GEMM on the
// gfx950 matrix cores, with the bias + activation + bf16 rounding epilogue
// fused in; for the last hidden layer the epilogue also applies the 1x1x1
// head and the threshold (logit > 0) and writes one flip nibble per voxel.
//
//   out[co][m] = act(bias[co] + sum_{tap, ci} W[co][ci][tap] * X[m + shift(tap)][ci])
//
// GEMM view (transposed so the epilogue holds 4 consecutive channels per
// lane): rows = c_out, columns = output voxels, K = 27 * c_in; weights are
// the A operand, activations the B operand of v_mfma_f32_32x32x16_bf16.
// Activations live in the zero-halo NTHWC layout of internal.h, so every tap
// is an index shift and the K loop has no bounds checks.
//
// Work split: persistent workgroups of 256 threads (4 wave64), two per CU, so
// each SIMD runs one wave of each and one workgroup's epilogue, barriers and
// staging stalls overlap the other's matrix work.  A tile is 256 output voxels
// x all c_out channels; a wave owns 128 voxels x 64 channels for c_out = 128
// (64 x 64 for c_out = 64): 4 (2) voxel blocks x 2 channel blocks of MFMA
// with fp32 accumulators, so each activation fragment read from LDS feeds two
// MFMAs and each weight fragment MB.
//   * The tile's input footprint is staged in LDS 16 input channels (32
//     bytes per voxel) at a time, double buffered, through registers: the
//     next chunk -- or, during the last chunk, the next tile's first chunk --
//     is loaded in 7 rounds spread over the current chunk's 27 k-steps (one
//     per tap) and written to the other buffer.
//   * A staged voxel occupies 48 bytes of LDS.  The LDS serves a 16-byte read
//     16 lanes at a time over 16 groups of 16 bytes; granule g of voxel v sits
//     in group (3 v + g) mod 16, so 16 consecutive staged voxels hit 16
//     distinct groups.  Flat tiles stage only the real columns; reads of the
//     left / right halo column are redirected to a 256-byte zero region with
//     the same low address bits (same group).
//   * The 27 k-steps of a chunk are unrolled and software pipelined:
//     activation fragments are read one step ahead, weight fragments
//     (arranged at create time in MFMA operand order, one coalesced 16-byte
//     load per lane; a layer is <= 0.9 MB and stays in L2) two steps ahead
//     through a 3-deep register ring that runs on across chunks and tiles.
//   * Epilogue: + bias, activation in fp32, bf16 (RNE); each wave transposes
//     its rows through its own slice of the staging buffer the tile read last
//     and writes whole 128-byte lines.  No barrier ends the tile: a wave
//     starts the next one at once, and only that tile's first staging store
//     (three k-steps in) waits for the others to leave the buffer.
#include "activation.h"
#include "internal.h"
#include "tiles.h"

namespace pd {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_w;
typedef __attribute__((address_space(3))) uint32_t lds_u32_w;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2_w;

constexpr int NT = 256;       // threads per workgroup: 4 wave64
constexpr int KC = 16;        // input channels per LDS chunk (one MFMA k-step)
constexpr int STEPS = 27;     // k-steps per chunk: one per tap
constexpr int BRING = 3;      // weight-fragment ring depth (prefetch distance BRING - 1)
constexpr int VSTRIDE = 48;   // LDS bytes per staged voxel (32 of channels + 16 of padding)
constexpr int BUF_VOX = 800;            // staged voxels a staging buffer holds
constexpr int MAX_SPAN = BUF_VOX - 1;    // staged voxels per tile (the last slot takes overflow writes)
// Every chunk is staged with RMAX rounds of NT 16-byte granules, stored
// unconditionally (a conditional store would let the compiler sink the load
// next to it): granules past the footprint load zeros into slots past the
// footprint, and granules past the buffer all go to its last slot.
constexpr int RMAX = 7;
static_assert(RMAX * NT >= 2 * MAX_SPAN && (RMAX * NT) % 32 == 0, "staging rounds cover the largest footprint");
static_assert(STEPS % BRING == 0, "the weight ring lines up with chunk boundaries");
static_assert(RMAX * 3 + 3 <= STEPS, "staging rounds fit in a chunk");
constexpr int ABUF = BUF_VOX * VSTRIDE;  // bytes per staging buffer

// Staging granule q = NT k + tid: in each run of 32, the first 16 take
// granule 0 of 16 consecutive staged voxels and the next 16 their granule 1,
// so the 16 lanes of an LDS write cycle hit 16 distinct bank groups.
__host__ __device__ inline int stage_voxel(int q) { return ((q >> 5) << 4) | (q & 15); }
__host__ __device__ inline int stage_gran(int q) { return (q >> 4) & 1; }

// LDS byte (relative to a staging buffer) of staging granule q; voxels past
// the buffer all go to its last slot.
__host__ __device__ inline int stage_slot(int q) {
  const int v = stage_voxel(q);
  return (v < BUF_VOX - 1 ? v : BUF_VOX - 1) * VSTRIDE + stage_gran(q) * 16;
}

// Epilogue modes: the activations of a hidden layer, a hidden layer with the
// 1x1x1 head fused in, or the 3x3x3 output layer itself (4 filters, padded to
// one block of 32 MFMA rows); EPI_PARK: one part of a split K loop, whose
// fp32 sums are parked for split_finish_kernel.  Only EPI_PARK kernels split
// (the others see a split of 1 at compile time and keep their registers for
// the epilogue).
enum Epi { EPI_ACT = 0, EPI_HEAD = 1, EPI_OUT = 2, EPI_PARK = 3 };

// Wave split of the 256 x COUT output tile: WN waves across the channels
// (NB blocks of 32 each: 2, or 1 for the 32-row output layer), WM across the
// voxels (ROWS each, MB blocks of 32).
template <int COUT>
struct Split {
  static constexpr int NB = COUT >= 64 ? 2 : 1;
  static constexpr int WN = COUT / (32 * NB);
  static constexpr int WM = (NT / 64) / WN;
  static constexpr int ROWS = kTileRows / WM;
  static constexpr int MB = ROWS / 32;
  static_assert(WM * WN * 64 == NT && WN * NB * 32 == COUT && WM * MB * 32 == kTileRows, "wave split");
  static_assert(MB % 2 == 0, "the epilogue transposes row blocks in pairs");
};

// LDS layout of one workgroup (byte offsets): two staging buffers, a
// 256-byte zero region (256-aligned, for halo-column reads), the bias
// [COUT] and the head weights [4][COUT].  The head epilogue puts its
// partial sums in the staging buffer the tile read last.
template <int COUT>
struct Lds {
  static constexpr int zero = 2 * ABUF;
  static constexpr int bias = zero + 256;
  static constexpr int headw = bias + COUT * 4;
  static constexpr int total = headw + 4 * COUT * 4;
  static_assert(zero % 256 == 0, "zero region must be 256-aligned");
  static_assert(2 * total <= 160 * 1024, "two workgroups per CU");
  static_assert(Split<COUT>::WN * kTileRows * 4 * 4 <= ABUF, "head partials fit a staging buffer");
  static_assert((NT / 64) * 64 * 128 <= ABUF, "epilogue transposition slices fit a staging buffer");
};

// Staging granule q = NT k + tid is granule stage_gran(q) (16 bytes) of
// staged voxel stage_voxel(q), bound for LDS byte stage_slot(q).  The loads are
// buffer loads relative to the tile's staging base (a padded voxel index no
// larger than any voxel the tile stages): per round, a lane's byte offset is
// the same for every chunk of the tile.  Granules past the footprint, and
// voxels outside the volume, get an offset past the buffer's range, for
// which the load returns zeros.
constexpr uint32_t kNoVoxel = 0x80000000u;
constexpr uint32_t kStageRange = 0x7FFFFFF0u;  // buffer range in bytes; every real offset is far below

// A value the whole wave agrees on, marked as such for the compiler (the
// 64-bit index arithmetic would otherwise leave it in vector registers, and
// a buffer resource built from it would need a per-lane loop).
__host__ __device__ inline long long wave_uniform(long long v) {
#ifndef __HIP_DEVICE_COMPILE__
  return v;
#else
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((unsigned long long)v >> 32));
  return (long long)(((unsigned long long)hi << 32) | lo);
#endif
}

template <int MODE>
__host__ __device__ inline long long stage_base(const Geom& g, const StageSrc& src) {
  if constexpr (MODE == 0) return wave_uniform(src.origin <= 0 ? 0 : line_to_padded(g, src.origin));
  return wave_uniform(src.origin);
}

template <int CIN, int MODE>
__host__ __device__ inline uint32_t stage_offset(const Geom& g, const Tiling& tl, const StageSrc& src,
                                                 long long base, long long limit, int span, int k, int tid) {
  const int q = k * NT + tid;
  const int vv = stage_voxel(q);
  const long long gv = staged_voxel_fast<MODE>(g, tl, src, vv, limit);
  return (vv < span && gv >= 0) ? (uint32_t)((gv - base) * (CIN * 2) + stage_gran(q) * 16) : kNoVoxel;
}

// Buffer resource over the activations from padded voxel `base`, channel
// offset `ch` on.
template <int CIN>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stage_rsrc(const uint16_t* x, long long base, int ch) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)(x + base * CIN + ch), 0, kStageRange, 0x00020000);
}

template <int CIN, int COUT, int EPI, int MODE>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
conv_hidden_kernel(Geom g, Tiling tl, int act, const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                   int ystride, const u32x4* __restrict__ wfrag, const float* __restrict__ bias,
                   const float* __restrict__ head_w, const float* __restrict__ head_b,
                   const int32_t* __restrict__ tables, uint8_t* __restrict__ nib,
                   float* __restrict__ logits, int batch, int kshift_arg, float* __restrict__ partial) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  using W = Split<COUT>;
  using L = Lds<COUT>;
  constexpr int MB = W::MB;
  constexpr int NB = W::NB;
  constexpr int NBT = COUT / 32;  // 32-channel blocks in total
  constexpr int NCHUNK = CIN / KC;
  constexpr int TSTEPS = NCHUNK * STEPS;  // k-steps of the layer
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % W::WM, wn = wave / W::WM;
  const int half = lane >> 5, l32 = lane & 31;
  const int ntiles = (int)tl.ntiles;
  const long long limit = (long long)batch * g.S;
  // Work units: (tile, part); part p of a tile runs its chunks [p NCU, (p+1) NCU)
  // with ksplit = 2^kshift parts per tile (EPI_PARK only: small batches).
  // With parts, each unit parks its fp32 sums in `partial` (unit u at
  // u * 256 * COUT floats) and split_finish_kernel does the epilogue.
  const int kshift = EPI == EPI_PARK ? kshift_arg : 0;
  const int ksplit = 1 << kshift;
  const int NCU = NCHUNK >> kshift;  // chunks per unit
  const int nunits = ntiles << kshift;

  lds_char* const lds = (lds_char*)smem;
  lds_char* const zero = lds + L::zero;
  lds_float* const bias_s = (lds_float*)(lds + L::bias);
  lds_float* const headw_s = (lds_float*)(lds + L::headw);
  for (int e = tid; e < COUT; e += NT) bias_s[e] = bias[e];
  if (tid < 64) ((lds_u32_w*)zero)[tid] = 0u;
  const uint32_t zero_addr = (uint32_t)(uintptr_t)zero;
  if (EPI == EPI_HEAD)
    for (int e = tid; e < 4 * COUT; e += NT) headw_s[e] = head_w[e];

  // Bias, activation and output of one tile from its accumulators (lane
  // holds channels co .. co + 3, co = 64 wn + 32 nb + 8 q + 4 half, of voxel
  // row wm ROWS + 32 mb + l32); ebuf: a staging buffer free for the
  // transposition / head partials.
  auto finish_tile = [&](int tile, lds_char* const ebuf, f32x16 (&acc)[MB][NB]) {
      // output row of each row block (recomputed: not kept live through the K loop)
      int pidx[MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        long long p = -1, o;
        int lb;
        pidx[mb] = tile_row(g, tl, tile, wm * W::ROWS + mb * 32 + l32, batch, &p, &lb, &o) ? (int)p : -1;
      }

      // ---- epilogue: lane holds channels co .. co + 3 (co = 64 wn + 32 nb +
      // 8 q + 4 half) of voxel row wm ROWS + 32 mb + l32 ----
      if constexpr (EPI == EPI_OUT) {
        // the output layer: rows 0..3 of the channel block are the four logits
        // (+ bias, no activation), held by the lanes of the first half-wave
        if (half == 0) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            int b, t, i, j;
            if (tile_row_coords(g, tl, tile, wm * W::ROWS + mb * 32 + l32, batch, &b, &t, &i, &j)) {
              const float lg[4] = {acc[mb][0][0] + bias_s[0], acc[mb][0][1] + bias_s[1], acc[mb][0][2] + bias_s[2],
                                   acc[mb][0][3] + bias_s[3]};
              const int HH = g.H * g.H;
              const int s = i * g.H + j;
              nib[(long long)b * g.V + (long long)t * HH + s] = (uint8_t)flip_nibble(g, tables, i, j, lg);
              if (logits) {
#pragma unroll
                for (int o = 0; o < 4; ++o) logits[(((long long)b * 4 + o) * g.T + t) * HH + s] = lg[o];
              }
            }
          }
        }
      } else if constexpr (EPI == EPI_ACT) {
        // bias + activation + bf16, transposed through this wave's slice of
        // the staging buffer the tile read last (64 rows x 128 bytes, granule
        // c of row r at c ^ (r % 8)), then stored as whole 128-byte halves of
        // voxel rows, 8 rows per instruction.  The next tile's first staging
        // store waits at a barrier until every wave is done here.
        lds_char* const tb = ebuf + wave * (64 * 128);
        with_activation(act, [&](auto A) {
          constexpr int ACT = decltype(A)::value;
#pragma unroll
          for (int ps = 0; ps < MB / 2; ++ps) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int c = nb * 4 + q;  // 16-byte granule of the wave's 64 channels
                const int co = wn * 64 + c * 8 + half * 4;
                const float4 bv = {bias_s[co], bias_s[co + 1], bias_s[co + 2], bias_s[co + 3]};
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                  const int mb = 2 * ps + m;
                  const float v0 = act_fn<ACT>(acc[mb][nb][4 * q + 0] + bv.x);
                  const float v1 = act_fn<ACT>(acc[mb][nb][4 * q + 1] + bv.y);
                  const float v2 = act_fn<ACT>(acc[mb][nb][4 * q + 2] + bv.z);
                  const float v3 = act_fn<ACT>(acc[mb][nb][4 * q + 3] + bv.w);
                  u32x2 packed;
                  packed.x = bf16_pack(v0, v1);
                  packed.y = bf16_pack(v2, v3);
                  const int r = m * 32 + l32;
                  *(lds_u32x2_w*)(tb + r * 128 + ((c ^ (r & 7)) << 4) + half * 8) = packed;
                }
              }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's rows are in LDS
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int it2 = 0; it2 < 8; ++it2) {
              const int gi = it2 * 64 + lane;
              const int r = gi >> 3, c = gi & 7;
              const u32x4 v = *(lds_u32x4*)(tb + r * 128 + ((c ^ (r & 7)) << 4));
              const int pr = __shfl(pidx[2 * ps + (it2 >> 2)], r & 31);
              if (pr >= 0) *reinterpret_cast<u32x4*>(y + (long long)pr * ystride + wn * 64 + c * 8) = v;
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // the reads are done before the next pass writes
            __builtin_amdgcn_wave_barrier();
          }
        });
      } else {
        // 1x1x1 head on the bf16-rounded activations: partial sums over this
        // lane's channels, then over the half-waves, then over the channel
        // waves through LDS (the buffer this tile read last)
        lds_float* const head_part = (lds_float*)(ebuf);  // [WN][256][4]
        float part[MB][4];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int o = 0; o < 4; ++o) part[mb][o] = 0.0f;
        with_activation(act, [&](auto A) {
          constexpr int ACT = decltype(A)::value;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int co = (wn * NB + nb) * 32 + q * 8 + half * 4;
              const float4 bv = {bias_s[co], bias_s[co + 1], bias_s[co + 2], bias_s[co + 3]};
              float4 hw[4];
#pragma unroll
              for (int o = 0; o < 4; ++o)
                hw[o] = {headw_s[o * COUT + co], headw_s[o * COUT + co + 1], headw_s[o * COUT + co + 2],
                         headw_s[o * COUT + co + 3]};
#pragma unroll
              for (int mb = 0; mb < MB; ++mb) {
                const float a0 = bf16_round(act_fn<ACT>(acc[mb][nb][4 * q + 0] + bv.x));
                const float a1 = bf16_round(act_fn<ACT>(acc[mb][nb][4 * q + 1] + bv.y));
                const float a2 = bf16_round(act_fn<ACT>(acc[mb][nb][4 * q + 2] + bv.z));
                const float a3 = bf16_round(act_fn<ACT>(acc[mb][nb][4 * q + 3] + bv.w));
#pragma unroll
                for (int o = 0; o < 4; ++o)
                  part[mb][o] += hw[o].x * a0 + hw[o].y * a1 + hw[o].z * a2 + hw[o].w * a3;
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
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): partials written
        __builtin_amdgcn_s_barrier();
        // one thread per voxel row: logits, threshold, flip nibble
        static_assert(NT == kTileRows, "one thread per tile row");
        {
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
      }
  };

  int unit = tile_of(blockIdx.x, gridDim.x, 0, nunits);
  if (unit < 0) return;
  int tile = unit >> kshift;

  auto source_of = [&](int t) {
    StageSrc src;
    long long p;
    int lb;
    tile_row(g, tl, t, 0, batch, &p, &lb, &src.origin);
    src.bo = box_origin(g, tl, src.origin);
    return src;
  };
  long long cur_base = stage_base<MODE>(g, source_of(tile));
  uint32_t soff[RMAX];  // this lane's staging offsets of the tile being staged
  {
    const StageSrc src = source_of(tile);
#pragma unroll
    for (int k = 0; k < RMAX; ++k) soff[k] = stage_offset<CIN, MODE>(g, tl, src, cur_base, limit, tl.span, k, tid);
  }

  // First tile: stage its first chunk synchronously.
  {
    const __amdgpu_buffer_rsrc_t rs = stage_rsrc<CIN>(x, cur_base, (unit & (ksplit - 1)) * NCU * KC);
#pragma unroll
    for (int k = 0; k < RMAX; ++k) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, soff[k], 0, 0);
      *(lds_u32x4_w*)(lds + stage_slot(k * NT + tid)) = v;
    }
  }

  // weight fragment (tile-step gs, block nb of this wave's channels): a
  // buffer load with this lane's 16-byte slot as the vector offset and the
  // fragment's offset as the scalar one (no per-load address arithmetic)
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc((void*)wfrag, 0, TSTEPS * NBT * 1024, 0x00020000);
  const uint32_t woff = (uint32_t)((wn * NB * 64 + lane) * 16);
  auto wload = [&](int gs, int nb) -> u32x4 {
    return __builtin_amdgcn_raw_buffer_load_b128(wres, woff, (gs * NBT + nb) * 1024, 0);
  };
  // weight-fragment ring: slot k holds the k-step gs (of the layer's
  // NCHUNK x 27), gs % BRING == k
  u32x4 bq[BRING][NB];
#pragma unroll
  for (int st = 0; st < BRING - 1; ++st)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bq[st][nb] = wload((unit & (ksplit - 1)) * NCU * STEPS + st, nb);
  __syncthreads();  // staged chunk, bias, zero region and head weights visible

  int gchunk = 0;  // chunks processed by this workgroup (selects the LDS buffer)
  for (int it = 0; unit >= 0; ++it) {
    const int c0 = (unit & (ksplit - 1)) * NCU;  // first chunk of this unit
    const int next_unit = tile_of(blockIdx.x, gridDim.x, it + 1, nunits);
    const int next = next_unit >= 0 ? next_unit >> kshift : -1;
    const int next_c0 = next_unit >= 0 ? (next_unit & (ksplit - 1)) * NCU : 0;
    const StageSrc next_src = source_of(next >= 0 ? next : tile);
    const long long next_base = stage_base<MODE>(g, next_src);
    // rows of this lane: voxel wm ROWS + 32 mb + l32 of the tile; LDS
    // offset of the row's (0,0,0) tap within a staging buffer (plus this
    // lane's granule) and, for flat tiles, the masks that send reads of the
    // left / right halo column to `zero`
    uint32_t rrel[MB], em0[MB], em2[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      long long p = -1, o;
      int lb = 0, col = -1;
      tile_row(g, tl, tile, wm * W::ROWS + mb * 32 + l32, batch, &p, &lb, &o, &col);
      rrel[mb] = (uint32_t)(lb * VSTRIDE + half * 16);
      em0[mb] = (MODE == 0 && col == 0) ? 0xFFFFFF00u : 0u;
      em2[mb] = (MODE == 0 && col == g.H - 1) ? 0xFFFFFF00u : 0u;
    }

    f32x16 acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[mb][nb][v] = 0.0f;

    for (int chunk = 0; chunk < NCU; ++chunk, ++gchunk) {
      lds_char* const cur = lds + (gchunk & 1) * ABUF;
      lds_char* const oth = lds + ((gchunk + 1) & 1) * ABUF;
      const int cc = c0 + chunk;  // the channel chunk this step loop reads
      // the chunk staged next: the following chunk of this unit, else the
      // first chunk of the next unit, else nothing
      const bool more = chunk + 1 < NCU;
      const int sspan = (more || next >= 0) ? tl.span : 0;  // staged voxels of the chunk staged next
      // the next tile's offsets replace soff round by round during the
      // last chunk (past the last tile: none, every granule empty)
      const __amdgpu_buffer_rsrc_t srs =
          more ? stage_rsrc<CIN>(x, cur_base, (cc + 1) * KC) : stage_rsrc<CIN>(x, next_base, next_c0 * KC);
      u32x4 stg;

      uint32_t rbase[MB];
      const uint32_t cur_u = (uint32_t)(uintptr_t)cur;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) rbase[mb] = cur_u + rrel[mb];
      // LDS address of the fragment of row block mb for tap st: the tap's
      // voxel offset is common to the wave; halo-column taps of flat tiles go
      // to the zero region (v_bfi keeps the low 8 address bits: same bank
      // group, so the read stays conflict-free).  rbase is made opaque before
      // each use so that every step computes its own addresses instead of
      // the compiler computing all of them at the top of the chunk.
      auto frag_read = [&](int mb, int st) -> u32x4 {
        asm volatile("" : "+v"(rbase[mb]));
        const int dt = st / 9, di = (st / 3) % 3, dj = st % 3;
        const uint32_t toff = (uint32_t)((dt * tl.sa + di * tl.sb + dj) * VSTRIDE);
        uint32_t a = rbase[mb] + toff;
        if (MODE == 0 && dj != 1) {
          uint32_t r;
          asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(dj == 0 ? em0[mb] : em2[mb]), "s"(zero_addr), "v"(a));
          a = r;
        }
        return *(lds_u32x4*)(uintptr_t)a;
      };
      // One register set of activation fragments: av[mb] is re-read for the
      // next step as soon as this step's two MFMAs on it have issued, so it
      // has the other row blocks' MFMAs to arrive.  Weight fragments are
      // loaded two steps ahead, staging rounds in the shadow of row block 0.
      u32x4 av[MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) av[mb] = frag_read(mb, 0);
      const int gbase = cc * STEPS;              // k-step of this chunk's step 0
      const int nbase = next_c0 * STEPS - STEPS;  // ... of the next unit's first chunk, minus STEPS
#pragma unroll
      for (int st = 0; st < STEPS; ++st) {
        {
          // past the chunk's last step, the last chunk of a unit runs on
          // into the next unit's first steps
          const int gs = (st + BRING - 1 < STEPS || more ? gbase : nbase) + st + BRING - 1;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) bq[(st + BRING - 1) % BRING][nb] = wload(gs, nb);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bq[st % BRING][nb]),
                                                                  __builtin_bit_cast(bf16x8, av[mb]), acc[mb][nb],
                                                                  0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          if (st + 1 < STEPS) av[mb] = frag_read(mb, st + 1);
          if (mb == 0) {
            // staging of the next chunk: round k is loaded at step 3k and
            // stored to LDS at step 3k + 3, just before round k + 1 is loaded
            if (st >= 3 && st % 3 == 0 && st / 3 - 1 < RMAX) {
              // a tile's first chunk stages into the buffer the previous
              // epilogue used (transposition or head partials): wait for
              // every wave to leave it
              if (st == 3 && chunk == 0) __builtin_amdgcn_s_barrier();
              *(lds_u32x4_w*)(oth + stage_slot((st / 3 - 1) * NT + tid)) = stg;
            }
            if (st % 3 == 0 && st / 3 < RMAX) {
              const int k = st / 3;
              if (!more) soff[k] = stage_offset<CIN, MODE>(g, tl, next_src, next_base, limit, sspan, k, tid);
              stg = __builtin_amdgcn_raw_buffer_load_b128(srs, soff[k], 0, 0);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // every wave's staging writes done, every wave done reading `cur`
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
    }

    if constexpr (EPI == EPI_PARK) {
      // split K loop: park this unit's fp32 sums as [tile row][channel]; a
      // second kernel adds a tile's parts and applies the epilogue
      float* const mine = partial + (size_t)unit * kTileRows * COUT;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = wm * W::ROWS + mb * 32 + l32, co = (wn * NB + nb) * 32 + q * 8 + half * 4;
            *reinterpret_cast<float4*>(mine + row * COUT + co) =
                float4{acc[mb][nb][4 * q], acc[mb][nb][4 * q + 1], acc[mb][nb][4 * q + 2], acc[mb][nb][4 * q + 3]};
          }
    } else {
      finish_tile(tile, lds + ((gchunk - 1) & 1) * ABUF, acc);
    }
    unit = next_unit;
    tile = next;
    cur_base = next_base;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Second kernel of a split K loop: one thread per (tile row, 8 channels)
// (activations) or per tile row (head, output layer) adds the tile's parts
// in part order, then applies the epilogue of the unsplit kernel: bias,
// activation, bf16 and a 16-byte store; or bias, activation, bf16 rounding,
// the 1x1x1 head and the threshold; or, for the output layer, bias and the
// threshold.
template <int EPI, int ACT>
__global__ void __launch_bounds__(256) split_finish_kernel(Geom g, Tiling tl, int cout, int kshift,
                                                           const float* __restrict__ partial,
                                                           const float* __restrict__ bias, uint16_t* __restrict__ y,
                                                           int ystride, const float* __restrict__ head_w,
                                                           const float* __restrict__ head_b,
                                                           const int32_t* __restrict__ tables,
                                                           uint8_t* __restrict__ nib, float* __restrict__ logits,
                                                           int batch) {
  const int groups = EPI == EPI_ACT ? cout / 8 : 1;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= tl.ntiles * kTileRows * groups) return;
  const int tile = (int)(gid / (kTileRows * groups));
  const int rem = (int)(gid - (long long)tile * kTileRows * groups);
  const int r = rem / groups, grp = rem - r * groups;
  const int ksplit = 1 << kshift;
  // sum of channels c .. c + 7 of this row over the tile's parts, part order
  auto sum8 = [&](int c, float (&v)[8]) {
    for (int p = 0; p < ksplit; ++p) {
      const float* src = partial + ((size_t)((tile << kshift) + p) * kTileRows + r) * cout + c;
      const float4 a = *reinterpret_cast<const float4*>(src);
      const float4 b = *reinterpret_cast<const float4*>(src + 4);
      const float t[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = p == 0 ? t[e] : v[e] + t[e];
    }
  };
  if constexpr (EPI == EPI_ACT) {
    long long pidx, o;
    int lb;
    if (!tile_row(g, tl, tile, r, batch, &pidx, &lb, &o)) return;
    float v[8];
    sum8(grp * 8, v);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = bf16_pack(act_fn<ACT>(v[2 * e] + bias[grp * 8 + 2 * e]),
                       act_fn<ACT>(v[2 * e + 1] + bias[grp * 8 + 2 * e + 1]));
    *reinterpret_cast<uint4*>(y + pidx * ystride + grp * 8) = uint4{w[0], w[1], w[2], w[3]};
  } else {
    int b, t, i, j;
    if (!tile_row_coords(g, tl, tile, r, batch, &b, &t, &i, &j)) return;
    float lg[4];
    if constexpr (EPI == EPI_OUT) {
      float v[8];
      sum8(0, v);
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) lg[o2] = v[o2] + bias[o2];
    } else {
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) lg[o2] = head_b[o2];
      for (int c = 0; c < cout; c += 8) {
        float v[8];
        sum8(c, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float a = bf16_round(act_fn<ACT>(v[e] + bias[c + e]));
#pragma unroll
          for (int o2 = 0; o2 < 4; ++o2) lg[o2] += head_w[o2 * cout + c + e] * a;
        }
      }
    }
    const int HH = g.H * g.H;
    const int s = i * g.H + j;
    nib[(long long)b * g.V + (long long)t * HH + s] = (uint8_t)flip_nibble(g, tables, i, j, lg);
    if (logits) {
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) logits[(((long long)b * 4 + o2) * g.T + t) * HH + s] = lg[o2];
    }
  }
}

// Launches one instance of the hidden kernel (the LDS size attribute set on
// its first use).
template <int CIN, int COUT, int EPI, int MODE>
hipError_t launch_hidden(const Geom& g, const Tiling& tl, int act, const void* x, void* y, int ystride,
                         const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                         const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_workgroups,
                         int kshift, float* partial, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)conv_hidden_kernel<CIN, COUT, EPI, MODE>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, Lds<COUT>::total);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long nwg = conv_workgroups(tl.ntiles << kshift, n_workgroups);
  hipLaunchKernelGGL((conv_hidden_kernel<CIN, COUT, EPI, MODE>), dim3((unsigned)nwg), dim3(NT),
                     (size_t)Lds<COUT>::total, stream, g, tl, act, (const uint16_t*)x, (uint16_t*)y, ystride,
                     (const u32x4*)wfrag, bias, head_w, head_b, tables, nib, logits, batch, kshift, partial);
  return hipSuccess;
}

template <int CIN, int COUT, int EPI, int MODE>
hipError_t launch_one(const Geom& g, const Tiling& tl, int act, const void* x, void* y, int ystride,
                      const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                      const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_workgroups,
                      const Split_k& sk, hipStream_t stream) {
  hipError_t e;
  if (sk.kshift == 0) {
    e = launch_hidden<CIN, COUT, EPI, MODE>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b, tables, nib,
                                            logits, batch, n_workgroups, 0, nullptr, stream);
    return e != hipSuccess ? e : hipGetLastError();
  }
  // K loops split: park the parts, then add them and finish the tiles
  e = launch_hidden<CIN, COUT, EPI_PARK, MODE>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b, tables, nib,
                                               logits, batch, n_workgroups, sk.kshift, sk.partial, stream);
  if (e != hipSuccess) return e;
  const long long threads = tl.ntiles * kTileRows * (EPI == EPI_ACT ? COUT / 8 : 1);
  with_activation(act, [&](auto A) {
    hipLaunchKernelGGL((split_finish_kernel<EPI, decltype(A)::value>), dim3((unsigned)((threads + 255) / 256)),
                       dim3(256), 0, stream, g, tl, COUT, sk.kshift, sk.partial, bias, (uint16_t*)y, ystride, head_w,
                       head_b, tables, nib, logits, batch);
  });
  return hipGetLastError();
}

}  // namespace

int conv_hidden_max_span() { return MAX_SPAN; }
size_t conv_hidden_partial_floats_per_unit() { return (size_t)kTileRows * 128; }
int conv_hidden_workgroups_per_cu() { return 2; }

#define PD_HIDDEN_CASE(CI, CO, E)                                                              \
  if (cin == CI && cout == CO && head == E) {                                                 \
    if (tl.mode == 0)                                                                          \
      return launch_one<CI, CO, E, 0>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b, \
                                      tables, nib, logits, batch, n_workgroups, sk, stream);   \
    return launch_one<CI, CO, E, 1>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,   \
                                    tables, nib, logits, batch, n_workgroups, sk, stream);     \
  }

hipError_t launch_conv_hidden(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x,
                              void* y, int ystride, const void* wfrag, const float* bias, int head,
                              const float* head_w, const float* head_b, const int32_t* tables, uint8_t* nib,
                              float* logits, int batch, int n_workgroups, const Split_k& sk,
                              hipStream_t stream) {
  if (tl.span <= 0 || tl.span > MAX_SPAN) return hipErrorInvalidValue;
  // parts per tile: a power of two dividing the layer's chunks, with room
  // for every unit's sums
  if (sk.kshift < 0 || (cin / KC) % (1 << sk.kshift) != 0 ||
      (sk.kshift > 0 && (tl.ntiles << sk.kshift) > sk.max_units))
    return hipErrorInvalidValue;
  PD_HIDDEN_CASE(64, 64, EPI_ACT)
  PD_HIDDEN_CASE(128, 128, EPI_ACT)
  PD_HIDDEN_CASE(64, 128, EPI_ACT)
  PD_HIDDEN_CASE(128, 64, EPI_ACT)
  PD_HIDDEN_CASE(256, 128, EPI_ACT)
  PD_HIDDEN_CASE(256, 64, EPI_ACT)
  PD_HIDDEN_CASE(64, 64, EPI_HEAD)
  PD_HIDDEN_CASE(128, 128, EPI_HEAD)
  PD_HIDDEN_CASE(64, 128, EPI_HEAD)
  PD_HIDDEN_CASE(128, 64, EPI_HEAD)
  if (cout == 4) cout = 32;  // the output layer's 4 filters fill one padded block
  PD_HIDDEN_CASE(64, 32, EPI_OUT)
  PD_HIDDEN_CASE(128, 32, EPI_OUT)
  PD_HIDDEN_CASE(256, 32, EPI_OUT)
  return hipErrorInvalidValue;
}

}  // namespace pd
