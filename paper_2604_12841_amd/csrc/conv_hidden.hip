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
//     over 16 groups of 16 bytes; granule g of voxel v sits in group
//     (3 v + g) mod 16, so 16 consecutive staged voxels hit 16 distinct
//     groups, and a fragment read of 32 consecutive staged voxels (flat
//     tiles) or the staging stores meet no group twice in one LDS cycle
//     (measured).  A read whose 32 voxels come from two rows of a box, with
//     the rows' halo voxels between them, costs a few cycles more, which the
//     LDS pipe absorbs (it is less than half busy here).  Flat tiles stage
//     only the real columns; reads of the left / right halo column are
//     redirected to a 256-byte zero region with the same low address bits
//     (same group).
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
typedef __attribute__((ext_vector_type(8))) uint32_t u32x8;
typedef __attribute__((ext_vector_type(8))) int i32x8;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_w;
typedef __attribute__((address_space(3))) uint32_t lds_u32_w;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2_w;

constexpr int NT = 256;       // threads per workgroup: 4 wave64
constexpr int KC = 16;        // input channels per LDS chunk (one MFMA k-step)
constexpr int VSTRIDE = 48;   // LDS bytes per staged voxel (32 of channels + 16 of padding)

// Per kernel size KS (3 or 5): the k-steps of a bf16 chunk (one per tap), the
// weight-fragment ring depth (prefetch distance RING - 1; it divides the
// k-steps of a chunk so that ring slots line up with chunk boundaries), the
// staged voxels a staging buffer holds (the last slot takes overflow writes)
// and the workgroups per CU.  KS = 3: two workgroups per CU, so each SIMD
// runs one wave of each and one workgroup's epilogue, barriers and staging
// stalls overlap the other's matrix work.  KS = 5: a 256-voxel tile's halo
// of two makes its footprint about 4.5 times the tile (a 4 x 8 x 8 box
// stages 8 x 12 x 12 voxels), so one workgroup per CU with larger staging
// buffers; its 125-step chunks keep the matrix pipe busy between barriers.
template <int KS>
struct Conv {
  static constexpr int TAPS = KS * KS * KS;
  static constexpr int BRING = KS == 3 ? 3 : 5;
  static constexpr int BUF_VOX = KS == 3 ? 800 : 1600;
  static constexpr int MAX_SPAN = BUF_VOX - 1;
  static constexpr int WG_PER_CU = KS == 3 ? 2 : 1;
  // Every chunk is staged with RMAX rounds of NT 16-byte granules, stored
  // unconditionally (a conditional store would let the compiler sink the
  // load next to it): granules past the footprint load zeros into slots
  // past the footprint, and granules past the buffer all go to its last
  // slot.
  static constexpr int RMAX = (2 * MAX_SPAN + NT - 1) / NT;
  static constexpr int ABUF = BUF_VOX * VSTRIDE;  // bytes per staging buffer
  static_assert(RMAX * NT >= 2 * MAX_SPAN && (RMAX * NT) % 32 == 0, "staging rounds cover the largest footprint");
  static_assert(TAPS % BRING == 0, "the weight ring lines up with chunk boundaries");
  static_assert(RMAX * 3 + 3 <= TAPS, "staging rounds fit in a chunk");
};

// The fp8 (E4M3) variant keeps the 32 staged bytes per voxel and chunk, now
// 32 channels, and runs v_mfma_f32_32x32x64_f8f6f4: k = 64 is two taps x 32
// channels, the first half-wave's lanes holding a voxel's 32 channels at tap
// 2 s, the second half-wave's at tap 2 s + 1 (the tap past the last does not
// exist: its weights are zero).  ceil(taps / 2) k-steps per chunk (14 for
// 3x3x3); staging round k loads at step 2 k and stores at step 2 k + 2 (the
// last one after the chunk's last step); the weight ring is 2 deep (32
// bytes per lane and block).
template <bool F8, int KS>
struct Prec {
  static constexpr int KCH = F8 ? 32 : KC;                                  // input channels per chunk
  static constexpr int NSTEP = F8 ? (Conv<KS>::TAPS + 1) / 2 : Conv<KS>::TAPS;  // k-steps per chunk
  static constexpr int RING = F8 ? (KS == 3 ? 2 : 3) : Conv<KS>::BRING;     // weight ring depth
  static constexpr int SG = F8 ? 2 : 3;           // steps between staging rounds
  static constexpr int ESZ = F8 ? 1 : 2;          // bytes per activation value
  static constexpr int WFRAG = F8 ? 2048 : 1024;  // bytes of one weight fragment (64 lanes)
  static_assert(NSTEP % RING == 0, "the weight ring lines up with chunk boundaries");
  static_assert(SG * (Conv<KS>::RMAX - 1) < NSTEP, "staging rounds load within a chunk");
  static_assert(KCH * ESZ == 32, "a chunk stages 32 bytes per voxel");
};

// Staging granule q = NT k + tid: in each run of 32, the first 16 take
// granule 0 of 16 consecutive staged voxels and the next 16 their granule 1,
// so the 16 lanes of an LDS write cycle hit 16 distinct bank groups.
__host__ __device__ inline int stage_voxel(int q) { return ((q >> 5) << 4) | (q & 15); }
__host__ __device__ inline int stage_gran(int q) { return (q >> 4) & 1; }

// LDS byte (relative to a staging buffer) of staging granule q; voxels past
// the buffer all go to its last slot.
template <int KS>
__host__ __device__ inline int stage_slot(int q) {
  constexpr int BV = Conv<KS>::BUF_VOX;
  const int v = stage_voxel(q);
  return (v < BV - 1 ? v : BV - 1) * VSTRIDE + stage_gran(q) * 16;
}

// Epilogue modes: the activations of a hidden layer, a hidden layer with the
// 1x1x1 head fused in, or the 5x5x5 output layer itself (4 filters, padded to
// one block of 32 MFMA rows; the 3x3x3 one has a kernel of its own); EPI_PARK: one part of a split K loop, whose
// fp32 sums are parked for split_finish_kernel.  Only EPI_PARK kernels split
// (the others see a split of 1 at compile time and keep their registers for
// the epilogue).  EPI_ADD: EPI_ACT with the block's shortcut added to the
// pre-activation (the second conv of a residual block): the bf16 row of sc
// at the output voxel (fp8: E4M3 codes), or, when head_w is given, its 1x1x1
// projection computed here from the sc_stride (<= 8) channels of sc's row
// (head_w [c_out][sc_stride] and head_b [c_out] in those slots:
// bf16(head_b + sum_ci head_w x_ci), an fp32 FMA chain in channel order;
// fp8: E4M3 of the same).
enum Epi { EPI_ACT = 0, EPI_HEAD = 1, EPI_OUT = 2, EPI_PARK = 3, EPI_ADD = 4 };

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
// 512-byte zero region (256-aligned, for halo-column reads; an fp8 lane
// reads 32 bytes from a redirected address), the bias [COUT] and the
// per-channel weight scales [COUT] (fp8) and the head weights [4][COUT].
// The head epilogue puts its partial sums in the staging buffer the tile
// read last.
// output-channel slices of one launch: up to 8 of 32 channels (a 256-wide
// layer), else up to 4
__host__ __device__ constexpr int max_slices(int cout) { return cout == 32 ? 8 : 4; }

template <int COUT, int KS>
struct Lds {
  static constexpr int ABUF = Conv<KS>::ABUF;
  static constexpr int zero = 2 * ABUF;
  // biases (fp8: then the weight scales) of up to max_slices(COUT)
  // output-channel slices; a head's weights (never sliced) follow one slice's
  static constexpr int bias = zero + 512;
  static constexpr int headw = bias + 2 * COUT * 4;
  // two unit numbers handed between the waves (dynamic scheduling)
  static constexpr int sched = bias + (2 * max_slices(COUT) > 6 ? 2 * max_slices(COUT) : 6) * COUT * 4;
  static constexpr int total = sched + 16;
  static_assert(zero % 256 == 0, "zero region must be 256-aligned");
  static_assert(Conv<KS>::WG_PER_CU * total <= 160 * 1024, "the workgroups of a CU fit its LDS");
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

// ROW: bytes per activation voxel row (c_in values).
template <int ROW, int MODE>
__host__ __device__ inline uint32_t stage_offset(const Geom& g, const Tiling& tl, const StageSrc& src,
                                                 long long base, long long limit, int span, int k, int tid) {
  const int q = k * NT + tid;
  const int vv = stage_voxel(q);
  const long long gv = staged_voxel_fast<MODE>(g, tl, src, vv, limit);
  return (vv < span && gv >= 0) ? (uint32_t)((gv - base) * ROW + stage_gran(q) * 16) : kNoVoxel;
}

// Buffer resource over the activations from padded voxel `base`, byte
// `cb` of the row on (rows of ROW bytes).
template <int ROW>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stage_rsrc(const void* x, long long base, int cb) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)((const char*)x + base * ROW + cb), 0, kStageRange, 0x00020000);
}

// The projected shortcut of channels co .. co + N - 1 at padded voxel p:
// b[c] + sum_ci w[c][ci] x[p][ci] over the pc channels of x's row (the
// network's input planes, bf16 on both paths), an fp32 FMA chain in channel
// order, rounded to bf16 (F8: to E4M3).
template <int N, bool F8>
__device__ __forceinline__ void project_shortcut(const uint16_t* __restrict__ x, int pc, long long p,
                                                 const float* __restrict__ w, const float* __restrict__ b, int co,
                                                 float (&s)[N]) {
  float a[N];
#pragma unroll
  for (int o = 0; o < N; ++o) a[o] = b[co + o];
  for (int ci = 0; ci < pc; ++ci) {
    const float xv = __uint_as_float((uint32_t)x[p * pc + ci] << 16);
#pragma unroll
    for (int o = 0; o < N; ++o) a[o] = __builtin_fmaf(w[(co + o) * pc + ci], xv, a[o]);
  }
#pragma unroll
  for (int o = 0; o < N; o += 2) {
    if constexpr (F8) {
      s[o] = e4m3_round(a[o]);
      s[o + 1] = e4m3_round(a[o + 1]);
    } else {
      const uint32_t pk = bf16_pack(a[o], a[o + 1]);
      s[o] = __uint_as_float(pk << 16);
      s[o + 1] = __uint_as_float(pk & 0xFFFF0000u);
    }
  }
}

// The block's shortcut of channels co .. co + N - 1 at padded voxel p: its
// stored row in sc (bf16, or F8 E4M3 codes), or with w given its
// projection from sc's few channels (the input planes).
template <int N, bool F8>
__device__ __forceinline__ void shortcut_of(const uint16_t* __restrict__ sc, int sc_stride, long long p,
                                            const float* __restrict__ w, const float* __restrict__ b, int co,
                                            float (&s)[N]) {
  if (w) {
    project_shortcut<N, F8>(sc, sc_stride, p, w, b, co, s);
  } else if constexpr (F8) {
    const uint8_t* r = (const uint8_t*)sc + p * sc_stride + co;
#pragma unroll
    for (int o = 0; o < N; o += 4) {
      const uint32_t q = *reinterpret_cast<const uint32_t*>(r + o);
      s[o] = __builtin_amdgcn_cvt_f32_fp8((int)q, 0);
      s[o + 1] = __builtin_amdgcn_cvt_f32_fp8((int)q, 1);
      s[o + 2] = __builtin_amdgcn_cvt_f32_fp8((int)q, 2);
      s[o + 3] = __builtin_amdgcn_cvt_f32_fp8((int)q, 3);
    }
  } else {
    const uint16_t* r = sc + p * sc_stride + co;
#pragma unroll
    for (int o = 0; o < N; o += 4) {
      const u32x2 q = *reinterpret_cast<const u32x2*>(r + o);
      s[o] = __uint_as_float(q.x << 16);
      s[o + 1] = __uint_as_float(q.x & 0xFFFF0000u);
      s[o + 2] = __uint_as_float(q.y << 16);
      s[o + 3] = __uint_as_float(q.y & 0xFFFF0000u);
    }
  }
}

// F8: E4M3 activations and weights (bias holds [COUT] biases then [COUT]
// per-channel weight scales; y and x hold one byte per value).  KS: the
// kernel size, 3 or 5 (5: box tiles on a halo of two).
template <int CIN, int COUT, int EPI, int MODE, bool F8, int KS>
__global__ void __launch_bounds__(NT)
__attribute__((amdgpu_waves_per_eu(Conv<KS>::WG_PER_CU, Conv<KS>::WG_PER_CU)))
conv_hidden_kernel(Geom g, Tiling tl, int act, const void* __restrict__ x, void* __restrict__ y,
                   int ystride, const u32x4* __restrict__ wfrag, const float* __restrict__ bias,
                   const float* __restrict__ head_w, const float* __restrict__ head_b,
                   const int32_t* __restrict__ tables, uint8_t* __restrict__ nib,
                   float* __restrict__ logits, int batch, int kshift_arg, float* __restrict__ partial,
                   const uint16_t* __restrict__ sc, int sc_stride, int lsl, uint32_t* __restrict__ sched,
                   int nstat) {
  static_assert(KS == 3 || MODE == 1, "5x5x5 layers run on box tiles");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  using W = Split<COUT>;
  using L = Lds<COUT, KS>;
  constexpr int MB = W::MB;
  constexpr int NB = W::NB;
  constexpr int NBT = COUT / 32;  // 32-channel blocks in total
  using P = Prec<F8, KS>;
  constexpr int KCH = P::KCH, NSTEP = P::NSTEP, SG = P::SG;
  // weight ring depth: 32-channel slices (small batches, one workgroup per
  // CU, two MFMAs per k-step) prefetch a third of a chunk ahead, since the
  // short steps alone cannot cover a load's latency
  constexpr int RING = (COUT == 32 && KS == 3) ? (F8 ? 7 : 9) : P::RING;
  static_assert(NSTEP % RING == 0, "the weight ring lines up with chunk boundaries");
  constexpr int RMAX = Conv<KS>::RMAX, ABUF = L::ABUF, TAPS = Conv<KS>::TAPS;
  constexpr int ROW = CIN * P::ESZ;  // bytes per input voxel row
  constexpr int NCHUNK = CIN / KCH;
  constexpr int TSTEPS = NCHUNK * NSTEP;  // k-steps of the layer
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % W::WM, wn = wave / W::WM;
  const int half = lane >> 5, l32 = lane & 31;
  const uint32_t hmask = half ? 0xFFFFFFFFu : 0u;  // fp8: selects the half-wave's tap
  const int ntiles = (int)tl.ntiles;
  const long long limit = (long long)batch * g.S;
  // Work units: (tile, part); part p of a tile runs its chunks [p NCU, (p+1) NCU)
  // with ksplit = 2^kshift parts per tile (EPI_PARK only: small batches).
  // With parts, each unit parks its fp32 sums in `partial` (unit u at
  // u * 256 * COUT floats) and split_finish_kernel does the epilogue.
  const int kshift = EPI == EPI_PARK ? kshift_arg : 0;
  const int ksplit = 1 << kshift;
  const int NCU = NCHUNK >> kshift;  // chunks per unit
  // Output-channel slices (a layer wider than COUT in one launch): 2^lsl
  // slices of COUT channels, unit u = ((tile << lsl | slice) << kshift) | part;
  // slice q has its own weight fragments (the layer's TSTEPS k-steps, after
  // q slices' worth), biases (COUT, fp8: and COUT scales) and output
  // columns (and shortcut columns, or projection rows).
  const int nunits = ntiles << (kshift + lsl);
  constexpr int BSL = (F8 ? 2 : 1) * COUT;  // bias floats per slice
  auto slice_of = [&](int u) { return (u >> kshift) & ((1 << lsl) - 1); };

  lds_char* const lds = (lds_char*)smem;
  lds_char* const zero = lds + L::zero;
  lds_float* const bias_s = (lds_float*)(lds + L::bias);
  lds_float* const scale_s = bias_s + COUT;  // fp8: per-channel weight scales
  lds_float* const headw_s = (lds_float*)(lds + L::headw);
  for (int e = tid; e < (BSL << lsl); e += NT) bias_s[e] = bias[e];
  if (tid < 128) ((lds_u32_w*)zero)[tid] = 0u;
  const uint32_t zero_addr = (uint32_t)(uintptr_t)zero;
  if (EPI == EPI_HEAD)
    for (int e = tid; e < 4 * COUT; e += NT) headw_s[e] = head_w[e];

  // Bias, activation and output of one tile from its accumulators (lane
  // holds channels co .. co + 3, co = 64 wn + 32 nb + 8 q + 4 half, of voxel
  // row wm ROWS + 32 mb + l32); ebuf: a staging buffer free for the
  // transposition / head partials.
  auto finish_tile = [&](int tile, int slice, lds_char* const ebuf, f32x16 (&acc)[MB][NB]) {
      // this slice's output columns, and its shortcut columns or projection rows
      char* const ysl = (char*)y + (size_t)slice * COUT * P::ESZ;
      const uint16_t* const scs = head_w ? sc : (const uint16_t*)((const char*)sc + (size_t)slice * COUT * P::ESZ);
      const float* const hws = head_w ? head_w + (size_t)slice * COUT * sc_stride : nullptr;
      const float* const hbs = head_w ? head_b + (size_t)slice * COUT : nullptr;
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
              float lg[4];
#pragma unroll
              for (int o = 0; o < 4; ++o)
                lg[o] = F8 ? __builtin_fmaf(acc[mb][0][o], scale_s[o], bias_s[o]) : acc[mb][0][o] + bias_s[o];
              if (sc) {  // residual shortcut of the last block: 4 bf16 channels
                const u32x2 sv = *reinterpret_cast<const u32x2*>(sc + padded_index(g, b, t, i, j) * sc_stride);
                lg[0] += __uint_as_float(sv.x << 16);
                lg[1] += __uint_as_float(sv.x & 0xFFFF0000u);
                lg[2] += __uint_as_float(sv.y << 16);
                lg[3] += __uint_as_float(sv.y & 0xFFFF0000u);
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
      } else if constexpr (EPI == EPI_ACT || EPI == EPI_ADD) {
        // bias + activation + bf16, transposed through this wave's slice of
        // the staging buffer the tile read last (64 rows x 128 bytes, granule
        // c of row r at c ^ (r % 8)), then stored as the wave's whole part of
        // each voxel row (NB x 32 channels: 128 bytes, 8 rows per
        // instruction, for NB = 2).  The next tile's first staging store
        // waits at a barrier until every wave is done here.
        // (fp8: one byte per channel, 16-byte granules of 16 channels)
        lds_char* const tb = ebuf + wave * (64 * 128);
        constexpr int GR = (F8 ? 2 : 4) * NB;  // 16-byte granules of a row's NB x 32 channels
        constexpr int LGR = GR == 8 ? 3 : (GR == 4 ? 2 : 1);
        static_assert((1 << LGR) == GR, "granules per row: a power of two");
        with_activation(act, [&](auto A) {
          constexpr int ACT = decltype(A)::value;
#pragma unroll
          for (int ps = 0; ps < MB / 2; ++ps) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int c8 = nb * 4 + q;  // 8-channel group of the wave's NB x 32 channels
                const int co = wn * NB * 32 + c8 * 8 + half * 4;
                const lds_float* const bsl = bias_s + slice * BSL;  // this slice's biases, then scales
                const float4 bv = {bsl[co], bsl[co + 1], bsl[co + 2], bsl[co + 3]};
                float4 sv = {1.0f, 1.0f, 1.0f, 1.0f};
                if constexpr (F8) sv = float4{bsl[COUT + co], bsl[COUT + co + 1], bsl[COUT + co + 2], bsl[COUT + co + 3]};
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                  const int mb = 2 * ps + m;
                  const int r = m * 32 + l32;
                  if constexpr (F8) {
                    float sh[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                    if constexpr (EPI == EPI_ADD) {  // the block's shortcut, 4 channels of this row
                      if (pidx[mb] >= 0) shortcut_of<4, true>(scs, sc_stride, pidx[mb], hws, hbs, co, sh);
                    }
                    const float v0 = act_fn<ACT>(__builtin_fmaf(acc[mb][nb][4 * q + 0], sv.x, bv.x) + sh[0]);
                    const float v1 = act_fn<ACT>(__builtin_fmaf(acc[mb][nb][4 * q + 1], sv.y, bv.y) + sh[1]);
                    const float v2 = act_fn<ACT>(__builtin_fmaf(acc[mb][nb][4 * q + 2], sv.z, bv.z) + sh[2]);
                    const float v3 = act_fn<ACT>(__builtin_fmaf(acc[mb][nb][4 * q + 3], sv.w, bv.w) + sh[3]);
                    const int c = c8 >> 1;  // granule; byte (c8 & 1) 8 + 4 half within it
                    *(lds_u32_w*)(tb + r * 128 + ((c ^ (r & 7)) << 4) + (c8 & 1) * 8 + half * 4) =
                        e4m3_pack4(v0, v1, v2, v3);
                  } else {
                    float4 sh = {0.0f, 0.0f, 0.0f, 0.0f};
                    if constexpr (EPI == EPI_ADD) {  // the block's shortcut, 4 channels of this row
                      if (pidx[mb] >= 0) {
                        float pj[4];
                        shortcut_of<4, false>(scs, sc_stride, pidx[mb], hws, hbs, co, pj);
                        sh = float4{pj[0], pj[1], pj[2], pj[3]};
                      }
                    }
                    const float v0 = act_fn<ACT>(acc[mb][nb][4 * q + 0] + bv.x + sh.x);
                    const float v1 = act_fn<ACT>(acc[mb][nb][4 * q + 1] + bv.y + sh.y);
                    const float v2 = act_fn<ACT>(acc[mb][nb][4 * q + 2] + bv.z + sh.z);
                    const float v3 = act_fn<ACT>(acc[mb][nb][4 * q + 3] + bv.w + sh.w);
                    u32x2 packed;
                    packed.x = bf16_pack(v0, v1);
                    packed.y = bf16_pack(v2, v3);
                    *(lds_u32x2_w*)(tb + r * 128 + ((c8 ^ (r & 7)) << 4) + half * 8) = packed;
                  }
                }
              }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's rows are in LDS
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int it2 = 0; it2 < GR; ++it2) {
              const int gi = it2 * 64 + lane;
              const int r = gi >> LGR, c = gi & (GR - 1);
              const u32x4 v = *(lds_u32x4*)(tb + r * 128 + ((c ^ (r & 7)) << 4));
              const int pr = __shfl(pidx[2 * ps + (it2 >> (LGR - 1))], r & 31);  // rows 32.. from it2 = GR / 2
              if (pr >= 0)
                *reinterpret_cast<u32x4*>(ysl + ((long long)pr * ystride + wn * NB * 32) * P::ESZ + c * 16) = v;
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
              float4 sv = {1.0f, 1.0f, 1.0f, 1.0f};
              if constexpr (F8) sv = float4{scale_s[co], scale_s[co + 1], scale_s[co + 2], scale_s[co + 3]};
              float4 hw[4];
#pragma unroll
              for (int o = 0; o < 4; ++o)
                hw[o] = {headw_s[o * COUT + co], headw_s[o * COUT + co + 1], headw_s[o * COUT + co + 2],
                         headw_s[o * COUT + co + 3]};
#pragma unroll
              for (int mb = 0; mb < MB; ++mb) {
                // the head's input: the activation rounded as the next layer would read it
                auto rnd = [&](float v, float sc, float bb) {
                  if constexpr (F8) return e4m3_round(act_fn<ACT>(__builtin_fmaf(v, sc, bb)));
                  else return bf16_round(act_fn<ACT>(v + bb));
                };
                const float a0 = rnd(acc[mb][nb][4 * q + 0], sv.x, bv.x);
                const float a1 = rnd(acc[mb][nb][4 * q + 1], sv.y, bv.y);
                const float a2 = rnd(acc[mb][nb][4 * q + 2], sv.z, bv.z);
                const float a3 = rnd(acc[mb][nb][4 * q + 3], sv.w, bv.w);
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

  // Units: each XCD takes a contiguous range (tile_of).  A workgroup's first
  // nstat units are fixed (the k-th, (k + n)-th, ... of its XCD's range, n =
  // the XCD's workgroups); with `sched` (a launch of more units than two per
  // workgroup), the rest are taken in turn from a per-XCD counter, so that
  // workgroups that run faster take more of them (fixed shares left the
  // last workgroups of an XCD finishing 10-20 % of the layer after the
  // first).  Thread 0 takes unit it + 2 at the top of iteration it and hands
  // it over in LDS slot it % 2 at the end of the iteration's first chunk,
  // read by every wave at the top of iteration it + 1 (a chunk's barrier in
  // between).  Counters sit in separate 64-byte lines (grab, then done, per
  // XCD); the last workgroup of an XCD to finish puts both back to zero for
  // the next launch.  Box tiles fix two units (c5: about 3 % less time);
  // flat tiles fix seven eighths of a workgroup's share: fixed shares keep
  // an XCD's workgroups on neighbouring tiles' chunks together, whose lines
  // L2 then serves to all of them, and counters from the third unit on
  // fetched half as much again from HBM (c3: 1.7 % less time); from seven
  // eighths on, 7 % more for 2.2 % less time.  Only the 128-wide 3x3x3
  // activation instances and the bf16 head ones take counters (fp8: 0.5 %
  // less time at c3, 1.4 % at c5): the 64-wide layers gained nothing, and the
  // counters' registers made the fp8 head instance spill in its K loop (and
  // the shortcut-adding ones spill more).
  constexpr bool DYN = COUT == 128 && KS == 3 && (EPI == EPI_ACT || (EPI == EPI_HEAD && !F8));
  if (!DYN) sched = nullptr;
  const int xcd = blockIdx.x & 7, nwx = gridDim.x >> 3, per_xcd = (nunits + 7) >> 3;
  uint32_t* const grab = sched ? sched + xcd * 32 : nullptr;
  uint32_t* const done = sched ? sched + xcd * 32 + 16 : nullptr;
  lds_u32_w* const dyn_s = (lds_u32_w*)(lds + L::sched);
  auto finish_sched = [&]() {
    if (sched && tid == 0 &&
        __hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)nwx - 1) {
      __hip_atomic_store(grab, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  };
  auto dyn_unit = [&](uint32_t c) -> int {  // unit of the c-th counter value (-1: none left)
    const long long local = (long long)nstat * nwx + c;
    if (local >= per_xcd) return -1;
    const long long u = (long long)xcd * per_xcd + local;
    return u < nunits ? (int)u : -1;
  };

  int unit = tile_of(blockIdx.x, gridDim.x, 0, nunits);
  if (unit < 0) {
    finish_sched();
    return;
  }
  int tile = unit >> (kshift + lsl);

  auto source_of = [&](int t) { return tile_source(g, tl, t, batch); };
  long long cur_base = stage_base<MODE>(g, source_of(tile));
  uint32_t soff[RMAX];  // this lane's staging offsets of the tile being staged
  {
    const StageSrc src = source_of(tile);
#pragma unroll
    for (int k = 0; k < RMAX; ++k) soff[k] = stage_offset<ROW, MODE>(g, tl, src, cur_base, limit, tl.span, k, tid);
  }

  // weight fragment (k-step gs, block nb of this wave's channels): buffer
  // loads with this lane's slot (16 bytes; fp8: 32) as the vector offset and
  // the fragment's offset as the scalar one (no per-load address arithmetic)
  constexpr int WQ = F8 ? 2 : 1;  // 16-byte pieces per lane and fragment
  const uint32_t wbytes = (uint32_t)(TSTEPS * NBT * P::WFRAG) << lsl;
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc((void*)wfrag, 0, wbytes, 0x00020000);

  // Small-batch launches of 32-channel slices have one workgroup per CU or
  // fewer, whose short k-steps would each wait on their weight fragments
  // coming from memory one after the other.  First the XCD's workgroups warm
  // its L2 with all the layer's fragments, each loading a share at once (up
  // to 32 KB), alongside the first chunk's staging; the values are folded
  // into one register, kept to the end of the prologue.  (fp8 at d = 25,
  // batch 1: 8 % less time per round.  Split K loops, whose k-steps are
  // four times as long, gained nothing from it.)
  constexpr bool WARM = COUT == 32 && KS == 3;
  uint32_t warm = 0;
  if constexpr (WARM) {
    const uint32_t per = (gridDim.x >> 3) > 0 ? (gridDim.x >> 3) : 1u;  // this XCD's workgroups
    const uint32_t share = ((wbytes + per - 1) / per + NT * 16 - 1) / (NT * 16) * (NT * 16);
    const uint32_t b0 = (blockIdx.x >> 3) * share;
    u32x4 pf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)  // offsets past the fragments read zeros
      pf[i] = (uint32_t)i * NT * 16 < share ? __builtin_amdgcn_raw_buffer_load_b128(wres, b0 + (i * NT + tid) * 16, 0, 0)
                                             : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) warm ^= pf[i].x;
  }

  // First tile: stage its first chunk synchronously.
  {
    const __amdgpu_buffer_rsrc_t rs = stage_rsrc<ROW>(x, cur_base, (unit & (ksplit - 1)) * NCU * 32);
#pragma unroll
    for (int k = 0; k < RMAX; ++k) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, soff[k], 0, 0);
      *(lds_u32x4_w*)(lds + stage_slot<KS>(k * NT + tid)) = v;
    }
  }
  if constexpr (WARM) asm volatile("" ::"v"(warm));
  const uint32_t woff = (uint32_t)((wn * NB * 64 + lane) * 16 * WQ);
  auto wload = [&](int gs, int nb, u32x4 (&dst)[WQ]) {
#pragma unroll
    for (int h = 0; h < WQ; ++h)
      dst[h] = __builtin_amdgcn_raw_buffer_load_b128(wres, woff + 16 * h, (gs * NBT + nb) * P::WFRAG, 0);
  };
  // weight-fragment ring: slot k holds the k-step gs (of the layer's
  // NCHUNK x NSTEP), gs % RING == k
  u32x4 bq[RING][NB][WQ];
#pragma unroll
  for (int st = 0; st < RING - 1; ++st)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      wload(slice_of(unit) * TSTEPS + (unit & (ksplit - 1)) * NCU * NSTEP + st, nb, bq[st][nb]);
  __syncthreads();  // staged chunk, bias, zero region and head weights visible

  int gchunk = 0;  // chunks processed by this workgroup (selects the LDS buffer)
  for (int it = 0; unit >= 0; ++it) {
    const int c0 = (unit & (ksplit - 1)) * NCU;  // first chunk of this unit
    const int slice = slice_of(unit);
    int next_unit;
    if (!sched || it + 1 < nstat) {
      next_unit = tile_of(blockIdx.x, gridDim.x, it + 1, nunits);
    } else {
      next_unit = (int)__builtin_amdgcn_readfirstlane(dyn_s[(it - 1) & 1]);
    }
    // unit it + 2 (written to LDS at the end of the first chunk, so that no
    // wave waits here for the counter)
    uint32_t grabbed = 0;
    if (sched && tid == 0 && it + 2 >= nstat)
      grabbed = __hip_atomic_fetch_add(grab, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int next = next_unit >= 0 ? next_unit >> (kshift + lsl) : -1;
    const int next_c0 = next_unit >= 0 ? (next_unit & (ksplit - 1)) * NCU : 0;
    const int next_slice = next_unit >= 0 ? slice_of(next_unit) : 0;
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
      // (fp8: both granules of the voxel, the tap set by the half-wave)
      rrel[mb] = (uint32_t)(lb * VSTRIDE + (F8 ? 0 : half * 16));
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
          more ? stage_rsrc<ROW>(x, cur_base, (cc + 1) * 32) : stage_rsrc<ROW>(x, next_base, next_c0 * 32);
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
      // LDS offset of tap `tap` relative to a row's (0,0,0) tap, and the
      // mask that sends a halo-column tap of a flat tile to `zero`
      auto tap_off = [&](int tap) -> uint32_t {
        const int dt = tap / (KS * KS), di = (tap / KS) % KS, dj = tap % KS;
        return (uint32_t)((dt * tl.sa + di * tl.sb + dj) * VSTRIDE);
      };
      auto tap_mask = [&](int mb, int tap) -> uint32_t {
        const int dj = tap % 3;
        return dj == 0 ? em0[mb] : (dj == 2 ? em2[mb] : 0u);
      };
      auto redirect = [&](uint32_t a, uint32_t m) -> uint32_t {
        uint32_t r;
        asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "s"(zero_addr), "v"(a));
        return r;
      };
      // B fragment of row block mb for k-step st (bf16: tap st, this lane's
      // granule; fp8: tap 2 st + half, both granules): the tap's voxel offset
      // is common to the (half-)wave; halo-column taps of flat tiles go to
      // the zero region (v_bfi keeps the low 8 address bits: same bank group,
      // so the read stays conflict-free).  rbase is made opaque before each
      // use so that every step computes its own addresses instead of the
      // compiler computing all of them at the top of the chunk.
      constexpr int AQ = F8 ? 2 : 1;  // 16-byte pieces of a B fragment
      auto frag_read = [&](int mb, int st, u32x4 (&dst)[AQ]) {
        asm volatile("" : "+v"(rbase[mb]));
        if constexpr (F8) {
          // the half-wave's tap and halo mask are selected with the lane's
          // half mask, made opaque here so that no per-step selection is
          // hoisted out of the chunk loop (it would hold 14 x 4 registers)
          uint32_t hm = hmask;
          asm volatile("" : "+v"(hm));
          const int t0 = 2 * st, t1 = 2 * st + 1 < TAPS ? 2 * st + 1 : 2 * st;  // the tap past the last: zero weights
          const uint32_t o0 = tap_off(t0), o1 = tap_off(t1);
          uint32_t a = rbase[mb] + o0 + ((o1 - o0) & hm);
          if (MODE == 0) {
            const int dj0 = t0 % 3, dj1 = t1 % 3;
            const uint32_t m0 = tap_mask(mb, t0), m1 = tap_mask(mb, t1);
            if (dj0 != 1 && dj1 != 1) {
              uint32_t m;
              asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(m) : "v"(hm), "v"(m1), "v"(m0));
              a = redirect(a, m);
            } else if (dj0 != 1) {
              a = redirect(a, m0 & ~hm);
            } else if (dj1 != 1) {
              a = redirect(a, m1 & hm);
            }
          }
          dst[0] = *(lds_u32x4*)(uintptr_t)a;
          dst[AQ - 1] = *(lds_u32x4*)(uintptr_t)(a + 16);
        } else {
          uint32_t a = rbase[mb] + tap_off(st);
          if (MODE == 0 && st % 3 != 1) a = redirect(a, tap_mask(mb, st));
          dst[0] = *(lds_u32x4*)(uintptr_t)a;
        }
      };
      auto mfma = [&](const u32x4 (&w)[WQ], const u32x4 (&a)[AQ], f32x16 c) -> f32x16 {
        if constexpr (F8) {
          const i32x8 wa = __builtin_bit_cast(i32x8, u32x8{w[0].x, w[0].y, w[0].z, w[0].w, w[WQ - 1].x,
                                                           w[WQ - 1].y, w[WQ - 1].z, w[WQ - 1].w});
          const i32x8 ab = __builtin_bit_cast(i32x8, u32x8{a[0].x, a[0].y, a[0].z, a[0].w, a[AQ - 1].x,
                                                           a[AQ - 1].y, a[AQ - 1].z, a[AQ - 1].w});
          return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wa, ab, c, 0, 0, 0, 0, 0, 0);
        } else {
          return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w[0]),
                                                         __builtin_bit_cast(bf16x8, a[0]), c, 0, 0, 0);
        }
      };
      // One register set of activation fragments (two for 32-channel
      // slices): av[mb] is re-read for the next step as soon as this step's
      // two MFMAs on it have issued, so it has the other row blocks' MFMAs to
      // arrive.  Weight fragments are loaded RING - 1 steps ahead, staging
      // rounds in the shadow of row block 0.
      // AD: steps between a fragment's read and its use -- two for 32-channel
      // slices, whose two MFMAs per step alone do not cover a read's latency
      constexpr int AD = (COUT == 32 && KS == 3) ? 2 : 1;
      u32x4 av[AD][MB][AQ];
      // Wave priority: a SIMD runs one wave of each of the two workgroups on
      // the CU; the one in its K loop goes ahead of one in staging waits or
      // the epilogue (1), and a wave about to issue MFMAs ahead of both (2),
      // which keeps the matrix pipe fed (about 2.5% less time per layer).
      // The fp8 loop, with half the MFMA cycles per fragment read, also
      // issues the next fragment reads at 2 (a further 2.5% at d = 13; no
      // gain in bf16).
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int d = 0; d < AD; ++d)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) frag_read(mb, d, av[d][mb]);
      const int gbase = slice * TSTEPS + cc * NSTEP;                  // k-step of this chunk's step 0
      const int nbase = next_slice * TSTEPS + next_c0 * NSTEP - NSTEP;  // ... of the next unit's first chunk, minus NSTEP
      // staging of the next chunk: round k is loaded at step SG k and stored
      // to LDS at step SG (k + 1), just before round k + 1 is loaded (a round
      // that would be stored past the last step is stored after it)
      auto stage_store = [&](int k) {
        // a tile's first chunk stages into the buffer the previous epilogue
        // used (transposition or head partials): wait for every wave to
        // leave it
        if (k == 0 && chunk == 0) __builtin_amdgcn_s_barrier();
        *(lds_u32x4_w*)(oth + stage_slot<KS>(k * NT + tid)) = stg;
      };
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) {
        {
          // past the chunk's last step, the last chunk of a unit runs on
          // into the next unit's first steps
          const int gs = (st + RING - 1 < NSTEP || more ? gbase : nbase) + st + RING - 1;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) wload(gs, nb, bq[(st + RING - 1) % RING][nb]);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          __builtin_amdgcn_s_setprio(2);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma(bq[st % RING][nb], av[st % AD][mb], acc[mb][nb]);
          if constexpr (!F8) __builtin_amdgcn_s_setprio(1);
          __builtin_amdgcn_sched_barrier(0);
          if (st + AD < NSTEP) frag_read(mb, st + AD, av[st % AD][mb]);
          if constexpr (F8) __builtin_amdgcn_s_setprio(1);  // fp8: the fragment reads go out at 2 too
          if (mb == 0) {
            if (st >= SG && st % SG == 0 && st / SG - 1 < RMAX) stage_store(st / SG - 1);
            if (st % SG == 0 && st / SG < RMAX) {
              const int k = st / SG;
              if (!more) soff[k] = stage_offset<ROW, MODE>(g, tl, next_src, next_base, limit, sspan, k, tid);
              stg = __builtin_amdgcn_raw_buffer_load_b128(srs, soff[k], 0, 0);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
      if constexpr (SG * RMAX >= NSTEP) stage_store(RMAX - 1);
      if (sched && tid == 0 && chunk == 0 && it + 2 >= nstat) dyn_s[it & 1] = (uint32_t)dyn_unit(grabbed);
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
      finish_tile(tile, slice, lds + ((gchunk - 1) & 1) * ABUF, acc);
    }
    unit = next_unit;
    tile = next;
    cur_base = next_base;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  finish_sched();
}

// Second kernel of a split K loop: one thread per (tile row, 8 channels)
// (activations) or per tile row (head, output layer) adds the tile's parts
// in part order, then applies the epilogue of the unsplit kernel: bias,
// activation, bf16 and a 16-byte store; or bias, activation, bf16 rounding,
// the 1x1x1 head and the threshold; or, for the output layer, bias and the
// threshold.  F8: the sums are scaled by the channel's weight scale (bias
// + cout) before the bias, and activations are stored as E4M3.
template <int EPI, int ACT, bool F8>
__global__ void __launch_bounds__(256) split_finish_kernel(Geom g, Tiling tl, int cout, int kshift,
                                                           const float* __restrict__ partial,
                                                           const float* __restrict__ bias, void* __restrict__ y,
                                                           int ystride, const float* __restrict__ head_w,
                                                           const float* __restrict__ head_b,
                                                           const int32_t* __restrict__ tables,
                                                           uint8_t* __restrict__ nib, float* __restrict__ logits,
                                                           int batch, const uint16_t* __restrict__ sc, int sc_stride,
                                                           int lsl) {
  constexpr bool ROWS8 = EPI == EPI_ACT || EPI == EPI_ADD;  // one thread per (row, 8 channels)
  // the head: one thread per (row, 8 channels) too, of every slice of the
  // row (hsl: the slices a row's lanes span), the rows' partial head sums
  // reduced over the row's consecutive lanes
  const int hsl = EPI == EPI_HEAD ? lsl : 0, tsl = lsl - hsl;
  const int groups = (ROWS8 || EPI == EPI_HEAD) ? (cout << hsl) / 8 : 1;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= ((long long)tl.ntiles << tsl) * kTileRows * groups) return;
  // (tile, output-channel slice) of this thread: activations only; the head
  // and the output layer take whole rows
  const int ts = (int)(gid / (kTileRows * groups));
  const int tile = ts >> tsl, slice = ts & ((1 << tsl) - 1);
  const int rem = (int)(gid - (long long)ts * kTileRows * groups);
  const int r = rem / groups, grp = rem - r * groups;
  const int ksplit = 1 << kshift;
  if (tsl) {  // this slice's biases, outputs, and shortcut columns or projection rows
    bias += (size_t)slice * (F8 ? 2 : 1) * cout;
    y = (char*)y + (size_t)slice * cout * (F8 ? 1 : 2);
    if (head_w) {
      head_w += (size_t)slice * cout * sc_stride;
      head_b += (size_t)slice * cout;
    } else if (sc) {
      sc = (const uint16_t*)((const char*)sc + (size_t)slice * cout * (F8 ? 1 : 2));
    }
  }
  // pre-activation of channels c .. c + 7 of this row in the slice whose
  // units are u << kshift .. (part p: + p) and biases bs: the sum over the
  // tile's parts in part order (fp8: times the channel's weight scale), plus
  // the bias
  // Parts are added strictly in part order; from four parts on they are read
  // four at a time, so the four reads go out together.
  auto sum8 = [&](int u, const float* bs, int c, float (&v)[8]) {
    if (ksplit < 4) {
      for (int p = 0; p < ksplit; ++p) {
        const float* src = partial + ((size_t)((u << kshift) + p) * kTileRows + r) * cout + c;
        const float4 a = *reinterpret_cast<const float4*>(src);
        const float4 b = *reinterpret_cast<const float4*>(src + 4);
        const float t[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = p == 0 ? t[e] : v[e] + t[e];
      }
    }
    for (int p0 = 0; p0 < ksplit && ksplit >= 4; p0 += 4) {
      float4 a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int p = p0 + q;  // < ksplit: ksplit is a power of two >= 4
        const float* src = partial + ((size_t)((u << kshift) + p) * kTileRows + r) * cout + c;
        a[q] = *reinterpret_cast<const float4*>(src);
        b[q] = *reinterpret_cast<const float4*>(src + 4);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int p = p0 + q;
        const float t[8] = {a[q].x, a[q].y, a[q].z, a[q].w, b[q].x, b[q].y, b[q].z, b[q].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = p == 0 ? t[e] : v[e] + t[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = F8 ? __builtin_fmaf(v[e], bs[cout + c + e], bs[c + e]) : v[e] + bs[c + e];
  };
  if constexpr (ROWS8) {
    long long pidx, o;
    int lb;
    if (!tile_row(g, tl, tile, r, batch, &pidx, &lb, &o)) return;
    float v[8];
    sum8(ts, bias, grp * 8, v);
    if constexpr (EPI == EPI_ADD) {  // the block's shortcut
      float pj[8];
      shortcut_of<8, F8>(sc, sc_stride, pidx, head_w, head_b, grp * 8, pj);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += pj[e];
    }
    if constexpr (F8) {
      const uint32_t w0 = e4m3_pack4(act_fn<ACT>(v[0]), act_fn<ACT>(v[1]), act_fn<ACT>(v[2]), act_fn<ACT>(v[3]));
      const uint32_t w1 = e4m3_pack4(act_fn<ACT>(v[4]), act_fn<ACT>(v[5]), act_fn<ACT>(v[6]), act_fn<ACT>(v[7]));
      *reinterpret_cast<uint2*>((uint8_t*)y + pidx * ystride + grp * 8) = uint2{w0, w1};
    } else {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = bf16_pack(act_fn<ACT>(v[2 * e]), act_fn<ACT>(v[2 * e + 1]));
      *reinterpret_cast<uint4*>((uint16_t*)y + pidx * ystride + grp * 8) = uint4{w[0], w[1], w[2], w[3]};
    }
  } else {
    int b, t, i, j;
    if (!tile_row_coords(g, tl, tile, r, batch, &b, &t, &i, &j)) return;
    float lg[4];
    if constexpr (EPI == EPI_OUT) {
      float v[8];
      sum8(ts, bias, 0, v);
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) lg[o2] = v[o2];
      if (sc) {  // residual shortcut of the last block
        const uint2 sv = *reinterpret_cast<const uint2*>(sc + padded_index(g, b, t, i, j) * sc_stride);
        lg[0] += __uint_as_float(sv.x << 16);
        lg[1] += __uint_as_float(sv.x & 0xFFFF0000u);
        lg[2] += __uint_as_float(sv.y << 16);
        lg[3] += __uint_as_float(sv.y & 0xFFFF0000u);
      }
    } else {
      // this lane's 8 channels (of slice c / cout), then the sum over the
      // row's groups (consecutive lanes, all active: a row is in range for
      // all or none)
      const int c = grp * 8, sl = c / cout, cl = c - sl * cout;
      float v[8];
      sum8((tile << hsl) | sl, bias + (size_t)sl * (F8 ? 2 : 1) * cout, cl, v);
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) lg[o2] = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = F8 ? e4m3_round(act_fn<ACT>(v[e])) : bf16_round(act_fn<ACT>(v[e]));
#pragma unroll
        for (int o2 = 0; o2 < 4; ++o2) lg[o2] += head_w[o2 * (cout << hsl) + c + e] * a;
      }
      for (int m = groups >> 1; m >= 1; m >>= 1)
#pragma unroll
        for (int o2 = 0; o2 < 4; ++o2) lg[o2] += __shfl_xor(lg[o2], m);
      if (grp != 0) return;
#pragma unroll
      for (int o2 = 0; o2 < 4; ++o2) lg[o2] += head_b[o2];
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
template <int CIN, int COUT, int EPI, int MODE, bool F8, int KS>
hipError_t launch_hidden(const Geom& g, const Tiling& tl, int act, const void* x, void* y, int ystride,
                         const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                         const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_workgroups,
                         int kshift, float* partial, const uint16_t* sc, int sc_stride, int lsl,
                         uint32_t* sched, hipStream_t stream) {
  using L = Lds<COUT, KS>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)conv_hidden_kernel<CIN, COUT, EPI, MODE, F8, KS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::total);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long nunits = tl.ntiles << (kshift + lsl);
  const long long nwg = conv_workgroups(nunits, n_workgroups);
  if (nunits <= 2 * nwg) sched = nullptr;  // every unit is one of the two fixed ones
  // fixed units per workgroup before the counters: two on box tiles; on flat
  // tiles seven eighths of a workgroup's share
  const long long share = (nunits + 7) / 8 / (nwg / 8);
  const int nstat = tl.mode == 0 ? (int)std::max(2ll, share * 7 / 8) : 2;
  hipLaunchKernelGGL((conv_hidden_kernel<CIN, COUT, EPI, MODE, F8, KS>), dim3((unsigned)nwg), dim3(NT),
                     (size_t)L::total, stream, g, tl, act, x, y, ystride, (const u32x4*)wfrag, bias, head_w,
                     head_b, tables, nib, logits, batch, kshift, partial, sc, sc_stride, lsl, sched, nstat);
  return hipSuccess;
}

template <int CIN, int COUT, int EPI, int MODE, bool F8, int KS>
hipError_t launch_one(const Geom& g, const Tiling& tl, int act, const void* x, void* y, int ystride,
                      const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                      const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_workgroups,
                      const Split_k& sk, const uint16_t* sc, int sc_stride, hipStream_t stream) {
  hipError_t e;
  // a head over output slices (a small batch): every unit parks its
  // slice's sums, and the second kernel finishes whole rows, head and
  // threshold included (32-channel slices exist only for this)
  constexpr bool PARK_ONLY = EPI == EPI_HEAD && COUT == 32;
  if constexpr (!PARK_ONLY) {
    if (sk.kshift == 0 && !(EPI == EPI_HEAD && sk.lsl > 0)) {
      e = launch_hidden<CIN, COUT, EPI, MODE, F8, KS>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,
                                                      tables, nib, logits, batch, n_workgroups, 0, nullptr, sc,
                                                      sc_stride, sk.lsl, sk.sched, stream);
      return e != hipSuccess ? e : hipGetLastError();
    }
  }
  // K loops split: park the parts, then add them and finish the tiles
  e = launch_hidden<CIN, COUT, EPI_PARK, MODE, F8, KS>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,
                                                       tables, nib, logits, batch, n_workgroups, sk.kshift,
                                                       sk.partial, nullptr, 0, sk.lsl, sk.sched, stream);
  if (e != hipSuccess) return e;
  const long long threads = ((long long)tl.ntiles << sk.lsl) * kTileRows *
                            (EPI == EPI_ACT || EPI == EPI_ADD || EPI == EPI_HEAD ? COUT / 8 : 1);
  static_assert(EPI != EPI_HEAD || (64 % (COUT / 8) == 0), "a row's head lanes lie in one wave");
  if (EPI == EPI_HEAD && (COUT << sk.lsl) / 8 > 64) return hipErrorInvalidValue;
  with_activation(act, [&](auto A) {
    hipLaunchKernelGGL((split_finish_kernel<EPI, decltype(A)::value, F8>), dim3((unsigned)((threads + 255) / 256)),
                       dim3(256), 0, stream, g, tl, COUT, sk.kshift, sk.partial, bias, y, ystride, head_w, head_b,
                       tables, nib, logits, batch, sc, sc_stride, sk.lsl);
  });
  return hipGetLastError();
}

template <bool F8>
hipError_t launch_case(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x, void* y,
                       int ystride, const void* wfrag, const float* bias, int head, const float* head_w,
                       const float* head_b, const int32_t* tables, uint8_t* nib, float* logits, int batch,
                       int n_workgroups, const Split_k& sk, const uint16_t* sc, int sc_stride, int ks,
                       hipStream_t stream) {
#define PD_HIDDEN_CASE(CI, CO, E)                                                                      \
  if (ks == 3 && cin == CI && cout == CO && head == E) {                                              \
    if (tl.mode == 0)                                                                                  \
      return launch_one<CI, CO, E, 0, F8, 3>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,  \
                                             tables, nib, logits, batch, n_workgroups, sk, sc,          \
                                             sc_stride, stream);                                         \
    return launch_one<CI, CO, E, 1, F8, 3>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,    \
                                           tables, nib, logits, batch, n_workgroups, sk, sc, sc_stride, \
                                           stream);                                                      \
  }
// 5x5x5 layers (Model 3 of Table models): box tiles only
#define PD_HIDDEN_CASE5(CI, CO, E)                                                                     \
  if (ks == 5 && cin == CI && cout == CO && head == E && tl.mode == 1)                                \
    return launch_one<CI, CO, E, 1, F8, 5>(g, tl, act, x, y, ystride, wfrag, bias, head_w, head_b,    \
                                           tables, nib, logits, batch, n_workgroups, sk, sc, sc_stride, \
                                           stream);
  PD_HIDDEN_CASE(64, 64, EPI_ACT)
  PD_HIDDEN_CASE(64, 32, EPI_ACT)   // 64- to 256-wide layers in 32-channel slices (small batches)
  PD_HIDDEN_CASE(128, 32, EPI_ACT)
  PD_HIDDEN_CASE(256, 32, EPI_ACT)
  PD_HIDDEN_CASE(128, 128, EPI_ACT)
  PD_HIDDEN_CASE(64, 128, EPI_ACT)
  PD_HIDDEN_CASE(128, 64, EPI_ACT)
  PD_HIDDEN_CASE(256, 128, EPI_ACT)
  PD_HIDDEN_CASE(256, 64, EPI_ACT)
  PD_HIDDEN_CASE(64, 64, EPI_HEAD)
  PD_HIDDEN_CASE(128, 128, EPI_HEAD)
  PD_HIDDEN_CASE(64, 128, EPI_HEAD)
  PD_HIDDEN_CASE(128, 64, EPI_HEAD)
  PD_HIDDEN_CASE(64, 32, EPI_HEAD)  // the head layer in 32-channel slices (small batches)
  PD_HIDDEN_CASE(128, 32, EPI_HEAD)
  // the residual network's layers (bf16 and fp8)
  PD_HIDDEN_CASE(512, 128, EPI_ACT)
  PD_HIDDEN_CASE(64, 64, EPI_ADD)
  PD_HIDDEN_CASE(128, 128, EPI_ADD)
  PD_HIDDEN_CASE(256, 128, EPI_ADD)
  PD_HIDDEN_CASE(512, 128, EPI_ADD)
  if constexpr (!F8) {
    PD_HIDDEN_CASE5(64, 64, EPI_ACT)
    PD_HIDDEN_CASE5(128, 128, EPI_ACT)
  }
  if (cout == 4) cout = 32;  // the output layer's 4 filters fill one padded block
  if constexpr (!F8) {
    // the 5x5x5 output layer (3x3x3 ones run on launch_conv_out)
    PD_HIDDEN_CASE5(64, 32, EPI_OUT)
    PD_HIDDEN_CASE5(128, 32, EPI_OUT)
  }
#undef PD_HIDDEN_CASE
#undef PD_HIDDEN_CASE5
  return hipErrorInvalidValue;
}

}  // namespace

int conv_hidden_max_span(int ks) { return ks == 5 ? Conv<5>::MAX_SPAN : Conv<3>::MAX_SPAN; }
size_t conv_hidden_partial_floats_per_unit() { return (size_t)kTileRows * 128; }
int conv_hidden_workgroups_per_cu(int ks) { return ks == 5 ? Conv<5>::WG_PER_CU : Conv<3>::WG_PER_CU; }

hipError_t launch_conv_hidden(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x,
                              void* y, int ystride, const void* wfrag, const float* bias, int head,
                              const float* head_w, const float* head_b, const int32_t* tables, uint8_t* nib,
                              float* logits, int batch, int n_workgroups, const Split_k& sk, int fp8,
                              const uint16_t* sc, int sc_stride, int ks, hipStream_t stream) {
  if (ks != 3 && ks != 5) return hipErrorInvalidValue;
  if (tl.span <= 0 || tl.span > conv_hidden_max_span(ks)) return hipErrorInvalidValue;
  // a shortcut projected in the epilogue: from at most 8 channels of sc
  if (head == 4 && head_w && (!head_b || !sc || sc_stride < 1 || sc_stride > 8)) return hipErrorInvalidValue;
  // the halo holds every tap: a 5x5x5 layer needs the two-voxel halo (and box tiles)
  if ((ks - 1) / 2 > g.pad || (tl.mode == 0 && g.pad != 1)) return hipErrorInvalidValue;
  // parts per tile: a power of two dividing the layer's chunks, with room
  // for every unit's sums
  const int nchunk = cin / (fp8 ? Prec<true, 3>::KCH : Prec<false, 3>::KCH);
  if (sk.kshift < 0 || nchunk % (1 << sk.kshift) != 0 ||
      (sk.kshift > 0 && (tl.ntiles << (sk.kshift + sk.lsl)) > sk.max_units))
    return hipErrorInvalidValue;
  // output-channel slices: up to max_slices, of activation layers, or of 32
  // or 64 channels for a head (whose rows the second kernel finishes; an
  // output layer needs every channel of a voxel in one unit)
  const bool head_slices = head == EPI_HEAD && (cout == 32 || (cout == 64 && sk.lsl > 0));
  if (sk.lsl < 0 || (1 << sk.lsl) > max_slices(cout) ||
      (sk.lsl > 0 && head != EPI_ACT && head != EPI_ADD && !head_slices))
    return hipErrorInvalidValue;
  // a sliced head parks every unit's sums, also with whole K loops
  if (head_slices && (!sk.partial || (tl.ntiles << (sk.kshift + sk.lsl)) > sk.max_units)) return hipErrorInvalidValue;
  if (fp8)
    return launch_case<true>(g, tl, cin, cout, act, x, y, ystride, wfrag, bias, head, head_w, head_b, tables, nib,
                             logits, batch, n_workgroups, sk, sc, sc_stride, ks, stream);
  return launch_case<false>(g, tl, cin, cout, act, x, y, ystride, wfrag, bias, head, head_w, head_b, tables, nib,
                            logits, batch, n_workgroups, sk, sc, sc_stride, ks, stream);
}

int conv_hidden_chunk_channels(int fp8) { return fp8 ? Prec<true, 3>::KCH : Prec<false, 3>::KCH; }

}  // namespace pd
