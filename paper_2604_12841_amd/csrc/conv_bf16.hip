// conv_bf16.hip -- K2 + K3 (+ K4 for the last layer): one 3x3x3 conv3d layer
// (Sec. IV.B, Fig. ConvArch; stride 1, zero padding, cross-correlation) as an
// implicit GEMM on the gfx950 matrix cores, with the bias + activation + bf16
// rounding epilogue fused in; for the last hidden layer the epilogue also
// applies the 1x1x1 head and the threshold (logit > 0) and writes one flip
// nibble per voxel instead of the activations.
//
//   out[co][m] = act(bias[co] + sum_{tap, ci} W[co][ci][tap] * X[m + shift(tap)][ci])
//
// GEMM view (transposed so the epilogue holds 4 consecutive channels per
// lane): rows = c_out, columns = output voxels, K = 27 * c_in.  Activations
// live in the zero-halo NTHWC layout of internal.h, so every tap is an index
// shift and the K loop has no bounds checks.
//
// Work split: persistent workgroups of 512 threads (8 wave64, two per SIMD),
// one per CU.  A tile is 256 output voxels x all c_out channels; wave w owns
// voxels [128 (w % 2), +128) and channels [32 (w / 2), +32) for c_out = 128
// (64-voxel x 32-channel blocks for c_out = 64), i.e. 4 (2) blocks of
// v_mfma_f32_32x32x16_bf16 with fp32 accumulators.
//   * The input footprint of a tile is staged in LDS 32 input channels (64
//     bytes per voxel) at a time, double buffered, through registers: the
//     next chunk -- or, during the last chunk, the next tile's first chunk --
//     is loaded from HBM/L2 in 7 rounds spread over the current chunk's
//     k-steps and written to the other buffer.
//   * A staged voxel occupies 80 bytes of LDS (its 64 bytes of channels plus
//     16 of padding).  The LDS serves a 16-byte read 16 lanes at a time over
//     64 banks (16 groups of 16 bytes); granule g of voxel v sits in bank
//     group (5 v + g) mod 16, so any 16 consecutive staged voxels hit 16
//     distinct groups, and the tilings keep the 16 voxels of a read
//     consecutive (flat tiles stage only the real columns; box tiles are 16
//     voxels wide in j).  Addresses stay linear: a fragment address is a
//     per-lane base plus a tap offset common to the wave.
//   * The 54 k-steps of a chunk (27 taps x 2) are fully unrolled and software
//     pipelined: activation fragments are read from LDS one step ahead, weight
//     fragments (pre-arranged at create time in MFMA operand order, one
//     coalesced 16-byte load per lane; a layer is <= 0.9 MB and stays in L2)
//     five steps ahead through a 6-deep register ring.
//   * Epilogue: + bias, activation in fp32, bf16 (RNE), written to an LDS
//     copy of the output tile and stored as whole voxel rows with 16-byte
//     stores into the interior of the output (the halo is never written).
// Layer 1 (c_in = 2) uses the same tiles with K = 27 taps x 2 channels padded
// to 64 (4 k-steps): each lane gathers 4 taps x 2 channels per fragment.
#include "internal.h"

namespace pd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) const uint32_t lds_u32;
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_w;
typedef __attribute__((address_space(3))) uint32_t lds_u32_w;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2_w;
typedef __attribute__((address_space(3))) int lds_i32;

constexpr int KC = 32;     // input channels per LDS chunk
constexpr int STEPS = 54;  // k-steps per chunk: 27 taps x 2 (16 channels each)
constexpr int BRING = 6;   // weight-fragment ring depth (prefetch distance BRING - 1)
constexpr int NT = 512;    // threads per workgroup: 8 wave64, two per SIMD
// Every chunk is staged with exactly RMAX rounds of NT 16-byte granules (896
// voxels at most); rounds past the footprint load voxel 0 and store to a
// scratch region, so every wave issues the same fixed sequence.
constexpr int RMAX = 7;
constexpr int VSTRIDE = 80;                            // LDS bytes per staged voxel
constexpr int ABUF = RMAX * (NT / 4) * VSTRIDE;        // bytes per staging buffer
constexpr int PLANE_RMAX = 2;                          // layer 1: rounds of NT voxels x 4 bytes
constexpr int TRASH = NT * 16;                         // destination of unused rounds

// Wave split of the 256 x COUT output tile: WN waves across the channels (32
// each), WM across the voxels (ROWS each, MB blocks of 32).
template <int COUT>
struct WaveSplit {
  static constexpr int WN = COUT / 32;
  static constexpr int WM = (NT / 64) / WN;
  static constexpr int ROWS = 256 / WM;
  static constexpr int MB = ROWS / 32;
};

// LDS layout of one workgroup (byte offsets): two staging buffers, the
// scratch round, a 256-byte zero region (256-aligned, for halo-column reads),
// the bias [COUT] and the head weights [4][COUT].  The epilogues reuse the
// staging buffer the tile read last (output tile, row table, head partials).
template <int COUT>
struct LdsLayout {
  static constexpr int buf1 = ABUF;
  static constexpr int trash = 2 * ABUF;
  static constexpr int zero = trash + TRASH;
  static constexpr int bias = zero + 256;
  static constexpr int headw = bias + COUT * 4;
  static constexpr int total = headw + 4 * COUT * 4;
  static_assert(zero % 256 == 0, "zero region must be 256-aligned");
  static_assert(total <= 160 * 1024, "LDS budget");
};

__device__ __forceinline__ float activation(float y, int act) {
  if (act == 1) {  // GELU, tanh form: 0.5 y (1 + tanh(u)) = y / (1 + exp(-2u))
    const float k0 = 0.7978845608028654f;          // sqrt(2 / pi)
    const float kl = -2.0f * 1.4426950408889634f;  // -2 log2(e)
    float u = k0 * (y + 0.044715f * y * y * y);
    float e = __builtin_amdgcn_exp2f(kl * u);
    return y * __builtin_amdgcn_rcpf(1.0f + e);
  }
  if (act == 2) return y > 0.0f ? y : 0.0f;
  return y;
}

__device__ __forceinline__ uint32_t bf16_bits(float v) {
  __bf16 h = (__bf16)v;
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float bf16_round(float v) { return __uint_as_float(bf16_bits(v) << 16); }

// Row r (0..255) of tile `tile`: false if the row is outside the volume,
// else its padded output index (pidx) and its column j (col).  Also the LDS
// voxel of the row's (0,0,0) tap (lds_base) and the staging origin: the
// line-space index of staged voxel 0 (mode 0) or its padded index (mode 1).
// 32-bit voxel counts: the host guarantees max_batch * V < 2^31.
__host__ __device__ inline bool tile_row(const Geom& g, const Tiling& tl, int tile, int r, int batch,
                                         long long* pidx, int* lds_base, long long* stage_origin,
                                         int* col = nullptr) {
  const int HH = g.H * g.H;
  if (tl.mode == 0) {
    const int seg = tile / tl.tiles_per_seg;
    const int k0 = (tile - seg * tl.tiles_per_seg) * kTileRows;
    const int u0 = seg * (int)tl.seg_len + k0;
    const int b0 = u0 / g.V;
    const int v0 = u0 - b0 * g.V;
    const int t0 = v0 / HH, s0 = v0 - t0 * HH;
    const long long l0 = line_index(g, b0, t0, s0 / g.H, s0 % g.H);
    *stage_origin = l0 - (line_plane(g) + g.H + 1);
    const int u = u0 + r;
    if (k0 + r >= tl.seg_len || u >= batch * g.V) {
      *lds_base = 0;
      if (col) *col = -1;
      return false;
    }
    const int b = u / g.V;
    const int v = u - b * g.V;
    const int t = v / HH, s = v - t * HH;
    const int i = s / g.H, j = s - i * g.H;
    *pidx = padded_index(g, b, t, i, j);
    *lds_base = (int)(line_index(g, b, t, i, j) - l0);
    if (col) *col = j;
    return true;
  } else {
    const int per = tl.ntT * tl.ntI * tl.ntJ;
    const int b = tile / per;
    const int rem = tile - b * per;
    const int tt = rem / (tl.ntI * tl.ntJ);
    const int ti = (rem / tl.ntJ) % tl.ntI;
    const int tj = rem % tl.ntJ;
    const int t0 = tt * tl.BT, i0 = ti * tl.BI, j0 = tj * tl.BJ;
    *stage_origin = (long long)b * g.S + (long long)t0 * g.P + (long long)i0 * g.Wp + j0;
    const int bij = tl.BI * tl.BJ;
    const int a = r / bij, c = (r / tl.BJ) % tl.BI, e = r % tl.BJ;
    const int t = t0 + a, i = i0 + c, j = j0 + e;
    const bool ok = (r < tl.BT * bij) && t < g.T && i < g.H && j < g.H;
    *lds_base = ok ? (a * (tl.BI + 2) + c) * (tl.BJ + 2) + e : 0;
    if (col) *col = ok ? j : -1;
    if (!ok) return false;
    *pidx = padded_index(g, b, t, i, j);
    return true;
  }
}

// Padded (t, i, j) of a box-mode tile's staging origin.
struct BoxOrigin {
  int t0, i0, j0;
};

__host__ __device__ inline BoxOrigin box_origin(const Geom& g, const Tiling& tl, long long origin) {
  BoxOrigin bo{0, 0, 0};
  if (tl.mode == 1) {
    const long long rem = origin % g.S;
    bo.t0 = (int)(rem / g.P);
    const int r2 = (int)(rem - (long long)bo.t0 * g.P);
    bo.i0 = r2 / g.Wp;
    bo.j0 = r2 - bo.i0 * g.Wp;
  }
  return bo;
}

// Global padded voxel of staged voxel vv (clamped to voxel 0, a zero halo
// voxel, when outside the batch or outside the sample's padded box).
__host__ __device__ inline long long staged_voxel(const Geom& g, const Tiling& tl, long long origin,
                                                  const BoxOrigin& bo, int vv, long long limit) {
  if (tl.mode == 0) {
    const long long p = line_to_padded(g, origin + vv);
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

// Tile handled by persistent workgroup `wg` at iteration `it`: the 8 XCDs
// receive workgroups round-robin, so workgroup wg runs on XCD wg % 8; each
// XCD gets a contiguous range of tiles (neighbouring tiles share halo voxels
// in its L2) and its workgroups stride through it.  -1 when done.
__host__ __device__ inline int tile_of(int wg, int nwg, int it, int ntiles) {
  const int xcd = wg & 7, k = wg >> 3, per_xcd_wg = nwg >> 3;
  const int per_xcd = (ntiles + 7) >> 3;
  const int idx = k + it * per_xcd_wg;
  if (idx >= per_xcd) return -1;
  const int t = xcd * per_xcd + idx;
  return t < ntiles ? t : -1;
}

// Staging source of a tile: its staging origin (see tile_row) and box origin.
struct StageSrc {
  long long origin;
  BoxOrigin bo;
};

// Global padded voxel of staged voxel vv; -1 when it is outside the batch or
// the sample's padded box (such voxels only feed rows that are discarded).
template <int MODE>
__host__ __device__ inline long long staged_voxel_fast(const Geom& g, const Tiling& tl, const StageSrc& src,
                                                       int vv, long long limit) {
  if constexpr (MODE == 0) {
    const uint32_t u = (uint32_t)(src.origin + vv);  // < 2^31 (host check)
    const uint32_t tp = fastdiv(u, tl.div_a);
    const uint32_t rem = u - tp * (uint32_t)tl.sa;
    const uint32_t ip = fastdiv(rem, tl.div_b);
    const uint32_t jj = rem - ip * (uint32_t)g.H;
    const long long p = (long long)tp * g.P + (long long)ip * g.Wp + jj + 1;
    return p < limit ? p : -1;
  } else {
  const int a = (int)fastdiv((uint32_t)vv, tl.div_a);
  const int rem = vv - a * tl.sa;
  const int c = (int)fastdiv((uint32_t)rem, tl.div_b);
  const int e = rem - c * tl.sb;
  if (src.bo.t0 + a >= g.T + 2 || src.bo.i0 + c >= g.Wp || src.bo.j0 + e >= g.Wp) return -1;
  return src.origin + (long long)a * g.P + (long long)c * g.Wp + e;
  }
}

// Staging granule q = NT k + tid is granule q & 3 (16 bytes) of
// staged voxel vv = q >> 2 (of 32-channel chunk `chunk`); it goes to LDS byte
// vv * VSTRIDE + 16 (q & 3).  Granules past the footprint (or of voxels
// outside the volume) read voxel 0 instead.
template <int CIN, int MODE>
__device__ __forceinline__ u32x4 stage_load(const Geom& g, const Tiling& tl, const uint16_t* __restrict__ x,
                                            const StageSrc& src, long long limit, int chunk, int ngran, int k,
                                            int tid) {
  const int q = k * NT + tid;
  const int vv = q >> 2;
  const int sg = q & 3;
  long long gv = staged_voxel_fast<MODE>(g, tl, src, vv, limit);
  gv = (q < ngran && gv >= 0) ? gv : 0;
  return *reinterpret_cast<const u32x4*>(x + gv * CIN + chunk * KC + sg * 8);
}

// Layer 1: both channels (4 bytes) of staged voxel NT k + tid.
__device__ __forceinline__ uint32_t plane_load(const Geom& g, const Tiling& tl, const uint16_t* __restrict__ x,
                                               const StageSrc& src, long long limit, int k, int tid) {
  const int vv = k * NT + tid;
  const long long gv = staged_voxel(g, tl, src.origin, src.bo, vv < tl.span ? vv : 0, limit);
  return reinterpret_cast<const uint32_t*>(x)[gv];
}

template <int CIN, int COUT, bool HEAD, int MODE>
__global__ void __launch_bounds__(NT) conv_bf16_kernel(Geom g, Tiling tl, int act,
                                                       const uint16_t* __restrict__ x,
                                                       uint16_t* __restrict__ y,
                                                       const u32x4* __restrict__ wfrag,
                                                       const float* __restrict__ bias,
                                                       const float* __restrict__ head_w,
                                                       const float* __restrict__ head_b,
                                                       const int32_t* __restrict__ comp_of_site,
                                                       uint8_t* __restrict__ nib, float* __restrict__ logits,
                                                       int batch) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  using W = WaveSplit<COUT>;
  constexpr int MB = W::MB;       // 32-voxel blocks per wave
  constexpr int NBT = COUT / 32;  // 32-channel blocks in total (one per column wave)
  constexpr int NCHUNK = (CIN == 2) ? 1 : CIN / KC;
  constexpr int TSTEPS = NCHUNK * STEPS;  // k-steps per tile (hidden layers)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % W::WM, wn = wave / W::WM;
  const int half = lane >> 5, l32 = lane & 31;
  const int ntiles = (int)tl.ntiles;
  const long long limit = (long long)batch * g.S;
  const int ngran = tl.span * 4;  // 16-byte granules of a staged chunk

  using L = LdsLayout<COUT>;
  lds_char* const lds = (lds_char*)smem;
  lds_char* const trash = lds + L::trash;
  lds_char* const zero = lds + L::zero;
  lds_float* const bias_s = (lds_float*)(lds + L::bias);
  lds_float* const headw_s = (lds_float*)(lds + L::headw);
  for (int e = tid; e < COUT; e += NT) bias_s[e] = bias[e];
  if (tid < 64) ((lds_u32_w*)zero)[tid] = 0u;
  const uint32_t zero_addr = (uint32_t)(uintptr_t)zero;
  if (HEAD)
    for (int e = tid; e < 4 * COUT; e += NT) headw_s[e] = head_w[e];

  int tile = tile_of(blockIdx.x, gridDim.x, 0, ntiles);
  if (tile < 0) return;

  auto source_of = [&](int t) {
    StageSrc src;
    long long p;
    int lb;
    tile_row(g, tl, t, 0, batch, &p, &lb, &src.origin);
    src.bo = box_origin(g, tl, src.origin);
    return src;
  };
  StageSrc cur_src = source_of(tile);

  // First tile: stage its first chunk synchronously.
  if constexpr (CIN == 2) {
#pragma unroll
    for (int k = 0; k < PLANE_RMAX; ++k) {
      const uint32_t v = plane_load(g, tl, x, cur_src, limit, k, tid);
      *(lds_u32_w*)(lds + (k * NT + tid) * 4) = v;
    }
  } else {
#pragma unroll
    for (int k = 0; k < RMAX; ++k) {
      const u32x4 v = stage_load<CIN, MODE>(g, tl, x, cur_src, limit, 0, ngran, k, tid);
      const int q = k * NT + tid;
      *(lds_u32x4_w*)(lds + (q >> 2) * VSTRIDE + (q & 3) * 16) = v;
    }
  }

  // weight fragment (tile-step gs) of this wave's 32 channels: a uniform base
  // plus this lane's 16-byte slot, so the load can use a scalar base
  const uint32_t woff = (uint32_t)((wn * 64 + lane) * 16);
  auto wload = [&](int gs) -> u32x4 {
    return *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(wfrag) + (size_t)gs * NBT * 1024 + woff);
  };
  // weight-fragment ring (hidden layers): slot k holds tile-step gs, gs % BRING == k
  u32x4 bq[BRING];
  if constexpr (CIN != 2) {
#pragma unroll
    for (int st = 0; st < BRING - 1; ++st) bq[st] = wload(st);
  }
  __syncthreads();  // staged chunk, bias and head weights visible

  int gchunk = 0;  // chunks processed by this workgroup (selects the LDS buffer)
  for (int it = 0; tile >= 0; ++it) {
    const int next = tile_of(blockIdx.x, gridDim.x, it + 1, ntiles);
    const StageSrc next_src = source_of(next >= 0 ? next : tile);
    // rows of this lane: voxel wm ROWS + 32 mb + l32 of the tile
    int rb[MB];
    int pidx[MB];
    uint32_t em0[MB], em2[MB];  // flat tiles: reads of the left / right halo column go to `zero`
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      long long p = -1, o;
      int lb = 0, col = -1;
      bool ok = tile_row(g, tl, tile, wm * W::ROWS + mb * 32 + l32, batch, &p, &lb, &o, &col);
      rb[mb] = lb;
      pidx[mb] = ok ? (int)p : -1;
      em0[mb] = (MODE == 0 && col == 0) ? 0xFFFFFF00u : 0u;
      em2[mb] = (MODE == 0 && col == g.H - 1) ? 0xFFFFFF00u : 0u;
    }

    f32x16 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][v] = 0.0f;

    if constexpr (CIN == 2) {
      lds_char* const cur = lds + (gchunk & 1) * ABUF;
      lds_char* const oth = (next >= 0) ? lds + ((gchunk + 1) & 1) * ABUF : trash;
      // next tile's planes into registers while this tile computes
      uint32_t nxt[PLANE_RMAX];
#pragma unroll
      for (int k = 0; k < PLANE_RMAX; ++k) nxt[k] = plane_load(g, tl, x, next_src, limit, k, tid);
      lds_u32* a32 = (lds_u32*)cur;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u32x4 wf = wload(ks);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          u32x4 av;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int tap = ks * 8 + half * 4 + q;
            uint32_t val = 0;
            if (tap < 27) {
              const int dt = tap / 9, di = (tap / 3) % 3, dj = tap % 3;
              val = a32[rb[mb] + dt * tl.sa + di * tl.sb + dj];
              if ((dj == 0 && em0[mb]) || (dj == 2 && em2[mb])) val = 0;
            }
            av[q] = val;
          }
          acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wf),
                                                            __builtin_bit_cast(bf16x8, av), acc[mb], 0, 0, 0);
        }
      }
#pragma unroll
      for (int k = 0; k < PLANE_RMAX; ++k)
        *(lds_u32_w*)(oth + ((next >= 0 ? k * NT : 0) + tid) * 4) = nxt[k];
      ++gchunk;
    } else {
      for (int chunk = 0; chunk < NCHUNK; ++chunk, ++gchunk) {
        lds_char* const cur = lds + (gchunk & 1) * ABUF;
        // the chunk staged next: the following chunk of this tile, else the
        // first chunk of the next tile, else nothing (scratch)
        const bool more = chunk + 1 < NCHUNK;
        const bool real = more || next >= 0;
        const StageSrc& ssrc = more ? cur_src : next_src;
        const int schunk = more ? chunk + 1 : 0;
        const int sgran = real ? ngran : 0;
        lds_char* const oth = lds + ((gchunk + 1) & 1) * ABUF;
        u32x4 stg;

        // Per-lane LDS bases of the row blocks (this lane's voxel, its
        // granule half) -- opaque so the per-step addresses are not hoisted
        // out of the chunk loop -- and the halo-column masks.
        uint32_t rbase[MB], e0c[MB], e2c[MB];
        const uint32_t cur_u = (uint32_t)(uintptr_t)cur;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          rbase[mb] = cur_u + (uint32_t)(rb[mb] * VSTRIDE + half * 16);
          e0c[mb] = em0[mb];
          e2c[mb] = em2[mb];
          asm volatile("" : "+v"(rbase[mb]), "+v"(e0c[mb]), "+v"(e2c[mb]));
        }
        // LDS address of the fragment of row block mb for k-step st: the
        // tap's voxel offset and the k-step's granule pair are common to the
        // wave; halo-column taps of flat tiles go to the zero region (same
        // bank group, so the read stays conflict-free)
        auto frag_addr = [&](int mb, int st) -> uint32_t {
          const int tap = st >> 1, ks = st & 1;
          const int dt = tap / 9, di = (tap / 3) % 3, dj = tap % 3;
          const uint32_t toff = (uint32_t)((dt * tl.sa + di * tl.sb + dj) * VSTRIDE + ks * 32);
          uint32_t a = rbase[mb] + toff;
          if (MODE == 0 && dj == 0) a = (a & ~e0c[mb]) | (zero_addr & e0c[mb]);
          if (MODE == 0 && dj == 2) a = (a & ~e2c[mb]) | (zero_addr & e2c[mb]);
          return a;
        };
        // Each step has two scheduling regions: (A) the LDS reads of the next
        // step's activation fragments (addresses computed a step earlier) and
        // the weight load five steps ahead; (B) this step's MFMAs, with the
        // address arithmetic for two steps ahead and the staging work in
        // their shadow.  The other wave of the SIMD fills the gaps.
        u32x4 av[2][MB];
        uint32_t an[MB];  // LDS addresses of the fragments of step st + 1
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) av[0][mb] = *(lds_u32x4*)(uintptr_t)frag_addr(mb, 0);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) an[mb] = frag_addr(mb, 1);
        const int gbase = chunk * STEPS;  // tile-step of this chunk's step 0
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
          // ---- region A ----
          if (st + 1 < STEPS) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) av[(st + 1) & 1][mb] = *(lds_u32x4*)(uintptr_t)an[mb];
          }
          {
            int gs = gbase + st + BRING - 1;  // wraps into the next tile's steps
            if (gs >= TSTEPS) gs -= TSTEPS;
            bq[(st + BRING - 1) % BRING] = wload(gs);
          }
          __builtin_amdgcn_sched_barrier(0);
          // ---- region B ----
          if (st + 2 < STEPS) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) an[mb] = frag_addr(mb, st + 2);
          }
          // staging of the next chunk: round k is loaded at step 6k and
          // stored to LDS at step 6k + 6, just before round k + 1 is loaded
          if (st >= 6 && st % 6 == 0 && st / 6 - 1 < RMAX) {
            const int k = st / 6 - 1;
            const int q = k * NT + tid;
            lds_char* dst = (k * NT < sgran) ? oth + (q >> 2) * VSTRIDE + (q & 3) * 16 : trash + tid * 16;
            *(lds_u32x4_w*)dst = stg;
          }
          if (st % 6 == 0 && st / 6 < RMAX)
            stg = stage_load<CIN, MODE>(g, tl, x, ssrc, limit, schunk, sgran, st / 6, tid);
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bq[st % BRING]),
                                                              __builtin_bit_cast(bf16x8, av[st & 1][mb]), acc[mb],
                                                              0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
        // every wave's staging writes done, every wave done reading `cur`
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
      }
    }

    // ---- epilogue: lane holds channels co .. co + 3 (co = 32 wn + 8 q +
    // 4 half) of voxel row wm ROWS + 32 mb + l32; the buffer this tile read
    // last is free for the output tile / head partials ----
    lds_char* const obuf = lds + ((gchunk - 1) & 1) * ABUF;
    if constexpr (CIN == 2) {
      // layer 1 read its planes from this buffer: every wave must be done
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_s_barrier();
    }
    if constexpr (!HEAD) {
      // bias + activation + bf16 into an LDS copy of the output tile, then
      // whole voxel rows go out as coalesced 16-byte stores (full cache lines)
      constexpr int OSTR = COUT * 2 + 16;  // padded row stride of the output tile
      static_assert(256 * OSTR + 256 * 4 <= ABUF, "output tile fits a staging buffer");
      lds_i32* const orow = (lds_i32*)(obuf + 256 * OSTR);  // padded output index per row, -1 if none
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int co = wn * 32 + q * 8 + half * 4;
        const float4 bv = {bias_s[co], bias_s[co + 1], bias_s[co + 2], bias_s[co + 3]};
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const float v0 = activation(acc[mb][4 * q + 0] + bv.x, act);
          const float v1 = activation(acc[mb][4 * q + 1] + bv.y, act);
          const float v2 = activation(acc[mb][4 * q + 2] + bv.z, act);
          const float v3 = activation(acc[mb][4 * q + 3] + bv.w, act);
          u32x2 packed;
          packed.x = bf16_bits(v0) | (bf16_bits(v1) << 16);
          packed.y = bf16_bits(v2) | (bf16_bits(v3) << 16);
          const int row = wm * W::ROWS + mb * 32 + l32;
          *(lds_u32x2_w*)(obuf + row * OSTR + co * 2) = packed;
        }
      }
      if (wn == 0 && half == 0) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) orow[wm * W::ROWS + mb * 32 + l32] = pidx[mb];
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
      constexpr int GPR = COUT / 8;  // 16-byte granules per voxel row
#pragma unroll
      for (int it2 = 0; it2 < 256 * GPR / NT; ++it2) {
        const int qq = it2 * NT + tid;
        const int row = qq / GPR, c = qq % GPR;
        const int p = orow[row];
        const u32x4 v = *(lds_u32x4*)(obuf + row * OSTR + c * 16);
        if (p >= 0) *reinterpret_cast<u32x4*>(y + (long long)p * COUT + c * 8) = v;
      }
    } else {
      // 1x1x1 head on the bf16-rounded activations: partial sums over this
      // lane's channels, then over the half-waves, then over the column waves
      lds_float* const head_part = (lds_float*)obuf;  // [WN][256][4]
      float part[MB][4];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int o = 0; o < 4; ++o) part[mb][o] = 0.0f;
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
          const float a0 = bf16_round(activation(acc[mb][4 * q + 0] + bv.x, act));
          const float a1 = bf16_round(activation(acc[mb][4 * q + 1] + bv.y, act));
          const float a2 = bf16_round(activation(acc[mb][4 * q + 2] + bv.z, act));
          const float a3 = bf16_round(activation(acc[mb][4 * q + 3] + bv.w, act));
#pragma unroll
          for (int o = 0; o < 4; ++o) part[mb][o] += hw[o].x * a0 + hw[o].y * a1 + hw[o].z * a2 + hw[o].w * a3;
        }
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int o = 0; o < 4; ++o) part[mb][o] += __shfl_xor(part[mb][o], 32);
      if (half == 0) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          lds_float* hp = head_part + (wn * 256 + wm * W::ROWS + mb * 32 + l32) * 4;
          hp[0] = part[mb][0];
          hp[1] = part[mb][1];
          hp[2] = part[mb][2];
          hp[3] = part[mb][3];
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): partials written
      __builtin_amdgcn_s_barrier();
      // one thread per voxel row: logits, threshold, flip nibble
      if (tid < 256) {
        const int r = tid;
        long long p = -1, o2;
        int lb;
        if (tile_row(g, tl, tile, r, batch, &p, &lb, &o2)) {
          float lg[4] = {head_b[0], head_b[1], head_b[2], head_b[3]};
#pragma unroll
          for (int w2 = 0; w2 < W::WN; ++w2) {
            const lds_float* hp = head_part + (w2 * 256 + r) * 4;
            lg[0] += hp[0];
            lg[1] += hp[1];
            lg[2] += hp[2];
            lg[3] += hp[3];
          }
          // padded index -> (b, t, i, j)
          const int b = (int)(p / g.S);
          const int rem = (int)(p - (long long)b * g.S);
          const int t = rem / g.P - 1;
          const int r2 = rem - (t + 1) * g.P;
          const int i = r2 / g.Wp - 1, j = r2 - (i + 1) * g.Wp - 1;
          const int HH = g.H * g.H;
          const int s = i * g.H + j;
          const int n = comp_of_site[s];
          const bool data = (i < g.d) && (j < g.d);
          unsigned bits = 0;
          if (data && lg[0] > 0.0f) bits |= 1u;
          if (data && lg[1] > 0.0f) bits |= 2u;
          if (n >= 0 && n < g.K && lg[2] > 0.0f) bits |= 4u;
          if (n >= g.K && lg[3] > 0.0f) bits |= 8u;
          nib[(long long)b * g.V + (long long)t * HH + s] = (uint8_t)bits;
          if (logits) {
#pragma unroll
            for (int o = 0; o < 4; ++o) logits[(((long long)b * 4 + o) * g.T + t) * HH + s] = lg[o];
          }
        }
      }
    }
    // the epilogue's buffer is where the next tile's second chunk is staged
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
    tile = next;
    cur_src = next_src;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// LDS bytes of one launch (layout at the top of the kernel).
static size_t lds_bytes(int cout) {
  return cout == 64 ? (size_t)LdsLayout<64>::total : (size_t)LdsLayout<128>::total;
}

size_t conv_bf16_lds_bytes(int cin, int span) {
  (void)cin;
  (void)span;
  return lds_bytes(128);
}

int conv_bf16_max_span() { return RMAX * NT / 4; }

template <int CIN, int COUT, bool HEAD, int MODE>
static hipError_t launch_one(const Geom& g, const Tiling& tl, int act, const void* x, void* y,
                             const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                             const int32_t* comp_of_site, uint8_t* nib, float* logits, int batch,
                             int n_workgroups, hipStream_t stream) {
  const size_t lds = lds_bytes(COUT);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)conv_bf16_kernel<CIN, COUT, HEAD, MODE>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const long long nwg = conv_workgroups(tl.ntiles, n_workgroups);
  hipLaunchKernelGGL((conv_bf16_kernel<CIN, COUT, HEAD, MODE>), dim3((unsigned)nwg), dim3(NT), lds, stream, g, tl,
                     act, (const uint16_t*)x, (uint16_t*)y, (const u32x4*)wfrag, bias, head_w, head_b,
                     comp_of_site, nib, logits, batch);
  return hipGetLastError();
}

#define PD_CONV_CASE(CI, CO)                                                                                 \
  if (cin == CI && cout == CO) {                                                                            \
    if (head && tl.mode == 0)                                                                                \
      return launch_one<CI, CO, true, 0>(g, tl, act, x, y, wfrag, bias, head_w, head_b, comp_of_site, nib,    \
                                         logits, batch, n_workgroups, stream);                               \
    if (head)                                                                                                \
      return launch_one<CI, CO, true, 1>(g, tl, act, x, y, wfrag, bias, head_w, head_b, comp_of_site, nib,    \
                                         logits, batch, n_workgroups, stream);                               \
    if (tl.mode == 0)                                                                                        \
      return launch_one<CI, CO, false, 0>(g, tl, act, x, y, wfrag, bias, head_w, head_b, comp_of_site, nib,   \
                                          logits, batch, n_workgroups, stream);                              \
    return launch_one<CI, CO, false, 1>(g, tl, act, x, y, wfrag, bias, head_w, head_b, comp_of_site, nib,     \
                                        logits, batch, n_workgroups, stream);                                \
  }

hipError_t launch_conv_bf16(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x, void* y,
                            const void* wfrag, const float* bias, int head, const float* head_w,
                            const float* head_b, const int32_t* comp_of_site, uint8_t* nib, float* logits,
                            int batch, int n_workgroups, hipStream_t stream) {
  PD_CONV_CASE(2, 64)
  PD_CONV_CASE(2, 128)
  PD_CONV_CASE(64, 64)
  PD_CONV_CASE(128, 128)
  PD_CONV_CASE(64, 128)
  PD_CONV_CASE(128, 64)
  return hipErrorInvalidValue;
}

}  // namespace pd
