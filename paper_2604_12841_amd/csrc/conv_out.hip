// conv_out.hip -- K4 of the paper's layout: the 3x3x3 output layer with its
// four filters (X / Z data-qubit flip and X / Z measurement flip logits,
// Table models), the threshold (logit > 0) and, for the last block of a
// residual network, the block's shortcut fused in.
//
// Four output channels make a poor matrix shape: as an implicit GEMM with
// the filters on the MFMA rows, 28 of every 32 rows are padding, and every
// weight fragment feeds a single 32-voxel block.  Here the rows are (tap,
// filter) pairs instead -- 27 x 4 = 108 of 128 rows in four row blocks -- and
// the K dimension is the input channels alone:
//
//   P[v][tap][co] = sum_ci W[co][ci][tap] * X[v][ci]      (one GEMM per voxel v)
//   logit[u][co]  = bias[co] + sum_tap P[u + shift(tap)][tap][co]
//
// so each input voxel's partial products are computed once (not once per
// tap) and each output sums 27 of its neighbours' partials.  The sum runs
// over the partials in LDS.
//
// Work unit: one sample, a range of output rounds t and a rectangle of the
// D x D grid (a strip of rows, the whole width when it fits).  The unit
// walks its input rounds in order (its output rounds plus the neighbour
// round on each side): for each input round it computes P for the round's
// voxels under the rectangle plus a one-voxel rim (at most 256 voxels, 8
// blocks of 32), stores P in LDS (27 taps x 256 voxels x 4 filters, fp32),
// and each of up to 256 threads adds the partials of its output voxel's
// neighbours in that round to three running sums (output rounds t - 1, t,
// t + 1).  Output round t - 1 is then complete: + bias (fp8: x the filter's
// weight scale first), + the shortcut (residual networks), threshold, flip
// nibble and logits.  Input rounds are shared by consecutive output rounds,
// so the only recomputation is the rim (and one round at each end of a
// range of rounds).
//
// Residual networks: the last block's shortcut is added to the logits --
// the block input itself, or its 1x1x1 projection (c_in -> 4) computed here
// as more k-steps of the same GEMM: the wave groups take alternate chunks of
// the block input's channels against projection fragments whose rows 0..3
// are the four filters, into an accumulator of their own; the two groups'
// sums land in two more LDS slots and the output's own voxel adds them,
// scales them (fp8), adds the projection's bias and rounds to the stored
// precision (bf16, or E4M3), the shortcut of the unfused path.
//
// Waves: wave w takes row blocks 2 (w % 2), 2 (w % 2) + 1 and voxel blocks
// w / 2, w / 2 + 2, ...: each weight fragment feeds up to four MFMAs and
// each activation fragment two.  With c_in <= 128 the weight fragments of
// the wave's two row blocks (64 registers for 128 bf16 channels) are loaded
// once per unit; wider inputs run in chunks of 64 channels, each chunk's
// fragments loaded per round.  The activation fragments are read from
// global memory (L2) straight into registers, 16 bytes per lane (fp8: 32).
#include <algorithm>

#include "activation.h"
#include "internal.h"

namespace pd {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) uint32_t u32x8;
typedef __attribute__((ext_vector_type(8))) int i32x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;

constexpr int NT = 256;      // threads per workgroup: 4 wave64
constexpr int TAPS = 27;
constexpr int NRB = 4;       // row blocks of 32 rows: row 32 rb + m is tap 8 rb + m / 4, filter m % 4
// Units stage at most MV = 256 voxels of a round (8 blocks of 32; one
// workgroup per CU).  P in LDS: [32 row slots of 4 filters][MV + 1] float4,
// tap-major; slot MV of every tap holds zeros (read for neighbours outside
// the grid), and row slots 27..31 take the zero rows of the last row block.
// (Units of 128 voxels, two workgroups per CU, measured slower: their rims
// stage more voxels and the second workgroup hides little, the sums and
// stores being short next to the matrix work.)
constexpr int MV = 256;
constexpr int PSTR = MV + 1;
constexpr int BPW = MV / 64;  // voxel blocks per wave
// LDS bytes: 32 row slots, and 2 more for the projection's halves
constexpr size_t lds_bytes(bool proj) { return (size_t)(proj ? 34 : 32) * PSTR * 16; }
static_assert(lds_bytes(true) <= 160 * 1024, "P fits the LDS of a CU");

template <bool F8>
struct OutPrec {
  static constexpr int KSTEP = F8 ? 64 : 16;  // input channels per MFMA
  static constexpr int LQ = F8 ? 2 : 1;       // 16-byte pieces per lane of a fragment
};

__device__ __forceinline__ f32x16 mma(const u32x4 (&a)[2], const u32x4 (&b)[2], f32x16 c, bool f8) {
  if (f8) {
    const i32x8 wa = __builtin_bit_cast(i32x8, u32x8{a[0].x, a[0].y, a[0].z, a[0].w, a[1].x, a[1].y, a[1].z, a[1].w});
    const i32x8 xb = __builtin_bit_cast(i32x8, u32x8{b[0].x, b[0].y, b[0].z, b[0].w, b[1].x, b[1].y, b[1].z, b[1].w});
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wa, xb, c, 0, 0, 0, 0, 0, 0);
  }
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[0]), __builtin_bit_cast(bf16x8, b[0]),
                                                 c, 0, 0, 0);
}

// Unit u of the launch: sample b, output rounds [t0, t1), rows [i0, i1) and
// columns [j0, j1) of the grid (even splits of T, H and H into nch, nsi and
// nsj parts).
struct Unit {
  int b, t0, t1, i0, i1, j0, j1;
};

__device__ __forceinline__ Unit unit_of(const Geom& g, int u, int nch, int nsi, int nsj) {
  Unit r;
  const int sj = u % nsj;
  u /= nsj;
  const int si = u % nsi;
  u /= nsi;
  const int c = u % nch;
  r.b = u / nch;
  r.t0 = c * g.T / nch;
  r.t1 = (c + 1) * g.T / nch;
  r.i0 = si * g.H / nsi;
  r.i1 = (si + 1) * g.H / nsi;
  r.j0 = sj * g.H / nsj;
  r.j1 = (sj + 1) * g.H / nsj;
  return r;
}

// wfrag: [rb][k-step][lane] fragments of LQ x 16 bytes (rows past tap 26 are
// zero); bias: [4] biases, then [4] weight scales (1 on the bf16 path).
// PROJ: px holds the block input (CIN channels, the layout of x), pfrag its
// projection fragments [k-step][lane] (LQ x 16 bytes, rows 0..3 the
// filters), pbias the projection's 4 biases then its 4 weight scales.
template <int CIN, bool F8, bool PROJ>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
conv_out_kernel(Geom g, int nch, int nsi, int nsj, const void* __restrict__ x, const u32x4* __restrict__ wfrag,
                const float* __restrict__ bias, const int32_t* __restrict__ tables, uint8_t* __restrict__ nib,
                float* __restrict__ logits, const uint16_t* __restrict__ sc, int sc_stride,
                const void* __restrict__ px, const u32x4* __restrict__ pfrag, const float* __restrict__ pbias) {
  using PR = OutPrec<F8>;
  constexpr int KSTEP = PR::KSTEP, LQ = PR::LQ;
  constexpr int ESZ = F8 ? 1 : 2;
  constexpr int ROW = CIN * ESZ;                      // bytes per activation row
  // input channels per chunk: all of them up to 128 (weights loaded once per
  // unit), else (and with a projection, whose chunks reload them) 64
  constexpr int CH = (CIN <= 128 && !PROJ) ? CIN : 64;
  constexpr int NCH = CIN / CH;                       // chunks
  constexpr int KPC = CH / KSTEP;                     // k-steps per chunk
  constexpr int NKS = CIN / KSTEP;                    // k-steps in all
  extern __shared__ __attribute__((aligned(16))) char smem[];
  lds_f32x4* const pl = (lds_f32x4*)smem;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int rp = wave & 1, bh = wave >> 1;  // row blocks 2 rp, 2 rp + 1; voxel blocks bh, bh + 2, ...
  // chunks of a round: the conv's, then (PROJ) the projection chunks rp,
  // rp + 2, ... of the block input
  const int nct = NCH + (PROJ ? (NCH - rp + 1) / 2 : 0);

  const Unit un = unit_of(g, blockIdx.x, nch, nsi, nsj);
  const int H = g.H;
  // the staged rectangle: the unit's rows and columns plus a rim of one
  // (inside the grid)
  const int ia = un.i0 > 0 ? un.i0 - 1 : 0, ib = un.i1 < H ? un.i1 + 1 : H;
  const int ja = un.j0 > 0 ? un.j0 - 1 : 0, jb = un.j1 < H ? un.j1 + 1 : H;
  const int ncol = jb - ja, nst = (ib - ia) * ncol;  // <= MV (host check)
  const int nblk = (nst + 31) >> 5;
  // input rounds: the output rounds and one on each side, inside the volume
  const int ta = un.t0 > 0 ? un.t0 - 1 : 0, tb = un.t1 < g.T ? un.t1 + 1 : g.T;

  // this lane's voxel of each of its blocks: its row in round 0 of the
  // sample, at the lane's k offset (voxels past the rectangle read the
  // sample's first padded voxels, zero halo voxels; their partials are
  // never summed)
  const char* bsrc[BPW];
#pragma unroll
  for (int k = 0; k < BPW; ++k) {
    const int v = (bh + 2 * k) * 32 + l32;
    long long off = 0;
    if (v < nst) {
      const int ri = v / ncol, rj = v - ri * ncol;
      off = (long long)g.pad * g.P + (long long)(ia + ri + g.pad) * g.Wp + (ja + rj + g.pad);
    }
    bsrc[k] = (const char*)x + ((long long)un.b * g.S + off) * ROW + half * (KSTEP / 2) * ESZ;
  }
  const int nbw = nblk > bh ? (nblk - bh + 1) >> 1 : 0;  // blocks this wave computes (<= BPW)

  // the output voxel this thread sums (if any), and the staged index of each
  // neighbour (oi + ki - 1, oj + kj - 1) in a round, MV (the zero slot)
  // outside the grid
  const int ow = un.j1 - un.j0, nout = (un.i1 - un.i0) * ow;
  const bool owner = tid < nout;
  const int oi = owner ? un.i0 + tid / ow : 0, oj = owner ? un.j0 + tid % ow : 0;
  int nbr[9];
#pragma unroll
  for (int ki = 0; ki < 3; ++ki)
#pragma unroll
    for (int kj = 0; kj < 3; ++kj) {
      const int ii = oi + ki - 1, jj = oj + kj - 1;
      const bool in = ii >= 0 && ii < H && jj >= 0 && jj < H;
      nbr[3 * ki + kj] = in ? (ii - ia) * ncol + (jj - ja) : MV;
    }
  if (tid < 32) pl[tid * PSTR + MV] = f32x4{0.f, 0.f, 0.f, 0.f};
  const unsigned allowed = owner ? flip_allowed(g, tables, oi, oj) : 0u;
  float bs[4], sca[4];
#pragma unroll
  for (int o = 0; o < 4; ++o) {
    bs[o] = bias[o];
    sca[o] = bias[4 + o];
  }

  // weight fragments of one chunk for the wave's two row blocks (a
  // projection chunk: its fragments in wa[0])
  u32x4 wa[2][KPC][LQ];
  auto load_w = [&](int c) {
    if (PROJ && c >= NCH) {
      const int k0 = (rp + 2 * (c - NCH)) * KPC;
#pragma unroll
      for (int s = 0; s < KPC; ++s)
#pragma unroll
        for (int q = 0; q < LQ; ++q) wa[0][s][q] = pfrag[((size_t)(k0 + s) * 64 + lane) * LQ + q];
      return;
    }
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int s = 0; s < KPC; ++s)
#pragma unroll
        for (int q = 0; q < LQ; ++q)
          wa[r][s][q] = wfrag[(((size_t)(2 * rp + r) * NKS + c * KPC + s) * 64 + lane) * LQ + q];
  };
  if constexpr (NCH == 1) load_w(0);

  f32x4 run[3];  // running sums of output rounds tin - 1, tin, tin + 1
  f32x4 shr[2];  // PROJ: the projected shortcuts of output rounds tin - 1, tin
#pragma unroll
  for (int k = 0; k < 3; ++k) run[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  shr[0] = shr[1] = f32x4{0.f, 0.f, 0.f, 0.f};
  float pbs[4], psc[4];
#pragma unroll
  for (int o = 0; o < 4; ++o) {
    pbs[o] = PROJ ? pbias[o] : 0.0f;
    psc[o] = PROJ ? pbias[4 + o] : 1.0f;
  }

  auto emit = [&](int t, const f32x4& s, const f32x4& sh) {
    if (!owner || t < un.t0 || t >= un.t1) return;
    float lg[4];
#pragma unroll
    for (int o = 0; o < 4; ++o) lg[o] = F8 ? __builtin_fmaf(s[o], sca[o], bs[o]) : s[o] + bs[o];
    if (PROJ) {
#pragma unroll
      for (int o = 0; o < 4; ++o) lg[o] += sh[o];
    } else if (sc) {  // residual shortcut of the last block: 4 channels (bf16, or E4M3 codes)
      const long long pi = padded_index(g, un.b, t, oi, oj) * sc_stride;
      if constexpr (F8) {
        const uint32_t q = *reinterpret_cast<const uint32_t*>((const uint8_t*)sc + pi);
        lg[0] += __builtin_amdgcn_cvt_f32_fp8((int)q, 0);
        lg[1] += __builtin_amdgcn_cvt_f32_fp8((int)q, 1);
        lg[2] += __builtin_amdgcn_cvt_f32_fp8((int)q, 2);
        lg[3] += __builtin_amdgcn_cvt_f32_fp8((int)q, 3);
      } else {
        const uint2 sv = *reinterpret_cast<const uint2*>(sc + pi);
        lg[0] += __uint_as_float(sv.x << 16);
        lg[1] += __uint_as_float(sv.x & 0xFFFF0000u);
        lg[2] += __uint_as_float(sv.y << 16);
        lg[3] += __uint_as_float(sv.y & 0xFFFF0000u);
      }
    }
    const int HH = H * H, s2 = oi * H + oj;
    nib[(long long)un.b * g.V + (long long)t * HH + s2] = (uint8_t)flip_bits(allowed, lg);
    if (logits) {
#pragma unroll
      for (int o = 0; o < 4; ++o) logits[(((long long)un.b * 4 + o) * g.T + t) * HH + s2] = lg[o];
    }
  };

  // activation fragments of the current (round, chunk) for the wave's
  // blocks; block k's registers are refilled with the next (round, chunk)
  // as soon as its MFMAs have issued, so the loads run under the rest of
  // the round (the other blocks, the partials' store and the sums)
  u32x4 xb[BPW][KPC][LQ];
  const long long pdelta = PROJ ? (const char*)px - (const char*)x : 0;  // the block input's rows
  auto load_x = [&](int k, int t, int c) {
    const char* src = bsrc[k] + (long long)t * g.P * ROW;
    if (PROJ && c >= NCH)
      src += pdelta + (rp + 2 * (c - NCH)) * CH * ESZ;
    else
      src += c * CH * ESZ;
#pragma unroll
    for (int s = 0; s < KPC; ++s)
#pragma unroll
      for (int q = 0; q < LQ; ++q) xb[k][s][q] = *reinterpret_cast<const u32x4*>(src + s * KSTEP * ESZ + q * 16);
  };
#pragma unroll
  for (int k = 0; k < BPW; ++k)
    if (k < nbw) load_x(k, ta, 0);

#pragma unroll 1
  for (int tin = ta; tin < tb; ++tin) {
    // ---- partials of round tin: P = W x for the wave's blocks and row blocks
    f32x16 acc[BPW][2];
    f32x16 accp[PROJ ? BPW : 1];  // the projection's half (rows 0..3)
#pragma unroll
    for (int k = 0; k < BPW; ++k)
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[k][r][e] = 0.0f;
#pragma unroll
    for (int k = 0; k < (PROJ ? BPW : 1); ++k)
#pragma unroll
      for (int e = 0; e < 16; ++e) accp[k][e] = 0.0f;
#pragma unroll 1
    for (int c = 0; c < nct; ++c) {
      if (NCH > 1 || PROJ) load_w(c);
      const bool more = c + 1 < nct || tin + 1 < tb;  // a next (round, chunk) to prefetch
      const int tn = c + 1 < nct ? tin : tin + 1, cn = c + 1 < nct ? c + 1 : 0;
#pragma unroll
      for (int k = 0; k < BPW; ++k) {
        if (k >= nbw) break;  // uniform per wave
        if (PROJ && c >= NCH) {
#pragma unroll
          for (int s = 0; s < KPC; ++s) {
            u32x4 a2[2] = {wa[0][s][0], wa[0][s][LQ - 1]};
            u32x4 b2[2] = {xb[k][s][0], xb[k][s][LQ - 1]};
            accp[k] = mma(a2, b2, accp[k], F8);
          }
        } else {
#pragma unroll
          for (int s = 0; s < KPC; ++s)
#pragma unroll
            for (int r = 0; r < 2; ++r) {
              u32x4 a2[2] = {wa[r][s][0], wa[r][s][LQ - 1]};
              u32x4 b2[2] = {xb[k][s][0], xb[k][s][LQ - 1]};
              acc[k][r] = mma(a2, b2, acc[k][r], F8);
            }
        }
        if (more) load_x(k, tn, cn);
      }
    }
    // lane holds rows 8 q + 4 half + e of each row block: row slot (tap) 8
    // rb + 2 q + half, filter e, for voxel 32 blk + l32
#pragma unroll
    for (int k = 0; k < BPW; ++k) {
      if (k >= nbw) break;
      const int v = (bh + 2 * k) * 32 + l32;
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int slot = 8 * (2 * rp + r) + 2 * q + half;
          pl[slot * PSTR + v] = f32x4{acc[k][r][4 * q], acc[k][r][4 * q + 1], acc[k][r][4 * q + 2],
                                      acc[k][r][4 * q + 3]};
        }
      // the projection's half: rows 0..3 (the first half-wave's q = 0) into slot 32 + rp
      if (PROJ && half == 0)
        pl[(32 + rp) * PSTR + v] = f32x4{accp[k][0], accp[k][1], accp[k][2], accp[k][3]};
    }
    // LDS-only barriers: a full fence would also wait for the prefetch loads
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's partials are in LDS
    __builtin_amdgcn_s_barrier();
    // ---- sums: tap (kt, ki, kj) of output round tin + 1 - kt reads round tin
    if (owner) {
#pragma unroll
      for (int kt = 0; kt < 3; ++kt) {
        f32x4 p[9];
#pragma unroll
        for (int n = 0; n < 9; ++n) p[n] = pl[(9 * kt + n) * PSTR + nbr[n]];
#pragma unroll
        for (int n = 0; n < 9; ++n) run[2 - kt] += p[n];
      }
      if (PROJ) {  // the output's own voxel in round tin: its projected shortcut, rounded as stored
        const f32x4 a = pl[32 * PSTR + nbr[4]], b = pl[33 * PSTR + nbr[4]];
        float sp[4];
#pragma unroll
        for (int o = 0; o < 4; ++o) sp[o] = __builtin_fmaf(a[o] + b[o], psc[o], pbs[o]);
        if constexpr (F8) {
          shr[1] = f32x4{e4m3_round(sp[0]), e4m3_round(sp[1]), e4m3_round(sp[2]), e4m3_round(sp[3])};
        } else {
          const uint32_t p01 = bf16_pack(sp[0], sp[1]), p23 = bf16_pack(sp[2], sp[3]);
          shr[1] = f32x4{__uint_as_float(p01 << 16), __uint_as_float(p01 & 0xFFFF0000u),
                         __uint_as_float(p23 << 16), __uint_as_float(p23 & 0xFFFF0000u)};
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the sums' reads are done before the next stores
    __builtin_amdgcn_s_barrier();
    // output round tin - 1 is complete
    emit(tin - 1, run[0], shr[0]);
    run[0] = run[1];
    run[1] = run[2];
    run[2] = f32x4{0.f, 0.f, 0.f, 0.f};
    shr[0] = shr[1];
  }
  // the last round when no round follows it
  if (tb == g.T) emit(tb - 1, run[0], shr[0]);
}

}  // namespace

size_t conv_out_fragment_bytes(int cin, int fp8) {
  return (size_t)NRB * (cin / (fp8 ? 64 : 16)) * 64 * (fp8 ? 32 : 16);
}

bool conv_out_supported(int cin, int fp8, int ks, int H) {
  if (ks != 3) return false;
  if (!(cin == 64 || cin == 128 || cin == 256 || cin == 512)) return false;
  int nsi, nsj;
  return conv_out_split(H, MV, &nsi, &nsj) > 0;
}

// Rectangles of the grid: the split into nsi x nsj parts whose staged
// rectangles (a part and its rim of one) hold at most maxv voxels and add
// up to the fewest staged voxels; returns that number (per round and
// sample), 0 if no split fits.
long long conv_out_split(int H, int maxv, int* nsi, int* nsj) {
  long long best = 0;
  for (int sj = 1; sj <= H; ++sj) {
    const int cols = sj == 1 ? H : std::min(H, (H + sj - 1) / sj + 2);
    for (int si = 1; si <= H; ++si) {
      const int rows = si == 1 ? H : std::min(H, (H + si - 1) / si + 2);
      if (rows * cols > maxv) continue;
      const long long cost = (long long)si * sj * rows * cols;
      if (best == 0 || cost < best) {
        best = cost;
        *nsi = si;
        *nsj = sj;
      }
      break;  // more rows only adds rims
    }
  }
  return best;
}

hipError_t launch_conv_out(const Geom& g, int cin, const void* x, const void* wfrag, const float* bias,
                           const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_cu, int fp8,
                           const uint16_t* sc, int sc_stride, const void* px, const void* pfrag,
                           const float* pbias, hipStream_t stream) {
  if (g.pad != 1 || batch < 1 || !conv_out_supported(cin, fp8, 3, g.H)) return hipErrorInvalidValue;
  const bool proj = px != nullptr;
  if (proj && (!pfrag || !pbias || sc)) return hipErrorInvalidValue;
  // Rectangles and rounds per unit: from the split with the fewest staged
  // voxels up to three more parts each way, and every split of T, the one
  // that minimises (units per CU, rounded up) x (input rounds per unit) x
  // (staged voxels per round + a fixed cost per round of about 128 voxels'
  // worth).  Large batches keep the fewest staged voxels; small ones take
  // smaller rectangles, which fill more of the chip.
  int s0i = 1, s0j = 1;
  conv_out_split(g.H, MV, &s0i, &s0j);
  int nsi = s0i, nsj = s0j, nch = 1;
  long long best = -1;
  for (int sj = s0j; sj <= std::min(g.H, s0j + 3); ++sj) {
    const int cols = sj == 1 ? g.H : std::min(g.H, (g.H + sj - 1) / sj + 2);
    for (int si = s0i; si <= std::min(g.H, s0i + 3); ++si) {
      const int rows = si == 1 ? g.H : std::min(g.H, (g.H + si - 1) / si + 2);
      if (rows * cols > MV) continue;
      const long long per = (long long)batch * si * sj;
      for (int c = 1; c <= g.T; ++c) {
        const long long units = per * c;
        if (units > 0x7fffffffLL) break;
        const long long waves = (units + n_cu - 1) / n_cu;
        const long long rounds = (g.T + c - 1) / c + (c > 1 ? 2 : 0);
        const long long cost = waves * rounds * (rows * cols + 128);
        if (best < 0 || cost < best) {
          best = cost;
          nsi = si;
          nsj = sj;
          nch = c;
        }
      }
    }
  }
  const long long units = (long long)batch * nsi * nsj * nch;
  if (units > 0x7fffffffLL) return hipErrorInvalidValue;
  auto go = [&](auto kern, bool p) -> hipError_t {
    const size_t lds = lds_bytes(p);
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)units), dim3(NT), lds, stream, g, nch, nsi, nsj, x,
                       (const u32x4*)wfrag, bias, tables, nib, logits, sc, sc_stride, px, (const u32x4*)pfrag,
                       pbias);
    return hipGetLastError();
  };
  if (proj && fp8) {
    switch (cin) {
      case 64: return go(conv_out_kernel<64, true, true>, true);
      case 128: return go(conv_out_kernel<128, true, true>, true);
      case 256: return go(conv_out_kernel<256, true, true>, true);
      case 512: return go(conv_out_kernel<512, true, true>, true);
    }
  } else if (proj) {
    switch (cin) {
      case 64: return go(conv_out_kernel<64, false, true>, true);
      case 128: return go(conv_out_kernel<128, false, true>, true);
      case 256: return go(conv_out_kernel<256, false, true>, true);
      case 512: return go(conv_out_kernel<512, false, true>, true);
    }
  } else if (fp8) {
    switch (cin) {
      case 64: return go(conv_out_kernel<64, true, false>, false);
      case 128: return go(conv_out_kernel<128, true, false>, false);
      case 256: return go(conv_out_kernel<256, true, false>, false);
      case 512: return go(conv_out_kernel<512, true, false>, false);
    }
  } else {
    switch (cin) {
      case 64: return go(conv_out_kernel<64, false, false>, false);
      case 128: return go(conv_out_kernel<128, false, false>, false);
      case 256: return go(conv_out_kernel<256, false, false>, false);
      case 512: return go(conv_out_kernel<512, false, false>, false);
    }
  }
  return hipErrorInvalidValue;
}

size_t conv_out_proj_fragment_bytes(int cin, int fp8) { return (size_t)(cin / (fp8 ? 64 : 16)) * 64 * (fp8 ? 32 : 16); }

}  // namespace pd
