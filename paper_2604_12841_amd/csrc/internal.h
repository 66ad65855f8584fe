// internal.h -- shared declarations between the C-ABI host code and the
// gfx950 kernels of the pre-decoder.  Not installed; the public contract is
// include/predecoder.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/predecoder.h"

namespace pd {

// Padded activation layout (NTHWC with a zero halo of `pad` voxels in t, i
// and j -- 1, or 2 for a network with 5x5x5 layers; H = d + 1 on the
// plaquette grid, d on the paper layout):
//   voxel (b, t, i, j), 0 <= t < T, 0 <= i, j < H, lives at padded index
//   b * S + (t + pad) * P + (i + pad) * Wp + (j + pad),  Wp = H + 2 pad,
//   P = Wp^2, S = (T + 2 pad) * P,
// channels contiguous.  The halo is zeroed once at create and never written,
// so a k x k x k tap (k <= 2 pad + 1) is a pure index shift.
struct Geom {
  int d, T, H, Wp, P;
  int pad;      // halo width
  long long S;  // padded voxels per sample
  int V;        // interior voxels per sample, T * H * H
  int K;        // stabilizers of each type, (d^2 - 1) / 2
  int nstab;    // d^2 - 1
  int nflip;    // 3 d^2 - 1
  long long Wd, Wf;  // packed words per sample
  // Input layout: 0 = plaquette grid, H = d + 1, two channels (detector events
  // at their stabilizer sites); 1 = the paper's own layout (Sec. IV.B.1), H = d
  // (the data qubits), four channels (x_type, z_type, x_present, z_present),
  // every stabilizer drawn onto one qubit of its support.
  int layout;
  // Basis prepared before round 0 / measured after round T-1 (0 none, 1 Z,
  // 2 X): in the paper's layout, Z clears x_present and X clears z_present
  // in that round.
  int first, last;
};

__host__ __device__ inline long long padded_index(const Geom& g, int b, int t, int i, int j) {
  return (long long)b * g.S + (long long)(t + g.pad) * g.P + (long long)(i + g.pad) * g.Wp + (j + g.pad);
}

// Output-row tiling of one conv launch.  A tile is up to 256 output voxels:
//  mode 0 (flat): 256 consecutive voxels of a segment of `seg_len` voxels in
//    (b, t, i, j) order (seg_len = V keeps tiles inside one sample, B * V lets
//    them cross samples).  The staged input lives in "line space": voxel
//    (b, t, i, j) with -1 <= t <= T, -1 <= i <= d+1 and only the real columns
//    0 <= j <= d has line-space index
//        u = (b (T+2) + t + 1) * PU + (i + 1) * H + j,   PU = (H+2) H,
//    which is linear in (t, i, j), so consecutive output voxels are
//    consecutive staged voxels.  The zero halo columns are not staged: a tap
//    that falls on one reads a zero region instead.  The staged span runs
//    from u(first row) - (PU + H + 1) to u(last row) + (PU + H + 1).
//    (Mode 0 needs pad = 1.)
//  mode 1 (box): a BT x BI x BJ box of (t, i, j); the staged input is the
//    (BT+2 pad) x (BI+2 pad) x (BJ+2 pad) padded box around it, halo
//    included.
// In both modes the LDS voxel of row r for tap (dt, di, dj) in {0..k-1}^3 is
// row_base(r) + dt * sa + di * sb + dj.
// Division by a runtime constant d >= 2 for numerators n < 2^31:
// q = mulhi(n, m) >> s with s = ceil(log2 d) - 1, m = floor(2^(32+s) / d) + 1.
// (m < 2^32 because 2^s < d; the error m d - 2^(32+s) <= d keeps
// n (m d - 2^(32+s)) < 2^(32+s) for n < 2^31 <= 2^(32+s) / d.)
struct FastDiv {
  uint32_t m;
  int s;
};

inline FastDiv make_fastdiv(uint32_t d) {
  if (d < 2) return FastDiv{0u, 0};  // unused divisor; fastdiv is only valid for d >= 2
  int c = 0;
  while ((1u << c) < d) ++c;  // ceil(log2 d)
  FastDiv f;
  f.s = c - 1;
  f.m = (uint32_t)((((unsigned long long)1) << (32 + f.s)) / d + 1);
  return f;
}

__host__ __device__ inline uint32_t fastdiv(uint32_t n, FastDiv f) {
#ifdef __HIP_DEVICE_COMPILE__
  return __umulhi(n, f.m) >> f.s;
#else
  return (uint32_t)(((unsigned long long)n * f.m) >> 32) >> f.s;
#endif
}

// n / d for any divisor d >= 1 (make_fastdiv(1) has m = 0: the quotient is n).
__host__ __device__ inline uint32_t fdiv(uint32_t n, FastDiv f) { return f.m ? fastdiv(n, f) : n; }

struct Tiling {
  int mode;
  long long seg_len;
  int tiles_per_seg;
  int BT, BI, BJ, ntT, ntI, ntJ;
  int sa, sb;
  int span;      // staged voxels per tile (upper bound), sizes the LDS buffers
  long long ntiles;
  FastDiv div_a, div_b;  // staging decode: mode 0 by PU and H; mode 1 by (BI+2)(BJ+2) and BJ+2
  // tile and row decoding (tiles.h): mode 0 by tiles_per_seg, V, H^2 and H;
  // mode 1 by the tiles per sample, ntI ntJ, ntJ, BI BJ and BJ
  FastDiv dv_tps, dv_V, dv_HH, dv_H, dv_per, dv_ntij, dv_ntj, dv_bij, dv_bj;
};

__host__ __device__ inline int line_plane(const Geom& g) { return (g.H + 2) * g.H; }

// Line-space index of voxel (b, t, i, j) (mode 0 staging, see Tiling).
__host__ __device__ inline long long line_index(const Geom& g, int b, int t, int i, int j) {
  return ((long long)b * (g.T + 2) + t + 1) * line_plane(g) + (long long)(i + 1) * g.H + j;
}

// Padded activation index of line-space voxel u.
__host__ __device__ inline long long line_to_padded(const Geom& g, long long u) {
  const int pu = line_plane(g);
  const long long tp = u / pu;
  const int rem = (int)(u - tp * pu);
  const int ip = rem / g.H;
  const int jj = rem - ip * g.H;
  return tp * g.P + (long long)ip * g.Wp + jj + 1;
}

constexpr int kTileRows = 256;

// Kernel launchers (all asynchronous on `stream`; return the launch error).
// Detector events -> input planes (c_in = 2 or 4 channels by layout).
hipError_t launch_unpack(const Geom& g, const int32_t* tables, const uint64_t* det, int batch, void* out,
                         int out_padded, int fp32, hipStream_t stream);

// The first 3x3x3 layer (c_in = 2 or 4, c_out = 64 or 128) when it is not
// also the last hidden layer: planes [batch * S][c_in] bf16, weight fragments
// [ceil(27 c_in / 16) k-steps][c_out / 32][64 lanes][8 bf16].  Output voxel
// rows are ystride channels apart (a wider layer is run as slices of c_out
// channels, y pointing at the slice's first channel).
// fp8: y holds E4M3 codes (one byte per value; the planes and the bf16
// weight fragments are unchanged, the weights being E4M3 values times their
// power-of-two scales, which bf16 represents exactly).
// ks: kernel size 3, or 5 (c_in = 4, bf16, a halo of two).
hipError_t launch_conv_first(const Geom& g, int cin, int cout, int act, const void* planes, void* y,
                             int ystride, const void* wfrag, const float* bias, int batch, int fp8, int ks,
                             hipStream_t stream);

// A network with one hidden layer: layer 1 (as launch_conv_first) with the
// 1x1x1 head (head_w [4][cout] fp32, bf16-valued; head_b [4]) and the
// threshold in its epilogue, which writes flip nibbles (and logits if
// non-null).  n_workgroups: one per CU.
hipError_t launch_conv_single(const Geom& g, const Tiling& tl, int cout, int act, const void* planes,
                              const void* wfrag, const float* bias, const float* head_w, const float* head_b,
                              const int32_t* tables, uint8_t* nib, float* logits, int batch,
                              int n_workgroups, hipStream_t stream);
int conv_single_max_span();  // staged voxels a tile may need

// A 3x3x3 layer on the zero-halo activations x (c_in in {64, 128, 256}),
// bf16, or fp8 (E4M3 activations and weight codes, bias holding c_out
// biases then c_out per-channel weight scales, one byte per value in x and
// y, fragments of conv_fragments_fp8 in 32-channel chunks).
//   head == 0: a hidden layer (c_out in {64, 128}) writing y, whose voxel rows
//              are ystride channels apart (a 256-wide layer runs as two slices
//              of 128, y pointing at the slice's first channel);
//   head == 1: a hidden layer whose epilogue applies the 1x1x1 head and the
//              threshold as launch_conv_single does, instead of writing y;
//   head == 2: the output layer itself (c_out = 4, no activation): its
//              outputs are the logits, thresholded into flip nibbles; with
//              sc non-null, the 4 bf16 channels of sc's row (sc_stride
//              values apart) are added to the logits first;
//   head == 4: a hidden layer with sc's row (bf16, sc_stride values apart,
//              pointing at the slice's first channel) added to the
//              pre-activation (residual blocks; bf16 only).
// Weight fragments in 16-channel chunks (conv_fragments in api.hip; c_out = 4
// padded to 32 channels, bias to 32 values); n_workgroups =
// conv_hidden_workgroups_per_cu() per CU.
// Small batches: each tile's K loop (its channel chunks) split into
// 2^kshift parts run by different workgroups of one launch, which park fp32
// sums in `partial` (max_units units of conv_hidden_partial_floats_per_unit()
// floats); a second launch adds each tile's parts in part order and runs the
// epilogue.  kshift = 0: no split, one launch.
struct Split_k {
  int kshift;
  float* partial;
  long long max_units;
  int lsl = 0;  // 2^lsl output-channel slices of c_out channels in one launch
  // 256 zeroed words (per XCD: a grab and a done counter, 64 bytes apart):
  // a launch of more than two units per workgroup takes its units after the
  // fixed ones from these counters and leaves them zero; null: fixed shares
  uint32_t* sched = nullptr;
};

// ks: kernel size 3, or 5 (box tiles, a halo of two; bf16 c_in / c_out of
// 64 or 128, activations and the output layer).
hipError_t launch_conv_hidden(const Geom& g, const Tiling& tl, int cin, int cout, int act, const void* x,
                              void* y, int ystride, const void* wfrag, const float* bias, int head,
                              const float* head_w, const float* head_b, const int32_t* tables, uint8_t* nib,
                              float* logits, int batch, int n_workgroups, const Split_k& sk, int fp8,
                              const uint16_t* sc, int sc_stride, int ks, hipStream_t stream);
int conv_hidden_max_span(int ks);         // staged voxels a tile may need
int conv_hidden_chunk_channels(int fp8);  // input channels per K-loop chunk
size_t conv_hidden_partial_floats_per_unit();
int conv_hidden_workgroups_per_cu(int ks);

// The 3x3x3 output layer of four filters with the threshold (and the last
// residual block's shortcut) fused in, over rectangles of the grid streamed
// through the rounds: fragments of conv_out_fragment_bytes(c_in, fp8) bytes
// ([row block][k-step][lane], rows (tap, filter)), bias [4] then the four
// weight scales (1 on the bf16 path); sc: optional bf16 shortcut rows (4
// channels at sc_stride; E4M3 codes on the fp8 path); px (no sc): the block
// input whose 1x1x1 projection is the shortcut, pfrag its fragments
// (conv_out_proj_fragment_bytes: [k-step][lane], 16 bytes (fp8: 32 of
// codes), rows 0..3 the filters) and pbias its 4 biases then 4 weight
// scales.  Supported: c_in 64, 128, 256 or 512, a halo of one, grids whose rectangles fit (conv_out_split: the
// split of an H x H grid into rectangles of at most maxv voxels with their
// rims).
hipError_t launch_conv_out(const Geom& g, int cin, const void* x, const void* wfrag, const float* bias,
                           const int32_t* tables, uint8_t* nib, float* logits, int batch, int n_cu, int fp8,
                           const uint16_t* sc, int sc_stride, const void* px, const void* pfrag,
                           const float* pbias, hipStream_t stream);
size_t conv_out_fragment_bytes(int cin, int fp8);
size_t conv_out_proj_fragment_bytes(int cin, int fp8);
bool conv_out_supported(int cin, int fp8, int ks, int H);
long long conv_out_split(int H, int maxv, int* nsi, int* nsj);

// Copies the interior voxel rows (row_bytes each, a multiple of 8) of a
// zero-halo activation buffer to out [batch][T][H][H] rows.
hipError_t launch_extract(const Geom& g, const void* act, int row_bytes, int batch, void* out, hipStream_t stream);

// Zeroes `bytes` (a multiple of 16) of device memory with a kernel (usable
// where a memset node is not wanted).
hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream);

// 1x1x1 projection shortcut (bf16): y[p][co] = bf16(b[co] + sum_ci w[co][ci]
// x[p][ci]) over the interior voxels of the zero-halo layout; w [cout][cin]
// fp32 holding bf16 values; strides in values (ystride a multiple of 4, and
// xstride of 8 when cin is), cout a multiple of 4.
hipError_t launch_proj(const Geom& g, const void* x, int cin, int xstride, const float* w, const float* b, int cout,
                       void* y, int ystride, int batch, hipStream_t stream);

// Temporal windows over a stream of rounds (Sec. VI, parallel windows in
// time): window k covers rounds [start, start + len) of every stream and
// commits its core rounds [core_start, core_start + core_len); it is row
// `slot * n_streams + s` of its group's batch (group: the windows of one
// length and boundary kind, run by one handle).
struct StreamWindow {
  int start, len, core_start, core_len, group, slot;
};

// Window detector rows from stream rows (row_words words per stream row,
// out_words per window row; S bits per round).
hipError_t launch_stream_gather(const uint64_t* det, long long row_words, const StreamWindow* win, int n_win,
                                int n_streams, int S, long long out_words, uint64_t* out, hipStream_t stream);
// Stream flip rows (row_words words each; F bits per round) from the
// windows' flip rows (group g: group_flips[g], group_words[g] words per row),
// each round taken from the window whose core holds it (window k's core
// starts at round k * core).
hipError_t launch_stream_scatter(const StreamWindow* win, const uint64_t* const* group_flips,
                                 const long long* group_words, int n_streams, int core, int n_rounds, int F,
                                 long long row_words, uint64_t* flips, hipStream_t stream);

// predecoder_run of handle h with its workspace laid out in the `bytes` of
// device memory at `base` instead of the handle's own (input planes,
// activation buffers, projection outputs, flip nibbles, then as many units of
// parked split-K sums as fit, at most the handle's own number): the planes
// and activation buffers are cleared with a fill kernel first; nothing is
// allocated.  PD_ERR_TOO_LARGE when the regions before the parked sums do not
// fit.  Asynchronous on st.
pd_status run_in_region(pd_predecoder* h, hipStream_t st, const uint64_t* det, int batch, uint64_t* flips,
                        uint64_t* residual, float* logits, void* base, size_t bytes);

// Persistent workgroups of a conv launch: one per CU (n_workgroups), a
// multiple of 8 (one per XCD round-robin slot), never more than the tiles
// need.
__host__ __device__ inline long long conv_workgroups(long long ntiles, long long n_workgroups) {
  long long cap = (ntiles + 7) / 8 * 8;
  long long n = (n_workgroups + 7) / 8 * 8;
  return n < cap ? n : cap;
}

hipError_t launch_conv_fp32(const Geom& g, int cin, int cout, int act, const float* x, float* y,
                            const float* w, const float* bias, int batch, hipStream_t stream);

hipError_t launch_head(const Geom& g, int cin, int fp32, const void* x, const float* w_head,
                       const float* b_head, const int32_t* tables, uint8_t* nib, float* logits,
                       int batch, hipStream_t stream);

hipError_t launch_residual_pack(const Geom& g, const int32_t* tables, const uint64_t* det,
                                const uint8_t* nib, uint64_t* flips, uint64_t* residual, int batch,
                                hipStream_t stream);

hipError_t launch_residual_from_flips(const Geom& g, const int32_t* tables, const uint64_t* det,
                                      const uint64_t* flips, uint64_t* residual, int batch,
                                      hipStream_t stream);

// Device tables (int32), one allocation, offsets in elements:
//   [0, nstab)           site_of[n]: grid index of compact stabilizer n -- where
//                        its detector event enters and its measurement flip is
//                        read (its plaquette site, or in the paper's layout the
//                        qubit it is drawn onto)
//   comp_x[H*H]          compact index of the X stabilizer at grid site s, or -1
//   comp_z[H*H]          the same for Z (in the paper's layout an X and a Z
//                        stabilizer can share a site)
//   supp[nstab][4]       grid indices of the data qubits of stabilizer n (data
//                        qubit (r, c) is grid site r*H+c), -1 pads
//   sten[nstab][4]       residual stencil of stabilizer n, 16-byte aligned:
//                        {site | mch << 16, q0 | q1 << 16, q2 | q3 << 16, 0},
//                        mch = 2 (X) or 3 (Z) the measurement channel; a
//                        weight-two stabilizer repeats q0 as q2 and q3, whose
//                        two reads then cancel in the XOR
//   fsite[nflip]         flip bit n of a round: site | channel << 16
__host__ __device__ inline int tables_site_of(const Geom&) { return 0; }
__host__ __device__ inline int tables_comp_x(const Geom& g) { return g.nstab; }
__host__ __device__ inline int tables_comp_z(const Geom& g) { return g.nstab + g.H * g.H; }
__host__ __device__ inline int tables_supp(const Geom& g) { return g.nstab + 2 * g.H * g.H; }
__host__ __device__ inline int tables_sten(const Geom& g) { return (5 * g.nstab + 2 * g.H * g.H + 3) & ~3; }
__host__ __device__ inline int tables_fsite(const Geom& g) { return tables_sten(g) + 4 * g.nstab; }
__host__ __device__ inline int tables_size(const Geom& g) { return tables_fsite(g) + g.nflip; }

// Flip nibble of grid site s (bit 0 Z data, 1 X data, 2 X measurement, 3 Z
// measurement correction) from the four logits, keeping each channel only
// where it is defined (Eqs. ZcorreJK..SynZCorrJK): data qubits for 0/1, the
// site of an X / Z stabilizer for 2 / 3; a logit of exactly 0 is no flip.
// The flip bits a grid site can carry (its data-qubit bits when it is a
// data qubit, a measurement bit per stabilizer type on it), and the nibble
// of a site from these and its four logits (threshold: logit > 0).
__device__ __forceinline__ unsigned flip_allowed(const Geom& g, const int32_t* __restrict__ tables, int i, int j) {
  const int s = i * g.H + j;
  unsigned m = (i < g.d && j < g.d) ? 3u : 0u;
  if (tables[tables_comp_x(g) + s] >= 0) m |= 4u;
  if (tables[tables_comp_z(g) + s] >= 0) m |= 8u;
  return m;
}

__device__ __forceinline__ unsigned flip_bits(unsigned allowed, const float* lg) {
  const unsigned b = (lg[0] > 0.0f ? 1u : 0u) | (lg[1] > 0.0f ? 2u : 0u) | (lg[2] > 0.0f ? 4u : 0u) |
                     (lg[3] > 0.0f ? 8u : 0u);
  return allowed & b;
}

__device__ __forceinline__ unsigned flip_nibble(const Geom& g, const int32_t* __restrict__ tables, int i, int j,
                                                const float* lg) {
  return flip_bits(flip_allowed(g, tables, i, j), lg);
}

}  // namespace pd
