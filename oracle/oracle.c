/*
 * oracle.c -- plain, slow CPU reference of the pre-decoder hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library.  It shares no code, header,
 * table or constant generator with the GPU path: it carries its own geometry,
 * bit packing, bf16 rounding and activation.
 *
 * Everything follows the definitions of arXiv 2604.12841 as written:
 *   - detector events d_{i,k} = s_{i,k} XOR s_{i,k-1} placed on a grid
 *     (Sec. IV.B.1, Eqs. encTrainX1/encTrainX2, Fig. StabMap);
 *   - a fully convolutional 3D CNN, output the same size as the input
 *     (Sec. IV.B, Fig. ConvArch), stride 1, zero padding;
 *   - GELU, tanh form (Table hyperparameters);
 *   - corrections read from the four output channels (Eqs. ZcorreJK,
 *     XcorreJK, SynXCorrJK, SynZCorrJK), thresholded at sigmoid > 1/2, i.e.
 *     logit > 0 (the BCE objective of Sec. IV.B.5 applies a sigmoid);
 *   - syndromes induced by the data corrections (Eqs. SXJK, SZJK) and the
 *     residual syndrome (Eqs. Resk1X, ReskG1X, Resk1Z, ReskG1Z).
 *
 * Floating point is fp64.  In bf16 mode the quantisation points of the GPU
 * path are reproduced (weights and every conv/head input rounded to bf16 with
 * round-to-nearest-even; the pre-activation is rounded to fp32 before the
 * activation; the activation is evaluated in fp64 and rounded to fp32 and then
 * to bf16; logits are rounded to fp32).  Products of bf16 values are exact in
 * fp64, so the only difference from an exact sum is fp64 rounding.
 *
 * In fp8 mode (the paper deploys its models in FP8, Sec. VI; it does not
 * state the scaling, the reading here is this file's): OCP E4M3 (4 exponent
 * bits, bias 7, 3 mantissa bits, no infinities, largest finite 448).  Weights
 * of every layer get one power-of-two scale per output channel, 2^e with e
 * the smallest integer such that max |w| / 2^e <= 448, and are stored as
 * e4m3(w / 2^e) (so w is used as e4m3(w / 2^e) * 2^e, exactly); every conv
 * or head input is rounded to e4m3 with no scale (the input planes, 0, 1/2
 * and 1, are exact); rounding is to nearest, ties to the even code, and
 * magnitudes above 448 saturate to 448.  The pre-activation is rounded to
 * fp32 and the activation evaluated in fp64 and rounded to fp32, then to
 * e4m3; biases and logits are fp32.
 *
 * Array layout is channel-major per sample (like PyTorch NCDHW):
 * x[b][c][t][i][j] with i, j in [0, d] on the (d+1) x (d+1) plaquette grid,
 * or, in the paper's own layout (Sec. IV.B.1), i, j in [0, d-1] on the D x D
 * data-qubit grid (D = d) with four input channels.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------- */
/* Geometry of the rotated surface code on the (d+1) x (d+1) plaquette grid */
/* (Sec. III, Fig. SurfaceCodeExamp: X_L horizontal, Z_L vertical; Fig. StabMap).           */
/* ---------------------------------------------------------------------- */

/* Kind of grid site (i, j): 1 = X stabilizer, 2 = Z stabilizer, 0 = none. */
int oracle_site_kind(int d, int i, int j) {
  if (i < 0 || j < 0 || i > d || j > d) return 0;
  if (((i + j) % 2 == 0) && i >= 1 && i <= d - 1) return 1;
  if (((i + j) % 2 == 1) && j >= 1 && j <= d - 1) return 2;
  return 0;
}

/* Data qubits acted on by plaquette (i, j): the corners (i-1, j-1), (i-1, j),
 * (i, j-1), (i, j) that lie in [0, d-1]^2.  Writes up to 4 (r, c) pairs into
 * rc[8] and returns how many. */
int oracle_plaquette_support(int d, int i, int j, int* rc) {
  int n = 0;
  for (int dr = -1; dr <= 0; ++dr)
    for (int dc = -1; dc <= 0; ++dc) {
      int r = i + dr, c = j + dc;
      if (r >= 0 && r < d && c >= 0 && c < d) {
        rc[2 * n] = r;
        rc[2 * n + 1] = c;
        ++n;
      }
    }
  return n;
}

/* Compact enumeration of stabilizers: the X sites in row-major (i, j) order,
 * then the Z sites in row-major order.  site_of[n] = i * (d+1) + j for
 * n < d^2 - 1; index_of[i * (d+1) + j] = n or -1.  Returns d^2 - 1. */
int oracle_stabilizer_order(int d, int* site_of, int* index_of) {
  int H = d + 1, n = 0;
  for (int s = 0; s < H * H; ++s) index_of[s] = -1;
  for (int kind = 1; kind <= 2; ++kind)
    for (int i = 0; i <= d; ++i)
      for (int j = 0; j <= d; ++j)
        if (oracle_site_kind(d, i, j) == kind) {
          site_of[n] = i * H + j;
          index_of[i * H + j] = n;
          ++n;
        }
  return n;
}

int64_t oracle_det_words(int d, int T) { return ((int64_t)T * (d * d - 1) + 63) / 64; }
int64_t oracle_flip_words(int d, int T) { return ((int64_t)T * (3 * d * d - 1) + 63) / 64; }

static int get_bit(const uint64_t* row, int64_t b) { return (int)((row[b >> 6] >> (b & 63)) & 1u); }
static void set_bit(uint64_t* row, int64_t b, int v) {
  if (v) row[b >> 6] |= (uint64_t)1 << (b & 63);
}

/* ---------------------------------------------------------------------- */
/* Unpack (Sec. IV.B.1): X-type detector events of round t at their X     */
/* sites in channel 0, Z-type at their Z sites in channel 1, 0 elsewhere.  */
/* planes: [B][2][T][d+1][d+1].                                            */
/* ---------------------------------------------------------------------- */
void oracle_unpack(int d, int T, int B, const uint64_t* det, double* planes) {
  int H = d + 1, S = d * d - 1;
  int64_t W = oracle_det_words(d, T);
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  for (int b = 0; b < B; ++b)
    for (int c = 0; c < 2; ++c)
      for (int t = 0; t < T; ++t)
        for (int i = 0; i < H; ++i)
          for (int j = 0; j < H; ++j) {
            int kind = oracle_site_kind(d, i, j);
            double v = 0.0;
            if (kind == c + 1) {
              int n = index_of[i * H + j];
              v = (double)get_bit(det + (int64_t)b * W, (int64_t)t * S + n);
            }
            planes[((((int64_t)b * 2 + c) * T + t) * H + i) * H + j] = v;
          }
  free(site_of);
  free(index_of);
}

/* ---------------------------------------------------------------------- */
/* The paper's own layout (Sec. IV.B.1, Fig. StabMap, Eqs. encTrainX1-4):  */
/* the grid is the D x D array of data qubits (D = d) and every stabilizer */
/* is drawn onto one data qubit of its support: a weight-four X (Z)        */
/* stabilizer onto its top-left (top-right) qubit, a weight-two X          */
/* stabilizer onto its top qubit and a weight-two Z stabilizer onto its    */
/* right qubit.                                                             */
/* ---------------------------------------------------------------------- */

/* Data qubit (r, c) of plaquette (i, j) under that drawing; returns 0 when
 * (i, j) holds no stabilizer.  "Top" is the smaller row, "left" the smaller
 * column. */
int oracle_stabilizer_qubit(int d, int i, int j, int* r, int* c) {
  int kind = oracle_site_kind(d, i, j);
  if (kind == 0) return 0;
  int rc[8];
  int n = oracle_plaquette_support(d, i, j, rc);
  /* the support in row-major order: rc[0..1] is the top-left qubit of a
   * weight-four plaquette and the top (left) qubit of a vertical (horizontal)
   * weight-two one */
  if (kind == 1) {
    *r = rc[0];
    *c = rc[1];
  } else {
    /* top-right of four; of a horizontal pair (same row), the right one */
    *r = rc[0];
    *c = (n == 4) ? rc[3] : rc[2 * (n - 1) + 1];
  }
  return kind;
}

/* Planes of the paper's layout: [B][4][T][d][d], channels
 *   0 x_type: X-type detector event of round t at its stabilizer's qubit,
 *   1 z_type: the same for Z-type,
 *   2 x_present: weight / 4 of the X stabilizer drawn at the qubit,
 *   3 z_present: the same for Z (Eqs. encTrainX1-encTrainX4),
 * and 0 wherever no stabilizer is drawn.  first / last (0 none, 1 Z, 2 X) is
 * the basis the qubit is prepared in before round 0 / measured in after round
 * T-1: preparing |0> (Z) or measuring Z clears x_present in that round,
 * preparing |+> (X) or measuring X clears z_present. */
void oracle_unpack_paper(int d, int T, int B, const uint64_t* det, int first, int last, double* planes) {
  int H = d + 1, S = d * d - 1;
  int64_t W = oracle_det_words(d, T);
  int64_t V = (int64_t)T * d * d;
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  memset(planes, 0, sizeof(double) * (size_t)B * 4 * V);
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < T; ++t)
      for (int i = 0; i <= d; ++i)
        for (int j = 0; j <= d; ++j) {
          int r, c, rc[8];
          int kind = oracle_stabilizer_qubit(d, i, j, &r, &c);
          if (kind == 0) continue;
          int n = index_of[i * H + j];
          double weight = (double)oracle_plaquette_support(d, i, j, rc) / 4.0;
          int cleared = (t == 0 && first == kind) || (t == T - 1 && last == kind);
          int64_t at = (int64_t)t * d * d + r * d + c;
          double* pb = planes + (int64_t)b * 4 * V;
          pb[(kind - 1) * V + at] = (double)get_bit(det + (int64_t)b * W, (int64_t)t * S + n);
          pb[(kind + 1) * V + at] = cleared ? 0.0 : weight;
        }
  free(site_of);
  free(index_of);
}

/* ---------------------------------------------------------------------- */
/* Number formats and the activation                                       */
/* ---------------------------------------------------------------------- */

/* fp32 -> bf16 -> fp32 with round-to-nearest, ties to even, on the fp32 bit
 * pattern (bf16 keeps the top 16 bits).  NaN stays NaN. */
float oracle_round_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) {
    u |= 0x00400000u; /* quiet NaN */
  } else {
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
  }
  u &= 0xffff0000u;
  float y;
  memcpy(&y, &u, 4);
  return y;
}

/* OCP E4M3 code -> value (Sec. VI deploys FP8; the format is the OCP 8-bit
 * floating point one): sign bit 7, exponent field bits 6..3 (bias 7),
 * mantissa bits 2..0; exponent field 0 is subnormal (m 2^-9); code 0x7f /
 * 0xff is NaN; there are no infinities. */
double oracle_e4m3_value(int code) {
  int sgn = (code >> 7) & 1, ex = (code >> 3) & 15, m = code & 7;
  double v;
  if (ex == 15 && m == 7) return NAN;
  if (ex == 0)
    v = ldexp((double)m, -9);
  else
    v = ldexp(1.0 + m / 8.0, ex - 7);
  return sgn ? -v : v;
}

/* fp32 -> E4M3 code: the nearest finite value, ties to the even code (the
 * one whose mantissa LSB is 0), |x| > 448 saturating to 448.  Found by
 * searching the 127 non-negative finite codes, whose values increase with
 * the code.  NaN gives 0x7f. */
int oracle_e4m3_code(float x) {
  if (isnan(x)) return 0x7f;
  int sgn = signbit(x) ? 0x80 : 0;
  double a = fabs((double)x);
  int lo = 0, hi = 0x7e; /* largest code with value <= a, by bisection */
  if (a >= oracle_e4m3_value(0x7e)) return sgn | 0x7e;
  while (lo < hi) {
    int mid = (lo + hi + 1) / 2;
    if (oracle_e4m3_value(mid) <= a)
      lo = mid;
    else
      hi = mid - 1;
  }
  double below = oracle_e4m3_value(lo), above = oracle_e4m3_value(lo + 1);
  int code;
  if (a - below < above - a)
    code = lo;
  else if (a - below > above - a)
    code = lo + 1;
  else
    code = (lo & 1) ? lo + 1 : lo;
  return sgn | code;
}

/* fp32 -> E4M3 -> value. */
double oracle_round_e4m3(float x) { return oracle_e4m3_value(oracle_e4m3_code(x)); }

/* Scale exponent of a weight row in fp8 mode: the smallest e with
 * amax / 2^e <= 448 (0 for an all-zero row). */
int oracle_e4m3_scale_exp(double amax) {
  if (amax == 0.0) return 0;
  int e = -160;
  while (ldexp(amax, -e) > 448.0) ++e;
  while (ldexp(amax, -(e - 1)) <= 448.0) --e;
  return e;
}

/* GELU, tanh approximation (Table hyperparameters):
 *   0.5 y (1 + tanh(u)),  u = sqrt(2/pi) (y + 0.044715 y^3),
 * evaluated as y / (1 + exp(-2u)), the same function (1 + tanh(u) =
 * 2 / (1 + exp(-2u))): in fp64, 1 + tanh(u) cancels once tanh(u) is within a
 * few ulps of -1 (u below about -18, y below about -5.5) and loses every
 * digit of the small result, which this form keeps. */
double oracle_gelu_tanh(double y) {
  const double pi = 3.14159265358979323846;
  double u = sqrt(2.0 / pi) * (y + 0.044715 * y * y * y);
  return y / (1.0 + exp(-2.0 * u));
}

enum { ACT_NONE = 0, ACT_GELU_TANH = 1, ACT_RELU = 2 };

static double activation(int act, double y) {
  if (act == ACT_GELU_TANH) return oracle_gelu_tanh(y);
  if (act == ACT_RELU) return y > 0.0 ? y : 0.0;
  return y;
}

int64_t oracle_weight_count(int n_layers, const int* spec) {
  int64_t n = 0;
  for (int l = 0; l < n_layers; ++l) {
    int64_t ci = spec[4 * l], co = spec[4 * l + 1], k = spec[4 * l + 2];
    n += co * ci * k * k * k + co;
  }
  return n;
}

/* ---------------------------------------------------------------------- */
/* Forward pass of the fully convolutional network (Sec. IV.B).           */
/*   y[co][t][i][j] = b[co] + sum_{ci,kt,ki,kj} w[co][ci][kt][ki][kj] *    */
/*                    x[ci][t+kt-p][i+ki-p][j+kj-p],  p = (k-1)/2,          */
/* with x = 0 outside [0,T) x [0,H) x [0,H); hidden layers apply their     */
/* activation, the last layer is linear (it gives the logits).              */
/* spec: n_layers x {c_in, c_out, k, act}.  weights: fp32, per layer        */
/* w[c_out][c_in][k][k][k] then b[c_out].  planes: [B][c_in0][T][H][H].     */
/* logits: [B][c_out_last][T][H][H].  prec: 0 exact (fp64), 1 bf16, 2 fp8:  */
/* the quantisation points described at the top of this file.               */
/* Samples and output channels are independent; they are spread over       */
/* OpenMP threads (the arithmetic of each output is unchanged).             */
/* ---------------------------------------------------------------------- */
/* Counter-based value in [-1, 1) (splitmix64 finaliser of the key). */
static double unit_hash(uint64_t key) {
  uint64_t z = key + 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (double)(z >> 11) * 0x1.0p-52 - 1.0;
}

/* eps > 0 (fp8 only; test infrastructure): every sum of products is moved
 * by u eps sum |products|, u in [-1, 1) hashed from (seed, layer, sample,
 * channel, voxel): a summation whose error is bounded by eps relative to the
 * sum of magnitudes, used to size the fp8 parity bounds.  Different seeds
 * give independent patterns of such errors. */
static void forward_impl(int H, int T, int B, const double* planes, int n_layers, const int* spec,
                         const float* weights, int prec, double eps, uint64_t seed, double* logits) {
  const int bf16 = prec == 1, fp8 = prec == 2;
  int64_t V = (int64_t)T * H * H;
  int cmax = spec[0];
  for (int l = 0; l < n_layers; ++l)
    if (spec[4 * l + 1] > cmax) cmax = spec[4 * l + 1];

  /* Per-layer weights in fp64 (rounded to bf16 first in bf16 mode; in fp8
   * mode e4m3(w / 2^e) * 2^e with one e per output channel). */
  double** w = (double**)malloc(sizeof(double*) * n_layers);
  double** bias = (double**)malloc(sizeof(double*) * n_layers);
  const float* src = weights;
  for (int l = 0; l < n_layers; ++l) {
    int ci = spec[4 * l], co = spec[4 * l + 1], k = spec[4 * l + 2];
    int64_t nw = (int64_t)co * ci * k * k * k;
    w[l] = (double*)malloc(sizeof(double) * nw);
    bias[l] = (double*)malloc(sizeof(double) * co);
    for (int64_t e = 0; e < nw; ++e) w[l][e] = bf16 ? (double)oracle_round_bf16(src[e]) : (double)src[e];
    if (fp8) {
      int64_t row = nw / co;
      for (int c = 0; c < co; ++c) {
        double amax = 0.0;
        for (int64_t e = 0; e < row; ++e) amax = fmax(amax, fabs((double)src[c * row + e]));
        int ex = oracle_e4m3_scale_exp(amax);
        for (int64_t e = 0; e < row; ++e)
          w[l][c * row + e] = ldexp(oracle_round_e4m3((float)ldexp((double)src[c * row + e], -ex)), ex);
      }
    }
    for (int e = 0; e < co; ++e) bias[l][e] = (double)src[nw + e];
    src += nw + co;
  }

  double* xa = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  double* xb = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  int c0 = spec[0];
  for (int b = 0; b < B; ++b)
    for (int64_t e = 0; e < c0 * V; ++e) {
      double v = planes[(int64_t)b * c0 * V + e];
      xa[(int64_t)b * cmax * V + e] =
          bf16 ? (double)oracle_round_bf16((float)v) : (fp8 ? oracle_round_e4m3((float)v) : v);
    }

  for (int l = 0; l < n_layers; ++l) {
    int ci_n = spec[4 * l], co_n = spec[4 * l + 1], k = spec[4 * l + 2], act = spec[4 * l + 3];
    int p = (k - 1) / 2, last = (l == n_layers - 1);
    const double* wl = w[l];
    const double* bl = bias[l];
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int co = 0; co < co_n; ++co) {
        const double* x = xa + (int64_t)b * cmax * V;
        double* y = xb + (int64_t)b * cmax * V + (int64_t)co * V;
        /* acc[v] = sum over (ci, kt, ki, kj), in that order, of w * x at the
         * tap's input voxel (taps outside the volume contribute nothing);
         * mag[v] the same sum of magnitudes.  The voxel loops sit inside the
         * tap loops so that each tap sweeps the input contiguously; every
         * output still adds its products in the order above. */
        double* acc = (double*)calloc((size_t)V, sizeof(double));
        double* mag = (double*)calloc((size_t)V, sizeof(double));
        for (int ci = 0; ci < ci_n; ++ci)
          for (int kt = 0; kt < k; ++kt)
            for (int ki = 0; ki < k; ++ki)
              for (int kj = 0; kj < k; ++kj) {
                const double wv = wl[(((int64_t)co * ci_n + ci) * k + kt) * k * k + ki * k + kj];
                for (int t = 0; t < T; ++t) {
                  int tt = t + kt - p;
                  if (tt < 0 || tt >= T) continue;
                  for (int i = 0; i < H; ++i) {
                    int ii = i + ki - p;
                    if (ii < 0 || ii >= H) continue;
                    const double* xr = x + (((int64_t)ci * T + tt) * H + ii) * H;
                    double* ar = acc + ((int64_t)t * H + i) * H;
                    double* mr = mag + ((int64_t)t * H + i) * H;
                    /* the j whose tap column j + kj - p lies in [0, H) */
                    const int j0 = p - kj > 0 ? p - kj : 0, j1 = H + p - kj < H ? H + p - kj : H;
                    for (int j = j0; j < j1; ++j) {
                      const double pr = wv * xr[j + kj - p];
                      ar[j] += pr;
                      mr[j] += fabs(pr);
                    }
                  }
                }
              }
        for (int t = 0; t < T; ++t)
          for (int i = 0; i < H; ++i)
            for (int j = 0; j < H; ++j) {
              const int64_t v = ((int64_t)t * H + i) * H + j;
              double a = acc[v];
              if (eps > 0.0) {
                const uint64_t key = ((((((uint64_t)l * 65536 + b) * 4096 + co) * 2048 + t) * 256 + i) * 256) + j;
                a += unit_hash(key ^ (seed * 0xd1b54a32d192ed03ull)) * eps * mag[v];
              }
              double out;
              if (fp8) {
                float pre = (float)(a + bl[co]);
                if (last) {
                  out = (double)pre; /* fp32 logit */
                } else {
                  float av = (float)activation(act, (double)pre);
                  out = oracle_round_e4m3(av);
                }
              } else if (bf16) {
                float pre = (float)(a + bl[co]);
                if (last) {
                  out = (double)pre; /* fp32 logit */
                } else {
                  float av = (float)activation(act, (double)pre);
                  out = (double)oracle_round_bf16(av);
                }
              } else {
                out = last ? a + bl[co] : activation(act, a + bl[co]);
              }
              y[v] = out;
            }
        free(acc);
        free(mag);
      }
    double* tmp = xa;
    xa = xb;
    xb = tmp;
  }
  int co_last = spec[4 * (n_layers - 1) + 1];
  for (int b = 0; b < B; ++b)
    memcpy(logits + (int64_t)b * co_last * V, xa + (int64_t)b * cmax * V, sizeof(double) * co_last * V);

  for (int l = 0; l < n_layers; ++l) {
    free(w[l]);
    free(bias[l]);
  }
  free(w);
  free(bias);
  free(xa);
  free(xb);
}

void oracle_forward_grid(int H, int T, int B, const double* planes, int n_layers, const int* spec,
                         const float* weights, int prec, double* logits) {
  forward_impl(H, T, B, planes, n_layers, spec, weights, prec, 0.0, 0, logits);
}

/* fp8 forward with the bounded summation error described at forward_impl
 * (eps = 0: the plain fp8 forward). */
void oracle_forward_grid_fp8_perturbed(int H, int T, int B, const double* planes, int n_layers, const int* spec,
                                       const float* weights, double eps, uint64_t seed, double* logits) {
  forward_impl(H, T, B, planes, n_layers, spec, weights, 2, eps, seed, logits);
}

/* The same on the (d+1) x (d+1) plaquette grid. */
void oracle_forward(int d, int T, int B, const double* planes, int n_layers, const int* spec,
                    const float* weights, int prec, double* logits) {
  oracle_forward_grid(d + 1, T, B, planes, n_layers, spec, weights, prec, logits);
}

/* ---------------------------------------------------------------------- */
/* Corrections and residual (Sec. IV.B.6).                                */
/* ---------------------------------------------------------------------- */

/* Residual of one sample from unpacked corrections on the grid:
 *   zc[t][r][c], xc[t][r][c]  data-qubit Z / X corrections (r, c < d),
 *   mx[t][i][j], mz[t][i][j]  X / Z measurement corrections at their sites.
 * R[t](s) = D[t](s) ^ m[t](s) ^ m[t-1](s) ^ (parity of the data corrections
 * on the support of s): M_X reads Z corrections, M_Z reads X corrections
 * (Eqs. SXJK, SZJK); a measurement correction in round t flips the outcome
 * in rounds t and t+1, so the detector of round t sees m[t] and m[t-1]
 * (Eqs. Resk1X..ReskG1Z; nothing before round 0). */
static void residual_one(int d, int T, const uint64_t* det, const uint8_t* zc, const uint8_t* xc,
                         const uint8_t* mx, const uint8_t* mz, uint64_t* res) {
  int H = d + 1, S = d * d - 1;
  int64_t W = oracle_det_words(d, T);
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  memset(res, 0, sizeof(uint64_t) * W);
  for (int t = 0; t < T; ++t)
    for (int n = 0; n < S; ++n) {
      int s = site_of[n], i = s / H, j = s % H;
      int kind = oracle_site_kind(d, i, j);
      const uint8_t* m = (kind == 1) ? mx : mz;
      const uint8_t* data = (kind == 1) ? zc : xc;
      int64_t b = (int64_t)t * S + n;
      int v = get_bit(det, b);
      v ^= m[(t * H + i) * H + j];
      if (t > 0) v ^= m[((t - 1) * H + i) * H + j];
      int rc[8];
      int q = oracle_plaquette_support(d, i, j, rc);
      for (int e = 0; e < q; ++e) v ^= data[(t * H + rc[2 * e]) * H + rc[2 * e + 1]];
      set_bit(res, b, v);
    }
  free(site_of);
  free(index_of);
}

/* Thresholds logits [B][4][T][H][H] (flip = logit > 0, Eqs. ZcorreJK..
 * SynZCorrJK with the sigmoid of Sec. IV.B.5), keeps each channel only where
 * it is defined (data qubits for 0/1, X sites for 2, Z sites for 3), packs the
 * flips and computes the residual. */
void oracle_flips_residual(int d, int T, int B, const double* logits, const uint64_t* det,
                           uint64_t* flips, uint64_t* residual) {
  int H = d + 1, S = d * d - 1, K = S / 2;
  int64_t V = (int64_t)T * H * H;
  int64_t Wd = oracle_det_words(d, T), Wf = oracle_flip_words(d, T);
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  uint8_t* f = (uint8_t*)malloc(4 * V);
  for (int b = 0; b < B; ++b) {
    const double* lg = logits + (int64_t)b * 4 * V;
    for (int ch = 0; ch < 4; ++ch)
      for (int t = 0; t < T; ++t)
        for (int i = 0; i < H; ++i)
          for (int j = 0; j < H; ++j) {
            int kind = oracle_site_kind(d, i, j);
            int defined = (ch < 2) ? (i < d && j < d) : (kind == ch - 1);
            int64_t e = ((int64_t)ch * T + t) * H * H + i * H + j;
            f[e] = (uint8_t)(defined && lg[e] > 0.0);
          }
    uint64_t* fr = flips + (int64_t)b * Wf;
    memset(fr, 0, sizeof(uint64_t) * Wf);
    for (int t = 0; t < T; ++t) {
      int64_t base = (int64_t)t * (3 * d * d - 1);
      for (int r = 0; r < d; ++r)
        for (int c = 0; c < d; ++c) {
          set_bit(fr, base + r * d + c, f[(0 * T + t) * H * H + r * H + c]);
          set_bit(fr, base + d * d + r * d + c, f[(1 * T + t) * H * H + r * H + c]);
        }
      for (int n = 0; n < S; ++n) {
        int s = site_of[n];
        int ch = (n < K) ? 2 : 3;
        set_bit(fr, base + 2 * d * d + n, f[((int64_t)ch * T + t) * H * H + s]);
      }
    }
    residual_one(d, T, det + (int64_t)b * Wd, f, f + V, f + 2 * V, f + 3 * V,
                 residual + (int64_t)b * Wd);
  }
  free(f);
  free(site_of);
  free(index_of);
}

/* The paper's layout: logits [B][4][T][d][d].  Channels 0/1 are the Z / X
 * data corrections of qubit (r, c) (Eqs. ZcorreJK, XcorreJK); channel 2 (3) at
 * the qubit an X (Z) stabilizer is drawn onto is that stabilizer's
 * measurement correction (Eqs. SynXCorrJK, SynZCorrJK).  Flips are packed as
 * in oracle_flips_residual and the residual is the same function of them. */
void oracle_flips_residual_paper(int d, int T, int B, const double* logits, const uint64_t* det,
                                 uint64_t* flips, uint64_t* residual) {
  int H = d + 1, S = d * d - 1;
  int64_t V = (int64_t)T * H * H, VD = (int64_t)T * d * d;
  int64_t Wd = oracle_det_words(d, T), Wf = oracle_flip_words(d, T);
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  uint8_t* f = (uint8_t*)malloc(4 * V); /* on the plaquette grid, as residual_one reads them */
  for (int b = 0; b < B; ++b) {
    const double* lg = logits + (int64_t)b * 4 * VD;
    memset(f, 0, 4 * V);
    uint64_t* fr = flips + (int64_t)b * Wf;
    memset(fr, 0, sizeof(uint64_t) * Wf);
    for (int t = 0; t < T; ++t) {
      int64_t base = (int64_t)t * (3 * d * d - 1);
      for (int r = 0; r < d; ++r)
        for (int c = 0; c < d; ++c)
          for (int ch = 0; ch < 2; ++ch) {
            int v = lg[ch * VD + (int64_t)t * d * d + r * d + c] > 0.0;
            f[ch * V + ((int64_t)t * H + r) * H + c] = (uint8_t)v;
            set_bit(fr, base + ch * d * d + r * d + c, v);
          }
      for (int n = 0; n < S; ++n) {
        int s = site_of[n], i = s / H, j = s % H, r, c;
        int kind = oracle_stabilizer_qubit(d, i, j, &r, &c);
        int ch = kind + 1; /* 2 for X, 3 for Z */
        int v = lg[ch * VD + (int64_t)t * d * d + r * d + c] > 0.0;
        f[ch * V + (int64_t)t * H * H + s] = (uint8_t)v;
        set_bit(fr, base + 2 * d * d + n, v);
      }
    }
    residual_one(d, T, det + (int64_t)b * Wd, f, f + V, f + 2 * V, f + 3 * V,
                 residual + (int64_t)b * Wd);
  }
  free(f);
  free(site_of);
  free(index_of);
}

/* Residual from packed flips (same format as oracle_flips_residual writes). */
void oracle_residual_from_flips(int d, int T, int B, const uint64_t* det, const uint64_t* flips,
                                uint64_t* residual) {
  int H = d + 1, S = d * d - 1, K = S / 2;
  int64_t V = (int64_t)T * H * H;
  int64_t Wd = oracle_det_words(d, T), Wf = oracle_flip_words(d, T);
  int* site_of = (int*)malloc(sizeof(int) * S);
  int* index_of = (int*)malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  uint8_t* f = (uint8_t*)malloc(4 * V);
  for (int b = 0; b < B; ++b) {
    const uint64_t* fr = flips + (int64_t)b * Wf;
    memset(f, 0, 4 * V);
    for (int t = 0; t < T; ++t) {
      int64_t base = (int64_t)t * (3 * d * d - 1);
      for (int r = 0; r < d; ++r)
        for (int c = 0; c < d; ++c) {
          f[(0 * T + t) * H * H + r * H + c] = (uint8_t)get_bit(fr, base + r * d + c);
          f[(1 * T + t) * H * H + r * H + c] = (uint8_t)get_bit(fr, base + d * d + r * d + c);
        }
      for (int n = 0; n < S; ++n) {
        int ch = (n < K) ? 2 : 3;
        f[((int64_t)ch * T + t) * H * H + site_of[n]] = (uint8_t)get_bit(fr, base + 2 * d * d + n);
      }
    }
    residual_one(d, T, det + (int64_t)b * Wd, f, f + V, f + 2 * V, f + 3 * V,
                 residual + (int64_t)b * Wd);
  }
  free(f);
  free(site_of);
  free(index_of);
}

/* ---------------------------------------------------------------------- */
/* Residual network (Model 6, Sec. VI, Fig. Model8Representation).        */
/* ---------------------------------------------------------------------- */

/* y[b][co][v] = bias[co] + sum_{ci, taps} w[co][ci][taps] x[b][ci][v + tap]
 * on a T x H x H volume with zero padding, k = 1 or 3; fp64 sums (acc32:
 * fp32 sums in this loop order, another valid summation).  eps > 0 (test
 * infrastructure, fp64 sums): each sum moved by u eps sum |products|, u in
 * [-1, 1) hashed from (seed, key, sample, channel, voxel), as in the fp8
 * forward above. */
static void conv_sums_eps(int H, int T, int B, const double* x, int ci_n, int co_n, int k, const double* w,
                          const double* bias, double* y, int acc32, double eps, uint64_t seed, uint64_t key) {
  const int64_t V = (int64_t)T * H * H;
  const int p = (k - 1) / 2;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int co = 0; co < co_n; ++co) {
      /* per output voxel, the products in (ci, kt, ki, kj) order; the voxel
       * loops sit inside the tap loops (each output's order is unchanged) */
      double* acc = (double*)calloc((size_t)V, sizeof(double));
      double* mag = eps > 0.0 ? (double*)calloc((size_t)V, sizeof(double)) : NULL;
      float* accf = (float*)calloc((size_t)V, sizeof(float));
      for (int ci = 0; ci < ci_n; ++ci)
        for (int kt = 0; kt < k; ++kt)
          for (int ki = 0; ki < k; ++ki)
            for (int kj = 0; kj < k; ++kj) {
              const double wv = w[(((int64_t)co * ci_n + ci) * k + kt) * k * k + ki * k + kj];
              for (int t = 0; t < T; ++t) {
                const int tt = t + kt - p;
                if (tt < 0 || tt >= T) continue;
                for (int i = 0; i < H; ++i) {
                  const int ii = i + ki - p;
                  if (ii < 0 || ii >= H) continue;
                  const double* xr = x + (((int64_t)b * ci_n + ci) * T + tt) * H * H + (int64_t)ii * H;
                  const int64_t o = ((int64_t)t * H + i) * H;
                  /* the j whose tap column j + kj - p lies in [0, H) */
                  const int j0 = p - kj > 0 ? p - kj : 0, j1 = H + p - kj < H ? H + p - kj : H;
                  if (acc32)
                    for (int j = j0; j < j1; ++j) accf[o + j] += (float)(wv * xr[j + kj - p]);
                  else
                    for (int j = j0; j < j1; ++j) acc[o + j] += wv * xr[j + kj - p];
                  if (mag)
                    for (int j = j0; j < j1; ++j) mag[o + j] += fabs(wv * xr[j + kj - p]);
                }
              }
            }
      for (int64_t v = 0; v < V; ++v) {
        double a = acc32 ? (double)accf[v] : acc[v];
        if (mag) {
          const uint64_t hk = (((key * 65536 + (uint64_t)b) * 4096 + (uint64_t)co) << 24) + (uint64_t)v;
          a += unit_hash(hk ^ (seed * 0xd1b54a32d192ed03ull)) * eps * mag[v];
        }
        y[((int64_t)b * co_n + co) * V + v] = a + bias[co];
      }
      free(acc);
      free(mag);
      free(accf);
    }
}

static void conv_sums(int H, int T, int B, const double* x, int ci_n, int co_n, int k, const double* w,
                      const double* bias, double* y, int acc32) {
  conv_sums_eps(H, T, B, x, ci_n, co_n, k, w, bias, y, acc32, 0.0, 0, 0);
}

/* conv_sums as a library entry (test infrastructure: pins its two
 * summation modes). */
void oracle_conv_sums(int H, int T, int B, const double* x, int ci_n, int co_n, int k, const double* w,
                      const double* bias, double* y, int acc32) {
  conv_sums(H, T, B, x, ci_n, co_n, k, w, bias, y, acc32);
}

/* Number of floats of a residual network's weights: per block (c_in, c_mid,
 * c_out): conv1 c_mid c_in 27 + c_mid, BatchNorm 4 c_mid (scale, shift,
 * running mean, running variance), conv2 c_out c_mid 27 + c_out, BatchNorm
 * 4 c_out, and a projection c_out c_in + c_out when c_in != c_out.  bn_per
 * channel = 2 counts the trainable parameters only (as the paper does). */
int64_t oracle_resnet_weight_count(int n_blocks, const int* spec, int bn_per_channel) {
  int64_t n = 0;
  for (int k = 0; k < n_blocks; ++k) {
    const int64_t ci = spec[4 * k], cm = spec[4 * k + 1], co = spec[4 * k + 2];
    n += cm * ci * 27 + cm + bn_per_channel * cm + co * cm * 27 + co + bn_per_channel * co;
    if (ci != co) n += co * ci + co;
  }
  return n;
}

/* Forward of a residual network: n_blocks blocks {c_in, c_mid, c_out, act},
 * each (conv1: c_in -> c_mid, conv2: c_mid -> c_out)
 *   h = act(BN1(conv1(x))), s = x (c_in == c_out) or P(x) (a 1x1x1
 *   projection with bias), y = act(BN2(conv2(h)) + s), the last block
 *   without its final act (its c_out = 4 channels are the logits);
 * BN(z) = (z - mean) / sqrt(var + 1e-5) * scale + shift, running statistics.
 * prec 0: exact, fp64, BatchNorm applied as written.  prec 1 (bf16): BatchNorm
 * folded into its conv (g = scale / sqrt(var + eps) in fp64, weights
 * bf16(fp32(w g)), bias fp32((b - mean) g + shift)), projection weights bf16
 * and bias fp32; every stored tensor (h, P(x), y) rounded to bf16 after
 * rounding the pre-activation (and the activation) to fp32; the sum
 * BN2(conv2 h) + s rounded to fp32 once.  prec 2: prec 1 with the conv sums
 * taken in fp32 (test infrastructure: another valid summation, which sizes
 * the parity tolerance of residual networks).  prec 3 (fp8): the fp8
 * reading of the plain networks applied to the folded convs -- weights
 * fp32(w g) quantised per output channel to e4m3(w / 2^e) 2^e (2^e the
 * smallest power of two with max |w| / 2^e <= 448), the projection's
 * weights likewise, biases fp32, every stored tensor (the input planes, h,
 * P(x), y) rounded to E4M3 after rounding to fp32, the sum BN2(conv2 h) + s
 * rounded to fp32 once; exact (fp64) sums.  planes [B][c_in0][T][H][H];
 * logits [B][4][T][H][H]. */
static void forward_resnet_impl(int H, int T, int B, const double* planes, int n_blocks, const int* spec,
                                const float* weights, int prec, double sum_eps, uint64_t seed, double* logits) {
  const double eps = 1e-5;
  const int64_t V = (int64_t)T * H * H;
  const int acc32 = prec == 2, fp8 = prec == 3;
  /* a stored tensor's value from its fp32 value, in the mode's precision */
#define STORE(v) (fp8 ? oracle_round_e4m3((float)(v)) : (double)oracle_round_bf16((float)(v)))
  int cmax = spec[0];
  for (int k = 0; k < n_blocks; ++k)
    for (int q = 1; q < 3; ++q) cmax = spec[4 * k + q] > cmax ? spec[4 * k + q] : cmax;
  double* x = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  double* h = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  double* s = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  double* y = (double*)malloc(sizeof(double) * (size_t)B * cmax * V);
  const int c0 = spec[0];
  for (int64_t e = 0; e < (int64_t)B * c0 * V; ++e) x[e] = prec ? STORE(planes[e]) : planes[e];
  const float* src = weights;
  for (int k = 0; k < n_blocks; ++k) {
    const int ci = spec[4 * k], cm = spec[4 * k + 1], co = spec[4 * k + 2], act = spec[4 * k + 3];
    const int last = k == n_blocks - 1;
    /* the two conv + BatchNorm pairs of the block, each as folded or as written */
    double* cw[2];
    double* cb[2];
    double* bnp[2]; /* scale, shift, mean, var */
    for (int c = 0; c < 2; ++c) {
      const int cin = c == 0 ? ci : cm, cout = c == 0 ? cm : co;
      const int64_t nw = (int64_t)cout * cin * 27;
      cw[c] = (double*)malloc(sizeof(double) * nw);
      cb[c] = (double*)malloc(sizeof(double) * cout);
      bnp[c] = (double*)malloc(sizeof(double) * 4 * cout);
      for (int e = 0; e < 4 * cout; ++e) bnp[c][e] = (double)src[nw + cout + e];
      for (int o = 0; o < cout; ++o) {
        const double g = bnp[c][o] / sqrt(bnp[c][3 * cout + o] + eps);
        double* row = cw[c] + o * (int64_t)cin * 27;
        for (int64_t e = 0; e < (int64_t)cin * 27; ++e) {
          const double wv = (double)src[o * (int64_t)cin * 27 + e];
          row[e] = fp8 ? (double)(float)(wv * g) : (prec ? (double)oracle_round_bf16((float)(wv * g)) : wv);
        }
        if (fp8) { /* one power-of-two scale per output channel */
          double amax = 0.0;
          for (int64_t e = 0; e < (int64_t)cin * 27; ++e) amax = fmax(amax, fabs(row[e]));
          const int ex = oracle_e4m3_scale_exp(amax);
          for (int64_t e = 0; e < (int64_t)cin * 27; ++e)
            row[e] = ldexp(oracle_round_e4m3((float)ldexp(row[e], -ex)), ex);
        }
        const double bv = (double)src[nw + o];
        cb[c][o] = prec ? (double)(float)((bv - bnp[c][2 * cout + o]) * g + bnp[c][cout + o]) : bv;
      }
      src += nw + cout + 4 * cout;
    }
    /* h = act(BN1(conv1 x)) */
    conv_sums_eps(H, T, B, x, ci, cm, 3, cw[0], cb[0], h, acc32, sum_eps, seed, 3 * (uint64_t)k);
    for (int b = 0; b < B; ++b)
      for (int o = 0; o < cm; ++o)
        for (int64_t v = 0; v < V; ++v) {
          double* z = &h[((int64_t)b * cm + o) * V + v];
          if (prec) {
            *z = STORE(activation(act, (double)(float)*z));
          } else {
            const double g = bnp[0][o] / sqrt(bnp[0][3 * cm + o] + eps);
            *z = activation(act, (*z - bnp[0][2 * cm + o]) * g + bnp[0][cm + o]);
          }
        }
    /* shortcut */
    if (ci != co) {
      const int64_t np = (int64_t)co * ci;
      double* pw = (double*)malloc(sizeof(double) * np);
      double* pb = (double*)malloc(sizeof(double) * co);
      for (int64_t e = 0; e < np; ++e) pw[e] = (prec && !fp8) ? (double)oracle_round_bf16(src[e]) : (double)src[e];
      if (fp8)
        for (int o = 0; o < co; ++o) { /* one power-of-two scale per output channel */
          double amax = 0.0;
          for (int e = 0; e < ci; ++e) amax = fmax(amax, fabs(pw[o * (int64_t)ci + e]));
          const int ex = oracle_e4m3_scale_exp(amax);
          for (int e = 0; e < ci; ++e)
            pw[o * (int64_t)ci + e] = ldexp(oracle_round_e4m3((float)ldexp(pw[o * (int64_t)ci + e], -ex)), ex);
        }
      for (int o = 0; o < co; ++o) pb[o] = (double)src[np + o];
      src += np + co;
      conv_sums_eps(H, T, B, x, ci, co, 1, pw, pb, s, acc32, sum_eps, seed, 3 * (uint64_t)k + 1);
      if (prec)
        for (int64_t e = 0; e < (int64_t)B * co * V; ++e) s[e] = STORE(s[e]);
      free(pw);
      free(pb);
    } else {
      memcpy(s, x, sizeof(double) * (size_t)B * co * V);
    }
    /* y = act(BN2(conv2 h) + s) */
    conv_sums_eps(H, T, B, h, cm, co, 3, cw[1], cb[1], y, acc32, sum_eps, seed, 3 * (uint64_t)k + 2);
    for (int b = 0; b < B; ++b)
      for (int o = 0; o < co; ++o)
        for (int64_t v = 0; v < V; ++v) {
          const int64_t e = ((int64_t)b * co + o) * V + v;
          double pre;
          if (prec) {
            pre = (double)(float)(y[e] + s[e]);
          } else {
            const double g = bnp[1][o] / sqrt(bnp[1][3 * co + o] + eps);
            pre = (y[e] - bnp[1][2 * co + o]) * g + bnp[1][co + o] + s[e];
          }
          if (last)
            y[e] = pre;
          else
            y[e] = prec ? STORE(activation(act, pre)) : activation(act, pre);
        }
    double* t = x;
    x = y;
    y = t;
    for (int c = 0; c < 2; ++c) {
      free(cw[c]);
      free(cb[c]);
      free(bnp[c]);
    }
  }
  memcpy(logits, x, sizeof(double) * (size_t)B * 4 * V);
  free(x);
  free(h);
  free(s);
  free(y);
#undef STORE
}

void oracle_forward_resnet(int H, int T, int B, const double* planes, int n_blocks, const int* spec,
                           const float* weights, int prec, double* logits) {
  forward_resnet_impl(H, T, B, planes, n_blocks, spec, weights, prec, 0.0, 0, logits);
}

/* The fp8 residual forward (prec 3) with every sum of products moved by up
 * to eps sum |products| (test infrastructure: sizes the fp8 parity bound of
 * residual networks; eps = 0 is the plain fp8 forward). */
void oracle_forward_resnet_fp8_perturbed(int H, int T, int B, const double* planes, int n_blocks, const int* spec,
                                         const float* weights, double eps, uint64_t seed, double* logits) {
  forward_resnet_impl(H, T, B, planes, n_blocks, spec, weights, 3, eps, seed, logits);
}

/* Threads an OpenMP parallel region of the oracle uses (reported with the
 * CPU timing; not part of the method). */
int oracle_num_threads(void) { return omp_get_max_threads(); }

/* Sets that number (the CPU timing's single-thread figure); n >= 1. */
void oracle_set_num_threads(int n) {
  if (n >= 1) omp_set_num_threads(n);
}
