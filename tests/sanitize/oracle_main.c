/* Drives every entry point of oracle/oracle.c on small inputs, for a build
 * under AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_sanitizers.py):
 * any out-of-bounds access, leak of uninitialised reads into control flow
 * caught by UBSan, or undefined arithmetic aborts the run.  It also checks
 * two invariants that need no reference: ground truth (zero logits) keeps
 * the residual equal to the detectors, and the exact, bf16 and fp8 forwards
 * agree to within the rounding of their precision points on a small net. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int64_t oracle_det_words(int d, int T);
int64_t oracle_flip_words(int d, int T);
int oracle_site_kind(int d, int i, int j);
int oracle_plaquette_support(int d, int i, int j, int* rc);
int oracle_stabilizer_order(int d, int* site_of, int* index_of);
void oracle_unpack(int d, int T, int B, const uint64_t* det, double* planes);
int oracle_stabilizer_qubit(int d, int i, int j, int* r, int* c);
void oracle_unpack_paper(int d, int T, int B, const uint64_t* det, int first, int last, double* planes);
float oracle_round_bf16(float x);
double oracle_e4m3_value(int code);
int oracle_e4m3_code(float x);
int oracle_e4m3_scale_exp(double amax);
double oracle_gelu_tanh(double y);
int64_t oracle_weight_count(int n_layers, const int* spec);
void oracle_forward_grid(int H, int T, int B, const double* planes, int n_layers, const int* spec,
                         const float* weights, int prec, double* logits);
void oracle_forward_grid_fp8_perturbed(int H, int T, int B, const double* planes, int n_layers, const int* spec,
                                       const float* weights, double eps, uint64_t seed, double* logits);
void oracle_forward(int d, int T, int B, const double* planes, int n_layers, const int* spec,
                    const float* weights, int prec, double* logits);
void oracle_flips_residual(int d, int T, int B, const double* logits, const uint64_t* det, uint64_t* flips,
                           uint64_t* residual);
void oracle_flips_residual_paper(int d, int T, int B, const double* logits, const uint64_t* det, uint64_t* flips,
                                 uint64_t* residual);
void oracle_residual_from_flips(int d, int T, int B, const uint64_t* det, const uint64_t* flips,
                                uint64_t* residual);
void oracle_conv_sums(int H, int T, int B, const double* x, int ci_n, int co_n, int k, const double* w,
                      const double* bias, double* y, int acc32);
int64_t oracle_resnet_weight_count(int n_blocks, const int* spec, int bn_per_channel);
void oracle_forward_resnet(int H, int T, int B, const double* planes, int n_blocks, const int* spec,
                           const float* weights, int prec, double* logits);
void oracle_forward_resnet_fp8_perturbed(int H, int T, int B, const double* planes, int n_blocks, const int* spec,
                                         const float* weights, double eps, uint64_t seed, double* logits);
void oracle_set_num_threads(int n);

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static double urand(void) {  /* splitmix64 in [0, 1) */
  uint64_t z = (rng += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (double)(z >> 11) * 0x1.0p-53;
}

static int fail(const char* what) {
  fprintf(stderr, "FAILED: %s\n", what);
  return 1;
}

int main(void) {
  oracle_set_num_threads(2);
  const int d = 5, T = 3, B = 2;
  const int H = d + 1;
  const int64_t Wd = oracle_det_words(d, T), Wf = oracle_flip_words(d, T);
  uint64_t* det = calloc((size_t)B * Wd, 8);
  const int64_t nbits = (int64_t)T * (d * d - 1);  /* bits per sample; the rest of the last word is padding */
  for (int s = 0; s < B; ++s)
    for (int64_t b = 0; b < nbits; ++b)
      if (urand() < 0.1) det[s * Wd + (b >> 6)] |= 1ull << (b & 63);
  /* geometry */
  int* site_of = malloc(sizeof(int) * (d * d - 1));
  int* index_of = malloc(sizeof(int) * H * H);
  oracle_stabilizer_order(d, site_of, index_of);
  int rc[8];
  for (int i = 0; i < H; ++i)
    for (int j = 0; j < H; ++j) {
      int r, c;
      (void)oracle_site_kind(d, i, j);
      (void)oracle_plaquette_support(d, i, j, rc);
      if (i < d && j < d) (void)oracle_stabilizer_qubit(d, i, j, &r, &c);
    }
  /* unpack, both layouts */
  double* pl = malloc(sizeof(double) * B * 2 * T * H * H);
  oracle_unpack(d, T, B, det, pl);
  double* pp = malloc(sizeof(double) * B * 4 * T * d * d);
  for (int first = 0; first < 3; ++first)
    for (int last = 0; last < 3; ++last) oracle_unpack_paper(d, T, B, det, first, last, pp);
  /* scalars */
  for (int k = 0; k < 1000; ++k) {
    const float x = (float)((urand() - 0.5) * 1000.0);
    (void)oracle_round_bf16(x);
    const int code = oracle_e4m3_code(x / 4);
    (void)oracle_e4m3_value(code);
    (void)oracle_gelu_tanh(x / 50);
  }
  for (int c = 0; c < 256; ++c) (void)oracle_e4m3_value(c);
  (void)oracle_e4m3_scale_exp(0.0);
  (void)oracle_e4m3_scale_exp(1000.0);
  /* forward: two layers of 3x3x3 (k = 3) and a 1x1x1 head, and a k = 5 net */
  const int spec[12] = {2, 8, 3, 1, 8, 8, 3, 2, 8, 4, 1, 0};
  const int64_t nw = oracle_weight_count(3, spec);
  float* w = malloc(sizeof(float) * nw);
  for (int64_t e = 0; e < nw; ++e) w[e] = (float)((urand() - 0.5) * 0.5);
  double* lg[3];
  for (int p = 0; p < 3; ++p) {
    lg[p] = malloc(sizeof(double) * B * 4 * T * H * H);
    oracle_forward(d, T, B, pl, 3, spec, w, p, lg[p]);
  }
  double* lq = malloc(sizeof(double) * B * 4 * T * H * H);
  oracle_forward_grid_fp8_perturbed(H, T, B, pl, 3, spec, w, 1e-3, 7, lq);
  for (int64_t e = 0; e < (int64_t)B * 4 * T * H * H; ++e) {
    if (!isfinite(lg[0][e]) || !isfinite(lq[e])) return fail("finite logits");
    if (fabs(lg[1][e] - lg[0][e]) > 0.1 * (1.0 + fabs(lg[0][e]))) return fail("bf16 forward near exact");
    if (fabs(lg[2][e] - lg[0][e]) > 0.5 * (1.0 + fabs(lg[0][e]))) return fail("fp8 forward near exact");
  }
  const int spec5[12] = {4, 8, 5, 1, 8, 8, 5, 1, 8, 4, 5, 0};
  const int64_t nw5 = oracle_weight_count(3, spec5);
  float* w5 = malloc(sizeof(float) * nw5);
  for (int64_t e = 0; e < nw5; ++e) w5[e] = (float)((urand() - 0.5) * 0.2);
  double* l5 = malloc(sizeof(double) * B * 4 * T * d * d);
  oracle_forward_grid(d, T, B, pp, 3, spec5, w5, 1, l5);
  /* conv sums, k = 1, 3, 5, both accumulations */
  const int ci = 3, co = 2;
  double* x = malloc(sizeof(double) * B * ci * T * H * H);
  for (int64_t e = 0; e < (int64_t)B * ci * T * H * H; ++e) x[e] = urand() - 0.5;
  double* cw = malloc(sizeof(double) * co * ci * 125);
  for (int e = 0; e < co * ci * 125; ++e) cw[e] = urand() - 0.5;
  double cb[2] = {0.25, -0.5};
  double* y = malloc(sizeof(double) * B * co * T * H * H);
  for (int k = 1; k <= 5; k += 2)
    for (int a = 0; a < 2; ++a) oracle_conv_sums(H, T, B, x, ci, co, k, cw, cb, y, a);
  /* flips and residual: zero logits keep the residual equal to the detectors */
  uint64_t* fl = malloc(8 * B * Wf);
  uint64_t* rs = malloc(8 * B * Wd);
  double* zero = calloc((size_t)B * 4 * T * H * H, sizeof(double));
  oracle_flips_residual(d, T, B, zero, det, fl, rs);
  if (memcmp(rs, det, 8 * B * Wd) != 0) return fail("zero flips keep the detectors");
  oracle_flips_residual(d, T, B, lg[0], det, fl, rs);
  oracle_residual_from_flips(d, T, B, det, fl, rs);
  oracle_flips_residual_paper(d, T, B, l5, det, fl, rs);
  /* residual network: two blocks with a projection and an identity shortcut */
  const int rspec[8] = {4, 8, 8, 1, 8, 8, 4, 0};
  const int64_t rn = oracle_resnet_weight_count(2, rspec, 4);
  float* rw = malloc(sizeof(float) * rn);
  for (int64_t e = 0; e < rn; ++e) rw[e] = (float)(0.5 + 0.4 * (urand() - 0.5));
  double* rl = malloc(sizeof(double) * B * 4 * T * d * d);
  for (int p = 0; p < 4; ++p) oracle_forward_resnet(d, T, B, pp, 2, rspec, rw, p, rl);
  oracle_forward_resnet_fp8_perturbed(d, T, B, pp, 2, rspec, rw, 1e-4, 3, rl);
  (void)oracle_resnet_weight_count(2, rspec, 2);
  free(det); free(site_of); free(index_of); free(pl); free(pp); free(w);
  for (int p = 0; p < 3; ++p) free(lg[p]);
  free(lq); free(w5); free(l5); free(x); free(cw); free(y); free(fl); free(rs); free(zero); free(rw); free(rl);
  printf("ok\n");
  return 0;
}
