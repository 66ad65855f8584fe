// api.hip -- host side of the C ABI declared in include/predecoder.h.
//
// create: validates the arguments on the host (no device call before that),
// builds the GPU-side geometry tables, plans the conv tiling, reorders the
// weights into MFMA fragment order (rounding to bf16 with round-to-nearest-
// even for the bf16 path), allocates the zero-halo activation buffers for
// max_batch samples and clears them once.
// run: enqueues unpack -> conv layers -> head -> residual/repack on the
// caller's stream and returns; it never synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/predecoder.h"
#include "internal.h"

using pd::Geom;
using pd::Tiling;

namespace {

constexpr size_t kSchedWords = 256;  // the hidden kernel's unit counters: 8 XCDs x 2 x 16 words

// Device memory one run works in besides its inputs, outputs, weights and
// tables: the input planes, the activation buffers, the projection outputs of
// residual blocks, the flip nibbles, the parked sums of split K loops and the
// hidden kernel's unit counters.
// A handle owns one (sized for max_batch at create); predecoder_run_static
// lays one over the library's static scratch array for each call.
struct Workspace {
  void* planes = nullptr;                      // [batch * S][c_in], zero halo
  void* act[3] = {nullptr, nullptr, nullptr};  // activations [batch * S][cmax]; act[2]: residual networks only
  void* pbuf = nullptr;                        // projection outputs [batch * S][pmax] (residual networks)
  uint8_t* nib = nullptr;                      // [batch][T][H][H] flip nibbles
  float* partial = nullptr;                    // split K loops of small batches: fp32 sums of up to max_units units
  long long max_units = 0;
  uint32_t* sched = nullptr;                   // the hidden kernel's unit counters (kSchedWords, zero between launches)
  size_t act_bytes = 0;                        // size of each activation buffer
  // Row width (bytes per voxel) of the data each activation buffer holds, 0
  // while it is all zero.  The 3x3x3 kernels read the zero halo around the
  // interior voxels; a buffer written with one row width and then with
  // another would show the old interior rows as halo, so it is zeroed first
  // (prepare_rows).
  int act_row[3] = {0, 0, 0};
};

}  // namespace

struct pd_predecoder {
  Geom g;                        // includes the layout and the boundary bases
  int dtype = 0;
  int max_batch = 0;
  int device = 0;
  std::vector<pd_layer> layers;
  int ks = 3;                    // kernel size of the conv layers: 3, or 5 (Model 3 of Table models)
  Tiling tiling{};               // shared by every k x k x k layer (bf16 and fp8 paths)
  Workspace ws;                  // sized for max_batch
  int32_t* tables = nullptr;
  std::vector<void*> wdev;       // per conv layer: fragments (bf16) or [tap][ci][co] (fp32)
  std::vector<size_t> wslice;    // per conv layer: bytes of the fragments of one 128-channel slice of a
                                 // 256-wide layer (run as two slices), 0 otherwise
  std::vector<float*> bdev;      // per conv layer: bias fp32 (a 3x3x3 output layer: [4] biases, [4] scales)
  // per conv layer of 64 to 256 input and output channels run by the hidden
  // kernel (else null): its fragments and biases (fp8: and scales) as slices
  // of 32 output channels, and (128 or 256 output channels) as slices of 64,
  // for small batches (more workgroups per layer)
  std::vector<void*> wnarrow, whalf;
  std::vector<float*> bnarrow, bhalf;
  float* head_w = nullptr;       // [4][c_in] fp32 (bf16-valued on the bf16 path)
  float* head_b = nullptr;       // [4]
  // residual network (predecoder_create_resnet): its blocks; wdev / wslice /
  // bdev hold conv1 and conv2 of block k at 2k and 2k + 1 (BatchNorm folded
  // in), proj_w / proj_b its projection (null for an identity shortcut)
  std::vector<pd_block> blocks;
  std::vector<float*> proj_w, proj_b;
  void* out_proj_frag = nullptr;  // the last block's projection as fragments of launch_conv_out (when it
                                  // runs there, fused into the output conv), else null
  float* out_proj_bias = nullptr; // ... its [4] biases and [4] weight scales
  int cmax = 0;                  // widest activation row (channels)
  int pmax = 0;                  // widest projection output (channels; residual networks)
  int n_cu = 256;                // compute units: one persistent conv workgroup each
};

// One recorded predecoder_run (predecoder_graph_create).
struct pd_graph {
  hipStream_t stream = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

namespace {

const int kMaxD = 63;
const int kMaxT = 1023;

bool layer_chain_ok(const pd_layer* l, int n, int layout) {
  if (n < 1) return false;
  if (l[0].c_in != (layout == PD_LAYOUT_PAPER ? 4 : 2)) return false;
  if (l[n - 1].c_out != 4) return false;
  if (l[n - 1].act != PD_ACT_NONE) return false;
  for (int i = 0; i < n; ++i) {
    if (l[i].c_in < 1 || l[i].c_out < 1) return false;
    if (l[i].k < 1 || (l[i].k % 2) == 0) return false;
    if (l[i].act < PD_ACT_NONE || l[i].act > PD_ACT_RELU) return false;
    if (i > 0 && l[i].c_in != l[i - 1].c_out) return false;
  }
  return true;
}

Geom make_geom(int d, int T, int layout = PD_LAYOUT_PLAQUETTE, int first = PD_BOUNDARY_NONE,
               int last = PD_BOUNDARY_NONE, int pad = 1) {
  Geom g;
  g.d = d;
  g.T = T;
  g.layout = layout;
  g.first = first;
  g.last = last;
  g.pad = pad;
  g.H = layout == PD_LAYOUT_PAPER ? d : d + 1;  // the data qubits, or the plaquettes
  g.Wp = g.H + 2 * pad;
  g.P = g.Wp * g.Wp;
  g.S = (long long)(T + 2 * pad) * g.P;
  g.V = T * g.H * g.H;
  g.nstab = d * d - 1;
  g.K = g.nstab / 2;
  g.nflip = 3 * d * d - 1;
  g.Wd = ((long long)T * g.nstab + 63) / 64;
  g.Wf = ((long long)T * g.nflip + 63) / 64;
  return g;
}

// GPU-side geometry tables (see internal.h).  Plaquette (i, j), 0 <= i, j <=
// d, holds an X stabilizer iff (i+j) is even and 1 <= i <= d-1, a Z
// stabilizer iff (i+j) is odd and 1 <= j <= d-1, and acts on the data qubits
// (i-1..i, j-1..j) inside [0, d-1]^2.  In the paper's layout (Sec. IV.B.1,
// Fig. StabMap) a stabilizer's events enter, and its measurement flip is read,
// at one qubit of its support: a weight-four X (Z) stabilizer at its top-left
// (top-right) qubit, a weight-two X stabilizer (on the left / right edge) at
// its upper qubit, a weight-two Z stabilizer (top / bottom edge) at its right
// qubit.
std::vector<int32_t> build_tables(const Geom& g) {
  std::vector<int32_t> t(pd::tables_size(g), -1);
  int32_t* site_of = t.data() + pd::tables_site_of(g);
  int32_t* comp_x = t.data() + pd::tables_comp_x(g);
  int32_t* comp_z = t.data() + pd::tables_comp_z(g);
  int32_t* supp = t.data() + pd::tables_supp(g);
  const int d = g.d, H = g.H;
  const bool paper = g.layout == PD_LAYOUT_PAPER;
  int n = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (int i = 0; i <= d; ++i)
      for (int j = 0; j <= d; ++j) {
        const bool x = ((i + j) & 1) == 0 && i >= 1 && i <= d - 1;
        const bool z = ((i + j) & 1) == 1 && j >= 1 && j <= d - 1;
        if (!((pass == 0 && x) || (pass == 1 && z))) continue;
        int q = 0;
        for (int r = i - 1; r <= i; ++r)
          for (int c = j - 1; c <= j; ++c)
            if (r >= 0 && r < d && c >= 0 && c < d) supp[n * 4 + q++] = r * H + c;
        int site = i * H + j;
        if (paper) {
          if (x)  // top-left of four; upper qubit of an edge pair (column 0 or d-1)
            site = (i - 1) * H + (j == 0 ? 0 : (j == d ? d - 1 : j - 1));
          else  // top-right of four; right qubit of an edge pair (row 0 or d-1)
            site = (i == 0 ? 0 : (i == d ? d - 1 : i - 1)) * H + j;
        }
        site_of[n] = site;
        (x ? comp_x : comp_z)[site] = n;
        ++n;
      }
  // residual stencils and flip-row sites (grid indices < 2^16: H <= 64)
  int32_t* sten = t.data() + pd::tables_sten(g);
  for (int k = 0; k < g.nstab; ++k) {
    const int32_t* q = supp + 4 * k;
    const int q2 = q[2] >= 0 ? q[2] : q[0], q3 = q[3] >= 0 ? q[3] : q[0];  // weight two: q2 = q3 cancel
    sten[4 * k] = site_of[k] | ((k < g.K ? 2 : 3) << 16);
    sten[4 * k + 1] = q[0] | (q[1] << 16);
    sten[4 * k + 2] = q2 | (q3 << 16);
    sten[4 * k + 3] = 0;
  }
  int32_t* fsite = t.data() + pd::tables_fsite(g);
  for (int k = 0; k < g.nflip; ++k) {
    const int dd = d * d;
    if (k < 2 * dd) {
      const int r = (k % dd) / d, c = (k % dd) % d;
      fsite[k] = (r * H + c) | ((k < dd ? 0 : 1) << 16);
    } else {
      const int m = k - 2 * dd;
      fsite[k] = site_of[m] | ((m < g.K ? 2 : 3) << 16);
    }
  }
  return t;
}

// fp32 -> bf16 bits, round to nearest even on the fp32 bit pattern.
uint16_t bf16_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
float bf16_value(float f) {
  uint32_t u = (uint32_t)bf16_bits(f) << 16;
  float r;
  std::memcpy(&r, &u, 4);
  return r;
}

// Tiling plan for the 3x3x3 layers: the candidate with the fewest MFMA rows
// per sample whose double-buffered 32-channel staging fits in LDS (cost 2 x
// rows; ties go to per-sample tiles, then boxes of 16-voxel rows, then the
// smaller span).

long long flat_span(const Geom& g, long long seg_len, long long nseg, int batch) {
  // exact maximum staged span (line space, see pd::Tiling) over all tiles of
  // `batch` samples
  long long best = 0, halo = pd::line_plane(g) + g.H + 1;
  long long tiles = (seg_len + pd::kTileRows - 1) / pd::kTileRows;
  for (long long s = 0; s < nseg; ++s)
    for (long long k = 0; k < tiles; ++k) {
      long long u0 = s * seg_len + k * pd::kTileRows;
      long long u1 = std::min(u0 + pd::kTileRows, std::min((s + 1) * seg_len, (long long)batch * g.V)) - 1;
      if (u1 < u0) continue;
      auto lidx = [&](long long u) {
        long long b = u / g.V, v = u % g.V;
        int HH = g.H * g.H;
        int t = (int)(v / HH), r = (int)(v % HH);
        return pd::line_index(g, (int)b, t, r / g.H, r % g.H);
      };
      best = std::max(best, lidx(u1) - lidx(u0) + 2 * halo + 1);
    }
  return best;
}

Tiling plan_tiling(const Geom& g, int max_batch, int ks = 3) {
  // 5x5x5 layers: their own (larger) staging buffers, box tiles on a halo of two
  const int kMaxSpan = ks == 3 ? std::min(pd::conv_single_max_span(), pd::conv_hidden_max_span(3))
                               : pd::conv_hidden_max_span(5);
  const int p = g.pad;
  Tiling best{};
  long long best_rows = -1;
  int best_span = 0;
  auto consider = [&](const Tiling& t, long long rows_per_sample) {
    if (t.span > kMaxSpan) return;
    if (best_rows < 0 || rows_per_sample < best_rows ||
        (rows_per_sample == best_rows && t.span < best_span)) {
      best = t;
      best_rows = rows_per_sample;
      best_span = t.span;
    }
  };
  // flat, tiles inside one sample (a halo of one only)
  if (p == 1) {
    Tiling t{};
    t.mode = 0;
    t.seg_len = g.V;
    t.tiles_per_seg = (g.V + pd::kTileRows - 1) / pd::kTileRows;
    t.sa = pd::line_plane(g);
    t.sb = g.H;
    t.span = (int)std::min<long long>(flat_span(g, g.V, 1, 1), 1 << 30);
    consider(t, 2ll * t.tiles_per_seg * pd::kTileRows);
  }
  // flat across samples (rows per sample ~ V); the span bound covers any batch
  if (max_batch > 1 && p == 1) {
    Tiling t{};
    t.mode = 0;
    t.seg_len = -1;  // set per run to batch * V
    t.tiles_per_seg = 0;
    t.sa = pd::line_plane(g);
    t.sb = g.H;
    int nb = std::min(max_batch, 256);
    t.span = (int)std::min<long long>(flat_span(g, (long long)nb * g.V, 1, nb), 1 << 30);
    consider(t, 2ll * g.V + 2);  // +2: prefer per-sample tiles at equal cost
  }
  // boxes
  for (int BJ = 1; BJ <= std::min(g.H, 256); ++BJ)
    for (int BI = 1; BI <= std::min(g.H, 256 / BJ); ++BI) {
      int BT = std::min(g.T, 256 / (BI * BJ));
      if (BT < 1) continue;
      Tiling t{};
      t.mode = 1;
      t.BT = BT;
      t.BI = BI;
      t.BJ = BJ;
      t.ntT = (g.T + BT - 1) / BT;
      t.ntI = (g.H + BI - 1) / BI;
      t.ntJ = (g.H + BJ - 1) / BJ;
      t.sa = (BI + 2 * p) * (BJ + 2 * p);
      t.sb = BJ + 2 * p;
      t.span = (BT + 2 * p) * (BI + 2 * p) * (BJ + 2 * p);
      // (a box row of BJ < 16 voxels, whose 16-lane LDS reads span two staged
      // lines, costs little: at d = T = 25 a 5x3x16 box and a 9x13x2 box
      // reach 0.54 and 0.53 of peak per MFMA row, so the row count decides,
      // and BJ = 16 only breaks ties)
      const long long rows = (long long)t.ntT * t.ntI * t.ntJ * pd::kTileRows;
      consider(t, 2 * rows + (BJ % 16 != 0));
    }
  return best;
}

void tiling_for_batch(Tiling* t, const Geom& g, int batch) {
  t->div_a = pd::make_fastdiv((uint32_t)t->sa);
  t->div_b = pd::make_fastdiv((uint32_t)t->sb);
  t->dv_V = pd::make_fastdiv((uint32_t)g.V);
  t->dv_HH = pd::make_fastdiv((uint32_t)(g.H * g.H));
  t->dv_H = pd::make_fastdiv((uint32_t)g.H);
  if (t->mode == 1) {
    t->dv_per = pd::make_fastdiv((uint32_t)(t->ntT * t->ntI * t->ntJ));
    t->dv_ntij = pd::make_fastdiv((uint32_t)(t->ntI * t->ntJ));
    t->dv_ntj = pd::make_fastdiv((uint32_t)t->ntJ);
    t->dv_bij = pd::make_fastdiv((uint32_t)(t->BI * t->BJ));
    t->dv_bj = pd::make_fastdiv((uint32_t)t->BJ);
  }
  if (t->mode == 0) {
    if (t->seg_len < 0 || t->tiles_per_seg == 0) {
      // flat across samples
      t->seg_len = (long long)batch * g.V;
      t->tiles_per_seg = (int)((t->seg_len + pd::kTileRows - 1) / pd::kTileRows);
      t->ntiles = t->tiles_per_seg;
    } else {
      t->ntiles = (long long)batch * t->tiles_per_seg;
    }
    t->dv_tps = pd::make_fastdiv((uint32_t)t->tiles_per_seg);
  } else {
    t->ntiles = (long long)batch * t->ntT * t->ntI * t->ntJ;
  }
}

// Kernel size of a network's conv layers: 5 when its first layer is 5x5x5
// (Model 3 of Table models), else 3.
int network_ks(const pd_layer* l) { return l[0].k == 5 ? 5 : 3; }

bool supported(const Geom& g, const pd_layer* l, int n, int dtype) {
  if (g.d > kMaxD || g.T > kMaxT) return false;
  if (n < 2) return false;  // at least one hidden 3x3x3 layer before the head
  if (network_ks(l) == 5) {
    // 5x5x5 networks (Model 3 of Table models): the paper layout, bf16, every
    // layer 5x5x5 (the output layer too), one hidden width, 64 or 128
    if (g.layout != PD_LAYOUT_PAPER || dtype != PD_DTYPE_BF16 || n < 3) return false;
    const int w = l[0].c_out;
    if (w != 64 && w != 128) return false;
    for (int i = 0; i < n; ++i) {
      if (l[i].k != 5) return false;
      if (i < n - 1 && l[i].c_out != w) return false;
    }
    return true;
  }
  if (g.layout == PD_LAYOUT_PAPER && dtype == PD_DTYPE_FP32) return false;
  const bool mfma = dtype != PD_DTYPE_FP32;
  // fp8 with a 1x1x1 head needs its head fused into a hidden layer after the
  // first (a lone hidden layer carrying the head runs in bf16 only)
  if (dtype == PD_DTYPE_FP8 && l[n - 1].k == 1 && n < 3) return false;
  bool wide = false;
  for (int i = 0; i < n - 1; ++i) {
    if (l[i].k != 3) return false;
    int co = l[i].c_out;
    if (mfma) {
      if (co != 64 && co != 128 && co != 256) return false;
      wide = wide || co == 256;
    } else {
      if (co % 8 != 0 || co > 128) return false;
    }
  }
  const pd_layer& out = l[n - 1];
  // 256-wide layers run as two 128-channel slices; a 1x1x1 head needs all
  // channels of its input in one workgroup, so they go with a 3x3x3 output layer
  if (wide && out.k != 3) return false;
  if (out.k == 3) return g.layout == PD_LAYOUT_PAPER;  // a 3x3x3 output layer (c_in 64 or 128, checked above)
  if (out.k != 1 || out.c_in > 128) return false;
  if (mfma && (out.c_in % 8) != 0) return false;
  return true;
}

// OCP E4M3 (fp8 path): the code of v, rounded to nearest with ties to even,
// magnitudes of 448 and above saturating to 448 (code 0x7e); NaN is never
// passed (weights are finite).
uint8_t e4m3_code(float v) {
  const uint8_t sgn = std::signbit(v) ? 0x80 : 0;
  const double a = std::fabs((double)v);
  if (a >= 448.0) return sgn | 0x7e;
  int ex;
  std::frexp(a, &ex);  // a = f 2^ex, f in [0.5, 1)
  if (a == 0.0 || ex - 1 < -6) {  // subnormal range: multiples of 2^-9
    const int q = (int)std::nearbyint(std::ldexp(a, 9));  // 8 becomes the smallest normal, code 0x08
    return sgn | (uint8_t)q;
  }
  int e = ex - 1;  // a = m 2^e, m in [1, 2)
  int m = (int)std::nearbyint((std::ldexp(a, -e) - 1.0) * 8.0);
  if (m == 8) {
    m = 0;
    ++e;
  }
  const int code = ((e + 7) << 3) | m;
  return sgn | (uint8_t)std::min(code, 0x7e);
}

float e4m3_value(uint8_t c) {
  const int ex = (c >> 3) & 15, m = c & 7;
  const double v = ex == 0 ? std::ldexp((double)m, -9) : std::ldexp(1.0 + m / 8.0, ex - 7);
  return (float)((c & 0x80) ? -v : v);
}

// Power-of-two scale exponent of a weight row: the smallest e with
// amax / 2^e <= 448 (0 for an all-zero row).
int e4m3_scale_exp(float amax) {
  if (amax == 0.0f) return 0;
  int ex;
  std::frexp((double)amax / 448.0, &ex);  // amax / 448 = f 2^ex, f in [0.5, 1)
  // 2^(ex-1) <= amax / 448 < 2^ex: e = ex, or ex - 1 when amax / 448 is exactly 2^(ex-1)
  return std::ldexp((double)amax, -(ex - 1)) <= 448.0 ? ex - 1 : ex;
}

// Weights of a layer in fp8: per output channel, codes e4m3(w / 2^e) and the
// scale 2^e; wq receives the values the codes stand for (e4m3 value x 2^e).
void quantize_e4m3(const float* w, int cout, size_t row, std::vector<uint8_t>* codes, std::vector<float>* scale,
                   std::vector<float>* wq) {
  codes->assign((size_t)cout * row, 0);
  scale->assign(cout, 1.0f);
  wq->assign((size_t)cout * row, 0.0f);
  for (int co = 0; co < cout; ++co) {
    float amax = 0.0f;
    for (size_t e = 0; e < row; ++e) amax = std::max(amax, std::fabs(w[co * row + e]));
    const int ex = e4m3_scale_exp(amax);
    (*scale)[co] = std::ldexp(1.0f, ex);
    for (size_t e = 0; e < row; ++e) {
      const uint8_t c = e4m3_code(std::ldexp(w[co * row + e], -ex));
      (*codes)[co * row + e] = c;
      (*wq)[co * row + e] = std::ldexp(e4m3_value(c), ex);
    }
  }
}

template <typename T>
pd_status dev_alloc(T** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc((void**)p, bytes);
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) {
    (void)hipGetLastError();
    return PD_ERR_OUT_OF_MEMORY;
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return PD_ERR_DEVICE;
  }
  return PD_OK;
}

template <typename T>
pd_status upload(T** p, const void* host, size_t bytes) {
  pd_status s = dev_alloc(p, bytes);
  if (s != PD_OK) return s;
  if (hipMemcpy(*p, host, bytes, hipMemcpyHostToDevice) != hipSuccess) return PD_ERR_DEVICE;
  return PD_OK;
}

void free_all(pd_predecoder* h) {
  auto f = [](void* p) {
    if (p) (void)hipFree(p);
  };
  f(h->ws.planes);
  f(h->ws.act[0]);
  f(h->ws.act[1]);
  f(h->ws.act[2]);
  f(h->ws.pbuf);
  for (float* p : h->proj_w) f(p);
  for (float* p : h->proj_b) f(p);
  f(h->out_proj_frag);
  f(h->out_proj_bias);
  h->out_proj_frag = nullptr;
  h->out_proj_bias = nullptr;
  h->ws.act[2] = h->ws.pbuf = nullptr;
  h->proj_w.clear();
  h->proj_b.clear();
  f(h->ws.nib);
  f(h->tables);
  for (void* p : h->wdev) f(p);
  for (float* p : h->bdev) f(p);
  for (void* p : h->wnarrow) f(p);
  for (float* p : h->bnarrow) f(p);
  for (void* p : h->whalf) f(p);
  for (float* p : h->bhalf) f(p);
  f(h->head_w);
  f(h->head_b);
  f(h->ws.partial);
  f(h->ws.sched);
  h->ws.planes = h->ws.act[0] = h->ws.act[1] = nullptr;
  h->ws.nib = nullptr;
  h->tables = nullptr;
  h->wdev.clear();
  h->wslice.clear();
  h->bdev.clear();
  h->wnarrow.clear();
  h->bnarrow.clear();
  h->whalf.clear();
  h->bhalf.clear();
  h->head_w = h->head_b = nullptr;
  h->ws.partial = nullptr;
  h->ws.sched = nullptr;
}

// bf16 A fragments (weights) for v_mfma_f32_32x32x16_bf16: lane l of
// fragment (k-step, channel block nb) holds W[co = 32 nb + l % 32][k0 + 8 (l / 32) + e],
// e = 0..7; output channels past c_out (the 4 filters of an output layer fill
// one block of 32) are zero.  Layer 1 (c_in = 2 or 4): k = c_in * tap + ci over
// ceil(k^3 c_in / 16) k-steps (taps past the last are zero).  Other layers:
// [chunk of 16 c_in][tap][nb] with ci = 16 chunk + 8 (l / 32) + e.
std::vector<uint16_t> conv_fragments(const float* w, int cin, int cout, int k = 3) {
  const int nbt = cout < 32 ? 1 : cout / 32;
  const int taps = k * k * k;
  std::vector<uint16_t> f;
  auto W = [&](int co, int ci, int tap) -> uint16_t {
    return co < cout ? bf16_bits(w[((size_t)co * cin + ci) * taps + tap]) : 0;
  };
  if (cin == 2 || cin == 4) {
    const int ks_n = (taps * cin + 15) / 16;
    f.assign((size_t)ks_n * nbt * 64 * 8, 0);
    for (int ks = 0; ks < ks_n; ++ks)
      for (int nb = 0; nb < nbt; ++nb)
        for (int l = 0; l < 64; ++l)
          for (int e = 0; e < 8; ++e) {
            int k = ks * 16 + 8 * (l / 32) + e;
            int tap = k / cin, ci = k % cin, co = nb * 32 + l % 32;
            f[(((size_t)ks * nbt + nb) * 64 + l) * 8 + e] = tap < taps ? W(co, ci, tap) : 0;
          }
  } else {
    const int nch = cin / 16;
    f.assign((size_t)nch * taps * nbt * 64 * 8, 0);
    for (int c = 0; c < nch; ++c)
      for (int tap = 0; tap < taps; ++tap)
        for (int nb = 0; nb < nbt; ++nb)
          for (int l = 0; l < 64; ++l)
            for (int e = 0; e < 8; ++e) {
              int ci = c * 16 + 8 * (l / 32) + e, co = nb * 32 + l % 32;
              size_t idx = ((((size_t)c * taps + tap) * nbt + nb) * 64 + l) * 8 + e;
              f[idx] = W(co, ci, tap);
            }
  }
  return f;
}

// fp8 A fragments (weight codes) for v_mfma_f32_32x32x64_f8f6f4: fragment
// (chunk of 32 c_in, k-step s, channel block nb), lane l holds 32 bytes,
// byte e = W[co = 32 nb + l % 32][ci = 32 chunk + e][tap 2 s + l / 32]
// (tap 27: zero); output channels past c_out are zero.
std::vector<uint8_t> conv_fragments_fp8(const uint8_t* codes, int cin, int cout) {
  const int nbt = cout < 32 ? 1 : cout / 32, nch = cin / 32, ns = 14;
  std::vector<uint8_t> f((size_t)nch * ns * nbt * 64 * 32, 0);
  for (int c = 0; c < nch; ++c)
    for (int st = 0; st < ns; ++st)
      for (int nb = 0; nb < nbt; ++nb)
        for (int l = 0; l < 64; ++l)
          for (int e = 0; e < 32; ++e) {
            const int co = nb * 32 + l % 32, ci = c * 32 + e, tap = 2 * st + l / 32;
            if (co < cout && tap < 27)
              f[((((size_t)c * ns + st) * nbt + nb) * 64 + l) * 32 + e] = codes[((size_t)co * cin + ci) * 27 + tap];
          }
  return f;
}

// Fragments of a 3x3x3 output layer of four filters for launch_conv_out:
// fragment (row block rb, k-step st), lane l: row m = l % 32 stands for tap
// 8 rb + m / 4 (zero past the last tap) and filter m % 4; bf16: 8 values,
// ci = 16 st + 8 (l / 32) + e; fp8 (codes): 32 codes, ci = 64 st + 32 (l /
// 32) + e.  Byte layout [rb][st][lane][16 or 32].
std::vector<uint8_t> out_fragments(const float* w, const uint8_t* codes, int cin, bool fp8) {
  const int kstep = fp8 ? 64 : 16, nks = cin / kstep, lb = fp8 ? 32 : 16;
  std::vector<uint8_t> f((size_t)4 * nks * 64 * lb, 0);
  for (int rb = 0; rb < 4; ++rb)
    for (int st = 0; st < nks; ++st)
      for (int l = 0; l < 64; ++l) {
        const int m = l % 32, tap = 8 * rb + m / 4, co = m % 4;
        if (tap >= 27) continue;
        uint8_t* dst = &f[(((size_t)rb * nks + st) * 64 + l) * lb];
        for (int e = 0; e < (fp8 ? 32 : 8); ++e) {
          const int ci = st * kstep + (fp8 ? 32 : 8) * (l / 32) + e;
          const size_t src = ((size_t)co * cin + ci) * 27 + tap;
          if (fp8) {
            dst[e] = codes[src];
          } else {
            const uint16_t v = bf16_bits(w[src]);
            std::memcpy(dst + 2 * e, &v, 2);
          }
        }
      }
  return f;
}

// bf16 fragments of a layer whose outputs run in slices of 128 channels
// when c_out > 128 (slices back to back; *slice = bytes of one slice, 0 when
// there is a single launch).
std::vector<uint16_t> fragments_sliced(const float* w, int cin, int cout, size_t* slice) {
  if (cout <= 128) {
    *slice = 0;
    return conv_fragments(w, cin, cout);
  }
  std::vector<uint16_t> f;
  for (int k = 0; k < cout / 128; ++k) {
    std::vector<uint16_t> fk = conv_fragments(w + (size_t)k * 128 * cin * 27, cin, 128);
    *slice = fk.size() * 2;
    f.insert(f.end(), fk.begin(), fk.end());
  }
  return f;
}

pd_status check_launch(hipError_t e) {
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return PD_ERR_DEVICE;
  }
  return PD_OK;
}

// Before a layer writes rows of row_bytes into activation buffer idx of ws:
// zero the buffer if it holds rows of another width (see act_row).
pd_status prepare_rows(Workspace& ws, int idx, int row_bytes, hipStream_t st) {
  if (ws.act_row[idx] != 0 && ws.act_row[idx] != row_bytes) {
    pd_status s = check_launch(pd::launch_zero(ws.act[idx], ws.act_bytes, st));
    if (s != PD_OK) return s;
  }
  ws.act_row[idx] = row_bytes;
  return PD_OK;
}

// Where a stopped run left the activations it was asked for (see
// enqueue_run's stop argument).
struct StopAt {
  const void* buf = nullptr;
  int row_bytes = 0;
};

// Split of a layer's K loop over 2^k workgroups per tile.  Only small
// batches split (tiles x parts within the workspace's units, one per compute
// unit for a handle's own: past that the parked fp32 sums cost more than the
// shorter loops gain); parts must divide the layer's input-channel chunks.
// Among the splits that fit, the one with the least estimated time of a
// workgroup's unit: its chunks, then either the tile's epilogue (bias,
// activation and stores, done by the tile's single workgroup) or parking the
// fp32 sums plus the second, elementwise kernel that finishes all tiles in
// parallel.  Microseconds per unit on MI355X at batch 1, from per-phase
// timestamps inside the kernel: a 16-channel chunk 2.5 (64 output channels)
// or 3.9 (128); the activation epilogue 3.3 or 7.3; parking 1.75 or 3.4;
// the finishing kernel with its launch about 8.  (For 64 channels at 25^3
// one unsplit launch beats two parts by 3 us; for 128 channels at 13^3 the
// split saves 20 us.)  fp8 chunks are 32 channels with about half a bf16
// chunk's matrix time per channel; a 5x5x5 chunk has 125 taps instead of 27.
// nsl: the layer's output-channel slices of cout channels, all in the one
// launch (each is a unit of its own per tile and part).  unit_us (optional):
// the estimate for an unsplit unit.
pd::Split_k split_for(const Workspace& ws, const Tiling& t, int cin, int cout, int fp8, int ks = 3, int nsl = 1,
                      double* unit_us = nullptr) {
  const int kch = pd::conv_hidden_chunk_channels(fp8);
  const int nch = cin / kch;
  const double wide = cout > 64 ? 1.0 : 0.0;
  const double chunk = (2.5 + 1.4 * wide) * (fp8 ? 1.1 : 1.0) * (ks * ks * ks) / 27.0;
  const double epi = 3.3 + 4.0 * wide, park = 1.75 + 1.65 * wide;
  const double finish = 8.0;
  pd::Split_k sk{0, ws.partial, ws.max_units};
  sk.sched = ws.sched;
  while ((1 << sk.lsl) < nsl) ++sk.lsl;
  double best = nch * chunk + epi;
  if (unit_us) *unit_us = best;
  for (int k = 1; nch % (1 << k) == 0 && (t.ntiles << (k + sk.lsl)) <= ws.max_units; ++k) {
    const double est = (nch >> k) * chunk + park + finish;
    if (est < best) {
      best = est;
      sk.kshift = k;
    }
  }
  return sk;
}

// One hidden-kernel layer over the batch (nsl output-channel slices of cw
// channels; see launch_conv_hidden for the rest).  Usually one launch.  When
// the layer's units (tiles x slices) fill the workgroup slots a few times
// over and leave a short remainder, two: the first samples, whose units fill
// whole rounds, unsplit; then the last few samples (a sub-batch: every
// per-sample pointer moved on by their offset) with their K loops split over
// the otherwise idle chip and finished by the second kernel.  A remainder of
// r units would otherwise take a whole unit's time on r slots (40 of 552
// units at Model 6's 13^3 batch 16 took about a third of the layer); the
// split saves that time but one fraction 2^-k, and costs the parked sums,
// the finishing kernel and one more kernel boundary: about 45 us in all,
// from MI355X timings of splits of 128 to 512 input channels (Models 1, 2
// and 6 at 13^3), so only long units split.  (Model 6 at 13^3 batch 16 in
// bf16: the last 2 of the 16 samples split in two, 5 % less time per round.)
constexpr long long kMaxTailRounds = 4;  // past this, a remainder costs little
constexpr double kTailCostUs = 45.0;

pd_status run_hidden(const pd_predecoder* h, Workspace& ws, const Tiling& tl, int cin, int cw, int nsl, int act,
                     const void* x, void* y, int ystride, const void* wfrag, const float* bias, int head,
                     const float* head_w, const float* head_b, float* logits, int batch, int fp8,
                     const uint16_t* sc, int sc_stride, int ks, hipStream_t st) {
  const Geom& g = h->g;
  const int slots = h->n_cu * pd::conv_hidden_workgroups_per_cu(ks);
  // samples b0 .. b0 + nb - 1 with tiling t and split sk
  auto launch = [&](const Tiling& t, const pd::Split_k& sk, int b0, int nb) {
    const int esz = fp8 ? 1 : 2;                  // bytes per activation value
    const long long pv = (long long)b0 * g.S;     // padded voxels before sample b0
    const uint16_t* scb = !sc ? nullptr
                              : (const uint16_t*)((const char*)sc + pv * sc_stride * (head_w ? 2 : esz));
    return check_launch(pd::launch_conv_hidden(
        g, t, cin, cw, act, (const char*)x + pv * cin * esz, y ? (char*)y + pv * ystride * esz : nullptr, ystride,
        wfrag, bias, head, head_w, head_b, h->tables, ws.nib + (long long)b0 * g.V,
        logits ? logits + (long long)b0 * 4 * g.T * g.H * g.H : nullptr, nb, slots, sk, fp8, scb, sc_stride, ks,
        st));
  };
  const pd::Split_k sk = split_for(ws, tl, cin, cw, fp8, ks, nsl);
  const long long units = tl.ntiles * nsl, q = units / slots, r = units % slots;
  if (sk.kshift == 0 && q >= 1 && q <= kMaxTailRounds && r > 0 && batch > 1) {
    // the most first samples whose tiles fit q full rounds (tiles grow with
    // the batch: per sample, or one flat run of batch x V voxels)
    const Tiling& base = h->tiling;
    const long long fit = q * slots / nsl;  // tiles
    const bool flat = base.mode == 0 && (base.seg_len < 0 || base.tiles_per_seg == 0);
    const long long per = base.mode == 1 ? (long long)base.ntT * base.ntI * base.ntJ : base.tiles_per_seg;
    const long long first = flat ? fit * pd::kTileRows / g.V : fit / per;
    if (first >= 1 && first < batch) {
      const int nb = batch - (int)first;
      Tiling th = base, tt = base;
      tiling_for_batch(&th, g, (int)first);
      tiling_for_batch(&tt, g, nb);
      double unit_us = 0.0;
      const pd::Split_k tsk = split_for(ws, tt, cin, cw, fp8, ks, nsl, &unit_us);
      if (tsk.kshift > 0 && unit_us * (1.0 - 1.0 / (1 << tsk.kshift)) > kTailCostUs) {
        const pd_status s = launch(th, sk, 0, batch - nb);
        return s != PD_OK ? s : launch(tt, tsk, batch - nb, nb);
      }
    }
  }
  return launch(tl, sk, 0, batch);
}

// The path of a residual network (Model 6, Sec. VI, Fig. Model8Representation):
// per block, conv1 (+ folded BatchNorm, activation) x -> hb, the shortcut (x,
// or its 1x1x1 projection into pbuf), conv2 (+ folded BatchNorm) hb -> the
// next x with the shortcut added before the activation; the last block's
// conv2 is the output layer (logits, threshold) with the shortcut added.
// Three activation buffers rotate so that x, hb and the output differ.
// stop >= 0: stop after conv number `stop` of the network (counting, block
// by block, conv1, the projection if the block has one, then conv2; the last
// conv2, the output layer, is not counted) and report its output in *at.
pd_status enqueue_resnet(pd_predecoder* h, Workspace& ws, hipStream_t st, const uint64_t* det, int batch,
                         uint64_t* flips, uint64_t* residual, float* logits, hipEvent_t* ev, int stop, StopAt* at) {
  const Geom& g = h->g;
  const int fp8 = h->dtype == PD_DTYPE_FP8;
  const int ae = fp8 ? 1 : 2;  // bytes per activation value
  int e = 0;
  auto mark = [&]() -> pd_status {
    if (ev && hipEventRecord(ev[e++], st) != hipSuccess) return PD_ERR_DEVICE;
    return PD_OK;
  };
  pd_status s;
  if ((s = mark()) != PD_OK) return s;
  if ((s = check_launch(pd::launch_unpack(g, h->tables, det, batch, ws.planes, 1, 0, st))) != PD_OK) return s;
  Tiling tl = h->tiling;
  tiling_for_batch(&tl, g, batch);
  const void* x = ws.planes;
  int xi = -1;     // index of x in ws.act (-1: the planes)
  int conv = 0;    // convs run so far (the numbering of `stop`)
  auto stopped = [&](const void* buf, int row_bytes) {
    if (conv++ != stop) return false;
    at->buf = buf;
    at->row_bytes = row_bytes;
    return true;
  };
  const int nb = (int)h->blocks.size();
  for (int k = 0; k < nb; ++k) {
    if ((s = mark()) != PD_OK) return s;
    const pd_block& B = h->blocks[k];
    const bool last = k == nb - 1;
    const int hi = (xi + 1) % 3, yi = (xi + 2 + (xi < 0 ? 1 : 0)) % 3;
    void* hb = ws.act[hi];
    void* yb = ws.act[yi];
    if ((s = prepare_rows(ws, hi, B.c_mid * ae, st)) != PD_OK) return s;
    if (!last && (s = prepare_rows(ws, yi, B.c_out * ae, st)) != PD_OK) return s;
    // conv1: x -> hb (a layer wider than 128 channels: slices of 128 output
    // channels, each with its fragments, biases (fp8: and scales) and output
    // columns; the hidden kernel runs all of them in one launch)
    {
      const int nsl = B.c_mid > 128 ? B.c_mid / 128 : 1, cw = B.c_mid / nsl;
      if (k == 0) {
        for (int q = 0; q < nsl && s == PD_OK; ++q) {
          const void* wq = (const char*)h->wdev[2 * k] + q * h->wslice[2 * k];
          void* yq = (char*)hb + (size_t)q * cw * ae;
          // layer 1 (fp8: bf16 matrix work on the dequantised weights, E4M3 output)
          s = check_launch(pd::launch_conv_first(g, B.c_in, cw, B.act, x, yq, B.c_mid, wq, h->bdev[2 * k] + q * cw,
                                                 batch, fp8, 3, st));
        }
      } else {
        s = run_hidden(h, ws, tl, B.c_in, cw, nsl, B.act, x, hb, B.c_mid, h->wdev[2 * k], h->bdev[2 * k], 0, nullptr,
                       nullptr, nullptr, batch, fp8, nullptr, 0, 3, st);
      }
      if (s != PD_OK) return s;
      if (stopped(hb, B.c_mid * ae)) return PD_OK;
    }
    // shortcut: the block input, or its 1x1x1 projection -- computed by the
    // epilogue of conv2 from an input of a few channels (the first block)
    // or by the output conv (the last block, its fragments built at create),
    // else by its own kernel (bf16), which also serves a caller that stops
    // at the projection
    const uint16_t* sc = (const uint16_t*)x;
    int sc_stride = B.c_in;
    const float* pw = nullptr;  // set: conv2 projects sc itself
    const float* pb = nullptr;
    if (h->proj_w[k]) {
      const bool fuse = (last ? h->out_proj_frag != nullptr : B.c_in <= 8) && stop != conv;
      if (fuse) {
        pw = h->proj_w[k];
        pb = h->proj_b[k];
        ++conv;  // the projection's stop number
      } else {
        if (fp8) return PD_ERR_UNSUPPORTED;  // no stored fp8 projection
        s = check_launch(pd::launch_proj(g, x, B.c_in, B.c_in, h->proj_w[k], h->proj_b[k], B.c_out, ws.pbuf,
                                         B.c_out, batch, st));
        if (s != PD_OK) return s;
        sc = (const uint16_t*)ws.pbuf;
        sc_stride = B.c_out;
        if (stopped(ws.pbuf, B.c_out * 2)) return PD_OK;
      }
    }
    // conv2: hb -> the next x (or the logits) with the shortcut added
    if (last && pw) {  // the projection fused into the output conv
      s = check_launch(pd::launch_conv_out(g, B.c_mid, hb, h->wdev[2 * k + 1], h->bdev[2 * k + 1], h->tables,
                                           ws.nib, logits, batch, h->n_cu, fp8, nullptr, 0, x, h->out_proj_frag,
                                           h->out_proj_bias, st));
    } else if (last) {
      s = check_launch(pd::launch_conv_out(g, B.c_mid, hb, h->wdev[2 * k + 1], h->bdev[2 * k + 1], h->tables,
                                           ws.nib, logits, batch, h->n_cu, fp8, sc, sc_stride, nullptr, nullptr,
                                           nullptr, st));
    } else {  // slices as for conv1, each also with its shortcut channels (or projection rows)
      const int nsl = B.c_out > 128 ? B.c_out / 128 : 1, cw = B.c_out / nsl;
      s = run_hidden(h, ws, tl, B.c_mid, cw, nsl, B.act, hb, yb, B.c_out, h->wdev[2 * k + 1], h->bdev[2 * k + 1], 4,
                     pw, pb, nullptr, batch, fp8, sc, sc_stride, 3, st);
    }
    if (s != PD_OK) return s;
    if (!last && stopped(yb, B.c_out * ae)) return PD_OK;
    x = yb;
    xi = yi;
  }
  if (stop >= 0) return PD_ERR_INVALID_ARG;  // no such conv
  if ((s = mark()) != PD_OK) return s;
  if ((s = check_launch(pd::launch_residual_pack(g, h->tables, det, ws.nib, flips, residual, batch, st))) != PD_OK)
    return s;
  return mark();
}

// Enqueues the whole path in workspace ws.  ev (optional) receives one event
// record before each stage and one after the last.  stop >= 0: stop after
// that hidden layer (residual networks: that conv, see enqueue_resnet), whose
// output activations are then written (no head fused into it) and reported
// in *at.
pd_status enqueue_run(pd_predecoder* h, Workspace& ws, hipStream_t st, const uint64_t* det, int batch,
                      uint64_t* flips, uint64_t* residual, float* logits, hipEvent_t* ev, int stop = -1,
                      StopAt* at = nullptr) {
  if (!h->blocks.empty()) return enqueue_resnet(h, ws, st, det, batch, flips, residual, logits, ev, stop, at);
  const Geom& g = h->g;
  const int fp32 = h->dtype == PD_DTYPE_FP32;
  const int fp8 = h->dtype == PD_DTYPE_FP8;
  const int aelem = fp8 ? 1 : 2;  // bytes per activation value (MFMA paths)
  const int n = (int)h->layers.size();
  // the last layer: a 1x1x1 head (fused into the last hidden layer's
  // epilogue on the MFMA paths) or a 3x3x3 (5x5x5) output layer of its own
  const bool out3 = h->layers[n - 1].k > 1;
  const int ks = h->ks;
  int e = 0;
  auto mark = [&]() -> pd_status {
    if (ev && hipEventRecord(ev[e++], st) != hipSuccess) return PD_ERR_DEVICE;
    return PD_OK;
  };
  pd_status s;
  if ((s = mark()) != PD_OK) return s;
  s = check_launch(pd::launch_unpack(g, h->tables, det, batch, ws.planes, 1, fp32, st));
  if (s != PD_OK) return s;
  const void* x = ws.planes;
  Tiling tl = h->tiling;
  if (!fp32) tiling_for_batch(&tl, g, batch);
  bool head_done = false;  // nibbles written by a fused head
  for (int l = 0; l < n - 1; ++l) {
    if ((s = mark()) != PD_OK) return s;
    void* y = ws.act[l & 1];
    const pd_layer& L = h->layers[l];
    const int row_bytes = L.c_out * (fp32 ? 4 : aelem);
    if ((s = prepare_rows(ws, l & 1, row_bytes, st)) != PD_OK) return s;
    const bool head_layer = !fp32 && !out3 && l == n - 2;  // carries the head unless the run stops at it
    const bool fuse_head = head_layer && stop < 0;
    if (fp32) {
      s = check_launch(pd::launch_conv_fp32(g, L.c_in, L.c_out, L.act, (const float*)x, (float*)y,
                                            (const float*)h->wdev[l], h->bdev[l], batch, st));
    } else if (l == 0 && fuse_head && L.c_in == 2) {  // one hidden layer: layer 1 carries the head
      s = check_launch(pd::launch_conv_single(g, tl, L.c_out, L.act, x, h->wdev[l], h->bdev[l], h->head_w,
                                              h->head_b, h->tables, ws.nib, logits, batch, h->n_cu, st));
      head_done = true;
    } else {
      // a 256-wide layer runs as two slices of 128 output channels over the
      // same input (slice k: its fragments, biases (fp8: and scales) and
      // output channels): two launches of layer 1's kernel, one of the
      // hidden kernel
      const int nsl = h->wslice[l] ? 2 : 1, cw = L.c_out / nsl;
      if (l == 0) {
        for (int k = 0; k < nsl && s == PD_OK; ++k) {
          const void* wk = (const char*)h->wdev[l] + k * h->wslice[l];
          void* yk = (char*)y + (size_t)k * cw * aelem;
          s = check_launch(pd::launch_conv_first(g, L.c_in, cw, L.act, x, yk, L.c_out, wk, h->bdev[l] + k * cw,
                                                 batch, fp8, ks, st));
        }
      } else if (l < (int)h->wnarrow.size() && h->wnarrow[l] && tl.ntiles * (L.c_out / 32) <= h->n_cu &&
                 (!head_layer || (L.c_in <= 128 && (tl.ntiles * (L.c_out / 32)) <= ws.max_units &&
                                  split_for(ws, tl, L.c_in, L.c_out, fp8, ks).kshift > 0))) {
        // a small batch: a 64- to 256-wide layer as 32-channel slices, two to
        // eight times the workgroups (still at most one per CU) for the same
        // staging, in place of splitting its K loops (a 256-channel input's
        // long loops may still split).  The layer that carries the head, when
        // unsliced it would split its K loops and finish in a second kernel
        // anyway: its slices park their sums and that kernel finishes whole
        // rows with the head (d = 13, batch 1, 8 x 128: 2.6 % less time per
        // round in bf16, 4 % in fp8; a head layer that runs whole in one
        // launch stays so, the extra kernel costing more: 3 % at d = 25,
        // 6 x 64).  A run that stops at it slices it the same way, so that
        // its exported activations are the ones the head reads.
        s = run_hidden(h, ws, tl, L.c_in, 32, L.c_out / 32, L.act, x, y, L.c_out, h->wnarrow[l], h->bnarrow[l],
                       fuse_head ? 1 : 0, fuse_head ? h->head_w : nullptr, fuse_head ? h->head_b : nullptr, logits,
                       batch, fp8, nullptr, 0, ks, st);
      } else if (l < (int)h->whalf.size() && h->whalf[l] && tl.ntiles * (L.c_out / 64) <= h->n_cu &&
                 (!head_layer || (L.c_in <= 128 && (tl.ntiles * (L.c_out / 64)) <= ws.max_units &&
                                  split_for(ws, tl, L.c_in, L.c_out, fp8, ks).kshift > 0))) {
        // ... or, with too many tiles for that, a 128- or 256-wide one as
        // slices of 64 (the head layer as above)
        s = run_hidden(h, ws, tl, L.c_in, 64, L.c_out / 64, L.act, x, y, L.c_out, h->whalf[l], h->bhalf[l],
                       fuse_head ? 1 : 0, fuse_head ? h->head_w : nullptr, fuse_head ? h->head_b : nullptr, logits,
                       batch, fp8, nullptr, 0, ks, st);
      } else {  // the last hidden layer may carry the head and the threshold in its epilogue
        s = run_hidden(h, ws, tl, L.c_in, cw, nsl, L.act, x, y, L.c_out, h->wdev[l], h->bdev[l], fuse_head ? 1 : 0,
                       h->head_w, h->head_b, logits, batch, fp8, nullptr, 0, ks, st);
      }
      head_done = fuse_head && l > 0;
    }
    if (s != PD_OK) return s;
    if (l == stop) {
      at->buf = y;
      at->row_bytes = row_bytes;
      return PD_OK;
    }
    x = y;
  }
  if (stop >= 0) return PD_ERR_INVALID_ARG;  // no such hidden layer
  if ((s = mark()) != PD_OK) return s;
  if (out3 && h->layers[n - 1].k == 3) {
    const pd_layer& L = h->layers[n - 1];
    s = check_launch(pd::launch_conv_out(g, L.c_in, x, h->wdev[n - 1], h->bdev[n - 1], h->tables, ws.nib, logits,
                                         batch, h->n_cu, fp8, nullptr, 0, nullptr, nullptr, nullptr, st));
  } else if (out3) {
    const pd_layer& L = h->layers[n - 1];
    s = run_hidden(h, ws, tl, L.c_in, L.c_out, 1, L.act, x, nullptr, 0, h->wdev[n - 1], h->bdev[n - 1], 2, nullptr,
                   nullptr, logits, batch, fp8, nullptr, 0, ks, st);
  } else if (!head_done) {  // fp32, or a one-hidden-layer network on the paper's layout
    s = check_launch(pd::launch_head(g, h->layers[n - 1].c_in, fp32, x, h->head_w, h->head_b, h->tables,
                                     ws.nib, logits, batch, st));
  }
  if (s != PD_OK) return s;
  if ((s = mark()) != PD_OK) return s;
  s = check_launch(pd::launch_residual_pack(g, h->tables, det, ws.nib, flips, residual, batch, st));
  if (s != PD_OK) return s;
  return mark();
}

// Number of convs predecoder_activations can stop after: the hidden layers,
// or for a residual network every conv but the output layer (conv1, the
// projection if any, conv2 per block).
int n_stop_points(const pd_predecoder* h) {
  if (h->blocks.empty()) return (int)h->layers.size() - 1;
  int n = 0;
  for (const pd_block& B : h->blocks) n += 2 + (B.c_in != B.c_out ? 1 : 0);
  return n - 1;
}

}  // namespace

extern "C" {

const char* predecoder_status_string(pd_status s) {
  switch (s) {
    case PD_OK: return "ok";
    case PD_ERR_INVALID_ARG: return "invalid argument";
    case PD_ERR_UNSUPPORTED: return "unsupported shape";
    case PD_ERR_OUT_OF_MEMORY: return "out of device memory";
    case PD_ERR_DEVICE: return "device error";
    case PD_ERR_TOO_LARGE: return "batch too large for the library's static scratch array";
  }
  return "unknown status";
}

int64_t predecoder_det_words(int32_t d, int32_t T) {
  if (d < 1 || T < 1) return -1;
  return ((int64_t)T * ((int64_t)d * d - 1) + 63) / 64;
}

int64_t predecoder_flip_words(int32_t d, int32_t T) {
  if (d < 1 || T < 1) return -1;
  return ((int64_t)T * (3 * (int64_t)d * d - 1) + 63) / 64;
}

size_t predecoder_weight_count(const pd_layer* layers, int32_t n_layers) {
  if (!layers || n_layers < 1) return 0;
  size_t n = 0;
  for (int i = 0; i < n_layers; ++i) {
    const pd_layer& l = layers[i];
    if (l.c_in < 1 || l.c_out < 1 || l.k < 1) return 0;
    n += (size_t)l.c_out * l.c_in * l.k * l.k * l.k + l.c_out;
  }
  return n;
}

int32_t predecoder_num_stages(const pd_predecoder* h) {
  if (!h) return -1;
  return (int32_t)(h->blocks.empty() ? h->layers.size() : h->blocks.size()) + 2;
}

pd_status predecoder_create(const float* weights, size_t n_weights, int32_t d, int32_t T,
                            const pd_layer* layers, int32_t n_layers, int32_t dtype, int32_t max_batch,
                            pd_predecoder** out) {
  return predecoder_create_ex(weights, n_weights, d, T, layers, n_layers, dtype, max_batch, nullptr, out);
}

pd_status predecoder_create_ex(const float* weights, size_t n_weights, int32_t d, int32_t T,
                               const pd_layer* layers, int32_t n_layers, int32_t dtype, int32_t max_batch,
                               const pd_options* opts, pd_predecoder** out) {
  if (!out) return PD_ERR_INVALID_ARG;
  *out = nullptr;
  if (!weights || !layers) return PD_ERR_INVALID_ARG;
  if (d < 3 || (d % 2) == 0 || T < 1) return PD_ERR_INVALID_ARG;
  if (dtype != PD_DTYPE_FP32 && dtype != PD_DTYPE_BF16 && dtype != PD_DTYPE_FP8) return PD_ERR_INVALID_ARG;
  if (max_batch < 1) return PD_ERR_INVALID_ARG;
  const pd_options o = opts ? *opts : pd_options{PD_LAYOUT_PLAQUETTE, PD_BOUNDARY_NONE, PD_BOUNDARY_NONE};
  if (o.layout != PD_LAYOUT_PLAQUETTE && o.layout != PD_LAYOUT_PAPER) return PD_ERR_INVALID_ARG;
  if (o.first_round < PD_BOUNDARY_NONE || o.first_round > PD_BOUNDARY_X || o.last_round < PD_BOUNDARY_NONE ||
      o.last_round > PD_BOUNDARY_X)
    return PD_ERR_INVALID_ARG;
  // the plaquette layout has no geometric channels to clear
  if (o.layout == PD_LAYOUT_PLAQUETTE && (o.first_round != PD_BOUNDARY_NONE || o.last_round != PD_BOUNDARY_NONE))
    return PD_ERR_INVALID_ARG;
  if (!layer_chain_ok(layers, n_layers, o.layout)) return PD_ERR_INVALID_ARG;
  if (n_weights != predecoder_weight_count(layers, n_layers)) return PD_ERR_INVALID_ARG;
  const int ks = network_ks(layers);
  // the zero halo holds every tap of a layer: one voxel, two for 5x5x5 layers
  Geom g = make_geom(d, T, o.layout, o.first_round, o.last_round, (ks - 1) / 2);
  if (!supported(g, layers, n_layers, dtype)) return PD_ERR_UNSUPPORTED;
  // kernels index voxels of a batch with 32-bit integers
  if ((long long)max_batch * g.V >= (1ll << 31) || (long long)max_batch * (g.Wd + g.Wf) >= (1ll << 31) ||
      (long long)max_batch * g.S >= (1ll << 31) ||
      (long long)max_batch * (T + 2) * pd::line_plane(g) >= (1ll << 31))
    return PD_ERR_UNSUPPORTED;

  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
    (void)hipGetLastError();
    return PD_ERR_DEVICE;
  }
  pd_predecoder* h = new (std::nothrow) pd_predecoder();
  if (!h) return PD_ERR_OUT_OF_MEMORY;
  h->g = g;
  h->dtype = dtype;
  h->max_batch = max_batch;
  h->layers.assign(layers, layers + n_layers);
  h->ks = ks;
  if (hipGetDevice(&h->device) != hipSuccess ||
      hipDeviceGetAttribute(&h->n_cu, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess ||
      h->n_cu < 1) {
    (void)hipGetLastError();
    delete h;
    return PD_ERR_DEVICE;
  }
  int cmax = 2;
  for (int i = 0; i < n_layers - 1; ++i) cmax = std::max(cmax, (int)layers[i].c_out);
  h->cmax = cmax;
  if (dtype != PD_DTYPE_FP32) {
    h->tiling = plan_tiling(g, max_batch, ks);
    const int max_span = ks == 3 ? std::min(pd::conv_single_max_span(), pd::conv_hidden_max_span(3))
                                 : pd::conv_hidden_max_span(5);
    if (h->tiling.span <= 0 || h->tiling.span > max_span) {
      delete h;
      return PD_ERR_UNSUPPORTED;
    }
  }

  pd_status s = PD_OK;
  // planes: fp32 or bf16; activations: fp32, bf16 or E4M3
  const size_t elem = dtype == PD_DTYPE_FP32 ? 4 : 2;
  const size_t aelem = dtype == PD_DTYPE_FP32 ? 4 : (dtype == PD_DTYPE_FP8 ? 1 : 2);
  const size_t vox = (size_t)max_batch * (size_t)g.S;
  auto fail = [&](pd_status st) {
    free_all(h);
    delete h;
    return st;
  };
  const size_t cin0 = (size_t)layers[0].c_in;
  if ((s = dev_alloc(&h->ws.planes, vox * cin0 * elem)) != PD_OK) return fail(s);
  h->ws.act_bytes = vox * cmax * aelem;
  if ((s = dev_alloc(&h->ws.act[0], vox * cmax * aelem)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.act[1], vox * cmax * aelem)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.nib, (size_t)max_batch * g.V)) != PD_OK) return fail(s);
  if (dtype != PD_DTYPE_FP32) {
    // parked fp32 sums of split K loops: room for one unit per compute unit
    h->ws.max_units = h->n_cu;
    if ((s = dev_alloc(&h->ws.partial, (size_t)h->ws.max_units * pd::conv_hidden_partial_floats_per_unit() * 4)) !=
        PD_OK)
      return fail(s);
    if ((s = dev_alloc(&h->ws.sched, kSchedWords * 4)) != PD_OK) return fail(s);
    if (hipMemset(h->ws.sched, 0, kSchedWords * 4) != hipSuccess) return fail(PD_ERR_DEVICE);
  }
  std::vector<int32_t> tab = build_tables(g);
  if ((s = upload(&h->tables, tab.data(), tab.size() * sizeof(int32_t))) != PD_OK) return fail(s);
  if (hipMemset(h->ws.planes, 0, vox * cin0 * elem) != hipSuccess ||
      hipMemset(h->ws.act[0], 0, vox * cmax * aelem) != hipSuccess ||
      hipMemset(h->ws.act[1], 0, vox * cmax * aelem) != hipSuccess)
    return fail(PD_ERR_DEVICE);

  const float* src = weights;
  for (int i = 0; i < n_layers; ++i) {
    const pd_layer& L = layers[i];
    const size_t nw = (size_t)L.c_out * L.c_in * L.k * L.k * L.k;
    const float* w = src;
    const float* b = src + nw;
    src += nw + L.c_out;
    // fp8: weight codes, per-channel scales and the values they stand for
    std::vector<uint8_t> codes;
    std::vector<float> scale, wq;
    if (dtype == PD_DTYPE_FP8) quantize_e4m3(w, L.c_out, nw / L.c_out, &codes, &scale, &wq);
    if (i == n_layers - 1 && L.k == 3) {  // a 3x3x3 output layer: rows (tap, filter)
      if (!pd::conv_out_supported(L.c_in, dtype == PD_DTYPE_FP8, 3, g.H)) return fail(PD_ERR_UNSUPPORTED);
      std::vector<uint8_t> f = out_fragments(w, codes.data(), L.c_in, dtype == PD_DTYPE_FP8);
      void* wd = nullptr;
      s = upload(&wd, f.data(), f.size());
      h->wdev.push_back(wd);
      h->wslice.push_back(0);
      if (s != PD_OK) return fail(s);
      std::vector<float> bp(8, 1.0f);
      for (int o2 = 0; o2 < 4; ++o2) {
        bp[o2] = b[o2];
        if (dtype == PD_DTYPE_FP8) bp[4 + o2] = scale[o2];
      }
      float* bd = nullptr;
      s = upload(&bd, bp.data(), bp.size() * 4);
      h->bdev.push_back(bd);
      if (s != PD_OK) return fail(s);
      break;
    }
    if (i == n_layers - 1 && L.k > 1) {  // a 5x5x5 output layer: 4 filters padded to one block of 32
      void* wd = nullptr;
      if (dtype == PD_DTYPE_FP8) {
        std::vector<uint8_t> f = conv_fragments_fp8(codes.data(), L.c_in, L.c_out);
        s = upload(&wd, f.data(), f.size());
      } else {
        std::vector<uint16_t> f = conv_fragments(w, L.c_in, L.c_out, L.k);
        s = upload(&wd, f.data(), f.size() * 2);
      }
      h->wdev.push_back(wd);
      h->wslice.push_back(0);
      if (s != PD_OK) return fail(s);
      // biases of the 32 padded channels, then (fp8) their weight scales
      std::vector<float> bp(64, 0.0f);
      for (int o2 = 0; o2 < L.c_out; ++o2) {
        bp[o2] = b[o2];
        bp[32 + o2] = dtype == PD_DTYPE_FP8 ? scale[o2] : 1.0f;
      }
      float* bd = nullptr;
      s = upload(&bd, bp.data(), bp.size() * 4);
      h->bdev.push_back(bd);
      if (s != PD_OK) return fail(s);
      break;
    }
    if (i == n_layers - 1) {
      std::vector<float> hw((size_t)4 * L.c_in);
      for (int o = 0; o < 4; ++o)
        for (int c = 0; c < L.c_in; ++c) {
          float v = w[(size_t)o * L.c_in + c];
          hw[(size_t)o * L.c_in + c] =
              dtype == PD_DTYPE_BF16 ? bf16_value(v) : (dtype == PD_DTYPE_FP8 ? wq[(size_t)o * L.c_in + c] : v);
        }
      if ((s = upload(&h->head_w, hw.data(), hw.size() * 4)) != PD_OK) return fail(s);
      if ((s = upload(&h->head_b, b, 4 * sizeof(float))) != PD_OK) return fail(s);
      break;
    }
    void* wd = nullptr;
    size_t slice = 0;
    std::vector<float> bias_dev(b, b + L.c_out);
    if (dtype == PD_DTYPE_FP8 && i > 0) {
      // E4M3 fragments; per 128-channel slice: its biases, then its scales
      const int cw = L.c_out == 256 ? 128 : L.c_out;
      std::vector<uint8_t> f = conv_fragments_fp8(codes.data(), L.c_in, cw);
      bias_dev.assign(b, b + cw);
      bias_dev.insert(bias_dev.end(), scale.begin(), scale.begin() + cw);
      if (L.c_out == 256) {
        slice = f.size();
        std::vector<uint8_t> f2 = conv_fragments_fp8(codes.data() + (size_t)128 * L.c_in * 27, L.c_in, 128);
        f.insert(f.end(), f2.begin(), f2.end());
        bias_dev.insert(bias_dev.end(), b + 128, b + 256);
        bias_dev.insert(bias_dev.end(), scale.begin() + 128, scale.end());
      }
      s = upload(&wd, f.data(), f.size());
    } else if (dtype != PD_DTYPE_FP32) {
      // bf16 fragments (fp8 layer 1: of the E4M3 values times their scales,
      // exact in bf16)
      const float* wv = dtype == PD_DTYPE_FP8 ? wq.data() : w;
      std::vector<uint16_t> f;
      if (L.c_out == 256) {  // two slices of 128 output channels, back to back
        f = conv_fragments(wv, L.c_in, 128);
        slice = f.size() * 2;
        std::vector<uint16_t> f2 = conv_fragments(wv + (size_t)128 * L.c_in * 27, L.c_in, 128);
        f.insert(f.end(), f2.begin(), f2.end());
      } else {
        f = conv_fragments(wv, L.c_in, L.c_out, L.k);
      }
      s = upload(&wd, f.data(), f.size() * 2);
    } else {
      std::vector<float> r((size_t)27 * L.c_in * L.c_out);
      for (int co = 0; co < L.c_out; ++co)
        for (int ci = 0; ci < L.c_in; ++ci)
          for (int tap = 0; tap < 27; ++tap)
            r[((size_t)tap * L.c_in + ci) * L.c_out + co] = w[((size_t)co * L.c_in + ci) * 27 + tap];
      s = upload(&wd, r.data(), r.size() * 4);
    }
    h->wdev.push_back(wd);
    h->wslice.push_back(slice);
    if (s != PD_OK) return fail(s);
    float* bd = nullptr;
    s = upload(&bd, bias_dev.data(), bias_dev.size() * 4);
    h->bdev.push_back(bd);
    if (s != PD_OK) return fail(s);
    // a 64- or 128-wide layer of the hidden kernel: also as slices of sw
    // output channels (fragments back to back; per slice its biases, then
    // (fp8) its scales)
    auto slices = [&](int sw, void** wn, float** bn) -> pd_status {
      std::vector<float> bq;
      pd_status st;
      if (dtype == PD_DTYPE_FP8) {
        std::vector<uint8_t> f;
        for (int q = 0; q < L.c_out / sw; ++q) {
          std::vector<uint8_t> fq = conv_fragments_fp8(codes.data() + (size_t)sw * q * L.c_in * 27, L.c_in, sw);
          f.insert(f.end(), fq.begin(), fq.end());
          bq.insert(bq.end(), b + sw * q, b + sw * (q + 1));
          bq.insert(bq.end(), scale.begin() + sw * q, scale.begin() + sw * (q + 1));
        }
        st = upload(wn, f.data(), f.size());
      } else {
        std::vector<uint16_t> f;
        for (int q = 0; q < L.c_out / sw; ++q) {
          std::vector<uint16_t> fq = conv_fragments(w + (size_t)sw * q * L.c_in * 27, L.c_in, sw);
          f.insert(f.end(), fq.begin(), fq.end());
        }
        st = upload(wn, f.data(), f.size() * 2);
        bq.assign(b, b + L.c_out);
      }
      return st != PD_OK ? st : upload(bn, bq.data(), bq.size() * 4);
    };
    for (auto* v : {&h->wnarrow, &h->whalf}) v->resize(h->wdev.size(), nullptr);
    for (auto* v : {&h->bnarrow, &h->bhalf}) v->resize(h->wdev.size(), nullptr);
    // (256 input channels: 32-channel slices in fp8 only, no 64-channel
    // ones -- in bf16 their 16-chunk K loops measured slower than the split
    // loops of 128-channel slices, at batch 1 of Models 2 and 5)
    auto width_ok = [](int c) { return c == 64 || c == 128 || c == 256; };
    if (i > 0 && L.k == 3 && width_ok(L.c_in) && width_ok(L.c_out) && dtype != PD_DTYPE_FP32) {
      if (L.c_in <= 128 || dtype == PD_DTYPE_FP8) s = slices(32, &h->wnarrow.back(), &h->bnarrow.back());
      if (s == PD_OK && L.c_in <= 128 && L.c_out >= 128) s = slices(64, &h->whalf.back(), &h->bhalf.back());
    }
    if (s != PD_OK) return fail(s);
  }
  if (hipDeviceSynchronize() != hipSuccess) return fail(PD_ERR_DEVICE);
  *out = h;
  return PD_OK;
}

size_t predecoder_resnet_weight_count(const pd_block* b, int32_t n) {
  if (!b || n < 1) return 0;
  size_t total = 0;
  for (int k = 0; k < n; ++k) {
    const size_t ci = b[k].c_in, cm = b[k].c_mid, co = b[k].c_out;
    if (b[k].c_in < 1 || b[k].c_mid < 1 || b[k].c_out < 1) return 0;
    total += cm * ci * 27 + cm + 4 * cm + co * cm * 27 + co + 4 * co;
    if (ci != co) total += co * ci + co;
  }
  return total;
}

pd_status predecoder_create_resnet(const float* weights, size_t n_weights, int32_t d, int32_t T,
                                   const pd_block* blocks, int32_t n_blocks, int32_t dtype, int32_t max_batch,
                                   const pd_options* opts, pd_predecoder** out) {
  if (!out) return PD_ERR_INVALID_ARG;
  *out = nullptr;
  if (!weights || !blocks || n_blocks < 1) return PD_ERR_INVALID_ARG;
  if (d < 3 || (d % 2) == 0 || T < 1 || max_batch < 1) return PD_ERR_INVALID_ARG;
  if (dtype != PD_DTYPE_FP32 && dtype != PD_DTYPE_BF16 && dtype != PD_DTYPE_FP8) return PD_ERR_INVALID_ARG;
  const pd_options o = opts ? *opts : pd_options{PD_LAYOUT_PLAQUETTE, PD_BOUNDARY_NONE, PD_BOUNDARY_NONE};
  if (o.layout != PD_LAYOUT_PLAQUETTE && o.layout != PD_LAYOUT_PAPER) return PD_ERR_INVALID_ARG;
  if (o.first_round < PD_BOUNDARY_NONE || o.first_round > PD_BOUNDARY_X || o.last_round < PD_BOUNDARY_NONE ||
      o.last_round > PD_BOUNDARY_X)
    return PD_ERR_INVALID_ARG;
  if (o.layout == PD_LAYOUT_PLAQUETTE && (o.first_round != PD_BOUNDARY_NONE || o.last_round != PD_BOUNDARY_NONE))
    return PD_ERR_INVALID_ARG;
  // the chain: input channels of the layout, widths that meet, 4 outputs
  if (blocks[0].c_in != (o.layout == PD_LAYOUT_PAPER ? 4 : 2) || blocks[n_blocks - 1].c_out != 4)
    return PD_ERR_INVALID_ARG;
  for (int k = 0; k < n_blocks; ++k) {
    const pd_block& B = blocks[k];
    if (B.c_in < 1 || B.c_mid < 1 || B.c_out < 1 || B.act < 0 || B.act > 2) return PD_ERR_INVALID_ARG;
    if (k > 0 && B.c_in != blocks[k - 1].c_out) return PD_ERR_INVALID_ARG;
  }
  if (n_weights != predecoder_resnet_weight_count(blocks, n_blocks)) return PD_ERR_INVALID_ARG;
  // what the kernels run: bf16 or fp8; widths 64, 128, 256 or 512 with
  // c_out = c_mid inside the network; fp8: projections only where they are
  // fused (the first block, from its few input channels, and the last, with
  // c_in = c_mid)
  if (dtype != PD_DTYPE_BF16 && dtype != PD_DTYPE_FP8) return PD_ERR_UNSUPPORTED;
  if (dtype == PD_DTYPE_FP8)
    for (int k = 0; k < n_blocks; ++k) {
      const pd_block& B = blocks[k];
      if (B.c_in == B.c_out) continue;
      const bool first_ok = k == 0 && B.c_in <= 8 && n_blocks > 1;
      const bool last_ok = k == n_blocks - 1 && B.c_in == B.c_mid;
      if (!first_ok && !last_ok) return PD_ERR_UNSUPPORTED;
    }
  auto width_ok = [](int c) { return c == 64 || c == 128 || c == 256 || c == 512; };
  // conv1 of a later block runs the hidden kernel from c_in to slices of
  // min(c_mid, 128) channels: the instantiated pairs
  auto conv1_ok = [](int ci, int cw) {
    return (ci == 64 && (cw == 64 || cw == 128)) || (ci == 128 && (cw == 64 || cw == 128)) ||
           (ci == 256 && (cw == 64 || cw == 128)) || (ci == 512 && cw == 128);
  };
  for (int k = 0; k < n_blocks; ++k) {
    const pd_block& B = blocks[k];
    if (!width_ok(B.c_mid)) return PD_ERR_UNSUPPORTED;
    if (k < n_blocks - 1 && B.c_out != B.c_mid) return PD_ERR_UNSUPPORTED;
    if (k > 0 && !conv1_ok(B.c_in, B.c_mid > 128 ? 128 : B.c_mid)) return PD_ERR_UNSUPPORTED;
  }
  Geom g = make_geom(d, T, o.layout, o.first_round, o.last_round);
  if (g.d > kMaxD || g.T > kMaxT) return PD_ERR_UNSUPPORTED;
  if ((long long)max_batch * g.V >= (1ll << 31) || (long long)max_batch * (g.Wd + g.Wf) >= (1ll << 31) ||
      (long long)max_batch * g.S >= (1ll << 31) ||
      (long long)max_batch * (T + 2) * pd::line_plane(g) >= (1ll << 31))
    return PD_ERR_UNSUPPORTED;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
    (void)hipGetLastError();
    return PD_ERR_DEVICE;
  }
  pd_predecoder* h = new (std::nothrow) pd_predecoder();
  if (!h) return PD_ERR_OUT_OF_MEMORY;
  h->g = g;
  h->dtype = dtype;
  h->max_batch = max_batch;
  h->blocks.assign(blocks, blocks + n_blocks);
  if (hipGetDevice(&h->device) != hipSuccess ||
      hipDeviceGetAttribute(&h->n_cu, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess ||
      h->n_cu < 1) {
    (void)hipGetLastError();
    delete h;
    return PD_ERR_DEVICE;
  }
  h->tiling = plan_tiling(g, max_batch);
  if (h->tiling.span <= 0 || h->tiling.span > pd::conv_hidden_max_span(3)) {
    delete h;
    return PD_ERR_UNSUPPORTED;
  }
  int cmax = 4, pmax = 4;
  for (int k = 0; k < n_blocks; ++k) {
    cmax = std::max(cmax, std::max((int)blocks[k].c_mid, (int)blocks[k].c_out));
    if (blocks[k].c_in != blocks[k].c_out) pmax = std::max(pmax, (int)blocks[k].c_out);
  }
  h->cmax = cmax;
  h->pmax = pmax;
  pd_status s = PD_OK;
  auto fail = [&](pd_status st) {
    free_all(h);
    delete h;
    return st;
  };
  const size_t vox = (size_t)max_batch * (size_t)g.S;
  const size_t cin0 = (size_t)blocks[0].c_in;
  if ((s = dev_alloc(&h->ws.planes, vox * cin0 * 2)) != PD_OK) return fail(s);
  h->ws.act_bytes = vox * cmax * 2;
  if ((s = dev_alloc(&h->ws.act[0], vox * cmax * 2)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.act[1], vox * cmax * 2)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.act[2], vox * cmax * 2)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.pbuf, vox * pmax * 2)) != PD_OK) return fail(s);
  if ((s = dev_alloc(&h->ws.nib, (size_t)max_batch * g.V)) != PD_OK) return fail(s);
  h->ws.max_units = h->n_cu;
  if ((s = dev_alloc(&h->ws.partial, (size_t)h->ws.max_units * pd::conv_hidden_partial_floats_per_unit() * 4)) != PD_OK)
    return fail(s);
  if ((s = dev_alloc(&h->ws.sched, kSchedWords * 4)) != PD_OK) return fail(s);
  if (hipMemset(h->ws.sched, 0, kSchedWords * 4) != hipSuccess) return fail(PD_ERR_DEVICE);
  std::vector<int32_t> tab = build_tables(g);
  if ((s = upload(&h->tables, tab.data(), tab.size() * sizeof(int32_t))) != PD_OK) return fail(s);
  if (hipMemset(h->ws.planes, 0, vox * cin0 * 2) != hipSuccess || hipMemset(h->ws.act[0], 0, vox * cmax * 2) != hipSuccess ||
      hipMemset(h->ws.act[1], 0, vox * cmax * 2) != hipSuccess || hipMemset(h->ws.act[2], 0, vox * cmax * 2) != hipSuccess ||
      hipMemset(h->ws.pbuf, 0, vox * pmax * 2) != hipSuccess)
    return fail(PD_ERR_DEVICE);
  // weights: per conv, BatchNorm folded in (g = scale / sqrt(var + 1e-5) in
  // fp64; weights fp32(w g), rounded to bf16 by the fragment builder or, on
  // the fp8 path, quantised per output channel to E4M3; bias fp32((b - mean)
  // g + shift))
  const bool fp8 = dtype == PD_DTYPE_FP8;
  const float* src = weights;
  for (int k = 0; k < n_blocks; ++k) {
    const pd_block& B = blocks[k];
    for (int c = 0; c < 2; ++c) {
      const int cin = c == 0 ? B.c_in : B.c_mid, cout = c == 0 ? B.c_mid : B.c_out;
      const size_t nw = (size_t)cout * cin * 27;
      const float* w = src;
      const float* b = src + nw;
      const float* bn = b + cout;  // scale, shift, mean, var
      src += nw + cout + 4 * (size_t)cout;
      std::vector<float> wf(nw), bf(cout > 4 ? cout : 32, 0.0f);
      for (int o2 = 0; o2 < cout; ++o2) {
        const double gg = (double)bn[o2] / std::sqrt((double)bn[3 * cout + o2] + 1e-5);
        for (size_t e = 0; e < (size_t)cin * 27; ++e) wf[o2 * (size_t)cin * 27 + e] = (float)((double)w[o2 * (size_t)cin * 27 + e] * gg);
        bf[o2] = (float)(((double)b[o2] - bn[2 * cout + o2]) * gg + bn[cout + o2]);
      }
      // fp8: the folded weights' E4M3 codes and per-channel scales (and the
      // values they stand for, for layer 1's bf16 fragments)
      std::vector<uint8_t> codes;
      std::vector<float> scale, wq;
      if (fp8) quantize_e4m3(wf.data(), cout, (size_t)cin * 27, &codes, &scale, &wq);
      size_t slice = 0;
      void* wd = nullptr;
      if (c == 1 && k == n_blocks - 1) {  // the output conv, 4 filters: rows (tap, filter)
        if (!pd::conv_out_supported(cin, fp8, 3, g.H)) return fail(PD_ERR_UNSUPPORTED);
        std::vector<uint8_t> f = out_fragments(wf.data(), codes.data(), cin, fp8);
        s = upload(&wd, f.data(), f.size());
        bf.resize(8);
        for (int o2 = 0; o2 < 4; ++o2) bf[4 + o2] = fp8 ? scale[o2] : 1.0f;  // [4] biases, then [4] weight scales
      } else if (fp8 && !(c == 0 && k == 0)) {
        // E4M3 fragments per 128-channel slice; per slice its biases, then its scales
        const int cw = cout > 128 ? 128 : cout, nsl = cout / cw;
        std::vector<uint8_t> f;
        std::vector<float> bd;
        for (int q = 0; q < nsl; ++q) {
          std::vector<uint8_t> fq = conv_fragments_fp8(codes.data() + (size_t)q * cw * cin * 27, cin, cw);
          if (nsl > 1) slice = fq.size();
          f.insert(f.end(), fq.begin(), fq.end());
          bd.insert(bd.end(), bf.begin() + (size_t)q * cw, bf.begin() + (size_t)(q + 1) * cw);
          bd.insert(bd.end(), scale.begin() + (size_t)q * cw, scale.begin() + (size_t)(q + 1) * cw);
        }
        bf = bd;
        s = upload(&wd, f.data(), f.size());
      } else {
        // bf16 fragments (fp8 layer 1: of the E4M3 values times their scales, exact in bf16)
        std::vector<uint16_t> f = fragments_sliced(fp8 ? wq.data() : wf.data(), cin, cout, &slice);
        s = upload(&wd, f.data(), f.size() * 2);
      }
      h->wdev.push_back(wd);
      h->wslice.push_back(slice);
      if (s != PD_OK) return fail(s);
      float* bd = nullptr;
      s = upload(&bd, bf.data(), bf.size() * 4);
      h->bdev.push_back(bd);
      if (s != PD_OK) return fail(s);
    }
    float* pw = nullptr;
    float* pb = nullptr;
    if (B.c_in != B.c_out) {
      // weights: bf16 values, or (fp8) E4M3 codes with per-channel scales and
      // the values they stand for
      const size_t np = (size_t)B.c_out * B.c_in;
      std::vector<uint8_t> pcodes;
      std::vector<float> pscale, pvals;
      if (fp8) {
        quantize_e4m3(src, B.c_out, B.c_in, &pcodes, &pscale, &pvals);
      } else {
        pvals.resize(np);
        for (size_t e = 0; e < np; ++e) pvals[e] = bf16_value(src[e]);
      }
      s = upload(&pw, pvals.data(), np * 4);
      if (s == PD_OK) s = upload(&pb, src + np, (size_t)B.c_out * 4);
      // the last block's projection (c_in = c_mid) runs inside the output
      // conv: fragments [k-step][lane], lane l's row l % 32 (filters 0..3,
      // the rest zero), bf16: ci = 16 k-step + 8 (l / 32) + e; fp8 codes:
      // ci = 64 k-step + 32 (l / 32) + e; then [4] biases and [4] scales
      if (s == PD_OK && k == n_blocks - 1 && B.c_in == B.c_mid) {
        const int kstep = fp8 ? 64 : 16, lb = fp8 ? 32 : 16, per = fp8 ? 32 : 8;
        std::vector<uint8_t> pf(pd::conv_out_proj_fragment_bytes(B.c_in, fp8), 0);
        for (int st = 0; st < B.c_in / kstep; ++st)
          for (int l = 0; l < 64; ++l)
            for (int e = 0; e < per; ++e) {
              const int co = l % 32, ci = st * kstep + per * (l / 32) + e;
              if (co >= B.c_out) continue;
              uint8_t* dst = &pf[((size_t)st * 64 + l) * lb];
              if (fp8) {
                dst[e] = pcodes[(size_t)co * B.c_in + ci];
              } else {
                const uint16_t v = bf16_bits(src[(size_t)co * B.c_in + ci]);
                std::memcpy(dst + 2 * e, &v, 2);
              }
            }
        s = upload(&h->out_proj_frag, pf.data(), pf.size());
        std::vector<float> pbias(8, 1.0f);
        for (int o2 = 0; o2 < 4; ++o2) {
          pbias[o2] = src[np + o2];
          if (fp8) pbias[4 + o2] = pscale[o2];
        }
        if (s == PD_OK) s = upload(&h->out_proj_bias, pbias.data(), pbias.size() * 4);
      }
      src += np + B.c_out;
    }
    h->proj_w.push_back(pw);
    h->proj_b.push_back(pb);
    if (s != PD_OK) return fail(s);
  }
  if (hipDeviceSynchronize() != hipSuccess) return fail(PD_ERR_DEVICE);
  *out = h;
  return PD_OK;
}

pd_status predecoder_run(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                         uint64_t* flips, uint64_t* residual, float* logits) {
  if (!h || !det || !flips || !residual) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  return enqueue_run(h, h->ws, (hipStream_t)hip_stream, det, batch, flips, residual, logits, nullptr);
}

}  // extern "C"

namespace pd {

pd_status run_in_region(pd_predecoder* h, hipStream_t st, const uint64_t* det, int batch, uint64_t* flips,
                        uint64_t* residual, float* logits, void* base, size_t bytes) {
  if (!h || !det || !flips || !residual || !base) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  const Geom& g = h->g;
  const bool resnet = !h->blocks.empty();
  const int fp32 = h->dtype == PD_DTYPE_FP32, fp8 = h->dtype == PD_DTYPE_FP8;
  const size_t elem = fp32 ? 4 : 2;                 // input planes
  const size_t aelem = fp32 ? 4 : (fp8 ? 1 : 2);   // activations
  const size_t cin0 = resnet ? (size_t)h->blocks[0].c_in : (size_t)h->layers[0].c_in;
  const size_t vox = (size_t)batch * (size_t)g.S;
  // regions of 256-byte aligned offsets: planes, activations, projection
  // outputs (residual networks), flip nibbles, then the parked sums
  size_t off = 0;
  auto carve = [&](size_t n) {
    const size_t at = (off + 255) & ~(size_t)255;
    off = at + ((n + 255) & ~(size_t)255);
    return at;
  };
  const size_t planes_bytes = vox * cin0 * elem, act_bytes = vox * (size_t)h->cmax * aelem;
  const size_t o_planes = carve(planes_bytes);
  size_t o_act[3] = {carve(act_bytes), carve(act_bytes), 0};
  size_t o_pbuf = 0;
  if (resnet) {
    o_act[2] = carve(act_bytes);
    o_pbuf = carve(vox * (size_t)h->pmax * 2);
  }
  const size_t o_nib = carve((size_t)batch * g.V);
  const size_t o_sched = fp32 ? 0 : carve(kSchedWords * 4);
  if (off > bytes) return PD_ERR_TOO_LARGE;
  char* b = (char*)base;
  Workspace ws;
  ws.planes = b + o_planes;
  for (int k = 0; k < (resnet ? 3 : 2); ++k) ws.act[k] = b + o_act[k];
  ws.pbuf = resnet ? (void*)(b + o_pbuf) : nullptr;
  ws.nib = (uint8_t*)(b + o_nib);
  ws.act_bytes = act_bytes;
  if (!fp32) {  // what is left holds the parked sums of up to the handle's own number of units
    const size_t unit = pd::conv_hidden_partial_floats_per_unit() * 4;
    const size_t o_part = carve(0);
    const long long fit = (long long)((bytes - std::min(bytes, o_part)) / unit);
    ws.max_units = std::min(h->ws.max_units, fit);
    ws.partial = (float*)(b + o_part);
  }
  // the zero halos the 3x3x3 layers read: the planes and every activation
  // buffer start all zero (a fill kernel, so that the call can be captured
  // into a graph); the other regions are written before they are read
  pd_status s = check_launch(launch_zero(ws.planes, (planes_bytes + 15) & ~(size_t)15, st));
  for (int k = 0; k < (resnet ? 3 : 2) && s == PD_OK; ++k)
    s = check_launch(launch_zero(ws.act[k], (act_bytes + 15) & ~(size_t)15, st));
  if (!fp32 && s == PD_OK) {  // the hidden kernel's unit counters start at zero (and stay so between launches)
    ws.sched = (uint32_t*)(b + o_sched);
    s = check_launch(launch_zero(ws.sched, kSchedWords * 4, st));
  }
  if (s != PD_OK) return s;
  return enqueue_run(h, ws, st, det, batch, flips, residual, logits, nullptr);
}

}  // namespace pd

extern "C" {

pd_status predecoder_residual(pd_predecoder* h, void* hip_stream, const uint64_t* det,
                              const uint64_t* flips, int32_t batch, uint64_t* residual) {
  if (!h || !det || !flips || !residual) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  return check_launch(
      pd::launch_residual_from_flips(h->g, h->tables, det, flips, residual, batch, (hipStream_t)hip_stream));
}

pd_status predecoder_activations(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                                 int32_t layer, void* out) {
  if (!h || !det || !out) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  if (layer < 0 || layer >= n_stop_points(h)) return PD_ERR_INVALID_ARG;
  if (h->dtype == PD_DTYPE_FP32) return PD_ERR_UNSUPPORTED;
  const hipStream_t st = (hipStream_t)hip_stream;
  StopAt at;
  pd_status s = enqueue_run(h, h->ws, st, det, batch, nullptr, nullptr, nullptr, nullptr, layer, &at);
  if (s != PD_OK) return s;
  return check_launch(pd::launch_extract(h->g, at.buf, at.row_bytes, batch, out, st));
}

pd_status predecoder_unpack(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                            void* planes) {
  if (!h || !det || !planes) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  return check_launch(pd::launch_unpack(h->g, h->tables, det, batch, planes, 0,
                                        h->dtype == PD_DTYPE_FP32, (hipStream_t)hip_stream));
}

pd_status predecoder_stage_times(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                                 uint64_t* flips, uint64_t* residual, int32_t n_iter, float* ms_per_stage) {
  if (!h || !det || !flips || !residual || !ms_per_stage) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch || n_iter < 1 || n_iter > 100000) return PD_ERR_INVALID_ARG;
  const int ns = predecoder_num_stages(h);
  const int ne = ns + 1;
  std::vector<hipEvent_t> ev((size_t)n_iter * ne, nullptr);
  pd_status s = PD_OK;
  for (auto& e : ev)
    if (hipEventCreate(&e) != hipSuccess) {
      s = PD_ERR_DEVICE;
      break;
    }
  hipStream_t st = (hipStream_t)hip_stream;
  for (int it = 0; it < n_iter && s == PD_OK; ++it)
    s = enqueue_run(h, h->ws, st, det, batch, flips, residual, nullptr, ev.data() + (size_t)it * ne);
  if (s == PD_OK && hipStreamSynchronize(st) != hipSuccess) s = PD_ERR_DEVICE;
  if (s == PD_OK) {
    for (int k = 0; k < ns; ++k) ms_per_stage[k] = 0.0f;
    for (int it = 0; it < n_iter && s == PD_OK; ++it)
      for (int k = 0; k < ns; ++k) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, ev[(size_t)it * ne + k], ev[(size_t)it * ne + k + 1]) != hipSuccess) {
          s = PD_ERR_DEVICE;
          break;
        }
        ms_per_stage[k] += ms / n_iter;
      }
  }
  for (auto& e : ev)
    if (e) (void)hipEventDestroy(e);
  (void)hipGetLastError();
  return s;
}

void predecoder_destroy(pd_predecoder* h) {
  if (!h) return;
  (void)hipDeviceSynchronize();
  free_all(h);
  delete h;
}

pd_status predecoder_graph_create(pd_predecoder* h, const uint64_t* det, int32_t batch, uint64_t* flips,
                                  uint64_t* residual, float* logits, pd_graph** out) {
  if (!out) return PD_ERR_INVALID_ARG;
  *out = nullptr;
  if (!h || !det || !flips || !residual) return PD_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->max_batch) return PD_ERR_INVALID_ARG;
  pd_graph* gr = new (std::nothrow) pd_graph();
  if (!gr) return PD_ERR_OUT_OF_MEMORY;
  auto fail = [&](pd_status e) {
    (void)hipGetLastError();
    if (gr->exec) (void)hipGraphExecDestroy(gr->exec);
    if (gr->graph) (void)hipGraphDestroy(gr->graph);
    if (gr->stream) (void)hipStreamDestroy(gr->stream);
    delete gr;
    return e;
  };
  // a stream of its own at the default priority (capture needs a stream
  // other than the null stream)
  if (hipStreamCreateWithFlags(&gr->stream, hipStreamNonBlocking) != hipSuccess) return fail(PD_ERR_DEVICE);
  // one run first: the handle's buffers reach the state every later run
  // starts from, so the recorded sequence (with any buffer clearing it
  // needs) is the one each replay repeats
  pd_status s = enqueue_run(h, h->ws, gr->stream, det, batch, flips, residual, logits, nullptr);
  if (s != PD_OK) return fail(s);
  if (hipStreamSynchronize(gr->stream) != hipSuccess) return fail(PD_ERR_DEVICE);
  if (hipStreamBeginCapture(gr->stream, hipStreamCaptureModeThreadLocal) != hipSuccess) return fail(PD_ERR_DEVICE);
  s = enqueue_run(h, h->ws, gr->stream, det, batch, flips, residual, logits, nullptr);
  hipGraph_t graph = nullptr;
  const hipError_t ec = hipStreamEndCapture(gr->stream, &graph);
  gr->graph = graph;
  if (s != PD_OK) return fail(s);
  if (ec != hipSuccess || !graph) return fail(PD_ERR_DEVICE);
  if (hipGraphInstantiate(&gr->exec, graph, nullptr, nullptr, 0) != hipSuccess) return fail(PD_ERR_DEVICE);
  *out = gr;
  return PD_OK;
}

pd_status predecoder_graph_launch(pd_graph* gr, void* hip_stream) {
  if (!gr || !gr->exec) return PD_ERR_INVALID_ARG;
  return check_launch(hipGraphLaunch(gr->exec, (hipStream_t)hip_stream));
}

void predecoder_graph_destroy(pd_graph* gr) {
  if (!gr) return;
  (void)hipDeviceSynchronize();
  if (gr->exec) (void)hipGraphExecDestroy(gr->exec);
  if (gr->graph) (void)hipGraphDestroy(gr->graph);
  if (gr->stream) (void)hipStreamDestroy(gr->stream);
  delete gr;
}

int32_t predecoder_stream_windows(int32_t n_rounds, int32_t core, int32_t buffer, int32_t* starts, int32_t* lengths,
                                  int32_t* core_starts, int32_t* core_lengths, int32_t capacity) {
  if (n_rounds < 1 || core < 1 || buffer < 0) return -1;
  const int32_t n = (n_rounds + core - 1) / core;
  if (!starts || !lengths || !core_starts || !core_lengths) return n;
  if (capacity < n) return -1;
  for (int32_t k = 0; k < n; ++k) {
    const int32_t c0 = k * core, c1 = std::min(n_rounds, c0 + core);
    const int32_t w0 = std::max(0, c0 - buffer), w1 = std::min(n_rounds, c1 + buffer);
    starts[k] = w0;
    lengths[k] = w1 - w0;
    core_starts[k] = c0;
    core_lengths[k] = c1 - c0;
  }
  return n;
}

}  // extern "C"

// Temporal window driver: windows of the planner grouped by (length,
// touches round 0, touches the last round); one handle per group runs all
// its windows of all streams as one batch.
struct pd_stream {
  int d = 0, n_rounds = 0, core = 0, buffer = 0, n_streams = 0;
  pd::Geom g;                          // the whole stream (for its residual)
  int32_t* tables = nullptr;           // its site tables
  std::vector<pd::StreamWindow> win;   // host copy
  pd::StreamWindow* win_dev = nullptr;
  struct Group {
    int len = 0, count = 0;
    pd_predecoder* h = nullptr;
    uint64_t *det = nullptr, *flips = nullptr, *res = nullptr;
    pd::StreamWindow* win_dev = nullptr;  // this group's windows, in slot order
  };
  std::vector<Group> groups;
  uint64_t** group_flips_dev = nullptr;
  long long* group_words_dev = nullptr;
};

namespace {
void stream_free(pd_stream* s) {
  for (auto& g : s->groups) {
    if (g.h) predecoder_destroy(g.h);
    if (g.det) (void)hipFree(g.det);
    if (g.flips) (void)hipFree(g.flips);
    if (g.res) (void)hipFree(g.res);
    if (g.win_dev) (void)hipFree(g.win_dev);
  }
  if (s->tables) (void)hipFree(s->tables);
  if (s->win_dev) (void)hipFree(s->win_dev);
  if (s->group_flips_dev) (void)hipFree(s->group_flips_dev);
  if (s->group_words_dev) (void)hipFree(s->group_words_dev);
  delete s;
}
}  // namespace

extern "C" {

pd_status predecoder_stream_create(const float* weights, size_t n_weights, int32_t d, int32_t n_rounds, int32_t core,
                                   int32_t buffer, const pd_layer* layers, int32_t n_layers, int32_t dtype,
                                   int32_t n_streams, const pd_options* opts, pd_stream** out) {
  if (!out) return PD_ERR_INVALID_ARG;
  *out = nullptr;
  if (!weights || !layers || n_rounds < 1 || core < 1 || buffer < 0 || n_streams < 1) return PD_ERR_INVALID_ARG;
  if (d < 3 || d % 2 == 0 || n_rounds > kMaxT) return d < 3 || d % 2 == 0 ? PD_ERR_INVALID_ARG : PD_ERR_UNSUPPORTED;
  const pd_options o = opts ? *opts : pd_options{PD_LAYOUT_PLAQUETTE, PD_BOUNDARY_NONE, PD_BOUNDARY_NONE};
  const int32_t nw = predecoder_stream_windows(n_rounds, core, buffer, nullptr, nullptr, nullptr, nullptr, 0);
  if (nw < 1) return PD_ERR_INVALID_ARG;
  std::vector<int32_t> st(nw), ln(nw), cs(nw), cl(nw);
  predecoder_stream_windows(n_rounds, core, buffer, st.data(), ln.data(), cs.data(), cl.data(), nw);
  pd_stream* s = new (std::nothrow) pd_stream();
  if (!s) return PD_ERR_OUT_OF_MEMORY;
  s->d = d;
  s->n_rounds = n_rounds;
  s->core = core;
  s->buffer = buffer;
  s->n_streams = n_streams;
  // group key: length, first-round window, last-round window (the paper
  // layout clears its geometric channels only at the stream's own ends)
  std::vector<std::array<int, 3>> keys;
  s->win.resize(nw);
  for (int k = 0; k < nw; ++k) {
    const std::array<int, 3> key{ln[k], st[k] == 0, st[k] + ln[k] == n_rounds};
    int gi = (int)(std::find(keys.begin(), keys.end(), key) - keys.begin());
    if (gi == (int)keys.size()) {
      keys.push_back(key);
      s->groups.emplace_back();
      s->groups.back().len = ln[k];
    }
    s->win[k] = pd::StreamWindow{st[k], ln[k], cs[k], cl[k], gi, s->groups[gi].count++};
  }
  pd_status r = PD_OK;
  auto fail = [&](pd_status e) {
    stream_free(s);
    return e;
  };
  for (size_t gi = 0; gi < s->groups.size(); ++gi) {
    auto& G = s->groups[gi];
    pd_options go = o;
    if (!keys[gi][1]) go.first_round = PD_BOUNDARY_NONE;
    if (!keys[gi][2]) go.last_round = PD_BOUNDARY_NONE;
    r = predecoder_create_ex(weights, n_weights, d, G.len, layers, n_layers, dtype, G.count * n_streams, &go, &G.h);
    if (r != PD_OK) return fail(r);
    const size_t rows = (size_t)G.count * n_streams;
    if ((r = dev_alloc(&G.det, rows * predecoder_det_words(d, G.len) * 8)) != PD_OK) return fail(r);
    if ((r = dev_alloc(&G.flips, rows * predecoder_flip_words(d, G.len) * 8)) != PD_OK) return fail(r);
    if ((r = dev_alloc(&G.res, rows * predecoder_det_words(d, G.len) * 8)) != PD_OK) return fail(r);
    std::vector<pd::StreamWindow> mine;
    for (const auto& w : s->win)
      if (w.group == (int)gi) mine.push_back(w);
    if ((r = upload(&G.win_dev, mine.data(), mine.size() * sizeof(pd::StreamWindow))) != PD_OK) return fail(r);
  }
  s->g = make_geom(d, n_rounds, o.layout, o.first_round, o.last_round);
  std::vector<int32_t> tab = build_tables(s->g);
  if ((r = upload(&s->tables, tab.data(), tab.size() * sizeof(int32_t))) != PD_OK) return fail(r);
  if ((r = upload(&s->win_dev, s->win.data(), s->win.size() * sizeof(pd::StreamWindow))) != PD_OK) return fail(r);
  std::vector<uint64_t*> gf;
  std::vector<long long> gw;
  for (auto& G : s->groups) {
    gf.push_back(G.flips);
    gw.push_back(predecoder_flip_words(d, G.len));
  }
  if ((r = upload(&s->group_flips_dev, gf.data(), gf.size() * sizeof(uint64_t*))) != PD_OK) return fail(r);
  if ((r = upload(&s->group_words_dev, gw.data(), gw.size() * sizeof(long long))) != PD_OK) return fail(r);
  if (hipDeviceSynchronize() != hipSuccess) return fail(PD_ERR_DEVICE);
  *out = s;
  return PD_OK;
}

pd_status predecoder_stream_run(pd_stream* s, void* hip_stream, const uint64_t* det, uint64_t* flips,
                                uint64_t* residual) {
  if (!s || !det || !flips || !residual) return PD_ERR_INVALID_ARG;
  const hipStream_t st = (hipStream_t)hip_stream;
  const int S = s->d * s->d - 1, F = 3 * s->d * s->d - 1;
  const long long det_words = predecoder_det_words(s->d, s->n_rounds);
  const long long flip_words = predecoder_flip_words(s->d, s->n_rounds);
  pd_status r;
  for (auto& G : s->groups) {
    r = check_launch(pd::launch_stream_gather(det, det_words, G.win_dev, G.count, s->n_streams, S,
                                              predecoder_det_words(s->d, G.len), G.det, st));
    if (r != PD_OK) return r;
    r = predecoder_run(G.h, hip_stream, G.det, G.count * s->n_streams, G.flips, G.res, nullptr);
    if (r != PD_OK) return r;
  }
  r = check_launch(pd::launch_stream_scatter(s->win_dev, s->group_flips_dev, s->group_words_dev, s->n_streams,
                                             s->core, s->n_rounds, F, flip_words, flips, st));
  if (r != PD_OK) return r;
  return check_launch(pd::launch_residual_from_flips(s->g, s->tables, det, flips, residual, s->n_streams, st));
}

void predecoder_stream_destroy(pd_stream* s) {
  if (!s) return;
  (void)hipDeviceSynchronize();
  stream_free(s);
}

}  // extern "C"
