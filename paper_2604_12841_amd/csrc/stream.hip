// stream.hip -- bit movers of the temporal window driver (Sec. VI, parallel
// windows in time): detector rows of a long stream -> rows of the windows
// that cover it, and the windows' committed flip rounds -> the stream's flip
// rows.  One thread per output word; every output word is written by exactly
// one thread (no races between windows that share a word).
#include "internal.h"

namespace pd {
namespace {

// n <= 64 bits of a packed row from bit position pos on (LSB first), the
// first of them in bit 0; reads at most the two words the run touches.
__device__ __forceinline__ uint64_t load_bits(const uint64_t* __restrict__ row, long long pos, int n) {
  const long long w = pos >> 6;
  const int sh = (int)(pos & 63);
  uint64_t v = row[w] >> sh;
  if (sh != 0 && sh + n > 64) v |= row[w + 1] << (64 - sh);
  return n == 64 ? v : (v & ((1ull << n) - 1));
}

// Window rows: out[(w * n_streams + s)][q] = bits [start_w * S + 64 q, ...) of
// stream s, limited to the window's len_w * S bits (the rest zero).
__global__ void __launch_bounds__(256) gather_kernel(const uint64_t* __restrict__ det, long long row_words,
                                                     const StreamWindow* __restrict__ win, int n_win, int n_streams,
                                                     int S, long long out_words, uint64_t* __restrict__ out) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)n_win * n_streams * out_words) return;
  const long long r = gid / out_words;
  const int q = (int)(gid - r * out_words);
  const int w = (int)(r / n_streams), s = (int)(r - (long long)w * n_streams);
  const long long nbits = (long long)win[w].len * S;
  const long long b0 = (long long)q * 64;
  uint64_t v = 0;
  if (b0 < nbits) {
    const int n = (int)(nbits - b0 < 64 ? nbits - b0 : 64);
    v = load_bits(det + (long long)s * row_words, (long long)win[w].start * S + b0, n);
  }
  out[gid] = v;
}

// Stream flip rows: word q of stream s takes each bit from the window whose
// core holds the bit's round (cores tile the stream: window k's core is
// rounds [k core, min((k+1) core, N))), in runs of at most two windows per word.
__global__ void __launch_bounds__(256) scatter_kernel(const StreamWindow* __restrict__ win,
                                                      const uint64_t* const* __restrict__ group_flips,
                                                      const long long* __restrict__ group_words, int n_streams,
                                                      int core, int n_rounds, int F, long long row_words,
                                                      uint64_t* __restrict__ flips) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)n_streams * row_words) return;
  const int s = (int)(gid / row_words);
  const long long q = gid - (long long)s * row_words;
  const long long total = (long long)n_rounds * F;
  long long b = q * 64;
  const long long bend = (b + 64 < total ? b + 64 : total);
  uint64_t v = 0;
  while (b < bend) {
    const int t = (int)(b / F);
    const int k = t / core;
    const StreamWindow& wk = win[k];
    const long long cend = (long long)(wk.core_start + wk.core_len) * F;  // end of the core's bits
    const int n = (int)((bend < cend ? bend : cend) - b);
    const uint64_t* row = group_flips[wk.group] + (long long)(wk.slot * n_streams + s) * group_words[wk.group];
    v |= load_bits(row, b - (long long)wk.start * F, n) << (b - q * 64);
    b += n;
  }
  flips[gid] = v;
}

}  // namespace

hipError_t launch_stream_gather(const uint64_t* det, long long row_words, const StreamWindow* win, int n_win,
                                int n_streams, int S, long long out_words, uint64_t* out, hipStream_t stream) {
  const long long total = (long long)n_win * n_streams * out_words;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, det, row_words, win,
                     n_win, n_streams, S, out_words, out);
  return hipGetLastError();
}

hipError_t launch_stream_scatter(const StreamWindow* win, const uint64_t* const* group_flips,
                                 const long long* group_words, int n_streams, int core, int n_rounds, int F,
                                 long long row_words, uint64_t* flips, hipStream_t stream) {
  const long long total = (long long)n_streams * row_words;
  hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, win, group_flips,
                     group_words, n_streams, core, n_rounds, F, row_words, flips);
  return hipGetLastError();
}

}  // namespace pd
