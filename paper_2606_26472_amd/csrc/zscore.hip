// Causal trailing-window smoothing and band combination.
//   Eq. 3:  z(t) = (x(t) - mu(t)) / (sigma(t) + eps)     (EPIKV_SMOOTH_Z)
//   Eq. 2:  mu(t)                                          (EPIKV_SMOOTH_MEAN)
// with mu and the population sigma over the last min(w, available) samples
// up to and including t; then s(t) = mean_A - mean_B over the signal rows
// (Fig. 1; the Lag-KV signal is a single row of weight +1).  s(t) is the
// token's frozen score (Sec. 3.3).
//
// One workgroup scores a tile of kZscoreTile tokens of one sequence.  For
// each signal row it stages the tile plus the w-1 samples before it in LDS
// (taken from the carried ring for the chunk's first tokens) and each thread
// computes its window's mean and variance in two passes over at most w
// values (fp32; the two-pass form avoids the E[x^2] - mu^2 cancellation when
// the signal's mean is large against its spread).
#include "epikv_internal.h"

namespace epikv {
namespace {

__global__ __launch_bounds__(kZscoreTile) void k_zscore(ZscoreArgs a) {
  __shared__ float xs[EPIKV_MAX_WINDOW - 1 + kZscoreTile];
  const int tid = threadIdx.x;
  const int tile = blockIdx.x;
  const int b = blockIdx.y;
  const int wm1 = a.w - 1;
  const int c = tile * kZscoreTile + tid;
  const int n_tok = max(a.n_tok_in[b], 0);
  // The first token of a fresh hidden-state stream has no predecessor and
  // hence no sample.
  const int c0 = (a.hs && n_tok == 0) ? 1 : 0;
  const int64_t prior = a.hs ? (int64_t)max(n_tok - 1, 0) : (int64_t)n_tok;
  const int cnt = (int)min((int64_t)wm1, prior);
  // Extended index space: X[j] = ring slot j for j < w-1, X[w-1+c] = sig of
  // token c.  Valid samples are X[vstart ..].
  const int vstart = wm1 - cnt + c0;
  const bool last_tile = (tile == (int)gridDim.x - 1);
  const int base = tile * kZscoreTile;   // X index held in xs[0]
  const int span = wm1 + kZscoreTile;
  const int64_t total_out = prior + (a.C - c0);
  const int cnt_out = (int)min((int64_t)wm1, total_out);

  float sum_a = 0.f, sum_b = 0.f;
  for (int l = 0; l < a.n_sig; ++l) {
    const float* ring = a.ring_in + ((int64_t)b * a.n_sig + l) * wm1;
    const float* sg = a.sig + ((int64_t)l * a.B + b) * a.C;
    for (int k = tid; k < span; k += kZscoreTile) {
      const int j = base + k;
      float v = 0.f;
      if (j < wm1)
        v = ring[j];
      else if (j - wm1 < a.C)
        v = sg[j - wm1];
      xs[k] = v;
    }
    __syncthreads();

    if (c < a.C) {
      const int j = wm1 + c;
      float v = 0.f;
      if (c >= c0) {
        const int lo = max(vstart, j - wm1);
        const float n = (float)(j - lo + 1);
        const float x = xs[j - base];
        if (a.mode == EPIKV_SMOOTH_RAW) {
          v = x;
        } else {
          float s = 0.f;
          for (int k = lo; k <= j; ++k) s += xs[k - base];
          const float mu = s / n;
          if (a.mode == EPIKV_SMOOTH_MEAN) {
            v = mu;
          } else {
            float q = 0.f;
            for (int k = lo; k <= j; ++k) {
              const float dlt = xs[k - base] - mu;
              q = fmaf(dlt, dlt, q);
            }
            v = (x - mu) / (sqrtf(q / n) + a.eps);
          }
        }
      }
      if (l < a.n_a)
        sum_a += v;
      else
        sum_b += v;
      if (a.smoothed) a.smoothed[((int64_t)l * a.B + b) * a.C + c] = v;
    }

    if (last_tile) {
      // Carry the last min(w-1, samples) samples, right-aligned: slot k
      // holds X[C + k].
      float* ro = a.ring_out + ((int64_t)b * a.n_sig + l) * wm1;
      for (int k = tid; k < wm1; k += kZscoreTile) {
        const bool valid = (wm1 - 1 - k) < cnt_out;
        ro[k] = valid ? xs[a.C + k - base] : 0.f;
      }
    }
    __syncthreads();
  }

  if (c < a.C) {
    float s = sum_a / (float)a.n_a;
    if (a.n_b > 0) s -= sum_b / (float)a.n_b;
    const int N = a.n_cached[b];
    if (N >= a.C && (int64_t)N <= a.ld_s)
      a.scores[(int64_t)b * a.ld_s + (N - a.C) + c] = s;
  }
  if (last_tile && tid == 0) a.n_tok_out[b] = n_tok + a.C;
}

}  // namespace

hipError_t launch_zscore(const ZscoreArgs& a, hipStream_t s) {
  dim3 grid((a.C + kZscoreTile - 1) / kZscoreTile, a.B);
  hipLaunchKernelGGL(k_zscore, grid, dim3(kZscoreTile), 0, s, a);
  return hipGetLastError();
}

}  // namespace epikv
