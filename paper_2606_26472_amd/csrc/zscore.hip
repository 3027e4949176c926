// Causal trailing-window smoothing and band combination.
//   Eq. 3:  z(t) = (x(t) - mu(t)) / (sigma(t) + eps)     (EPIKV_SMOOTH_Z)
//   Eq. 2:  mu(t)                                          (EPIKV_SMOOTH_MEAN)
// with mu and the population sigma over the last min(w, available) samples
// up to and including t; then s(t) = mean_A - mean_B over the signal rows
// (Fig. 1; the Lag-KV signal is a single row of weight +1).  s(t) is the
// token's frozen score (Sec. 3.3).
//
// One 1024-thread workgroup scores a tile of kZscoreTile (64) tokens of one
// sequence; each of its 16 wavefronts smooths one signal row at a time (lane
// = token), so the band layers are processed in parallel.  A wavefront
// stages its row's tile plus the w-1 samples before it in its own LDS slice
// (taken from the carried ring for the chunk's first tokens) and each lane
// computes its window's mean and variance in two passes over at most w
// values (fp32; the two-pass form avoids the E[x^2] - mu^2 cancellation when
// the signal's mean is large against its spread).  The per-row values meet
// in LDS for the band combination.
#include "epikv_internal.h"

namespace epikv {
namespace {

constexpr int kWaves = kZscoreThreads / 64;
constexpr int kZscoreWaves = kWaves;
constexpr int kSlice = EPIKV_MAX_WINDOW - 1 + kZscoreTile;

__global__ __launch_bounds__(kZscoreThreads) void k_zscore(ZscoreArgs a) {
  __shared__ float xs[kWaves][kSlice];
  __shared__ float vals[EPIKV_MAX_BAND][kZscoreTile];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int tile = blockIdx.x;
  const int b = blockIdx.y;
  const int wm1 = a.w - 1;
  const int c = tile * kZscoreTile + lane;
  const int n_tok = max(a.n_tok_in[b], 0);
  // The first token of a fresh hidden-state stream has no predecessor and
  // hence no sample.
  const int c0 = (a.hs && n_tok == 0) ? 1 : 0;
  const int64_t prior = a.hs ? (int64_t)max(n_tok - 1, 0) : (int64_t)n_tok;
  const int cnt = (int)min((int64_t)wm1, prior);
  // Extended index space: X[j] = ring slot j for j < w-1, X[w-1+c] = signal
  // of token c.  Valid samples are X[vstart ..].
  const int vstart = wm1 - cnt + c0;
  const bool last_tile = (tile == (int)gridDim.x - 1);
  const int base = tile * kZscoreTile;  // X index held in xs[wave][0]
  const int span = wm1 + kZscoreTile;
  const int64_t total_out = prior + (a.C - c0);
  const int cnt_out = (int)min((int64_t)wm1, total_out);
  float* x = xs[wave];

  // Every wavefront runs the same number of rounds so the barriers match.
  const int rounds = (a.n_sig + kWaves - 1) / kWaves;
  for (int rd = 0; rd < rounds; ++rd) {
    const int l = rd * kWaves + wave;
    const bool active = l < a.n_sig;
    if (active) {
      const float* ring = a.ring_in + ((int64_t)b * a.n_sig + l) * wm1;
      const float* sg = a.sig + ((int64_t)l * a.B + b) * a.C;
      for (int k = lane; k < span; k += 64) {
        const int j = base + k;
        float v = 0.f;
        if (j < wm1)
          v = ring[j];
        else if (j - wm1 < a.C)
          v = sg[j - wm1];
        x[k] = v;
      }
    }
    __syncthreads();
    if (active) {
      float v = 0.f;
      if (c < a.C && c >= c0) {
        const int j = wm1 + c;
        v = smooth_at(x, base, max(vstart, j - wm1), j, a.mode, a.eps);
      }
      vals[l][lane] = v;
      if (a.smoothed && c < a.C) a.smoothed[((int64_t)l * a.B + b) * a.C + c] = v;
      if (last_tile) {
        // Carry the last min(w-1, samples) samples, right-aligned: slot k
        // holds X[C + k].
        float* ro = a.ring_out + ((int64_t)b * a.n_sig + l) * wm1;
        for (int k = lane; k < wm1; k += 64) {
          const bool valid = (wm1 - 1 - k) < cnt_out;
          ro[k] = valid ? x[a.C + k - base] : 0.f;
        }
      }
    }
    __syncthreads();
  }

  if (tid < kZscoreTile && c < a.C) {
    const float s = band_combine<kZscoreTile>(vals, tid, a.n_a, a.n_sig, a.n_b);
    const int N = a.n_cached[b];
    if (N >= a.C && (int64_t)N <= a.ld_s) a.scores[(int64_t)b * a.ld_s + (N - a.C) + c] = s;
  }
  if (last_tile && tid == 0) a.n_tok_out[b] = n_tok + a.C;
  if (last_tile && tid < a.n_sig)
    a.ema_out[(int64_t)b * a.n_sig + tid] = a.ema_in[(int64_t)b * a.n_sig + tid];
}

// EMA smoothing (App. E): y(t) = alpha*y(t-1) + (1-alpha)*x(t), y = x at the
// stream's first sample.  One 1024-thread workgroup per sequence walks the
// chunk in 64-token tiles; for each signal row a wavefront turns its tile
// into per-token affine maps y -> A*y + Bc (a token without a sample is the
// identity) and composes them with a lane-wise inclusive scan, so the tile's
// averages follow exactly from the average carried in from the previous
// tile.  The per-row values meet in LDS for the band combination.
__global__ __launch_bounds__(kZscoreThreads) void k_ema(ZscoreArgs a) {
  __shared__ float carry[EPIKV_MAX_BAND];
  __shared__ float vals[EPIKV_MAX_BAND][kZscoreTile];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.y;
  const int wm1 = a.w - 1;
  const int n_tok = max(a.n_tok_in[b], 0);
  const int c0 = (a.hs && n_tok == 0) ? 1 : 0;
  const int64_t prior = a.hs ? (int64_t)max(n_tok - 1, 0) : (int64_t)n_tok;
  const float al = a.alpha, bl = 1.0f - a.alpha;
  if (tid < a.n_sig) carry[tid] = a.ema_in[(int64_t)b * a.n_sig + tid];
  const int N = a.n_cached[b];
  const bool write_scores = N >= a.C && (int64_t)N <= a.ld_s;
  const int rounds = (a.n_sig + kZscoreWaves - 1) / kZscoreWaves;
  const int tiles = (a.C + kZscoreTile - 1) / kZscoreTile;
  __syncthreads();
  for (int tile = 0; tile < tiles; ++tile) {
    const int c = tile * kZscoreTile + lane;
    const bool has = c < a.C && c >= c0;
    // the stream's first sample starts the average
    const bool first = prior == 0 && c == c0;
    for (int rd = 0; rd < rounds; ++rd) {
      const int l = rd * kZscoreWaves + wave;
      if (l < a.n_sig) {
        const float x = has ? a.sig[((int64_t)l * a.B + b) * a.C + c] : 0.f;
        const float y = ema_scan(x, has, first, al, bl, carry[l], lane);
        const float v = has ? y : 0.f;
        vals[l][lane] = v;
        if (a.smoothed && c < a.C) a.smoothed[((int64_t)l * a.B + b) * a.C + c] = v;
        const float y_last = __shfl(y, 63, 64);
        if (lane == 0) carry[l] = y_last;
      }
    }
    __syncthreads();
    if (tid < kZscoreTile && c < a.C && write_scores)
      a.scores[(int64_t)b * a.ld_s + (N - a.C) + c] =
          band_combine<kZscoreTile>(vals, tid, a.n_a, a.n_sig, a.n_b);
    __syncthreads();
  }
  // carried state: averages, sample ring, token count
  if (tid < a.n_sig) a.ema_out[(int64_t)b * a.n_sig + tid] = carry[tid];
  const int64_t total_out = prior + (a.C - c0);
  const int cnt_out = (int)min((int64_t)wm1, total_out);
  for (int i = tid; i < a.n_sig * wm1; i += kZscoreThreads) {
    const int l = i / wm1;
    const int k = i - l * wm1;
    const int j = a.C + k;  // index in [ring | chunk signal]
    float v = 0.f;
    if ((wm1 - 1 - k) < cnt_out)
      v = j < wm1 ? a.ring_in[((int64_t)b * a.n_sig + l) * wm1 + j]
                  : a.sig[((int64_t)l * a.B + b) * a.C + (j - wm1)];
    a.ring_out[((int64_t)b * a.n_sig + l) * wm1 + k] = v;
  }
  if (tid == 0) a.n_tok_out[b] = n_tok + a.C;
}

}  // namespace

hipError_t launch_zscore(const ZscoreArgs& a, hipStream_t s) {
  if (a.mode == EPIKV_SMOOTH_EMA) {
    hipLaunchKernelGGL(k_ema, dim3(1, a.B), dim3(kZscoreThreads), 0, s, a);
    return hipGetLastError();
  }
  dim3 grid((a.C + kZscoreTile - 1) / kZscoreTile, a.B);
  hipLaunchKernelGGL(k_zscore, grid, dim3(kZscoreThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace epikv
