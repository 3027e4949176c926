// Per-token scoring in one launch: for chunks of up to 64 new tokens (a
// decoder scoring each token as it is generated, Sec. 3.3) the hidden-state
// change of Eq. 1, the trailing-window smoothing of Eqs. 2-3 (or raw, or
// EMA, App. E) and the band combination of Fig. 1 run in a single
// workgroup per sequence, with the signal kept in LDS.
//
// The arithmetic is the separate kernels' own, in the same order: per band
// row a wavefront accumulates the squared differences of its 16-byte columns
// lane by lane and reduces them with the same butterfly as the score kernel,
// then smooths the row with the same window statistics as the zscore
// kernel, and the rows meet for the same band combination.  So this launch
// gives bit for bit the scores and carried state of epikv_score followed by
// epikv_zscore.
#include "epikv_internal.h"

namespace epikv {
namespace {

constexpr int kWaves = kZscoreThreads / 64;
constexpr int kSlice = EPIKV_MAX_WINDOW - 1 + kZscoreTile;

template <int VPW, int U>
__global__ __launch_bounds__(kZscoreThreads) void k_score_tokens(ScoreTokArgs a) {
  __shared__ float xs[kWaves][kSlice];
  __shared__ float vals[EPIKV_MAX_BAND][kZscoreTile];
  __shared__ float carry[EPIKV_MAX_BAND];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.x;
  const int wm1 = a.w - 1;
  const int nvec = a.D >> 3;
  const int n_tok = max(a.n_tok_in[b], 0);
  // The first token of a fresh stream has no predecessor and no sample.
  const bool fresh = n_tok == 0;
  const int c0 = fresh ? 1 : 0;
  const int64_t prior = (int64_t)max(n_tok - 1, 0);
  const int cnt = (int)min((int64_t)wm1, prior);
  const int vstart = wm1 - cnt + c0;
  const int64_t total_out = prior + (a.C - c0);
  const int cnt_out = (int)min((int64_t)wm1, total_out);
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const float al = a.alpha, bl = 1.0f - a.alpha;
  float* x = xs[wave];

  const int rounds = (a.n_band + kWaves - 1) / kWaves;
  for (int rd = 0; rd < rounds; ++rd) {
    const int l = rd * kWaves + wave;
    const bool active = l < a.n_band;
    if (active) {
      const int64_t row = (int64_t)b * a.n_band + l;
      // (the carried EMA value is loaded first: it is only used after the
      // rows, so its latency overlaps theirs)
      const float ema_c = a.ema_in[row];
      for (int k = lane; k < wm1; k += 64) x[k] = a.ring_in[row * wm1 + k];
      // Eq. 1 over the chunk's rows, the previous row in registers
      const uint16_t* rows = a.hidden[l] + (int64_t)b * a.ld_seq;
      const uint16_t* prow = a.h_prev_in + row * a.D;
      u32x4 prev[VPW];
#pragma unroll
      for (int i = 0; i < VPW; ++i) {
        const int v = lane + i * 64;
        prev[i] = (v < nvec && !fresh) ? ld_stream(prow + v * 8) : zero;
      }
      for (int c = 0; c < a.C; c += U) {
        u32x4 cur[U][VPW];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
          for (int i = 0; i < VPW; ++i) {
            const int v = lane + i * 64;
            cur[u][i] = (c + u < a.C && v < nvec)
                            ? ld_stream(rows + (int64_t)(c + u) * a.ld_tok + v * 8)
                            : zero;
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          float acc = 0.f;
#pragma unroll
          for (int i = 0; i < VPW; ++i)
            acc = sqdiff8(cur[u][i], u == 0 ? prev[i] : cur[u - 1][i], acc);
          const float g2 = wave_sum(acc);
          if (lane == 0 && c + u < a.C)
            x[wm1 + c + u] = (fresh && c + u == 0) ? 0.f : sqrtf(g2);
        }
        // (prev: the latest row of the chunk, so after the loop its last)
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (c + u < a.C)
#pragma unroll
            for (int i = 0; i < VPW; ++i) prev[i] = cur[u][i];
      }
      // the chunk's last row is the next call's predecessor (from registers)
      uint16_t* hout = a.h_prev_out + row * a.D;
#pragma unroll
      for (int i = 0; i < VPW; ++i) {
        const int v = lane + i * 64;
        if (v < nvec) *reinterpret_cast<u32x4*>(hout + v * 8) = prev[i];
      }
      if (lane == 0) carry[l] = ema_c;
    }
    __syncthreads();
    if (active) {
      const int row = b * a.n_band + l;
      const int c = lane;
      const bool has = c < a.C && c >= c0;
      float v = 0.f;
      if (a.mode == EPIKV_SMOOTH_EMA) {
        const float xv = has ? x[wm1 + c] : 0.f;
        const float y = ema_scan(xv, has, prior == 0 && c == c0, al, bl, carry[l], lane);
        v = has ? y : 0.f;
        const float y_last = __shfl(y, 63, 64);
        if (lane == 0) a.ema_out[row] = y_last;
      } else {
        if (has) {
          const int j = wm1 + c;
          v = smooth_at(x, 0, max(vstart, j - wm1), j, a.mode, a.eps);
        }
        if (lane == 0) a.ema_out[row] = carry[l];
      }
      vals[l][lane] = v;
      // carried samples: the last min(w-1, samples), right-aligned
      float* ro = a.ring_out + (int64_t)row * wm1;
      for (int k = lane; k < wm1; k += 64) ro[k] = ((wm1 - 1 - k) < cnt_out) ? x[a.C + k] : 0.f;
    }
    __syncthreads();
  }
  if (tid < a.C) {
    const float s = band_combine<kZscoreTile>(vals, tid, a.n_a, a.n_band, a.n_b);
    const int N = a.n_cached[b];
    if (N >= a.C && (int64_t)N <= a.ld_s) a.scores[(int64_t)b * a.ld_s + (N - a.C) + tid] = s;
  }
  if (tid == 0) a.n_tok_out[b] = n_tok + a.C;
}

template <int VPW, int U>
hipError_t launch(const ScoreTokArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_score_tokens<VPW, U>), dim3(a.B), dim3(kZscoreThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_tokens(const ScoreTokArgs& a, hipStream_t s) {
  const int nvec = a.D / 8;
  if (nvec <= 64) return launch<1, 4>(a, s);
  if (nvec <= 128) return launch<2, 2>(a, s);
  if (nvec <= 256) return launch<4, 2>(a, s);
  if (nvec <= 512) return launch<8, 1>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace epikv
