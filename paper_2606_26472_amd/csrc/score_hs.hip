// Band-layer hidden-state change, Sec. 3.2 Eq. 1:
//   g_l(t) = || h_l(t) - h_l(t-1) ||_2
// for every band layer l and every new token t of every sequence.
//
// Rows of up to 4096 elements (the usual case): one wavefront walks a
// segment of consecutive tokens of one (sequence, layer).  Lane l owns the
// 16-byte columns l, l+64, ... of the bf16 row, keeps the previous token's
// columns in registers and streams U rows ahead, so each hidden row is read
// from HBM once, plus one predecessor row per segment.  Squared differences
// are accumulated in fp32 per lane and reduced with a fixed butterfly: no LDS
// and no barrier, and the result is deterministic.
//
// Wider rows: one 256-thread workgroup per segment, the four wavefronts'
// partial sums combined through LDS in a fixed order.
#include "score_hs_impl.h"

namespace epikv {
namespace {

template <int VPT, int U>
__global__ __launch_bounds__(kScoreThreads) void k_score_hs(ScoreHsArgs a) {
  __shared__ float red[kScoreThreads / 64][U];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int seg = blockIdx.x;
  const int l = blockIdx.y;
  const int b = blockIdx.z;
  const int c0 = seg * a.seg_len;
  const int c1 = min(c0 + a.seg_len, a.C);
  const int nvec = a.D >> 3;
  const u32x4 zero = {0u, 0u, 0u, 0u};

  const uint16_t* rows = a.hidden[l] + (int64_t)b * a.ld_seq;
  const bool fresh = (c0 == 0) && (a.n_tok_in[b] <= 0);
  const uint16_t* prow =
      (c0 == 0) ? a.h_prev_in + ((int64_t)b * a.n_band + l) * a.D
                : rows + (int64_t)(c0 - 1) * a.ld_tok;

  u32x4 prev[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int v = tid + i * kScoreThreads;
    prev[i] = (v < nvec && !fresh) ? ld_stream(prow + v * 8) : zero;
  }

  for (int c = c0; c < c1; c += U) {
    u32x4 cur[U][VPT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) {
        const int v = tid + i * kScoreThreads;
        cur[u][i] = (c + u < c1 && v < nvec)
                        ? ld_stream(rows + (int64_t)(c + u) * a.ld_tok + v * 8)
                        : zero;
      }
    }
    float part[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < VPT; ++i)
        acc = sqdiff8(cur[u][i], u == 0 ? prev[i] : cur[u - 1][i], acc);
      part[u] = wave_sum(acc);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) prev[i] = cur[U - 1][i];
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) red[wave][u] = part[u];
    }
    __syncthreads();
    if (tid < U && c + tid < c1) {
      const float g2 = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
      const bool no_sample = fresh && (c + tid == 0);
      a.sig[((int64_t)l * a.B + b) * a.C + c + tid] = no_sample ? 0.f : sqrtf(g2);
    }
    __syncthreads();
  }

  // The segment holding the chunk's last token hands that row on as the
  // predecessor of the next call.
  if (c1 == a.C && c1 > c0) {
    const uint16_t* last = rows + (int64_t)(a.C - 1) * a.ld_tok;
    uint16_t* out = a.h_prev_out + ((int64_t)b * a.n_band + l) * a.D;
    for (int v = tid; v < nvec; v += kScoreThreads)
      *reinterpret_cast<u32x4*>(out + v * 8) = *reinterpret_cast<const u32x4*>(last + v * 8);
  }
}

template <int VPW, int U>
__global__ __launch_bounds__(kScoreThreads) void k_score_hs_wave(ScoreHsArgs a) {
  const int unit = blockIdx.x * (kScoreThreads / 64) + (threadIdx.x >> 6);
  score_impl::score_hs_unit<VPW, U>(a, unit, threadIdx.x & 63);
}

template <int VPW, int U>
hipError_t launch_wave(const ScoreHsArgs& a, hipStream_t s) {
  const int64_t units = score_impl::wave_units(a);
  const int per = kScoreThreads / 64;
  hipLaunchKernelGGL((k_score_hs_wave<VPW, U>), dim3((unsigned)((units + per - 1) / per)),
                     dim3(kScoreThreads), 0, s, a);
  return hipGetLastError();
}

template <int VPT, int U>
hipError_t launch(const ScoreHsArgs& a, hipStream_t s) {
  dim3 grid((a.C + a.seg_len - 1) / a.seg_len, a.n_band, a.B);
  hipLaunchKernelGGL((k_score_hs<VPT, U>), grid, dim3(kScoreThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_hs(const ScoreHsArgs& a, hipStream_t s) {
  const int nvec = a.D / 8;
  if (nvec <= 64 * 8) {
    ScoreHsArgs w = a;
    w.seg_len = score_impl::wave_seg_len(a);
    if (nvec <= 64) return launch_wave<1, 8>(w, s);
    if (nvec <= 128) return launch_wave<2, 8>(w, s);
    if (nvec <= 256) return launch_wave<4, 4>(w, s);
    return launch_wave<8, 2>(w, s);
  }
  const int vpt = (nvec + kScoreThreads - 1) / kScoreThreads;
  if (vpt <= 4) return launch<4, 4>(a, s);
  return launch<8, 2>(a, s);
}

}  // namespace epikv
