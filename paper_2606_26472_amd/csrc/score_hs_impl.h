// Eq. 1 for one (sequence, band layer, segment of tokens) on one wavefront,
// shared by the score kernel and the fused select + score launch of the
// eviction step (both must give the same bits).
#pragma once

#include "epikv_internal.h"

namespace epikv {
namespace score_impl {

// Wavefront variant for rows of at most 64*8*8 = 4096 elements: one
// wavefront owns one (sequence, layer, segment); lane l holds the 16-byte
// columns l, l+64, ... of the row, the previous row stays in registers and
// the squared differences are reduced with the wavefront butterfly alone (no
// LDS, no barrier), so any number of units can share a workgroup.
template <int VPW, int U>
__device__ __forceinline__ void score_hs_unit(const ScoreHsArgs& a, int unit, int lane) {
  const int n_seg = (a.C + a.seg_len - 1) / a.seg_len;
  const int seg = unit % n_seg;
  const int rest = unit / n_seg;
  const int l = rest % a.n_band;
  const int b = rest / a.n_band;
  if (b >= a.B) return;
  const int c0 = seg * a.seg_len;
  const int c1 = min(c0 + a.seg_len, a.C);
  const int nvec = a.D >> 3;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const uint16_t* rows = a.hidden[l] + (int64_t)b * a.ld_seq;
  const bool fresh = (c0 == 0) && (a.n_tok_in[b] <= 0);
  const uint16_t* prow =
      (c0 == 0) ? a.h_prev_in + ((int64_t)b * a.n_band + l) * a.D
                : rows + (int64_t)(c0 - 1) * a.ld_tok;
  u32x4 prev[VPW];
#pragma unroll
  for (int i = 0; i < VPW; ++i) {
    const int v = lane + i * 64;
    prev[i] = (v < nvec && !fresh) ? ld_stream(prow + v * 8) : zero;
  }
  float* out = a.sig + ((int64_t)l * a.B + b) * a.C;
  for (int c = c0; c < c1; c += U) {
    u32x4 cur[U][VPW];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int i = 0; i < VPW; ++i) {
        const int v = lane + i * 64;
        cur[u][i] = (c + u < c1 && v < nvec)
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
      if (lane == 0 && c + u < c1) {
        const bool no_sample = fresh && (c + u == 0);
        out[c + u] = no_sample ? 0.f : sqrtf(g2);
      }
    }
#pragma unroll
    for (int i = 0; i < VPW; ++i) prev[i] = cur[U - 1][i];
  }
  if (c1 == a.C && c1 > c0) {
    const uint16_t* last = rows + (int64_t)(a.C - 1) * a.ld_tok;
    uint16_t* dst = a.h_prev_out + ((int64_t)b * a.n_band + l) * a.D;
    for (int v = lane; v < nvec; v += 64)
      *reinterpret_cast<u32x4*>(dst + v * 8) = *reinterpret_cast<const u32x4*>(last + v * 8);
  }
}

// Longest segment (fewest re-read predecessor rows) that still gives about
// kScoreWavesWanted wavefronts; short chunks and small batches split down
// to 4 tokens per wavefront.
inline int wave_seg_len(const ScoreHsArgs& a) {
  int seg = kScoreSegWave;
  while (seg > 4 && (int64_t)((a.C + seg - 1) / seg) * a.n_band * a.B < kScoreWavesWanted) seg >>= 1;
  return seg;
}

__host__ __device__ inline int64_t wave_units(const ScoreHsArgs& a) {
  return (int64_t)((a.C + a.seg_len - 1) / a.seg_len) * a.n_band * a.B;
}

}  // namespace score_impl
}  // namespace epikv
