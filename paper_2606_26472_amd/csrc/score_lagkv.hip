// KV-vector signals, Sec. 3.3 and Table 1:
//   Lag-KV      x~ = (x - mn) / (mx - mn + eps) per channel, with (mn, mx) the
//               range of the previous chunk at the same (layer, K|V, head,
//               channel), for keys and values;
//   lag-kv-key  the same, keys only;
//   KV-key/val  x~ = x, keys (values) only;
//   v(t, l, kv, h) = population variance of x~ over the head dimension;
//   q(t) = mean over (layer, head) of the sum of v over the used tensors.
// For the lag-normalised signals the chunk's own per-channel range is written
// out as the next chunk's reference; the first chunk of a stream, with no
// previous chunk, is normalised by its own range.
//
// Kernel 1: 256-thread workgroups per (layer, K|V) plane and sequence, each
// streaming its share of the chunk's rows of that plane from the paged pool
// (planes of an unused tensor only zero their partial sums; the first chunk
// of a stream goes to one workgroup, which needs every row for the range).
// Thread i owns 8 channels (one 16-byte column) of a row and loads
// kLagRowsAhead rows (page-table entries first, then the rows) before using
// any; when a row spans whole wavefronts its index, page and address are
// wave-uniform and computed with scalar instructions.  The d/8 lanes of one
// head reduce the variance with DPP row operations (two passes: mean, then
// squared deviations), and per-(token, head) variances go to LDS.  The
// lag-normalised signals are a separate instantiation: it tracks the
// chunk's per-channel range with IEEE minimum/maximum (a NaN propagates, as
// in a plain minimum over the chunk) and multiplies by the reciprocal of the
// previous range.  The workgroup then writes per-token sums over its heads
// to partial[b][plane][c].
// Kernel 2 sums the 2L planes in a fixed order and divides by L*H, and
// combines the shares' channel ranges into the next chunk's reference.
#include "epikv_internal.h"

namespace epikv {
namespace {

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of `width` lanes (8, 16 or 32), every lane of a
// group ending with the same bits: each step adds two values that the
// partner lane adds in the other order.  DPP moves within a row of 16 lanes
// (rotations, half-row mirror, quad permutes) instead of LDS shuffles.
__device__ __forceinline__ float group_sum(float v, int width) {
  if (width == 8) {
    v += dpp<0x141>(v);  // row_half_mirror: lane i + lane 7-i
    v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    return v;
  }
  v += dpp<0x128>(v);    // row_ror:8
  v += dpp<0x124>(v);    // row_ror:4
  v += dpp<0x122>(v);    // row_ror:2
  v += dpp<0x121>(v);    // row_ror:1
  if (width == 32) v += __shfl_xor(v, 16, 64);
  return v;
}

// Channel ranges propagate NaN (IEEE minimum / maximum, one instruction on
// gfx950), as a plain minimum over the chunk does.
__device__ __forceinline__ float nan_min(float a, float b) {
  return __builtin_elementwise_minimum(a, b);
}
__device__ __forceinline__ float nan_max(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

__device__ __forceinline__ void unpack8(u32x4 w, float x[8]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    x[2 * k] = bf16_lo(w[k]);
    x[2 * k + 1] = bf16_hi(w[k]);
  }
}

// WR: a row spans whole wavefronts (at least 64 16-byte columns), so the
// row a wavefront works on, its page and its address are wave-uniform and
// live in scalar registers; the vector units only do the arithmetic.
template <bool LAG, bool WR>
__global__ __launch_bounds__(kScoreThreads) void k_score_lagkv(ScoreLagArgs a) {
  extern __shared__ float lds[];
  const int tid = threadIdx.x;
  const int lk = blockIdx.x;
  const int b = blockIdx.y;
  const int sp = blockIdx.z;                   // which share of the chunk's rows
  const int layer = lk >> 1;
  const int kv = lk & 1;
  const int HD = a.H * a.d;
  const int row_vec = HD >> 3;                 // 16-byte columns per row
  const int rpp = kScoreThreads / row_vec;     // rows per pass
  const int col = tid % row_vec;
  const int ro = WR ? __builtin_amdgcn_readfirstlane(tid / row_vec) : tid / row_vec;
  const int gl = a.d >> 3;                     // lanes per head
  const int head = col / gl;
  const int row_bytes = HD * 2;

  // Per-(head, row) variances, [H][C + 1]: the padding puts the heads of
  // one row, written together, in different banks, and the per-row sums
  // read consecutive rows.  The range combine holds [2][rpp][8][row_vec]:
  // lane = column, so every access is to consecutive words.
  const int vld = a.C + 1;
  float* vbuf = lds;
  float* cmb = lds + a.H * vld;
  float* part = a.partial + ((int64_t)b * 2 * a.L + lk) * a.C;
  if ((kv == 0 && !a.use_k) || (kv == 1 && !a.use_v)) {
    if (sp == 0)
      for (int r = tid; r < a.C; r += kScoreThreads) part[r] = 0.f;
    return;
  }

  const int N = a.n_cached[b];
  const int start = N - a.C;
  const bool seq_ok = start >= 0 && (int64_t)((N - 1) / a.page_size) < a.ld_pt;
  const char* plane = a.base + (int64_t)layer * a.s_layer + (int64_t)kv * a.s_kv;
  const int32_t* pt = a.pt + (int64_t)b * a.ld_pt;
  const int64_t half = (int64_t)a.B * a.L * 2 * HD;
  const int64_t rbase = (((int64_t)b * a.L + layer) * 2 + kv) * HD + col * 8;
  const bool fresh = LAG && a.n_tok_in[b] <= 0;
  // Rows [r_lo, r_hi) of the chunk are this workgroup's.  The first chunk of
  // a stream is normalised by its own range, which needs every row before
  // any variance: one workgroup takes it whole.
  int r_lo = 0, r_hi = 0;
  if (fresh) {
    r_hi = sp == 0 ? a.C : 0;
  } else {
    const int per = ((a.C + a.splits - 1) / a.splits + rpp - 1) / rpp * rpp;
    r_lo = min(a.C, sp * per);
    r_hi = min(a.C, r_lo + per);
  }

  // Page of chunk row r (-1 for none), then the address of this thread's
  // column of the row (nullptr for none).  Split so that a batch of rows
  // issues all its page-table loads before any row load waits on one.
  // (page sizes that are powers of two -- the usual case -- divide by a
  // shift: a division costs some thirty instructions per row and lane)
  auto row_page = [&](int r) -> int {
    if (!seq_ok || r >= r_hi) return -1;
    const int pos = start + r;
    return pt[a.page_shift >= 0 ? pos >> a.page_shift : pos / a.page_size];
  };
  auto row_ptr = [&](int r, int pg) -> const char* {
    if (pg < 0 || pg >= a.n_pages) return nullptr;
    const int pos = start + r;
    const int slot = a.page_shift >= 0 ? pos & (a.page_size - 1) : pos % a.page_size;
    return plane + (int64_t)pg * a.s_page + (int64_t)slot * row_bytes + col * 16;
  };

  float mn[8], mx[8], cmn[8], cmx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    cmn[e] = __builtin_huge_valf();
    cmx[e] = -__builtin_huge_valf();
  }

  // Combine the per-thread ranges of the rpp threads sharing a column.
  auto combine = [&]() {
    if (ro < rpp) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        cmb[(ro * 8 + e) * row_vec + col] = cmn[e];
        cmb[((rpp + ro) * 8 + e) * row_vec + col] = cmx[e];
      }
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float lo = cmb[e * row_vec + col], hi = cmb[(rpp * 8 + e) * row_vec + col];
      for (int q = 1; q < rpp; ++q) {
        lo = nan_min(lo, cmb[(q * 8 + e) * row_vec + col]);
        hi = nan_max(hi, cmb[((rpp + q) * 8 + e) * row_vec + col]);
      }
      cmn[e] = lo;
      cmx[e] = hi;
    }
    __syncthreads();
  };

  if (fresh) {
    for (int r0 = r_lo + ro; r0 < r_hi && ro < rpp; r0 += kLagRowsAhead * rpp) {
      u32x4 raw[kLagRowsAhead];
      bool got[kLagRowsAhead];
      int pg[kLagRowsAhead];
#pragma unroll
      for (int u = 0; u < kLagRowsAhead; ++u) pg[u] = row_page(r0 + u * rpp);
#pragma unroll
      for (int u = 0; u < kLagRowsAhead; ++u) {
        const char* p = row_ptr(r0 + u * rpp, pg[u]);
        got[u] = p != nullptr;
        if (got[u]) raw[u] = ld_stream(p);
      }
#pragma unroll
      for (int u = 0; u < kLagRowsAhead; ++u) {
        if (!got[u]) continue;
        float x[8];
        unpack8(raw[u], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          cmn[e] = nan_min(cmn[e], x[e]);
          cmx[e] = nan_max(cmx[e], x[e]);
        }
      }
    }
    combine();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = cmn[e];
      mx[e] = cmx[e];
    }
  } else if (LAG) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = a.range_in[rbase + e];
      mx[e] = a.range_in[half + rbase + e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = 0.f;
      mx[e] = 0.f;
    }
  }
  float den[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) den[e] = 1.0f / (mx[e] - mn[e] + a.eps);

  const float inv_d = 1.0f / (float)a.d;
  // All threads run the same trip count so that the head-group shuffles see
  // every lane of the group.
  // kLagRowsAhead rows per thread are loaded before any is used, so each
  // thread has that many 16-byte loads in flight.
  const int trips = (r_hi - r_lo + rpp - 1) / rpp;
  for (int it0 = 0; it0 < trips; it0 += kLagRowsAhead) {
    u32x4 raw[kLagRowsAhead];
    bool got[kLagRowsAhead];
    int pg[kLagRowsAhead];
#pragma unroll
    for (int u = 0; u < kLagRowsAhead; ++u) {
      const int r = r_lo + (it0 + u) * rpp + ro;
      pg[u] = ro < rpp ? row_page(r) : -1;
    }
#pragma unroll
    for (int u = 0; u < kLagRowsAhead; ++u) {
      const char* p = row_ptr(r_lo + (it0 + u) * rpp + ro, pg[u]);
      got[u] = p != nullptr;
      if (got[u]) raw[u] = ld_stream(p);
    }
#pragma unroll
    for (int u = 0; u < kLagRowsAhead; ++u) {
      const int r = r_lo + (it0 + u) * rpp + ro;
      const bool live = ro < rpp && r < r_hi;
      float x[8];
      if (got[u]) {
        unpack8(raw[u], x);
        if (LAG) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            cmn[e] = nan_min(cmn[e], x[e]);
            cmx[e] = nan_max(cmx[e], x[e]);
            x[e] = (x[e] - mn[e]) * den[e];
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = 0.f;
      }
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s += x[e];
      const float mu = group_sum(s, gl) * inv_d;
      float q = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float dlt = x[e] - mu;
        q = fmaf(dlt, dlt, q);
      }
      const float var = group_sum(q, gl) * inv_d;
      if (live && (col % gl) == 0) vbuf[head * vld + r] = got[u] ? var : 0.f;
    }
  }
  __syncthreads();
  if (LAG) {
    // this share's range of the chunk; the reduce kernel combines the shares
    combine();
    if (ro == 0) {
      float* pr = a.prange + (int64_t)sp * 2 * half;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pr[rbase + e] = cmn[e];
        pr[half + rbase + e] = cmx[e];
      }
    }
  }
  for (int r = r_lo + tid; r < r_hi; r += kScoreThreads) {
    float s = 0.f;
    for (int h = 0; h < a.H; ++h) s += vbuf[h * vld + r];
    part[r] = s;
  }
}

// Blocks [0, tok_blocks) of each sequence: q(t) = the 2L plane sums of
// token t in a fixed order, times 1/(L*H).  The remaining blocks (lag
// signals): each channel's range over the chunk = the min and max of the
// shares' partial ranges, in a fixed order.
__global__ __launch_bounds__(kScoreThreads) void k_lag_reduce(LagReduceArgs a) {
  const int b = blockIdx.y;
  const int tok_blocks = (a.C + kScoreThreads - 1) / kScoreThreads;
  if ((int)blockIdx.x < tok_blocks) {
    const int c = blockIdx.x * kScoreThreads + threadIdx.x;
    if (c >= a.C) return;
    const float* p = a.partial + (int64_t)b * a.n_lk * a.C + c;
    float s = 0.f;
#pragma unroll 8
    for (int lk = 0; lk < a.n_lk; ++lk) s += p[(int64_t)lk * a.C];
    a.sig[(int64_t)b * a.C + c] = s * a.inv_count;
    return;
  }
  const int i = ((int)blockIdx.x - tok_blocks) * kScoreThreads + threadIdx.x;
  if (i >= a.n_chan) return;
  const int64_t half = (int64_t)a.B * a.n_chan;
  const int64_t o = (int64_t)b * a.n_chan + i;
  const int kv = (i / (a.n_chan / a.n_lk)) & 1;
  float lo = 0.f, hi = 0.f;  // planes of an unused tensor carry no range
  if (kv == 0 ? a.use_k : a.use_v) {
    lo = a.prange[o];
    hi = a.prange[half + o];
    for (int sp = 1; sp < a.splits; ++sp) {
      lo = nan_min(lo, a.prange[sp * 2 * half + o]);
      hi = nan_max(hi, a.prange[sp * 2 * half + half + o]);
    }
  }
  a.range_out[o] = lo;
  a.range_out[half + o] = hi;
}

}  // namespace

size_t lagkv_lds_bytes(int C, int H, int d) {
  const int HD = H * d;
  const int rpp = kScoreThreads / (HD / 8);
  return (size_t)(C + 1) * H * 4 + (size_t)2 * rpp * HD * 4;
}

hipError_t launch_score_lagkv(const ScoreLagArgs& a, const LagReduceArgs& r, hipStream_t s) {
  const size_t lds = lagkv_lds_bytes(a.C, a.H, a.d);
  const dim3 grid(2 * a.L, a.B, a.splits);
  const bool wr = a.H * a.d / 8 >= 64;
  if (a.lag && wr)
    hipLaunchKernelGGL((k_score_lagkv<true, true>), grid, dim3(kScoreThreads), lds, s, a);
  else if (a.lag)
    hipLaunchKernelGGL((k_score_lagkv<true, false>), grid, dim3(kScoreThreads), lds, s, a);
  else if (wr)
    hipLaunchKernelGGL((k_score_lagkv<false, true>), grid, dim3(kScoreThreads), lds, s, a);
  else
    hipLaunchKernelGGL((k_score_lagkv<false, false>), grid, dim3(kScoreThreads), lds, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tok_blocks = (r.C + kScoreThreads - 1) / kScoreThreads;
  const int rng_blocks = r.lag ? (r.n_chan + kScoreThreads - 1) / kScoreThreads : 0;
  hipLaunchKernelGGL(k_lag_reduce, dim3(tok_blocks + rng_blocks, r.B), dim3(kScoreThreads), 0, s,
                     r);
  return hipGetLastError();
}

}  // namespace epikv
