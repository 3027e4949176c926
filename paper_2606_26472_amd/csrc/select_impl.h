// Selection of one sequence, shared by the select kernel and the fused
// select + score launch of the eviction step.
//
// Which positions survive an eviction step (Sec. 3.1, Sec. 3.3, App. D):
// the prefill [0, P), the recency window [N-R, N) and the M = K-P-R best
// positions of [P, N-R), exactly K in ascending order.
//
// Ranking key: the fp32 score mapped to an unsigned integer whose order is
// the ranking (higher score = larger key), with -0 folded onto +0 and every
// NaN mapped to 0, below -inf.  Equal keys rank by lower position.
//
// One 1024-thread workgroup per sequence:
//   1. radix select of the M-th largest key over 11/11/10-bit digits: each
//      pass histograms the keys that match the digits chosen so far (LDS
//      atomics), a block-wide suffix scan finds the digit holding the M-th
//      key.  After three passes the threshold T is exact and `need` says
//      how many keys equal to T are kept;
//   2. the kept positions in order: keys equal to T are ranked by position
//      with a prefix count (the first `need` of them are kept) and a second
//      prefix count gives every kept position its output slot, so keep_idx
//      comes out ascending without a sort.
// For N up to 32 Ki positions thread t keeps the keys of the contiguous
// positions [t*KPT, (t+1)*KPT) in registers for all four sweeps, so step 2
// needs two workgroup-wide scans in total.  Longer sequences re-read the
// scores from global memory (L2) in each sweep and produce the output in
// tiles of 8192 positions staged through LDS (two scans per tile).
#pragma once

#include "epikv_internal.h"

namespace epikv {
namespace select_impl {


constexpr int kWaves = kSelectThreads / 64;
constexpr int kOutPer = 8;                         // long rows: positions per thread per tile
constexpr int kOutTile = kOutPer * kSelectThreads;  // positions per output tile

__device__ __forceinline__ uint32_t rank_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN: lowest
  if (u == 0x80000000u) u = 0u;                     // -0 == +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive scan over the workgroup in thread order.
__device__ __forceinline__ uint32_t block_inclusive_scan(uint32_t v, uint32_t* wsum) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  if (lane == 63) wsum[wave] = v;
  __syncthreads();
  uint32_t add = 0;
  for (int w = 0; w < wave; ++w) add += wsum[w];
  __syncthreads();
  return v + add;
}

// Exclusive rank of this lane's flag among the workgroup's set flags, and
// the workgroup total.
__device__ __forceinline__ uint32_t block_flag_rank(bool flag, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  const uint32_t below = (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wave] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t pre = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t x = wsum[w];
    pre += (w < wave) ? x : 0u;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return pre + below;
}

// Exclusive prefix over the workgroup in thread order, and the total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum,
                                                         uint32_t* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(x, off, 64);
    if (lane >= off) x += t;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t pre = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t y = wsum[w];
    pre += (w < wave) ? y : 0u;
    tot += y;
  }
  __syncthreads();
  *total = tot;
  return pre + x - v;
}

// The digit holding the need-th largest key of a histogram of nb bins in
// LDS (nb a multiple of the workgroup size), and how many keys lie in
// higher digits; both land in *digit / *above.  Thread t owns the bpt bins
// just below nb - t*bpt (descending order), so the inclusive scan counts
// keys whose digit is >= its lowest bin.
__device__ __forceinline__ void find_digit(const uint32_t* hist, int nb, uint32_t need,
                                           uint32_t* wsum, uint32_t* digit, uint32_t* above_out) {
  const int bpt = nb / kSelectThreads;
  const int top = nb - 1 - (int)threadIdx.x * bpt;
  uint32_t local = 0u;
  for (int q = 0; q < bpt; ++q) local += hist[top - q];
  const uint32_t incl = block_inclusive_scan(local, wsum);
  const uint32_t excl = incl - local;
  if (excl < need && need <= incl) {
    uint32_t above = excl;
    int d = top - bpt + 1;
    for (int q = 0; q < bpt; ++q) {
      const uint32_t h = hist[top - q];
      if (above + h >= need) {
        d = top - q;
        break;
      }
      above += h;
    }
    *digit = (uint32_t)d;
    *above_out = above;
  }
}

// KPT > 0: positions [tid*KPT, (tid+1)*KPT) have their keys in registers.
// KPT == 0: keys are recomputed from global memory in every sweep.
template <int KPT>
__device__ __forceinline__ void select_seq(const SelectArgs& a, int b) {
  __shared__ uint32_t hist[2048];
  // staging tile of the long-row output phase (unused by the register path)
  __shared__ uint32_t out_tile[KPT > 0 ? 1 : kOutTile + kOutTile / kOutPer];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t sel_digit, sel_above;
  const int tid = threadIdx.x;
  const int N = a.n_cached[b];
  const int P = a.n_prefix[b];
  const int K = a.K;
  const int R = a.R;
  int32_t* out = a.keep_idx + (int64_t)b * K;

  if (N < a.min_n || (int64_t)N > a.ld_s || P < 0 || (KPT > 0 && N > KPT * kSelectThreads)) {
    if (tid == 0) {
      a.n_keep[b] = -1;
      a.seq_status[b] = EPIKV_SEQ_RANGE;
    }
    return;
  }
  if (N <= K) {
    for (int j = tid; j < N; j += kSelectThreads) out[j] = j;
    if (tid == 0) {
      a.n_keep[b] = N;
      a.seq_status[b] = EPIKV_SEQ_OK;
    }
    return;
  }
  if ((int64_t)P + R >= K) {
    if (tid == 0) {
      a.n_keep[b] = -1;
      a.seq_status[b] = EPIKV_SEQ_BUDGET;
    }
    return;
  }

  const float* s = a.scores + (int64_t)b * a.ld_s;
  const int lo = P, hi = N - R;  // eligible positions [lo, hi)
  constexpr int KR = KPT > 0 ? KPT : 1;
  uint32_t keys[KR];
  const int base = tid * KR;  // first position owned (register path)
  if (KPT > 0) {
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      const int i = base + k;
      keys[k] = (i >= lo && i < hi) ? rank_key(s[i]) : 0u;
    }
  }
  uint32_t prefix = 0u, mask = 0u;
  uint32_t need = (uint32_t)(K - P - R);  // rank (1-based) of the threshold key

  const int shifts[3] = {21, 10, 0};
  const int nbits[3] = {11, 11, 10};
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = shifts[pass];
    const int nb = 1 << nbits[pass];
    const uint32_t dmask = (uint32_t)nb - 1u;
    for (int i = tid; i < nb; i += kSelectThreads) hist[i] = 0u;
    __syncthreads();
    if (KPT > 0) {
#pragma unroll
      for (int k = 0; k < KR; ++k) {
        const int i = base + k;
        if (i >= lo && i < hi && (keys[k] & mask) == prefix)
          atomicAdd(&hist[(keys[k] >> shift) & dmask], 1u);
      }
    } else {
      // kOutPer scores per thread are loaded before any is counted
      for (int i0 = lo + tid; i0 < hi; i0 += kOutPer * kSelectThreads) {
        float v[kOutPer];
#pragma unroll
        for (int u = 0; u < kOutPer; ++u) {
          const int i = i0 + u * kSelectThreads;
          v[u] = i < hi ? s[i] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kOutPer; ++u) {
          const uint32_t key = rank_key(v[u]);
          if (i0 + u * kSelectThreads < hi && (key & mask) == prefix)
            atomicAdd(&hist[(key >> shift) & dmask], 1u);
        }
      }
    }
    __syncthreads();
    find_digit(hist, nb, need, wsum, &sel_digit, &sel_above);
    __syncthreads();
    prefix |= sel_digit << shift;
    mask |= dmask << shift;
    need -= sel_above;
    __syncthreads();
  }

  // need = keys equal to T that are kept, lowest positions first.
  const uint32_t T = prefix;
  uint32_t written = 0u;
  if (KPT > 0) {
    uint32_t n_eq = 0u;
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      const int i = base + k;
      n_eq += (i >= lo && i < hi && keys[k] == T) ? 1u : 0u;
    }
    uint32_t eq_tot;
    uint32_t eq_rank = block_exclusive_scan(n_eq, wsum, &eq_tot);
    uint64_t keep_bits = 0ull;
    uint32_t n_keep_t = 0u;
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      const int i = base + k;
      if (i < N) {
        const bool elig = i >= lo && i < hi;
        bool keep = !elig || keys[k] > T;
        if (elig && keys[k] == T) {
          keep = eq_rank < need;
          ++eq_rank;
        }
        if (keep) {
          keep_bits |= 1ull << k;
          ++n_keep_t;
        }
      }
    }
    uint32_t slot = block_exclusive_scan(n_keep_t, wsum, &written);
#pragma unroll
    for (int k = 0; k < KR; ++k) {
      if ((keep_bits >> k) & 1ull) {
        if (slot < (uint32_t)K) out[slot] = base + k;
        ++slot;
      }
    }
  } else {
    // Tiles of kOutTile positions: read coalesced into LDS (one pad word
    // after every kOutPer, so the strided reads below hit distinct banks),
    // then thread t takes the kOutPer contiguous positions
    // [t*kOutPer, (t+1)*kOutPer) of the tile, so that two workgroup scans
    // per tile rank the keys equal to T and place the kept positions in
    // order.
    float* tile_s = reinterpret_cast<float*>(out_tile);
    uint32_t eq_seen = 0u;
    float nxt[kOutPer];  // the next tile's scores, loaded while this one is ranked
#pragma unroll
    for (int u = 0; u < kOutPer; ++u) {
      const int k = u * kSelectThreads + tid;
      nxt[u] = k < N ? s[k] : 0.f;
    }
    for (int t0 = 0; t0 < N; t0 += kOutTile) {
#pragma unroll
      for (int u = 0; u < kOutPer; ++u) {
        const int k = u * kSelectThreads + tid;
        tile_s[k + k / kOutPer] = nxt[u];
        const int kn = t0 + kOutTile + k;
        nxt[u] = kn < N ? s[kn] : 0.f;
      }
      __syncthreads();
      const int q0 = tid * kOutPer;
      uint32_t key[kOutPer];
      uint32_t n_eq = 0u;
#pragma unroll
      for (int u = 0; u < kOutPer; ++u) {
        const int i = t0 + q0 + u;
        key[u] = rank_key(tile_s[q0 + tid + u]);  // padded: no bank conflicts
        n_eq += (i >= lo && i < hi && key[u] == T) ? 1u : 0u;
      }
      uint32_t eq_tot;
      uint32_t eq_rank = eq_seen + block_exclusive_scan(n_eq, wsum, &eq_tot);
      uint32_t keep_bits = 0u, n_keep_t = 0u;
#pragma unroll
      for (int u = 0; u < kOutPer; ++u) {
        const int i = t0 + q0 + u;
        if (i < N) {
          const bool elig = i >= lo && i < hi;
          bool keep = !elig || key[u] > T;
          if (elig && key[u] == T) {
            keep = eq_rank < need;
            ++eq_rank;
          }
          if (keep) {
            keep_bits |= 1u << u;
            ++n_keep_t;
          }
        }
      }
      uint32_t keep_tot;
      uint32_t slot = written + block_exclusive_scan(n_keep_t, wsum, &keep_tot);
#pragma unroll
      for (int u = 0; u < kOutPer; ++u) {
        if ((keep_bits >> u) & 1u) {
          if (slot < (uint32_t)K) out[slot] = t0 + q0 + u;
          ++slot;
        }
      }
      eq_seen += eq_tot;
      written += keep_tot;
      __syncthreads();  // the tile buffer is refilled next
    }
  }
  if (tid == 0) {
    const bool ok = written == (uint32_t)K;
    a.n_keep[b] = ok ? K : -1;
    a.seq_status[b] = ok ? EPIKV_SEQ_OK : EPIKV_SEQ_RANGE;
  }
}

}  // namespace select_impl
}  // namespace epikv
