// Order-preserving rebuild of the paged cache (App. H): for every kept slot
// j of sequence b, copy the K and V rows of position keep_idx[b][j] at every
// layer into slot j of the destination pages.  A token's row at one
// (layer, K|V) holds all KV heads (n_kv_heads * head_dim bf16, 2 KiB for
// 8 x 128), so the copy is a gather of 2 KiB rows: pure HBM streaming.
//
// Three kernels:
//   order    one workgroup ranks every (sequence, destination page) by its
//            page id, i.e. by physical address: the used pages first, in
//            ascending page id, then the unused ones.  Writing the rebuilt
//            cache in that order streams the writes through memory the way
//            a plain copy does even when the allocator scattered the
//            destination pages (measured on MI355X: 5.2 -> 6.2 TB/s for
//            randomly placed pages; a cache rebuilt into one run of pages
//            per sequence is already in that order).  When the used ids
//            already rise in logical order the ranks follow from two prefix
//            counts; otherwise the used ids are marked in an LDS bitmap over
//            their range, and a page's rank is the number of marked ids
//            below it.  A range too wide for the bitmap, or a page id used
//            twice, keeps the logical order (sequence, page).
//   resolve  one thread per slot of the budget's pages turns keep_idx and
//            the two page tables into the byte offsets of the source and
//            destination rows inside a plane, a 16-byte record written at
//            position rank(sequence, page) * page_size + slot (slots past
//            n_keep, and rows out of range, get an empty record), and copies
//            the slot's score and position;
//   gather   a 64-thread workgroup copies 64 16-byte columns (1 KiB: half a
//            2 KiB row) of one record in one (layer, K|V) plane: it reads the
//            record with a scalar load and streams the columns, one load
//            and one store per lane, non-temporal (each byte is touched
//            once).  Workgroups walk the records in order, so consecutive
//            workgroups write consecutive addresses.  (Measured on the
//            32 x 4096-row rebuild: 1 KiB workgroups 2% faster than four
//            2 KiB rows per 256-thread workgroup.)
#include "epikv_internal.h"

namespace epikv {
namespace {

constexpr int kOrderThreads = 1024;
constexpr int kOrderWords = 16384;  // bitmap words: page ids spanning up to 512 Ki

// Exclusive prefix sum of one value per thread over the workgroup, in
// thread order; *total gets the sum.  (wsum: kOrderThreads / 64 words.)
__device__ uint32_t block_exclusive_sum(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(x, off, 64);
    if (lane >= off) x += t;
  }
  __syncthreads();
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t base = 0, tot = 0;
  for (int w = 0; w < kOrderThreads / 64; ++w) {
    base += w < wave ? wsum[w] : 0u;
    tot += wsum[w];
  }
  *total = tot;
  return base + x - v;
}

__global__ __launch_bounds__(kOrderThreads) void k_compact_order(CompactArgs a) {
  __shared__ uint32_t bits[kOrderWords];
  __shared__ uint32_t pre[kOrderThreads];  // per-thread prefix of the bitmap chunks
  __shared__ uint32_t wsum[kOrderThreads / 64];
  __shared__ int s_lo, s_hi, s_logical, s_unsorted;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int n_pg = a.n_pg;
  const int64_t N = (int64_t)a.B * n_pg;
  int32_t* rank = a.rank;

  // Destination page of entry e = b * n_pg + m, or -1 if the page is not
  // used (past n_keep, a refused sequence) or out of range.
  auto page_of = [&](int64_t e) -> int {
    const int b = (int)(e / n_pg);
    const int m = (int)(e - (int64_t)b * n_pg);
    const int nk = min(a.n_keep[b], a.K);
    if (nk <= 0 || (int64_t)m * a.page_size >= nk || m >= a.ld_dst_pt) return -1;
    const int pg = a.dst_pt[(int64_t)b * a.ld_dst_pt + m];
    return (pg >= 0 && pg < a.d_npages) ? pg : -1;
  };

  // Each thread takes a contiguous range of entries: its used and unused
  // counts, and whether its used page ids rise strictly.
  const int64_t per = (N + kOrderThreads - 1) / kOrderThreads;
  const int64_t e0 = (int64_t)tid * per;
  const int64_t e1 = min(N, e0 + per);
  uint32_t n_use = 0, n_bad = 0;
  int first = -1, last = -1;
  bool rising = true;
  for (int64_t e = e0; e < e1; ++e) {
    const int pg = page_of(e);
    if (pg < 0) {
      ++n_bad;
    } else {
      if (last >= 0 && pg <= last) rising = false;
      if (first < 0) first = pg;
      last = pg;
      ++n_use;
    }
  }
  if (tid == 0) {
    s_lo = INT32_MAX;
    s_hi = -1;
    s_logical = 0;
    s_unsorted = 0;
  }
  uint32_t n_used, n_unused;
  uint32_t used_before = block_exclusive_sum(n_use, wsum, &n_used);
  uint32_t bad_before = block_exclusive_sum(n_bad, wsum, &n_unused);
  // The used page ids rise strictly over all entries iff every thread's do
  // and each thread's first exceeds the last of the threads before it.
  {
    int mx = last;  // inclusive prefix maximum of the threads' last ids
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int t = __shfl_up(mx, off, 64);
      if (lane >= off) mx = max(mx, t);
    }
    __syncthreads();
    if (lane == 63) wsum[tid >> 6] = (uint32_t)(mx + 1);
    __syncthreads();
    int before = __shfl_up(mx, 1, 64);
    if (lane == 0) before = -1;
    for (int w = 0; w < (tid >> 6); ++w) before = max(before, (int)wsum[w] - 1);
    if (!rising || (first >= 0 && first <= before)) atomicOr(&s_unsorted, 1);
    __syncthreads();
  }

  // Rising: a used page's rank (the number of used ids below it) is the
  // number of used entries before it; the unused entries follow, in
  // logical order.
  if (!s_unsorted) {
    for (int64_t e = e0; e < e1; ++e)
      rank[e] = page_of(e) >= 0 ? (int32_t)used_before++ : (int32_t)(n_used + bad_before++);
    return;
  }

  // Otherwise the ranks come from a bitmap of the used ids over their range.
  // 1. the range of the used page ids
  int lo = INT32_MAX, hi = -1;
  for (int64_t e = tid; e < N; e += kOrderThreads) {
    const int pg = page_of(e);
    if (pg >= 0) {
      lo = min(lo, pg);
      hi = max(hi, pg);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, __shfl_xor(lo, off, 64));
    hi = max(hi, __shfl_xor(hi, off, 64));
  }
  if (lane == 0) {
    atomicMin(&s_lo, lo);
    atomicMax(&s_hi, hi);
  }
  __syncthreads();
  lo = s_lo;
  hi = s_hi;
  const int64_t span = hi >= lo ? (int64_t)hi - lo + 1 : 0;
  const int words = (int)((span + 31) / 32);
  bool logical = span == 0 || words > kOrderWords;

  // 2. mark the used page ids (a page used twice keeps the logical order)
  if (!logical) {
    for (int w = tid; w < words; w += kOrderThreads) bits[w] = 0u;
    __syncthreads();
    for (int64_t e = tid; e < N; e += kOrderThreads) {
      const int pg = page_of(e);
      if (pg >= 0) {
        const uint32_t bit = 1u << ((pg - lo) & 31);
        if (atomicOr(&bits[(pg - lo) >> 5], bit) & bit) s_logical = 1;
      }
    }
    __syncthreads();
    logical = s_logical != 0;
  }

  // 3. ranks: a used page's is the number of used ids below it; the
  //    unused entries follow, in logical order
  const int chunk = (words + kOrderThreads - 1) / kOrderThreads;  // bitmap words per thread
  if (!logical) {
    uint32_t c = 0;
    for (int k = 0; k < chunk; ++k) {
      const int w = tid * chunk + k;
      if (w < words) c += __popc(bits[w]);
    }
    uint32_t tot;
    pre[tid] = block_exclusive_sum(c, wsum, &tot);
    __syncthreads();
  }
  for (int64_t e = e0; e < e1; ++e) {
    int32_t r;
    if (logical) {
      r = (int32_t)e;
    } else {
      const int pg = page_of(e);
      if (pg >= 0) {
        const int i = pg - lo;
        const int w = i >> 5;
        const int owner = w / chunk;
        uint32_t below = pre[owner];
        for (int k = owner * chunk; k < w; ++k) below += __popc(bits[k]);
        below += __popc(bits[w] & ((1u << (i & 31)) - 1u));
        r = (int32_t)below;
      } else {
        r = (int32_t)(n_used + bad_before++);
      }
    }
    rank[e] = r;
  }
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_resolve(CompactArgs a) {
  const int j = blockIdx.x * kCompactThreads + threadIdx.x;
  const int b = blockIdx.y;
  const int slots = a.n_pg * a.page_size;  // slots of the budget's pages
  if (j >= slots) return;
  const int m = j / a.page_size;
  const int slot_in = j - m * a.page_size;
  // A caller's n_keep above K is clamped so keep_idx is never read past the
  // sequence's row; n_keep < 0: sequence untouched.
  const int nk = min(a.n_keep[b], a.K);
  int64_t so = -1, dso = -1;
  int idx = -1;
  bool bad = false;
  if (j < nk) {
    idx = a.keep_idx[(int64_t)b * a.K + j];
    if (idx >= 0) {
      const int sp = idx / a.page_size;
      const int slot = idx - sp * a.page_size;
      if ((int64_t)sp < a.ld_src_pt) {
        const int pg = a.src_pt[(int64_t)b * a.ld_src_pt + sp];
        if (pg >= 0 && pg < a.s_npages) so = (int64_t)pg * a.s_page + (int64_t)slot * a.row_bytes;
      }
    }
    if ((int64_t)m < a.ld_dst_pt) {
      const int pg = a.dst_pt[(int64_t)b * a.ld_dst_pt + m];
      if (pg >= 0 && pg < a.d_npages) dso = (int64_t)pg * a.d_page + (int64_t)slot_in * a.row_bytes;
    }
    bad = so < 0 || dso < 0;
  }
  const bool ok = j < nk && !bad;
  const int64_t pos = (int64_t)a.rank[(int64_t)b * a.n_pg + m] * a.page_size + slot_in;
  int64_t* rec = a.offsets + 2 * pos;
  rec[0] = ok ? so : -1;
  rec[1] = ok ? dso : -1;
  if (bad) {
    if (a.seq_status) a.seq_status[b] = EPIKV_SEQ_RANGE;
    return;
  }
  if (ok && (int64_t)idx < a.ld_s && (int64_t)j < a.ld_s) {
    const int64_t si = (int64_t)b * a.ld_s + idx;
    const int64_t di = (int64_t)b * a.ld_s + j;
    if (a.dst_scores) a.dst_scores[di] = a.src_scores[si];
    if (a.dst_pos) a.dst_pos[di] = a.src_pos[si];
  }
}

// Workgroup x (linear over blockIdx.z, blockIdx.x): record x / units, its
// columns [64 u, 64 u + 64) with u = x % units, in plane blockIdx.y.  The
// record is wave-uniform (a scalar load); lanes past the row's columns idle.
__global__ __launch_bounds__(64) void k_compact(CompactArgs a, int64_t total) {
  const int lane = threadIdx.x;
  const int64_t x = (int64_t)blockIdx.z * gridDim.x + blockIdx.x;
  if (x >= total) return;
  const int64_t r = x / a.units;
  const int u = (int)(x - r * a.units);
  const int64_t* rec = a.offsets + 2 * r;
  const int64_t s0 = rec[0];
  const int64_t d0 = rec[1];
  if (s0 < 0) return;
  const int c = u * 64 + lane;
  if (c >= (a.row_bytes >> 4)) return;
  const int pl = blockIdx.y;
  const char* sb = a.src + (int64_t)(pl >> 1) * a.s_layer + (int64_t)(pl & 1) * a.s_kv + s0;
  char* db = a.dst + (int64_t)(pl >> 1) * a.d_layer + (int64_t)(pl & 1) * a.d_kv + d0;
  st_stream(db + (int64_t)c * 16, ld_stream(sb + (int64_t)c * 16));
}

}  // namespace

hipError_t launch_compact(const CompactArgs& args, hipStream_t s) {
  CompactArgs a = args;
  a.units = ((a.row_bytes >> 4) + 63) / 64;
  hipLaunchKernelGGL(k_compact_order, dim3(1), dim3(kOrderThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int slots = a.n_pg * a.page_size;
  hipLaunchKernelGGL(k_compact_resolve, dim3((slots + kCompactThreads - 1) / kCompactThreads, a.B),
                     dim3(kCompactThreads), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // workgroups (record, column group) in order, the linear index split as
  // blockIdx.z * gridDim.x + blockIdx.x
  const int64_t total = (int64_t)a.B * slots * a.units;
  const int64_t gx = total < kCompactGridX ? total : kCompactGridX;
  const int64_t gz = (total + gx - 1) / gx;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)gx, a.n_lk, (unsigned)gz), dim3(64), 0, s, a,
                     total);
  return hipGetLastError();
}

}  // namespace epikv
