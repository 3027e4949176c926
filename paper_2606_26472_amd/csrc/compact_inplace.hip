// Order-preserving rebuild of the cache inside the sequence's own pages: the
// move-minimising form of the App. H rebuild.  Slot j of sequence b receives
// the row of position keep_idx[b][j]; keep_idx is strictly ascending, so
// keep_idx[j] >= j and every row only moves towards the front.  Slots in
// front of the first hole (keep_idx[j] == j) already hold their row and are
// not touched, nor is anything at or past n_keep.
//
// Two kernels:
//   check  one 1024-thread workgroup per sequence verifies that keep_idx is
//          strictly ascending and that every page it reaches exists, writes
//          the byte offsets of each moved row (source and destination, inside
//          a plane) to the workspace together with the first hole, and moves
//          the scores and positions.  A sequence that fails the check is left
//          untouched and flagged RANGE.
//   move   one wavefront per (sequence, plane, column slice) walks the moved
//          slots in ascending order, a tile of T rows at a time (16 to 256,
//          deeper when there are few walks): it loads the tile's source rows,
//          waits until every load has returned, then stores them.  A store
//          to slot j can only overwrite a row that a slot <= j reads; slots
//          of this tile have read theirs, and slots of later tiles read rows
//          past the end of this tile (their sources are >= their own slots).
//          So one wavefront per column slice moves its bytes without any
//          barrier or second copy, and different slices, planes and
//          sequences touch disjoint bytes.  With 1 KiB slices the walk is
//          pipelined: the next tile's loads are in flight while this tile
//          is stored (they read past every slot written so far).
//
// With page remapping (epikv_compact_remap) the check kernel also rewrites
// the page table so that whole retained pages change places instead of being
// copied; the walk then skips their slots, and the ordering argument above
// still holds for every row that moves (see remap_pages).
#include "epikv_internal.h"

namespace epikv {
namespace {

// Every memory operation issued so far has completed: loaded values are in
// registers and earlier stores are done.  The builtin (rather than inline
// assembly) lets the compiler see that nothing is outstanding afterwards, so
// it adds no waits of its own between the stores that follow; the empty asm
// statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void wait_vmem() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int64_t shfl64(int64_t v, int src) {
  const int lo = __shfl((int)(uint32_t)(uint64_t)v, src);
  const int hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Exclusive rank of this thread's flag among the workgroup's set flags (in
// thread order), and the workgroup total.
__device__ __forceinline__ int flag_rank(bool flag, int* wsum, int* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  if (lane == 0) wsum[wave] = __popcll(m);
  __syncthreads();
  int pre = 0, tot = 0;
  for (int w = 0; w < kInplaceThreads / 64; ++w) {
    const int x = wsum[w];
    pre += (w < wave) ? x : 0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return pre + __popcll(m & ((1ull << lane) - 1ull));
}

// Index of `v` in the strictly ascending keep[0, n), or -1.
__device__ __forceinline__ int find_kept(const int32_t* keep, int n, int64_t v) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (keep[mid] < v) lo = mid + 1; else hi = mid;
  }
  return (lo < n && keep[lo] == v) ? lo : -1;
}

// Whole-page retention.  A destination page m (a full page of the rebuilt
// sequence) whose slots receive, in order, all rows of one source page p > m
// is not copied: the table entry m takes p's page.  The pages of such
// destinations that are not themselves such sources are released and go,
// k-th to k-th in ascending order, to the sources that are not themselves
// destinations, so the row stays a permutation of the sequence's pages.  A
// released page (that of m) then only receives rows at slots of a later
// page than m, after every slot that reads it in the front-to-back walk.
//
// Runs inside the check kernel once keep_idx is known to be valid: rewrites
// the destination half of the offset records of the moved slots, drops the
// records of remapped pages (their rows do not move) and then rewrites the
// table.  Per sequence, in the workspace, indexed by destination page:
//   src[m]  p if m is remapped, else -1
//   npg[m]  the page slot m*page_size.. writes to (remapped: the table value)
//   give[m] the rank, then the page, handed to position src[m] when that
//           position is not a destination itself, else -1
// and by rank: rel[k] the k-th released page.
__device__ void remap_pages(const InplaceArgs& a, int b, const int32_t* keep, const int32_t* pt,
                            int nk, int hole, int64_t* rec) {
  __shared__ int s_sum[kInplaceThreads / 64];
  const int tid = threadIdx.x;
  const int ps = a.page_size;
  const int npd = nk / ps;                // full destination pages
  const int ndp = (nk + ps - 1) / ps;     // destination pages
  const int m0 = hole / ps;               // the leading run's pages stay
  int32_t* src = a.remap_ws + (int64_t)b * 4 * a.n_pg;
  int32_t* npg = src + a.n_pg;
  int32_t* give = npg + a.n_pg;
  int32_t* rel = give + a.n_pg;

  for (int m = m0 + tid; m < ndp; m += kInplaceThreads) {
    int p = -1;
    if (m < npd) {
      const int k0 = keep[m * ps];
      const int k1 = keep[m * ps + ps - 1];
      // keep is strictly ascending, so a span of ps - 1 means consecutive
      if (k0 % ps == 0 && k0 > m * ps && k1 - k0 == ps - 1) p = k0 / ps;
    }
    src[m] = p;
    npg[m] = pt[p >= 0 ? p : m];
    give[m] = -1;
  }
  wait_vmem();
  __syncthreads();

  int n_rel = 0, n_give = 0;
  for (int t0 = m0; t0 < npd; t0 += kInplaceThreads) {
    const int m = t0 + tid;
    const int p = m < npd ? src[m] : -1;
    bool released = false, gives = false;
    if (p >= 0) {
      // m is itself a source if some remapped destination takes page m
      const int j = find_kept(keep, nk, (int64_t)m * ps);
      const bool is_src = j >= 0 && j % ps == 0 && j / ps >= m0 && j / ps < npd && src[j / ps] == m;
      released = !is_src;
      gives = !(p < npd && src[p] >= 0);
    }
    int tot_rel, tot_give;
    const int r_rel = n_rel + flag_rank(released, s_sum, &tot_rel);
    const int r_give = n_give + flag_rank(gives, s_sum, &tot_give);
    if (released) rel[r_rel] = pt[m];
    if (gives) give[m] = r_give;
    n_rel += tot_rel;
    n_give += tot_give;
  }
  // The two counts agree for every strictly ascending keep_idx; should they
  // not, the sequence is rebuilt without remapping rather than with a page
  // nobody handed over.
  if (n_rel != n_give) return;
  wait_vmem();
  __syncthreads();

  for (int m = m0 + tid; m < npd; m += kInplaceThreads) {
    const int r = give[m];
    if (r >= 0) {
      const int page = rel[r];
      give[m] = page;
      const int p = src[m];
      if (p < ndp) npg[p] = page;
    }
  }
  wait_vmem();
  __syncthreads();

  // The records of the rows that still move, packed in ascending slot order
  // from index `hole` on (the walk needs only their order), tile by tile:
  // every record of a tile is read before any is written, and a row's
  // packed index never exceeds its slot.
  int n_mv = 0;
  for (int j0 = hole; j0 < nk; j0 += kInplaceThreads) {
    const int j = j0 + tid;
    bool mv = false;
    int64_t so = -1, dso = -1;
    if (j < nk) {
      const int d = j / ps;
      mv = !(d < npd && src[d] >= 0);
      if (mv) {
        so = rec[2 * j];
        dso = (int64_t)npg[d] * a.s_page + (int64_t)(j - d * ps) * a.row_bytes;
      }
    }
    wait_vmem();
    int tot;
    const int k = hole + n_mv + flag_rank(mv, s_sum, &tot);
    if (mv) {
      rec[2 * k] = so;
      rec[2 * k + 1] = dso;
    }
    n_mv += tot;
  }
  if (tid == 0) a.info[2 * b + 1] = hole + n_mv;
  // every read of the old table is behind this barrier
  wait_vmem();
  __syncthreads();

  int32_t* out = a.pt_out + (int64_t)b * a.ld_pt;
  for (int m = m0 + tid; m < npd; m += kInplaceThreads) {
    const int p = src[m];
    if (p >= 0) {
      out[m] = npg[m];
      const int page = give[m];
      if (page >= 0) out[p] = page;
    }
  }
}

__global__ __launch_bounds__(kInplaceThreads) void k_inplace_check(InplaceArgs a) {
  __shared__ int s_bad[kInplaceThreads / 64];
  __shared__ int s_hole[kInplaceThreads / 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.x;
  int32_t* info = a.info + 2 * b;
  int nk = a.n_keep[b];
  if (nk <= 0) {  // nothing kept, or a sequence select already refused
    if (tid == 0) info[0] = info[1] = 0;
    return;
  }
  nk = min(nk, a.K);
  const int32_t* keep = a.keep_idx + (int64_t)b * a.K;
  const int32_t* pt = a.pt + (int64_t)b * a.ld_pt;
  int64_t* rec = a.offsets + 2 * (int64_t)b * a.K;
  const bool side = a.scores || a.pos;
  int bad = 0, hole = nk;
  for (int j = tid; j < nk; j += kInplaceThreads) {
    const int idx = keep[j];
    const int prev = j > 0 ? keep[j - 1] : -1;
    int64_t so = -1, dso = -1;
    if (idx > prev && !(side && (int64_t)idx >= a.ld_s)) {
      const int sp = idx / a.page_size;
      const int dp = j / a.page_size;
      if ((int64_t)sp < a.ld_pt) {  // dp <= sp since j <= idx
        const int ps = pt[sp];
        const int pd = pt[dp];
        if (ps >= 0 && ps < a.n_pages && pd >= 0 && pd < a.n_pages) {
          so = (int64_t)ps * a.s_page + (int64_t)(idx - sp * a.page_size) * a.row_bytes;
          dso = (int64_t)pd * a.s_page + (int64_t)(j - dp * a.page_size) * a.row_bytes;
        }
      }
    }
    if (so < 0) bad = 1;
    if (idx != j) hole = min(hole, j);
    rec[2 * j] = so;
    rec[2 * j + 1] = dso;
  }
  // block-wide "any bad" and "first hole"
  bad = __any(bad);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) hole = min(hole, __shfl_xor(hole, m));
  if (lane == 0) {
    s_bad[wave] = bad;
    s_hole[wave] = hole;
  }
  __syncthreads();
  bad = 0;
  hole = nk;
  for (int w = 0; w < kInplaceThreads / 64; ++w) {
    bad |= s_bad[w];
    hole = min(hole, s_hole[w]);
  }
  if (bad) {
    if (tid == 0) {
      info[0] = info[1] = 0;
      if (a.seq_status) a.seq_status[b] = EPIKV_SEQ_RANGE;
    }
    return;
  }
  if (tid == 0) {
    info[0] = hole;
    info[1] = nk;
  }
  if (a.remap) {
    remap_pages(a, b, keep, pt, nk, hole, rec);
    wait_vmem();
    __syncthreads();
  }
  if (!side) return;
  // Scores and positions follow their rows, in ascending tiles (the same
  // argument as the row move, with the workgroup barrier as the wait).
  float* sc = a.scores ? a.scores + (int64_t)b * a.ld_s : nullptr;
  int32_t* ps = a.pos ? a.pos + (int64_t)b * a.ld_s : nullptr;
  for (int j0 = hole; j0 < nk; j0 += kInplaceThreads) {
    const int j = j0 + tid;
    float v = 0.f;
    int32_t p = 0;
    if (j < nk) {
      const int idx = keep[j];
      if (sc) v = sc[idx];
      if (ps) p = ps[idx];
    }
    wait_vmem();
    __syncthreads();
    if (j < nk) {
      if (sc) sc[j] = v;
      if (ps) ps[j] = p;
    }
  }
}

template <int LPR, int NI>
__global__ __launch_bounds__(kCompactThreads) void k_inplace_move(InplaceArgs a) {
  constexpr int RPI = 64 / LPR;          // rows per load instruction
  constexpr int T = RPI * NI;            // rows per tile
  constexpr int RPL = (T + 63) / 64;     // records per lane
  static_assert(T <= 64 || T % 64 == 0, "a tile fills whole record registers");
  const int lane = threadIdx.x & 63;
  const int64_t unit = (int64_t)blockIdx.x * kCompactWaves + (threadIdx.x >> 6);
  const int64_t per_seq = (int64_t)a.n_lk * a.n_slices;
  const int b = (int)(unit / per_seq);
  if (b >= a.B) return;
  const int rem = (int)(unit - (int64_t)b * per_seq);
  const int pl = rem / a.n_slices;
  const int sl = rem - pl * a.n_slices;
  const int h = a.info[2 * b];
  const int nk = a.info[2 * b + 1];
  if (h >= nk) return;
  const int col = sl * LPR + lane % LPR;
  const bool col_ok = col < (a.row_bytes >> 4);
  const int rsub = lane / LPR;
  char* base = a.pool + (int64_t)(pl >> 1) * a.s_layer + (int64_t)(pl & 1) * a.s_kv + (int64_t)col * 16;
  const int64_t* rec = a.offsets + 2 * (int64_t)b * a.K;
  // register r of lane i holds the record of the tile's row r * 64 + i
  int64_t rs[RPL], rd[RPL];
#pragma unroll
  for (int r = 0; r < RPL; ++r) {
    const int t = r * 64 + lane;
    rs[r] = rd[r] = -1;
    if (t < T && h + t < nk) {
      rs[r] = rec[2 * (h + t)];
      rd[r] = rec[2 * (h + t) + 1];
    }
  }
  // (waiting here too keeps the loop head free of a wait for the previous
  // tile's stores)
  wait_vmem();
  for (int j0 = h; j0 < nk; j0 += T) {
    u32x4 v[NI];
    int64_t dd[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      // row i * RPI + rsub of the tile; RPI divides 64, so its register is
      // known at compile time
      const int r = (i * RPI) / 64;
      const int src = (i * RPI) % 64 + rsub;
      const int64_t s = shfl64(rs[r], src);
      dd[i] = shfl64(rd[r], src);
      if (s >= 0 && col_ok) v[i] = ld_stream(base + s);
    }
    // next tile's records, while this tile's rows are in flight
    int64_t ns[RPL], nd[RPL];
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
      const int t = r * 64 + lane;
      const int jn = j0 + T + t;
      ns[r] = nd[r] = -1;
      if (t < T && jn < nk) {
        ns[r] = rec[2 * jn];
        nd[r] = rec[2 * jn + 1];
      }
    }
    wait_vmem();
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (dd[i] >= 0 && col_ok) st_stream(base + dd[i], v[i]);
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
      rs[r] = ns[r];
      rd[r] = nd[r];
    }
  }
}

// The move for 1 KiB column slices (64 lanes per row, one row per
// instruction), software pipelined: tile k + 1's loads are issued before
// tile k's stores, and a tile's stores wait only for its own loads.  This
// keeps the ordering argument: tile k + 1 reads positions at or past its
// own slots, which lie past every slot tile k (or any earlier tile)
// writes, and tile k's stores follow its loads.  Every load and store is
// issued, a missing row or record through an empty buffer resource (its
// loads read 0 without a memory access, its stores are dropped), so that
// the operations in flight are the same on every path and each wait is
// exactly for the tile it needs.
// One (src, dst) record per lane for the rows of a tile: lane t < NI holds
// the tile's row t (a lane past the walk's rows loads the first record
// and is marked absent).
template <int NI>
struct WalkRecs {
  int64_t s, d;
  int in;
};

__device__ __forceinline__ void st_row_nt(char* row, uint32_t off, int n_bytes, u32x4 v) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, n_bytes, kBufferRsrcWord3);
  __builtin_amdgcn_raw_buffer_store_b128(v, rs, off, 0, kBufferNonTemporal);
}
__device__ __forceinline__ u32x4 ld_row_nt(const char* row, uint32_t off, int n_bytes) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, n_bytes, kBufferRsrcWord3);
  return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kBufferNonTemporal);
}

template <int NI>
__global__ __launch_bounds__(kCompactThreads) void k_inplace_walk(InplaceArgs a) {
  static_assert(NI <= 64, "a tile's records fit one register per lane");
  const int lane = threadIdx.x & 63;
  // (the wavefront index made explicitly uniform, so that everything derived
  // from it -- the walk's plane and slice, hence each row's buffer resource --
  // lives in scalar registers)
  const int64_t unit =
      (int64_t)blockIdx.x * kCompactWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t per_seq = (int64_t)a.n_lk * a.n_slices;
  const int b = (int)(unit / per_seq);
  if (b >= a.B) return;
  const int rem = (int)(unit - (int64_t)b * per_seq);
  const int pl = rem / a.n_slices;
  const int sl = rem - pl * a.n_slices;
  const int h = a.info[2 * b];
  const int nk = a.info[2 * b + 1];
  if (h >= nk) return;
  // this slice of a row: bytes [1024 sl, min(1024 sl + 1024, row_bytes))
  char* base = a.pool + (int64_t)(pl >> 1) * a.s_layer + (int64_t)(pl & 1) * a.s_kv + 1024 * sl;
  const int span = min(1024, a.row_bytes - 1024 * sl);
  const uint32_t off = 16u * lane;
  const int64_t* rec = a.offsets + 2 * (int64_t)b * a.K;
  auto load_recs = [&](int j0, WalkRecs<NI>& r) {
    const int t = j0 + lane;
    r.in = lane < NI && t < nk;
    const int tc = r.in ? t : h;
    r.s = rec[2 * tc];
    r.d = rec[2 * tc + 1];
  };
  // row i of a tile: its source (load) or destination (store) row base and
  // the bytes it spans, 0 when absent -- read from lane i into scalars, so
  // the row's buffer resource is wave-uniform
  auto row_at = [&](const WalkRecs<NI>& r, int i, bool dst, int& n) -> char* {
    const int64_t w = dst ? r.d : r.s;
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)(uint64_t)w, i);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)w >> 32), i);
    const int64_t v = (int64_t)(((uint64_t)hi << 32) | lo);
    const bool ok = __builtin_amdgcn_readlane(r.in, i) && v >= 0;
    n = ok ? span : 0;
    return ok ? base + v : base;
  };
  auto load_tile = [&](const WalkRecs<NI>& r, u32x4 (&v)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      int n;
      const char* q = row_at(r, i, false, n);
      v[i] = ld_row_nt(q, off, n);
    }
  };
  auto store_tile = [&](const WalkRecs<NI>& r, const u32x4 (&v)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      int n;
      char* q = row_at(r, i, true, n);
      st_row_nt(q, off, n, v[i]);
    }
  };
  WalkRecs<NI> r0, r1, r2;
  load_recs(h, r0);
  load_recs(h + NI, r1);
  u32x4 va[NI], vb[NI];
  load_tile(r0, va);  // (waits for r0 only)
  for (int j0 = h;; j0 += 2 * NI) {
    // tile at j0 in va (records r0), the next tile's records in r1
    load_recs(j0 + 2 * NI, r2);
    load_tile(r1, vb);
    store_tile(r0, va);
    if (j0 + NI >= nk) break;
    load_recs(j0 + 3 * NI, r0);
    load_tile(r2, va);
    store_tile(r1, vb);
    if (j0 + 2 * NI >= nk) break;
    r1 = r0;
    r0 = r2;
  }
}

template <int LPR, int NI>
hipError_t launch_move(const InplaceArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.B * a.n_lk * a.n_slices;
  const int64_t blocks = (units + kCompactWaves - 1) / kCompactWaves;
  hipLaunchKernelGGL((k_inplace_move<LPR, NI>), dim3((unsigned)blocks), dim3(kCompactThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compact_inplace(const InplaceArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_inplace_check, dim3(a.B), dim3(kInplaceThreads), 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (a.lanes_per_row * 1000 + a.tile_ni) {
    case 64016: {
      const int64_t units = (int64_t)a.B * a.n_lk * a.n_slices;
      const int64_t blocks = (units + kCompactWaves - 1) / kCompactWaves;
      hipLaunchKernelGGL((k_inplace_walk<8>), dim3((unsigned)blocks), dim3(kCompactThreads), 0, s, a);
      return hipGetLastError();
    }
    case 16008: return launch_move<16, 8>(a, s);
    case 16016: return launch_move<16, 16>(a, s);
    case 4004: return launch_move<4, 4>(a, s);
    case 4016: return launch_move<4, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace epikv
