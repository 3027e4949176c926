// Order-preserving rebuild of the paged cache (App. H): for every kept slot
// j of sequence b, copy the K and V rows of position keep_idx[b][j] at every
// layer into slot j of the destination pages.  A token's row at one
// (layer, K|V) holds all KV heads (n_kv_heads * head_dim bf16, 2 KiB for
// 8 x 128), so the copy is a gather of 2 KiB rows: pure HBM streaming.
//
// Two kernels:
//   resolve  one thread per kept slot turns keep_idx and the two page tables
//            into the byte offsets of the source and destination rows inside
//            a plane (one 16-byte record per slot, in the workspace), and
//            copies the slot's score and position;
//   gather   a 256-thread workgroup owns four consecutive slots of one
//            sequence (one wavefront per slot) for lk_per_block planes.  The
//            wavefront reads its slot's offset record with a scalar load and
//            then streams the row's 16-byte columns of every plane: a single
//            dependent load before the data, so short-lived workgroups keep
//            HBM busy.  Loads and stores are non-temporal: each byte is
//            touched once.  The hardware deals workgroups to the 8 XCDs
//            round-robin; the gather remaps its block index so that each XCD
//            streams one contiguous range of destination slots (measured
//            2-4% faster than the interleaved order).  The gather reserves
//            LDS it does not use so that at most six workgroups (24
//            wavefronts) share a CU: fewer requests in flight keep HBM more
//            efficient here (measured 2% faster than eight per CU, and
//            faster than five or seven).
#include "epikv_internal.h"

namespace epikv {
namespace {

__global__ __launch_bounds__(kCompactThreads) void k_compact_resolve(CompactArgs a) {
  const int j = blockIdx.x * kCompactThreads + threadIdx.x;
  const int b = blockIdx.y;
  // A caller's n_keep above K is clamped so keep_idx is never read past the
  // sequence's row.
  const int nk = min(a.n_keep[b], a.K);
  if (j >= nk) return;  // also n_keep < 0: sequence untouched
  const int idx = a.keep_idx[(int64_t)b * a.K + j];
  int64_t so = -1, dso = -1;
  if (idx >= 0) {
    const int sp = idx / a.page_size;
    const int slot = idx - sp * a.page_size;
    if ((int64_t)sp < a.ld_src_pt) {
      const int pg = a.src_pt[(int64_t)b * a.ld_src_pt + sp];
      if (pg >= 0 && pg < a.s_npages) so = (int64_t)pg * a.s_page + (int64_t)slot * a.row_bytes;
    }
  }
  {
    const int dp = j / a.page_size;
    const int dslot = j - dp * a.page_size;
    if ((int64_t)dp < a.ld_dst_pt) {
      const int pg = a.dst_pt[(int64_t)b * a.ld_dst_pt + dp];
      if (pg >= 0 && pg < a.d_npages) dso = (int64_t)pg * a.d_page + (int64_t)dslot * a.row_bytes;
    }
  }
  const bool ok = so >= 0 && dso >= 0;
  int64_t* rec = a.offsets + 2 * ((int64_t)b * a.K + j);
  rec[0] = ok ? so : -1;
  rec[1] = ok ? dso : -1;
  if (!ok) {
    if (a.seq_status) a.seq_status[b] = EPIKV_SEQ_RANGE;
    return;
  }
  if ((int64_t)idx < a.ld_s && (int64_t)j < a.ld_s) {
    const int64_t si = (int64_t)b * a.ld_s + idx;
    const int64_t di = (int64_t)b * a.ld_s + j;
    if (a.dst_scores) a.dst_scores[di] = a.src_scores[si];
    if (a.dst_pos) a.dst_pos[di] = a.src_pos[si];
  }
}

// One wavefront per destination row: the row's offset record, n_keep and
// the plane bases are wave-uniform (scalar loads), lane l streams the
// row's 16-byte columns l, l+64, ... (NV of them) of each plane.
template <int NV, int PL>
__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int b = blockIdx.z;
  // XCD-aware: hardware places block x on XCD x % 8; give each XCD a
  // contiguous range of slot groups.
  const int nx = gridDim.x;
  int bx = blockIdx.x;
  if ((nx & 7) == 0) bx = (bx & 7) * (nx >> 3) + (bx >> 3);
  const int j = bx * kCompactWaves + wave;
  const int row_vec = a.row_bytes >> 4;
  // The record of slot min(j, K-1) is always readable, so it is fetched
  // together with n_keep instead of after it.
  const int64_t* rec = a.offsets + 2 * ((int64_t)b * a.K + min(j, a.K - 1));
  const int64_t s0 = rec[0];
  const int64_t d0 = rec[1];
  const int nk = min(a.n_keep[b], a.K);
  if (j >= nk || s0 < 0) return;

  const int lk0 = blockIdx.y * a.lk_per_block;
  const int lk1 = min(a.n_lk, lk0 + a.lk_per_block);
  for (int lk = lk0; lk < lk1; lk += PL) {
    u32x4 val[PL][NV];
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const int pl = lk + p;
      if (pl < lk1) {
        const char* sb = a.src + (int64_t)(pl >> 1) * a.s_layer + (int64_t)(pl & 1) * a.s_kv + s0;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
          const int c = lane + q * 64;
          if (c < row_vec) val[p][q] = ld_stream(sb + (int64_t)c * 16);
        }
      }
    }
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const int pl = lk + p;
      if (pl < lk1) {
        char* db = a.dst + (int64_t)(pl >> 1) * a.d_layer + (int64_t)(pl & 1) * a.d_kv + d0;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
          const int c = lane + q * 64;
          if (c < row_vec) st_stream(db + (int64_t)c * 16, val[p][q]);
        }
      }
    }
  }
}

template <int NV, int PL>
hipError_t launch(const CompactArgs& a, hipStream_t s) {
  dim3 grid(a.blocks_per_seq, (a.n_lk + a.lk_per_block - 1) / a.lk_per_block, a.B);
  hipLaunchKernelGGL((k_compact<NV, PL>), grid, dim3(kCompactThreads), kCompactLdsCap, s, a);
  return hipGetLastError();
}

template <int PL>
hipError_t launch_nv(const CompactArgs& a, hipStream_t s) {
  const int row_vec = a.row_bytes >> 4;
  if (row_vec <= 64) return launch<1, PL>(a, s);
  if (row_vec <= 128) return launch<2, PL>(a, s);
  if (row_vec <= 256) return launch<4, PL>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_compact(const CompactArgs& args, hipStream_t s) {
  CompactArgs a = args;
  // One wavefront per destination row, four rows and one (layer, K|V) plane
  // per workgroup: measured best on MI355X among 2..16 rows x 1..64 planes
  // for 32 sequences keeping 4096 of 8k..32k tokens.  (A wavefront here has
  // one 1 KiB load in flight at a time -- the compiler waits between the
  // guarded loads; a branch-free variant with both loads in flight measured
  // 5% slower at eight workgroups per CU, and more planes per wavefront
  // slower still.)
  a.lk_per_block = 1;
  a.blocks_per_seq = (a.K + kCompactWaves - 1) / kCompactWaves;
  hipLaunchKernelGGL(k_compact_resolve, dim3((a.K + kCompactThreads - 1) / kCompactThreads, a.B),
                     dim3(kCompactThreads), 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_nv<1>(a, s);
}

}  // namespace epikv
