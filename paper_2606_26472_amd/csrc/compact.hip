// Order-preserving rebuild of the paged cache (App. H): for every kept slot
// j of sequence b, copy the K and V rows of position keep_idx[b][j] at every
// layer into slot j of the destination pages.  A token's row at one
// (layer, K|V) holds all KV heads (n_kv_heads * head_dim bf16, 2 KiB for
// 8 x 128), so the copy is a gather of 2 KiB rows: pure HBM streaming.
//
// One 256-thread workgroup owns one destination page of one sequence (up to
// page_size consecutive slots) for lk_per_block (layer, K|V) planes.  The
// page's source row offsets are resolved once (keep_idx -> page table) into
// LDS; every thread then holds up to NV 16-byte columns of the page tile and
// re-uses their source/destination offsets for each plane.  Loads and stores
// are non-temporal: the data is touched exactly once.  A destination page
// is written as one contiguous run per plane.
#include "epikv_internal.h"

namespace epikv {
namespace {

constexpr int kMaxPageRows = 1024;

template <int NV>
__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a) {
  __shared__ int64_t soff[kMaxPageRows];
  __shared__ int64_t doff;
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int b = blockIdx.x / a.pages_per_seq;
  const int p = blockIdx.x - b * a.pages_per_seq;
  // A caller's n_keep above K is clamped so keep_idx is never read past the
  // sequence's row.
  const int nk = min(a.n_keep[b], a.K);
  const int j0 = p * a.page_size;
  if (nk <= j0) return;  // also n_keep < 0: sequence untouched
  const int rows = min(a.page_size, nk - j0);

  if (tid == 0) {
    bad = 0;
    const int pg = (int64_t)p < a.ld_dst_pt ? a.dst_pt[(int64_t)b * a.ld_dst_pt + p] : -1;
    doff = (pg >= 0 && pg < a.d_npages) ? (int64_t)pg * a.d_page : -1;
  }
  __syncthreads();
  for (int r = tid; r < rows; r += kCompactThreads) {
    const int idx = a.keep_idx[(int64_t)b * a.K + j0 + r];
    int64_t off = -1;
    if (idx >= 0) {
      const int sp = idx / a.page_size;
      const int slot = idx - sp * a.page_size;
      if ((int64_t)sp < a.ld_src_pt) {
        const int pg = a.src_pt[(int64_t)b * a.ld_src_pt + sp];
        if (pg >= 0 && pg < a.s_npages)
          off = (int64_t)pg * a.s_page + (int64_t)slot * a.row_bytes;
      }
    }
    soff[r] = off;
    if (off < 0 || doff < 0) bad = 1;
    if (blockIdx.y == 0 && off >= 0 && doff >= 0 && (int64_t)idx < a.ld_s &&
        (int64_t)(j0 + r) < a.ld_s) {
      const int64_t so = (int64_t)b * a.ld_s + idx;
      const int64_t dj = (int64_t)b * a.ld_s + j0 + r;
      if (a.dst_scores) a.dst_scores[dj] = a.src_scores[so];
      if (a.dst_pos) a.dst_pos[dj] = a.src_pos[so];
    }
  }
  __syncthreads();
  if (bad && a.seq_status && tid == 0) a.seq_status[b] = EPIKV_SEQ_RANGE;
  if (doff < 0) return;

  // Column c of the page tile (rows x row_vec 16-byte vectors) for this
  // thread's NV columns; offsets are the same for every plane.
  const int row_vec = a.row_bytes >> 4;
  const int nvec = rows * row_vec;
  int64_t so[NV];
  int64_t dof[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int v = tid + q * kCompactThreads;
    so[q] = -1;
    dof[q] = 0;
    if (v < nvec) {
      const int r = v / row_vec;
      const int col = v - r * row_vec;
      const int64_t s0 = soff[r];
      if (s0 >= 0) {
        so[q] = s0 + (int64_t)col * 16;
        dof[q] = doff + (int64_t)r * a.row_bytes + (int64_t)col * 16;
      }
    }
  }

  const int lk0 = blockIdx.y * a.lk_per_block;
  const int lk1 = min(a.n_lk, lk0 + a.lk_per_block);
  for (int lk = lk0; lk < lk1; ++lk) {
    const int layer = lk >> 1;
    const int kv = lk & 1;
    const char* sb = a.src + (int64_t)layer * a.s_layer + (int64_t)kv * a.s_kv;
    char* db = a.dst + (int64_t)layer * a.d_layer + (int64_t)kv * a.d_kv;
    u32x4 val[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q)
      if (so[q] >= 0) val[q] = ld_stream(sb + so[q]);
#pragma unroll
    for (int q = 0; q < NV; ++q)
      if (so[q] >= 0) st_stream(db + dof[q], val[q]);
  }
}

template <int NV>
hipError_t launch(const CompactArgs& a, hipStream_t s) {
  dim3 grid(a.B * a.pages_per_seq, (a.n_lk + a.lk_per_block - 1) / a.lk_per_block);
  hipLaunchKernelGGL((k_compact<NV>), grid, dim3(kCompactThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t s) {
  const int page_vec = a.page_size * (a.row_bytes >> 4);
  const int nv = (page_vec + kCompactThreads - 1) / kCompactThreads;
  if (nv <= 1) return launch<1>(a, s);
  if (nv <= 2) return launch<2>(a, s);
  if (nv <= 4) return launch<4>(a, s);
  if (nv <= 8) return launch<8>(a, s);
  if (nv <= 16) return launch<16>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace epikv
