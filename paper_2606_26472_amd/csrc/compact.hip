// Order-preserving rebuild of the paged cache (App. H): for every kept slot
// j of sequence b, copy the K and V rows of position keep_idx[b][j] at every
// layer into slot j of the destination pages.  A token's row at one
// (layer, K|V) holds all KV heads (n_kv_heads * head_dim bf16, 2 KiB for
// 8 x 128), so the copy is a gather of 2 KiB rows: pure HBM streaming.
//
// One 256-thread workgroup owns rows_per_block consecutive destination
// slots of one sequence for lk_per_block (layer, K|V) planes.  The slots'
// source and destination row offsets are resolved once (keep_idx -> page
// tables) into LDS; each thread then holds NV 16-byte columns of the
// rows x row_bytes tile and reuses their offsets for every plane.  Small
// tiles (one or two 16-byte vectors per thread) keep many workgroups in
// flight on every CU, which is what lets a streaming copy approach the HBM
// rate on gfx950.  Loads and stores are non-temporal: each byte is touched
// once.
#include "epikv_internal.h"

namespace epikv {
namespace {

template <int NV, int PL>
__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a) {
  __shared__ int64_t soff[kCompactMaxRows];
  __shared__ int64_t doff[kCompactMaxRows];
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int b = blockIdx.x / a.blocks_per_seq;
  const int cb = blockIdx.x - b * a.blocks_per_seq;
  // A caller's n_keep above K is clamped so keep_idx is never read past the
  // sequence's row.
  const int nk = min(a.n_keep[b], a.K);
  const int j0 = cb * a.rows_per_block;
  if (nk <= j0) return;  // also n_keep < 0: sequence untouched
  const int rows = min(a.rows_per_block, nk - j0);

  if (tid == 0) bad = 0;
  __syncthreads();
  for (int r = tid; r < rows; r += kCompactThreads) {
    const int j = j0 + r;
    const int idx = a.keep_idx[(int64_t)b * a.K + j];
    int64_t so = -1, dso = -1;
    if (idx >= 0) {
      const int sp = idx / a.page_size;
      const int slot = idx - sp * a.page_size;
      if ((int64_t)sp < a.ld_src_pt) {
        const int pg = a.src_pt[(int64_t)b * a.ld_src_pt + sp];
        if (pg >= 0 && pg < a.s_npages)
          so = (int64_t)pg * a.s_page + (int64_t)slot * a.row_bytes;
      }
    }
    {
      const int dp = j / a.page_size;
      const int dslot = j - dp * a.page_size;
      if ((int64_t)dp < a.ld_dst_pt) {
        const int pg = a.dst_pt[(int64_t)b * a.ld_dst_pt + dp];
        if (pg >= 0 && pg < a.d_npages)
          dso = (int64_t)pg * a.d_page + (int64_t)dslot * a.row_bytes;
      }
    }
    const bool ok = so >= 0 && dso >= 0;
    soff[r] = ok ? so : -1;
    doff[r] = dso;
    if (!ok) bad = 1;
    if (blockIdx.y == 0 && ok && (int64_t)idx < a.ld_s && (int64_t)j < a.ld_s) {
      const int64_t si = (int64_t)b * a.ld_s + idx;
      const int64_t di = (int64_t)b * a.ld_s + j;
      if (a.dst_scores) a.dst_scores[di] = a.src_scores[si];
      if (a.dst_pos) a.dst_pos[di] = a.src_pos[si];
    }
  }
  __syncthreads();
  if (bad && a.seq_status && tid == 0) a.seq_status[b] = EPIKV_SEQ_RANGE;

  // This thread's NV columns of the rows x row_vec tile; the offsets are the
  // same for every plane.
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
      const int64_t col = (int64_t)(v - r * row_vec) * 16;
      if (soff[r] >= 0) {
        so[q] = soff[r] + col;
        dof[q] = doff[r] + col;
      }
    }
  }

  // PL planes are loaded together before any of them is stored, so each
  // thread keeps PL * NV independent 16-byte loads in flight.
  const int lk0 = blockIdx.y * a.lk_per_block;
  const int lk1 = min(a.n_lk, lk0 + a.lk_per_block);
  for (int lk = lk0; lk < lk1; lk += PL) {
    u32x4 val[PL][NV];
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const int pl = lk + p;
      if (pl < lk1) {
        const char* sb = a.src + (int64_t)(pl >> 1) * a.s_layer + (int64_t)(pl & 1) * a.s_kv;
#pragma unroll
        for (int q = 0; q < NV; ++q)
          if (so[q] >= 0) val[p][q] = ld_stream(sb + so[q]);
      }
    }
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const int pl = lk + p;
      if (pl < lk1) {
        char* db = a.dst + (int64_t)(pl >> 1) * a.d_layer + (int64_t)(pl & 1) * a.d_kv;
#pragma unroll
        for (int q = 0; q < NV; ++q)
          if (so[q] >= 0) st_stream(db + dof[q], val[p][q]);
      }
    }
  }
}

template <int NV, int PL>
hipError_t launch(const CompactArgs& a, hipStream_t s) {
  dim3 grid(a.B * a.blocks_per_seq, (a.n_lk + a.lk_per_block - 1) / a.lk_per_block);
  hipLaunchKernelGGL((k_compact<NV, PL>), grid, dim3(kCompactThreads), 0, s, a);
  return hipGetLastError();
}

template <int PL>
hipError_t launch_nv(const CompactArgs& a, hipStream_t s) {
  const int tile_vec = a.rows_per_block * (a.row_bytes >> 4);
  const int nv = (tile_vec + kCompactThreads - 1) / kCompactThreads;
  if (nv <= 1) return launch<1, PL>(a, s);
  if (nv <= 2) return launch<2, PL>(a, s);
  if (nv <= 4) return launch<4, PL>(a, s);
  if (nv <= 8) return launch<8, PL>(a, s);
  if (nv <= 16) return launch<16, PL>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t s) {
  switch (a.planes_together) {
    case 1: return launch_nv<1>(a, s);
    case 2: return launch_nv<2>(a, s);
    case 4: return launch_nv<4>(a, s);
    case 8: return launch_nv<8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace epikv
