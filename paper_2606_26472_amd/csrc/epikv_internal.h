// Internal interface between the C-ABI host layer (epikv_api.hip) and the
// gfx950 kernels.  Each kernel takes one argument struct by value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "epikv.h"

namespace epikv {

// 16-byte vector used for every global load/store of bf16 rows.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ u32x4 ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st_stream(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// Buffer resources (gfx9 family): the fourth descriptor word of a raw
// buffer, and the cache-policy bit of a non-temporal access.
constexpr int kBufferRsrcWord3 = 0x00020000;
constexpr int kBufferNonTemporal = 2;

// Sum over the 64 lanes of a wavefront with a fixed butterfly order, so the
// result is identical on every lane and from run to run.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---------------------------------------------------------------------------
// Argument structs
// ---------------------------------------------------------------------------
struct ScoreHsArgs {
  const uint16_t* hidden[EPIKV_MAX_BAND];  // per band layer, Band A first
  int64_t ld_tok, ld_seq;                  // bf16 elements
  int32_t B, C, D, n_band, seg_len;
  const int32_t* n_tok_in;                 // state [B]
  const uint16_t* h_prev_in;               // state [B][n_band][D]
  uint16_t* h_prev_out;
  float* sig;                              // [n_band][B][C]
};

// Fused per-token scoring (Eq. 1 + smoothing + band combination) of chunks of
// at most kZscoreTile tokens with rows of at most 4096 elements.
struct ScoreTokArgs {
  const uint16_t* hidden[EPIKV_MAX_BAND];
  int64_t ld_tok, ld_seq;
  int32_t B, C, D, n_band, n_a, n_b, w, mode;
  float eps, alpha;
  const int32_t* n_cached;
  const int32_t* n_tok_in;
  const float* ring_in;
  const uint16_t* h_prev_in;
  const float* ema_in;
  int32_t* n_tok_out;
  float* ring_out;
  uint16_t* h_prev_out;
  float* ema_out;
  float* scores;
  int64_t ld_s;
};

struct ScoreLagArgs {
  const char* base;                        // pool
  int64_t s_layer, s_kv, s_page, n_pages;
  const int32_t* pt;
  int64_t ld_pt;
  const int32_t* n_cached;
  int32_t B, C, L, H, d, page_size;
  int32_t page_shift;                      // log2(page_size), or -1 if not a power of 2
  int32_t lag;                             // lag normalisation
  int32_t n_planes;                        // used planes: 2L (keys and values) or L
  int32_t two, kv0;                        // both tensors used; else the one used
  float eps;
  const int32_t* n_tok_in;
  const float* range_in;                   // [2][B][L][2][H][d] (lag only)
  float* range_out;
  float* partial;                          // [B][n_planes][segments][C]
  int32_t splits;                          // workgroups sharing one plane's rows
  float* prange;                           // [splits][2][B][L][2][H][d] partial ranges
};

struct LagReduceArgs {
  const float* partial;                    // [B][n_sums][C]
  float* sig;                              // [B][C]
  int32_t B, C, L, n_sums;                 // n_sums = used planes x row segments
  float inv_count;                         // 1 / (L*H)
  int32_t lag, use_k, use_v, splits, n_chan;  // n_chan = L*2*H*d channels per sequence
  const float* prange;
  float* range_out;                        // [2][B][L][2][H][d]
};

struct ZscoreArgs {
  const float* sig;                        // [n_sig][B][C]
  int32_t B, C, n_sig, n_a, n_b, w, mode, hs;
  float eps;
  const int32_t* n_cached;
  const int32_t* n_tok_in;
  const float* ring_in;                    // [B][n_sig][w-1]
  int32_t* n_tok_out;
  float* ring_out;
  const float* ema_in;                     // [B][n_sig] running averages
  float* ema_out;
  float alpha;                             // EMA weight of the previous average
  float* scores;
  int64_t ld_s;
  float* smoothed;                         // optional [n_sig][B][C]
};

struct SelectArgs {
  const float* scores;
  int64_t ld_s;
  const int32_t* n_cached;
  const int32_t* n_prefix;
  int32_t B, K, R, min_n;
  int32_t* keep_idx;                       // [B][K]
  int32_t* n_keep;
  int32_t* seq_status;
};

// One sequence's selection split over `groups` workgroups (select_multi.hip).
// scratch: per sequence kSelSeqWords words -- a 256-byte head (the 64-bit
// marker that the rest is clear, a give-up flag, a join count), then the
// three radix passes' histograms of 2048 bins -- followed by two words per
// workgroup of the grid (each zeroed by its workgroup first).
struct SelectMultiArgs {
  SelectArgs sel;
  uint32_t* scratch;
  int32_t groups;
};

struct CompactArgs {
  const char* src;
  int64_t s_layer, s_kv, s_page, s_npages;
  char* dst;
  int64_t d_layer, d_kv, d_page, d_npages;
  const int32_t* src_pt;
  int64_t ld_src_pt;
  const int32_t* dst_pt;
  int64_t ld_dst_pt;
  const int32_t* keep_idx;                 // [B][K]
  const int32_t* n_keep;
  const float* src_scores;
  float* dst_scores;
  const int32_t* src_pos;
  int32_t* dst_pos;
  int64_t ld_s;
  int32_t* seq_status;                     // optional
  int64_t* offsets;                        // workspace [B * n_pg * page_size][2]: src, dst
                                           // byte offsets, in destination-page rank order
  int32_t* rank;                           // workspace [B][n_pg]: rank of each destination page
  int32_t B, K, page_size, row_bytes, n_lk;
  int32_t n_pg;                            // pages of the budget: ceil(K / page_size)
  int32_t units;                           // 1 KiB column groups per row (set by launch_compact)
};

struct InplaceArgs {
  char* pool;
  int64_t s_layer, s_kv, s_page, n_pages;
  const int32_t* pt;                       // [B][ld_pt], source and destination
  int64_t ld_pt;
  const int32_t* keep_idx;                 // [B][K], strictly ascending
  const int32_t* n_keep;
  float* scores;                           // [B][ld_s], moved in place (optional)
  int32_t* pos;                            // [B][ld_s], moved in place (optional)
  int64_t ld_s;
  int32_t* seq_status;                     // optional
  int64_t* offsets;                        // workspace [B][K][2]: src, dst byte offsets
  int32_t* info;                           // workspace [B][2]: first hole, rows kept
  // Page remapping (whole retained pages change places in the table instead
  // of being copied): pt_out is the same table, written; remap_ws holds four
  // int32 arrays of n_pg = ceil(K / page_size) entries per sequence.
  int32_t remap;
  int32_t* pt_out;
  int32_t* remap_ws;                       // workspace [B][4][n_pg]
  int32_t n_pg;
  int32_t B, K, page_size, row_bytes, n_lk;
  int32_t lanes_per_row;                   // 64, 16 or 4 lanes share one row of a plane
  int32_t n_slices;                        // ceil(row_bytes / 16 / lanes_per_row)
  int32_t tile_ni;                         // row loads per lane and tile
};

struct FillArgs {
  uint32_t* p;
  int64_t n_words;
  uint32_t value;
};

// ---------------------------------------------------------------------------
// Arithmetic shared by kernels that must agree bit for bit (the fused
// per-token scorer and the separate score / zscore kernels)
// ---------------------------------------------------------------------------
// Accumulate the squared differences of eight bf16 pairs (Eq. 1), in order.
__device__ __forceinline__ float sqdiff8(u32x4 a, u32x4 b, float acc) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float d0 = bf16_lo(a[k]) - bf16_lo(b[k]);
    const float d1 = bf16_hi(a[k]) - bf16_hi(b[k]);
    acc = fmaf(d0, d0, acc);
    acc = fmaf(d1, d1, acc);
  }
  return acc;
}

// Smoothed value of the sample at extended index j over its window [lo, j]
// (Eq. 3 z-score, Eq. 2 mean, or the raw sample); x holds the extended
// samples from index `base` on.  Two passes over at most w values.
__device__ __forceinline__ float smooth_at(const float* x, int base, int lo, int j, int mode,
                                           float eps) {
  const float n = (float)(j - lo + 1);
  const float xv = x[j - base];
  if (mode == EPIKV_SMOOTH_RAW) return xv;
  // (unrolled so that the LDS reads issue ahead of the additions, which
  // stay in order)
  float s = 0.f;
#pragma unroll 8
  for (int k = lo; k <= j; ++k) s += x[k - base];
  const float mu = s / n;
  if (mode == EPIKV_SMOOTH_MEAN) return mu;
  float q = 0.f;
#pragma unroll 8
  for (int k = lo; k <= j; ++k) {
    const float dlt = x[k - base] - mu;
    q = fmaf(dlt, dlt, q);
  }
  return (xv - mu) / (sqrtf(q / n) + eps);
}

// EMA over one 64-token tile of a signal row (App. E): each lane's token is
// the affine map y -> A*y + Bc (the identity without a sample, y = x at the
// stream's first sample); an inclusive lane scan composes them and applies
// the result to the average carried into the tile.
__device__ __forceinline__ float ema_scan(float x, bool has, bool first, float al, float bl,
                                          float carry, int lane) {
  float A = has ? (first ? 0.f : al) : 1.f;
  float Bc = has ? (first ? x : bl * x) : 0.f;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float pa = __shfl_up(A, off, 64);
    const float pb = __shfl_up(Bc, off, 64);
    if (lane >= off) {
      Bc = fmaf(A, pb, Bc);
      A = A * pa;
    }
  }
  return fmaf(A, carry, Bc);
}

// s = mean over Band A rows - mean over Band B rows of token t (Fig. 1).
template <int TILE>
__device__ __forceinline__ float band_combine(const float (*vals)[TILE], int t, int n_a,
                                              int n_sig, int n_b) {
  float sa = 0.f, sb = 0.f;
  for (int l = 0; l < n_a; ++l) sa += vals[l][t];
  for (int l = n_a; l < n_sig; ++l) sb += vals[l][t];
  float s = sa / (float)n_a;
  if (n_b > 0) s -= sb / (float)n_b;
  return s;
}

// ---------------------------------------------------------------------------
// Launchers (return the HIP error of the launch; never synchronise)
// ---------------------------------------------------------------------------
hipError_t launch_score_hs(const ScoreHsArgs& a, hipStream_t s);
hipError_t launch_score_tokens(const ScoreTokArgs& a, hipStream_t s);
hipError_t launch_score_lagkv(const ScoreLagArgs& a, const LagReduceArgs& r,
                              hipStream_t s);
hipError_t launch_zscore(const ZscoreArgs& a, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
// The eviction step's selection: several workgroups per sequence when the
// batch is too small to fill the device with one each (scratch of
// select_scratch_bytes(B), kept between calls), else launch_select.
hipError_t launch_select_groups(const SelectArgs& a, void* scratch, hipStream_t s);
size_t select_scratch_bytes(int B);
// Selection and hidden-state scoring in one launch; valid only when
// select_score_fusable (the chunk lies inside the recency window).
bool select_score_fusable(const SelectArgs& sel, const ScoreHsArgs& sc);
hipError_t launch_select_score(const SelectArgs& sel, const ScoreHsArgs& sc, hipStream_t s);
hipError_t launch_compact(const CompactArgs& a, hipStream_t s);
hipError_t launch_compact_inplace(const InplaceArgs& a, hipStream_t s);
hipError_t launch_fill(const FillArgs& a, hipStream_t s);

// Tunables the host layer validates against.
constexpr int kScoreThreads = 256;
constexpr int kScoreSeg = 32;            // tokens per score_hs workgroup (wide rows)
constexpr int kScoreSegWave = 64;        // longest segment per score_hs wavefront (rows <= 4096)
constexpr int kScoreWavesWanted = 1024;  // shorten segments until this many wavefronts
constexpr int kZscoreTile = 64;          // tokens per zscore workgroup (one per lane)
constexpr int kZscoreThreads = 1024;     // 16 wavefronts: one signal row each
constexpr int kTokMaxRow = 4096;         // fused per-token scorer: widest hidden row
constexpr int kSelectThreads = 1024;
constexpr int kSelHeadWords = 64;                         // marker, flag, join count
constexpr uint32_t kSelMarkLo = 0x9E3779B9u;              // "this scratch is clear"
constexpr uint32_t kSelMarkHi = 0x7F4A7C15u;
constexpr int kSelSeqWords = kSelHeadWords + 3 * 2048;    // per-sequence scratch words
constexpr int kSelMaxGrid = 256;  // workgroups of a multi-workgroup selection, at most
constexpr int kCompactThreads = 256;      // resolve kernel; in-place move workgroups
constexpr int64_t kCompactGridX = 1 << 24;  // gather workgroups per grid row
constexpr int kCompactWaves = kCompactThreads / 64;  // walks per in-place move workgroup
constexpr int kLagWgWanted = 512;        // split a plane's rows until this many workgroups
constexpr int kLagPtCache = 1024;        // page-table entries a KV-scorer workgroup keeps in LDS
constexpr int kLagRowCache = kLagPtCache / 2;  // or row offsets (int64, the same LDS)

// KV-vector scorer shapes (lag: a lag-normalised signal).  Wavefronts per
// workgroup and rows each keeps in flight: 8 and 8 for the lag-normalised
// signals, whose four registers of per-channel state allow four
// wavefronts per SIMD (two workgroups per CU); 16 and 4 for the raw
// signals, which fit eight.  When the planes and sequences alone give at
// most kLagWgWanted / 2 workgroups (one lag-normalised tensor), its
// workgroups are "big": 16 wavefronts (one workgroup per CU) with 8 rows
// in flight each, which cover a plane's rows in half as many shares and
// so spare the partial ranges of the split rows.
// A lane takes 4 words (8 channels, 16 bytes) of a row, so a row spans
// H*d / 8 lanes; from 64 lanes on it is split into segments of 64 lanes,
// one wavefront each.
// LDS: the range slots (lag-normalised only; one [2][H*d] slot per row
// slot, or per row of a wavefront for narrow rows), then the transposed
// reduction's rows (row segments), then kLagPtCache page-table entries.
constexpr int kLagWords = 4;
__host__ __device__ inline int lagkv_row_lanes(int H, int d, bool) { return H * d / (2 * kLagWords); }
__host__ __device__ inline bool lagkv_wide(int H, int d, bool lag) {
  return lagkv_row_lanes(H, d, lag) >= 64;
}
__host__ __device__ inline int lagkv_segments(int H, int d, bool lag) {
  const int lanes = lagkv_row_lanes(H, d, lag);
  return lanes >= 64 ? lanes / 64 : 1;
}
// base: used planes x sequences
__host__ __device__ inline bool lagkv_big(int H, int d, bool lag, int64_t base) {
  return lag && lagkv_wide(H, d, lag) && base <= kLagWgWanted / 2;
}
__host__ __device__ constexpr int lagkv_waves(bool lag, bool big) { return lag && !big ? 8 : 16; }
__host__ __device__ constexpr int lagkv_threads(bool lag, bool big) {
  return 64 * lagkv_waves(lag, big);
}
__host__ __device__ constexpr int lagkv_ahead(bool lag) { return lag ? 8 : 4; }
__host__ __device__ inline int lagkv_range_floats(int H, int d, bool big) {
  const int lanes = lagkv_row_lanes(H, d, true);
  const int n_part = lanes >= 64 ? lagkv_waves(true, big) / lagkv_segments(H, d, true)
                                 : lagkv_waves(true, big) * (64 / lanes);
  return n_part * 2 * H * d;
}
// The transposed reduction's row of 64 (sum, sum of squares) pairs, with
// 4 words of padding after every 8 lanes.
constexpr int kRedRowWords = 64 * 2 + 8 * 4;
size_t lagkv_lds_bytes(int H, int d, bool lag, bool big);
constexpr int kInplaceThreads = 1024;    // per-sequence check + score move
constexpr int kInplaceUnitsWanted = 2048;  // narrow the column slices below this

}  // namespace epikv
