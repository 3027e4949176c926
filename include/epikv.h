/*
 * epikv.h -- C ABI of the EpiKV eviction step on AMD Instinct MI355X (gfx950).
 *
 * The step follows "Epiphany-Aware KV Cache Eviction Without the Attention
 * Matrix" (Kolawole & Smith, arXiv 2606.26472):
 *
 *   score    hidden-state change g_l(t) = ||h_l(t) - h_l(t-1)||_2 at the band
 *            layers (Sec. 3.2, Eq. 1), or a K/V-vector variance (Sec. 3.3:
 *            Lag-KV, KV-key, KV-val, lag-kv-key);
 *   zscore   causal trailing-window smoothing (Eq. 3 z-score, or the Eq. 2
 *            mean) and the band combination s = mean_A - mean_B (Fig. 1);
 *            the result is the token's frozen score (Sec. 3.3);
 *   select   keep the prefill, a recency window of R = min(128, K/4) and the
 *            best scores so that exactly K positions survive (Sec. 3.1,
 *            Sec. 3.3, App. D);
 *   compact  rebuild the paged cache from the kept positions, in order, for
 *            every layer, K and V and KV head (App. H; the cache holds
 *            2*L*H*d_h scalars per token, Sec. 3.1): into fresh pages, in
 *            place, or in place with whole retained pages remapped.
 *
 * epikv_evict_step runs the four in one call; epikv_score_tokens fuses score
 * and zscore for the online regime of scoring each token as it is generated
 * (Sec. 3.3), after which the step only selects and compacts.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are device pointers unless marked "host".  The caller owns
 *   every buffer.  The library allocates nothing, keeps no global state,
 *   never synchronises, and enqueues its kernels on `stream` (0 = the null
 *   stream).  Calls on different streams are independent.  (The one
 *   exception is epikv_evict_step_noalloc, whose scratch is a fixed
 *   per-GPU array inside the library: see there.)
 * - bf16 tensors are passed as raw 16-bit storage.
 * - Return value: EPIKV_OK (0) or a negative epikv_status.  Every negative
 *   code except EPIKV_ELAUNCH is detected on the host before anything is
 *   enqueued, so a failed call leaves device memory untouched.
 * - Per-sequence conditions that only the device sees (budget too small,
 *   lengths or page ids out of range) are reported in seq_status[b] with an
 *   epikv_seq_status value; the sequence's outputs are then left untouched.
 */
#ifndef EPIKV_H
#define EPIKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Host-detected errors. */
typedef enum epikv_status {
  EPIKV_OK = 0,
  EPIKV_EINVAL_NULL = -1,   /* a required pointer is NULL */
  EPIKV_EINVAL_SHAPE = -2,  /* a size is out of the supported range */
  EPIKV_EINVAL_PARAM = -3,  /* a parameter (budget, window, eps, enum) is invalid */
  EPIKV_EALIGN = -4,        /* a pointer, stride or leading dimension is misaligned */
  EPIKV_EWORKSPACE = -5,    /* workspace missing or smaller than required */
  EPIKV_EALIAS = -6,        /* an output overlaps an input it must not overlap */
  EPIKV_ELAUNCH = -7        /* the HIP runtime refused a kernel launch */
} epikv_status;

/* Per-sequence status written by the device. */
typedef enum epikv_seq_status {
  EPIKV_SEQ_OK = 0,
  EPIKV_SEQ_BUDGET = 1,     /* N > K but P + R >= K: no room for scored tokens */
  EPIKV_SEQ_RANGE = 2,      /* N, P, a kept index or a page id out of range */
  EPIKV_SEQ_SYNC = 3        /* the eviction step's selection of this sequence
                               runs on several workgroups that wait for each
                               other; one gave up waiting (about a second:
                               the device was so busy with other work that
                               they could not all run at once).  keep_idx
                               is not valid; n_keep = -1. */
} epikv_seq_status;

/* Which per-token signal is scored. */
typedef enum epikv_signal {
  EPIKV_SIGNAL_HS = 0,        /* band-layer hidden-state change, Sec. 3.2 Eq. 1 */
  EPIKV_SIGNAL_LAGKV = 1,     /* lag-normalised key + value variance, Sec. 3.3 */
  EPIKV_SIGNAL_KV_KEY = 2,    /* variance of the key vectors, Sec. 3.3 (KV-key) */
  EPIKV_SIGNAL_KV_VAL = 3,    /* variance of the value vectors, Sec. 3.3 (KV-val) */
  EPIKV_SIGNAL_LAGKV_KEY = 4  /* lag-normalised key variance (lag-kv-key, App. B) */
} epikv_signal;

/* How the per-token signal is smoothed over the trailing window. */
typedef enum epikv_smoothing {
  EPIKV_SMOOTH_Z = 0,       /* rolling z-score, Eq. 3 (EpiKV) */
  EPIKV_SMOOTH_MEAN = 1,    /* rolling mean, Eq. 2 (HS-variance, KV family) */
  EPIKV_SMOOTH_RAW = 2,     /* no smoothing (App. E "raw") */
  EPIKV_SMOOTH_EMA = 3      /* exponential moving average (App. E, alpha 0.9):
                               y = alpha*y_prev + (1-alpha)*x, y = x at the
                               stream's first sample */
} epikv_smoothing;

/* How epikv_evict_step rebuilds the cache (epikv_step_io.in_place). */
typedef enum epikv_compact_mode {
  EPIKV_COMPACT_OUT_OF_PLACE = 0,  /* epikv_compact into fresh pages (App. H) */
  EPIKV_COMPACT_IN_PLACE = 1,      /* epikv_compact_inplace */
  EPIKV_COMPACT_REMAP = 2          /* epikv_compact_remap (table rewritten) */
} epikv_compact_mode;

#define EPIKV_MAX_BAND 32   /* band layers per call */
#define EPIKV_MAX_WINDOW 256

/*
 * Configuration, passed by (host) pointer to every call.
 *
 * HS signal: n_band_a + n_band_b hidden-state layers are scored, Band A
 * (positive weight) first.  The paper's bands are layers 7..13 (A) and
 * 18..25 (B) of a 32-layer model (Sec. 3.2, App. A); the single-layer
 * preset A = {10}, B = {21} gives Eq. 3's z_10 - z_21.  n_band_b may be 0.
 * KV-vector signals (Lag-KV, KV-key, KV-val, lag-kv-key): one signal row per
 * sequence, weight +1; the band fields are ignored.
 */
typedef struct epikv_cfg {
  int32_t batch;        /* B >= 1 sequences */
  int32_t hidden;       /* D: hidden width for the HS signal, 8..16384, D % 8 == 0 */
  int32_t n_layers;     /* L: layers held in the KV pool, >= 1 */
  int32_t n_kv_heads;   /* H >= 1 */
  int32_t head_dim;     /* d: 64, 128 or 256; H*d <= 2048 */
  int32_t page_size;    /* tokens per KV page, 1..1024 */
  int32_t n_band_a;     /* HS: Band A layer count, >= 1 */
  int32_t n_band_b;     /* HS: Band B layer count, >= 0; A + B <= EPIKV_MAX_BAND */
  int32_t window;       /* w: trailing window in samples, 1..EPIKV_MAX_WINDOW (paper: 64) */
  float eps;            /* epsilon added to sigma (Eq. 3) and to the Lag-KV range, >= 0 */
  int32_t signal;       /* epikv_signal */
  int32_t smoothing;    /* epikv_smoothing */
  int32_t budget;       /* K >= 1: positions kept per sequence */
  int32_t recent;       /* R >= 0, or -1 for min(128, K/4) (App. D) */
  float ema_alpha;      /* EMA weight of the previous average, [0, 1] (paper: 0.9) */
} epikv_cfg;

/*
 * A paged bf16 KV pool.  The K (kv = 0) or V (kv = 1) row of the token in
 * slot s of page p at layer l starts at
 *     base + l*stride_layer + kv*stride_kv + p*stride_page + s*row_bytes
 * with row_bytes = n_kv_heads*head_dim*2: all KV heads of one token are one
 * contiguous row, heads outermost.  Strides are in bytes, multiples of 16,
 * and base is 16-byte aligned.  Valid page ids are [0, n_pages).
 */
typedef struct epikv_pool {
  void* base;
  int64_t stride_layer;
  int64_t stride_kv;
  int64_t stride_page;
  int64_t n_pages;
} epikv_pool;

/* Fill *cfg with the paper's setting: 32 layers, D = 4096, 8 KV heads x 128,
 * 16-token pages, Band A = 7 layers, Band B = 8 layers, w = 64, eps = 1e-6,
 * HS signal, z-score smoothing, R = min(128, K/4), EMA alpha = 0.9.  batch and budget are set
 * to 1 and 4096.  Returns EPIKV_EINVAL_NULL if cfg is NULL. */
int epikv_default_cfg(epikv_cfg* cfg);

/* Static description of a status code (never NULL). */
const char* epikv_strerror(int status);

/* Validate a configuration without touching the device. */
int epikv_check_cfg(const epikv_cfg* cfg);

/*
 * Scorer state carried from one call to the next (one flat device buffer,
 * caller-owned; checkpoint = copy it, resume = copy it back).  Sections,
 * each 256-byte aligned, at the offsets epikv_state_layout returns:
 *   [0] int32 n_tok[B]            tokens the scorer has consumed per sequence
 *   [1] float ring[B][n_sig][w-1] the last min(w-1, samples) signal samples,
 *                                 right-aligned (slot w-2 newest), unused
 *                                 slots 0
 *   [2] bf16  h_prev[B][n_band][D] HS: hidden state of the last token
 *   [3] float range[2][B][L][2][H][d] lag-normalised signals: per-channel
 *                                 min (first half) and max of the previous
 *                                 chunk
 *   [4] float ema[B][n_sig]       the running average after the last sample
 *                                 (EMA smoothing; carried unchanged in the
 *                                 other modes)
 * n_sig = n_band_a + n_band_b for HS, 1 for the KV-vector signals.  An HS
 * stream yields a sample for every token but its first (which has no
 * predecessor); a KV-vector stream for every token.  Sections a signal does
 * not use have size 0.  Returns the total size in bytes, or 0 for an invalid
 * cfg.
 */
size_t epikv_state_bytes(const epikv_cfg* cfg);

/* Byte offsets of the five state sections (host array of 5), see above.
 * Returns EPIKV_OK or a host error code. */
int epikv_state_layout(const epikv_cfg* cfg, size_t offsets[5]);

/* Device scratch that epikv_evict_step (and epikv_score) needs for a chunk
 * of `chunk` new tokens per sequence; for chunk = 0 (a step that only
 * selects and compacts) the selection's scratch and the compaction's
 * (epikv_select_workspace_bytes(cfg) + epikv_compact_workspace_bytes(cfg)).
 * 0 for an invalid cfg or chunk < 0. */
size_t epikv_workspace_bytes(const epikv_cfg* cfg, int32_t chunk);

/* Device scratch of epikv_compact, epikv_compact_inplace and
 * epikv_compact_remap: 16 bytes per slot of each sequence's budget pages,
 * B*ceil(K/page_size)*page_size*16 rounded up to 256, then 8 bytes per
 * sequence rounded up to 256, then 16 bytes per (sequence, page of the
 * budget), B*ceil(K/page_size)*16 rounded up to 256.  0 for an invalid cfg. */
size_t epikv_compact_workspace_bytes(const epikv_cfg* cfg);

/* Reset a state buffer of epikv_state_bytes(cfg) bytes to the start of a
 * stream (every section zero).  Uses a fill kernel, so it may be captured
 * in a HIP graph. */
int epikv_state_init(const epikv_cfg* cfg, void* state, hipStream_t stream);

/*
 * epikv_score -- per-token signal of `chunk` new tokens of every sequence.
 *
 * HS signal (Sec. 3.2, Eq. 1): sig[l][b][c] = ||h_l(b,c) - h_l(b,c-1)||_2 for
 * each band layer l, computed in fp32 from bf16 inputs.  h_l(b,-1) is
 * state_in.h_prev; for a fresh stream (n_tok = 0) the first token has no
 * sample and sig is 0 there.
 *   hidden      host array of n_band device pointers (Band A first); the
 *               row of token c of sequence b at layer l starts at
 *               hidden[l] + b*ld_seq + c*ld_tok (bf16 elements); pointers
 *               16-byte aligned, ld_tok and ld_seq multiples of 8, rows of
 *               D elements.
 *   pool, page_table, ld_pt, n_cached   unused (may be NULL / 0).
 * KV-vector signals (Sec. 3.3, Table 1): the chunk's tokens are positions
 * [n_cached[b] - chunk, n_cached[b]) of the paged cache (page_table int32
 * [B][ld_pt]).  For each used tensor (keys for KV-key and lag-kv-key, values
 * for KV-val, both for Lag-KV) the population variance over the head
 * dimension is taken per (layer, KV head) -- of the raw vectors, or for the
 * lag-normalised signals of (x - mn) / (mx - mn + eps) with (mn, mx) the
 * previous chunk's per-channel range from state_in (the first chunk of a
 * stream uses its own range) -- the used tensors' variances are summed and
 * averaged over layers and KV heads: sig[0][b][c].  hidden may be NULL.
 * Needs epikv_workspace_bytes(cfg, chunk) bytes of workspace (ignored for
 * HS).
 *
 * state_out receives h_prev (HS) or this chunk's range (lag-normalised
 * signals); its
 * counters and ring are written by epikv_zscore, so a step is complete only
 * after both calls.  state_in and state_out must not overlap.
 * sig: float [n_sig][B][chunk].
 * Sequences whose positions fall outside [0, ld_pt*page_size) or whose pages
 * are outside the pool get sig 0 for the affected tokens.
 */
int epikv_score(const epikv_cfg* cfg, int32_t chunk,
                const void* const* hidden, int64_t ld_tok, int64_t ld_seq,
                const epikv_pool* pool, const int32_t* page_table,
                int64_t ld_pt, const int32_t* n_cached,
                const void* state_in, void* state_out, float* sig,
                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * epikv_zscore -- smoothing and band combination (Eq. 3 or Eq. 2, Fig. 1).
 *
 * For each signal row the new samples follow the w-1 carried in
 * state_in.ring; each token's window is the last min(w, available) samples
 * up to and including its own.  Z: (x - mu) / (sigma + eps) with the
 * population sigma; MEAN: mu; RAW: x; EMA: the running average carried in
 * state_in.ema.  Tokens without a sample get 0.  The
 * frozen score s = mean over Band A rows - mean over Band B rows (KV-vector
 * signals: the single row) is written to scores[b*ld_s + n_cached[b] - chunk + c].
 * Sequences with n_cached < chunk or n_cached > ld_s are skipped.
 *   sig       float [n_sig][B][chunk] from epikv_score.
 *   smoothed  optional (may be NULL) float [n_sig][B][chunk]: per-row
 *             smoothed values.
 * state_out receives n_tok += chunk and the updated ring.
 */
int epikv_zscore(const epikv_cfg* cfg, int32_t chunk, const float* sig,
                 const int32_t* n_cached, const void* state_in,
                 void* state_out, float* scores, int64_t ld_s,
                 float* smoothed, hipStream_t stream);

/*
 * epikv_score_tokens -- epikv_score and epikv_zscore in one launch, for the
 * online regime of Sec. 3.3: a decoder scores each token (or a few) as it
 * is generated and freezes the score; an eviction then needs only
 * epikv_select + epikv_compact.
 *
 * Hidden-state signal only (cfg->signal == EPIKV_SIGNAL_HS), every
 * smoothing mode, 1 <= chunk <= 64, cfg->hidden <= 4096.  Arguments as for
 * epikv_score (hidden, ld_tok, ld_seq, state_in, state_out) and
 * epikv_zscore (n_cached, scores, ld_s); no signal buffer or workspace (the
 * signal stays on chip).  The scores written and the state_out produced are
 * bit for bit those of the two separate calls.  Errors: EINVAL_PARAM for
 * another signal, EINVAL_SHAPE for chunk or hidden out of range, and the
 * checks of epikv_score / epikv_zscore.
 */
int epikv_score_tokens(const epikv_cfg* cfg, int32_t chunk,
                       const void* const* hidden, int64_t ld_tok,
                       int64_t ld_seq, const int32_t* n_cached,
                       const void* state_in, void* state_out, float* scores,
                       int64_t ld_s, hipStream_t stream);

/*
 * epikv_select -- positions that survive (Sec. 3.1, Sec. 3.3, App. D).
 *
 * Per sequence with N = n_cached[b] and P = n_prefix[b]:
 *   N <= K          keep all: keep_idx = 0..N-1, n_keep = N;
 *   P + R >= K < N  seq_status BUDGET, n_keep = -1;
 *   otherwise       keep [0, P), [N-R, N) and the K-P-R best positions of
 *                   [P, N-R): higher score first, equal scores by lower
 *                   position, -0 equal to +0, NaN below every number.
 *                   n_keep = K.
 * keep_idx is int32 [B][K], ascending.  scores float [B][ld_s].
 * N < 0, N > ld_s, P < 0: seq_status RANGE, n_keep = -1.
 */
int epikv_select(const epikv_cfg* cfg, const float* scores, int64_t ld_s,
                 const int32_t* n_cached, const int32_t* n_prefix,
                 int32_t* keep_idx, int32_t* n_keep, int32_t* seq_status,
                 hipStream_t stream);

/* Device scratch of epikv_select_ws: for batches of up to 128 sequences,
 * per sequence 256 bytes (a marker, a flag, a count) and three histograms
 * of 2048 uint32 bins, B*24832 bytes, then 2048 bytes (two counts per
 * workgroup, at most 256 workgroups), rounded up to 256; 0 for a larger
 * batch (never split) or an invalid cfg. */
size_t epikv_select_workspace_bytes(const epikv_cfg* cfg);

/*
 * epikv_select_ws -- epikv_select with device scratch, so that one
 * sequence's selection can be split over several workgroups (Sec. 3.1,
 * Sec. 3.3, App. D; the results are those of epikv_select, bit for bit).
 *
 * Worth it when the batch is too small to fill the device with one
 * workgroup per sequence (a single long prefill, a small decode batch):
 * each sequence's positions are cut into slices of 1024 to 16384, one per
 * workgroup, as few per workgroup as keep the grid within one workgroup
 * per compute unit; rows that one workgroup covers anyway, and batches
 * where the grid would not fit, run epikv_select's kernel.  The workgroups of a
 * sequence wait for each other between the radix passes; if they cannot all
 * be resident at once because other work holds the device for about a
 * second, the sequence is flagged EPIKV_SEQ_SYNC (n_keep = -1) instead of
 * waiting longer.
 *
 * workspace: epikv_select_workspace_bytes(cfg) bytes of device memory,
 * 16-byte aligned (EPIKV_EALIGN), overlapping none of the other arguments
 * (EPIKV_EALIAS); EPIKV_EWORKSPACE if it is missing or too small (it may be
 * NULL when that size is 0).  Any contents are accepted: a small fill
 * kernel clears the scratch at the start of every split call, so nothing
 * depends on what the memory held before, and the call may be captured in
 * a HIP graph.  Calls that share a workspace must not overlap in time.
 * Other arguments and errors as for epikv_select.
 */
int epikv_select_ws(const epikv_cfg* cfg, const float* scores, int64_t ld_s,
                    const int32_t* n_cached, const int32_t* n_prefix,
                    int32_t* keep_idx, int32_t* n_keep, int32_t* seq_status,
                    void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * epikv_compact -- order-preserving rebuild of the cache (App. H).
 *
 * For every sequence with n_keep[b] >= 0 and every j < n_keep[b]: the row
 * of position keep_idx[b][j] (through src_pt, int32 [B][ld_src_pt]) is
 * copied bit for bit to slot j (through dst_pt, int32 [B][ld_dst_pt]) for
 * every layer, K and V.  Slots >= n_keep[b] are not written.  When
 * src_scores/dst_scores (float [B][ld_s]) are given, dst_scores[b][j] =
 * src_scores[b][keep_idx[b][j]]; likewise src_pos/dst_pos (int32 [B][ld_s]).
 * Out of place: destination pages must not be source pages of any sequence
 * (not checked), and dst_scores/dst_pos must not overlap their sources.
 * Rows whose index or page id is out of range are skipped and set
 * seq_status[b] = RANGE when seq_status is given.
 * workspace: 16-byte aligned device scratch of at least
 * epikv_compact_workspace_bytes(cfg) bytes (the resolved row offsets); it
 * must not overlap any other argument.
 */
int epikv_compact(const epikv_cfg* cfg, const epikv_pool* src,
                  const int32_t* src_pt, int64_t ld_src_pt,
                  const epikv_pool* dst, const int32_t* dst_pt,
                  int64_t ld_dst_pt, const int32_t* keep_idx,
                  const int32_t* n_keep, const float* src_scores,
                  float* dst_scores, const int32_t* src_pos, int32_t* dst_pos,
                  int64_t ld_s, int32_t* seq_status, void* workspace,
                  size_t workspace_bytes, hipStream_t stream);

/*
 * epikv_compact_inplace -- the same rebuild inside the sequence's own pages
 * (the move-minimising form of App. H's rebuild; no second pool).
 *
 * page_table (int32 [B][ld_pt]) maps the sequence's positions to pages of
 * `pool` both before and after the call.  For every sequence with
 * n_keep[b] > 0 and every j < min(n_keep[b], K): slot j receives, bit for
 * bit, the row that position keep_idx[b][j] held before the call, for every
 * layer, K and V.  keep_idx must be strictly ascending (as epikv_select
 * writes it), so rows only move towards the front.  Slots before the first
 * hole (the first j with keep_idx[b][j] != j) are not written, nor is any
 * slot >= n_keep[b]: pages wholly inside that leading run -- for instance
 * prefill pages shared between sequences and protected by n_prefix -- are
 * never touched, and pages past ceil(n_keep / page_size) may be released by
 * the caller afterwards.  scores (float [B][ld_s]) and pos (int32 [B][ld_s])
 * are optional and move the same way, in place.
 *
 * Pages of one sequence must not be pages of another sequence unless they
 * lie in that leading run.  A sequence whose keep_idx is not strictly
 * ascending, reaches a page id outside [0, n_pages) or past ld_pt, or (with
 * scores/pos) a position >= ld_s, is left untouched and flagged
 * seq_status[b] = RANGE (when seq_status is given).  Sequences with
 * n_keep[b] <= 0 are skipped.
 * workspace: 16-byte aligned device scratch of at least
 * epikv_compact_workspace_bytes(cfg) bytes, overlapping no other argument.
 */
int epikv_compact_inplace(const epikv_cfg* cfg, const epikv_pool* pool,
                          const int32_t* page_table, int64_t ld_pt,
                          const int32_t* keep_idx, const int32_t* n_keep,
                          float* scores, int32_t* pos, int64_t ld_s,
                          int32_t* seq_status, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/*
 * epikv_compact_remap -- epikv_compact_inplace with whole-page retention
 * (the page-table form of the move-minimising rebuild of App. H).
 *
 * The result, read through the page table after the call, is the same as
 * epikv_compact_inplace's: slot j < min(n_keep[b], K) holds the row position
 * keep_idx[b][j] held before, for every layer, K and V.  But a full
 * destination page m whose page_size slots receive, in order, every row of
 * one source page p > m is not copied: page_table[b][m] takes that page.  The
 * pages of such destinations that are not themselves such sources go, k-th
 * to k-th in ascending position order, to the positions of the sources that
 * are not themselves such destinations.  page_table[b] stays a permutation
 * of its old entries (only positions below ceil((keep_idx[b][n_keep-1]+1) /
 * page_size) change), so the sequence owns the same pages; rows are written
 * only at slots >= the first hole that lie outside remapped pages.  Evicting
 * whole aligned pages therefore moves no row at all.
 *
 * page_table (int32 [B][ld_pt]) is read and rewritten on the device; it must
 * overlap neither keep_idx, n_keep nor the workspace (EPIKV_EALIAS).  Everything else -- arguments,
 * checks, flagged sequences (left untouched, table included), the optional
 * scores and pos, the workspace -- is as for epikv_compact_inplace.
 */
int epikv_compact_remap(const epikv_cfg* cfg, const epikv_pool* pool,
                        int32_t* page_table, int64_t ld_pt,
                        const int32_t* keep_idx, const int32_t* n_keep,
                        float* scores, int32_t* pos, int64_t ld_s,
                        int32_t* seq_status, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* Arguments of one eviction step (host struct; pointers as above). */
typedef struct epikv_step_io {
  int32_t chunk;                /* new tokens per sequence (eviction cadence) */
  const void* const* hidden;    /* HS: host array of n_band device pointers */
  int64_t ld_tok, ld_seq;
  const int32_t* n_cached;      /* [B] cached tokens incl. the new chunk */
  const int32_t* n_prefix;      /* [B] prefill tokens, always kept */
  epikv_pool src;               /* cache before the step */
  const int32_t* src_pt;
  int64_t ld_src_pt;
  epikv_pool dst;               /* cache after the step (disjoint pages) */
  const int32_t* dst_pt;
  int64_t ld_dst_pt;
  float* scores;                /* [B][ld_s] frozen scores; the chunk's are written */
  float* dst_scores;            /* [B][ld_s] compacted scores (optional) */
  const int32_t* src_pos;       /* [B][ld_s] optional token ids ... */
  int32_t* dst_pos;             /* ... and their compacted copy */
  int64_t ld_s;
  const void* state_in;
  void* state_out;
  int32_t* keep_idx;            /* [B][K] */
  int32_t* n_keep;              /* [B] */
  int32_t* seq_status;          /* [B] */
  void* workspace;
  size_t workspace_bytes;       /* >= epikv_workspace_bytes(cfg, chunk) */
  int32_t in_place;             /* EPIKV_COMPACT_OUT_OF_PLACE (0): epikv_compact
                                   from src/src_pt into dst/dst_pt.
                                   EPIKV_COMPACT_IN_PLACE (1): compact with
                                   epikv_compact_inplace on src/src_pt; dst
                                   and dst_pt are ignored, scores always
                                   follow their rows in place, dst_scores
                                   must be NULL or scores, and dst_pos must
                                   equal src_pos (moved in place).
                                   EPIKV_COMPACT_REMAP (2): the same with
                                   epikv_compact_remap: src_pt is rewritten
                                   on the device, so it must point to
                                   writable memory (and overlap neither
                                   keep_idx, n_keep nor the workspace).
                                   Other values: EPIKV_EINVAL_PARAM. */
} epikv_step_io;

/*
 * epikv_evict_step -- score, zscore, select and compact in one call, all on
 * `stream`, with no host synchronisation.  Equivalent to the four calls
 * above with the signal in the workspace; sequences with n_cached < chunk
 * are flagged RANGE by the select stage.
 * chunk = 0 is the step of the online regime (Sec. 3.3), where every token
 * was scored as it was generated (epikv_score_tokens) and its score is
 * already frozen in `scores`: select and compact only.  hidden, state_in
 * and state_out are then not used (may be NULL), and the workspace needs
 * epikv_workspace_bytes(cfg, 0) bytes.
 * The selection runs epikv_select_ws's kernels with their scratch at the
 * start of the workspace, where it is kept from one step to the next (when
 * the chunk lies inside the recency window it runs epikv_select's instead,
 * beside the scoring).
 */
int epikv_evict_step(const epikv_cfg* cfg, const epikv_step_io* io,
                     hipStream_t stream);

/* Size of the scratch array behind epikv_evict_step_noalloc (per GPU). */
#define EPIKV_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * epikv_evict_step_noalloc -- epikv_evict_step for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.
 *
 * Same arguments and results as epikv_evict_step, except that
 * io->workspace and io->workspace_bytes are ignored: the step's scratch is
 * a file-scope device array of EPIKV_NOALLOC_SCRATCH_BYTES (16 MiB) inside
 * the library, one per GPU, held until the process ends.  A step that needs
 * more than that (epikv_workspace_bytes(cfg, io->chunk) above the limit)
 * returns EPIKV_EWORKSPACE before anything is enqueued.  Nothing is
 * allocated.
 *
 * The first call on a device looks the array's device address up
 * (hipGetSymbolAddress, with that device current); make it outside stream
 * capture.  `stream` must belong to the calling thread's current device
 * (else EPIKV_EINVAL_PARAM); the address lookup failing returns
 * EPIKV_ELAUNCH.  Every call on one GPU shares its array, which keeps the
 * last call's contents (the step writes everything it reads from it, the
 * selection's scratch through a clearing kernel): calls that overlap in
 * time on one GPU -- on two streams, or from two threads -- race and must
 * not be issued.
 */
int epikv_evict_step_noalloc(const epikv_cfg* cfg, const epikv_step_io* io,
                             hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* EPIKV_H */
