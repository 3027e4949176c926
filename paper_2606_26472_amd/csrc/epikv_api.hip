// C-ABI host layer: argument validation, state/workspace layout and kernel
// launches.  Every host-detectable error is returned before anything is
// enqueued; nothing here allocates, synchronises or keeps global state.
#include <math.h>

#include <algorithm>
#include <string.h>

#include "epikv_internal.h"

#define EPIKV_EXPORT extern "C" __attribute__((visibility("default")))

namespace epikv {


namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int n_band(const epikv_cfg* c) { return c->n_band_a + c->n_band_b; }

int n_sig(const epikv_cfg* c) { return c->signal == EPIKV_SIGNAL_HS ? n_band(c) : 1; }

bool is_kv(int signal) { return signal != EPIKV_SIGNAL_HS; }

bool uses_range(int signal) {
  return signal == EPIKV_SIGNAL_LAGKV || signal == EPIKV_SIGNAL_LAGKV_KEY;
}

int recent_of(const epikv_cfg* c) {
  return c->recent >= 0 ? c->recent : (c->budget / 4 < 128 ? c->budget / 4 : 128);
}

int row_bytes(const epikv_cfg* c) { return c->n_kv_heads * c->head_dim * 2; }

int pages_for(int64_t tokens, int page_size) { return (int)((tokens + page_size - 1) / page_size); }

constexpr int kSections = 5;

struct Layout {
  size_t off[kSections];
  size_t size[kSections];
  size_t total;
};

Layout state_layout(const epikv_cfg* c) {
  Layout L;
  const size_t B = (size_t)c->batch;
  L.size[0] = 4 * B;
  L.size[1] = 4 * B * (size_t)n_sig(c) * (size_t)(c->window - 1);
  L.size[2] = c->signal == EPIKV_SIGNAL_HS ? 2 * B * (size_t)n_band(c) * (size_t)c->hidden : 0;
  L.size[3] = uses_range(c->signal)
                  ? 4 * 2 * B * (size_t)c->n_layers * 2 * (size_t)c->n_kv_heads * (size_t)c->head_dim
                  : 0;
  L.size[4] = 4 * B * (size_t)n_sig(c);
  size_t o = 0;
  for (int i = 0; i < kSections; ++i) {
    L.off[i] = o;
    o = align_up(o + L.size[i]);
  }
  L.total = o;
  return L;
}

size_t sig_bytes(const epikv_cfg* c, int chunk) {
  return align_up(4 * (size_t)n_sig(c) * (size_t)c->batch * (size_t)chunk);
}

int budget_pages(const epikv_cfg* c) {
  return (int)(((int64_t)c->budget + c->page_size - 1) / c->page_size);
}

// Row offset records, 16 bytes per slot of the budget's pages (out of
// place: in destination-page rank order; in place: [B][K]), then (in place)
// [B][2] int32, then [B][4][ceil(K / page_size)] int32 (page remapping;
// out of place, the first [B][ceil(K / page_size)] hold the destination
// pages' ranks).
size_t compact_records_bytes(const epikv_cfg* c) {
  return align_up(16 * (size_t)c->batch * (size_t)budget_pages(c) * (size_t)c->page_size);
}

size_t compact_ws_bytes(const epikv_cfg* c) {
  return compact_records_bytes(c) + align_up(8 * (size_t)c->batch) +
         align_up(16 * (size_t)c->batch * (size_t)budget_pages(c));
}

// Planes the KV-vector scorer reads: every (layer, K|V) for Lag-KV, the
// layers of the one tensor otherwise.
int lag_planes(const epikv_cfg* c) {
  return (c->signal == EPIKV_SIGNAL_LAGKV ? 2 : 1) * c->n_layers;
}

// Workgroups sharing the rows of one (sequence, plane) in the KV-vector
// scorer: enough for about kLagWgWanted workgroups, each wavefront keeping
// at least its rows in flight busy.
int lag_splits(const epikv_cfg* c, int chunk) {
  const bool lag = uses_range(c->signal);
  const int64_t base = (int64_t)lag_planes(c) * c->batch;
  const bool big = lagkv_big(c->n_kv_heads, c->head_dim, lag, base);
  const int64_t wanted = big ? kLagWgWanted / 2 : kLagWgWanted;
  const int64_t s = (wanted + base - 1) / base;
  const int64_t cap = std::max<int64_t>(1, chunk / (lagkv_waves(lag, big) * lagkv_ahead(lag)));
  return (int)std::max<int64_t>(1, std::min(s, cap));
}

// Partial channel ranges of the shares, when a plane's rows are split.
size_t prange_bytes(const epikv_cfg* c, int chunk) {
  if (!uses_range(c->signal) || lag_splits(c, chunk) == 1) return 0;
  return align_up(4 * (size_t)lag_splits(c, chunk) * 2 * (size_t)c->batch * (size_t)c->n_layers *
                  2 * (size_t)c->n_kv_heads * (size_t)c->head_dim);
}


// Per-(sequence, plane, row segment, token) sums of the heads' variances,
// then the shares' partial channel ranges.
size_t plane_sums_bytes(const epikv_cfg* c, int chunk) {
  const int segs = lagkv_segments(c->n_kv_heads, c->head_dim, uses_range(c->signal));
  return align_up(4 * (size_t)c->batch * (size_t)lag_planes(c) * (size_t)segs * (size_t)chunk);
}

size_t partial_bytes(const epikv_cfg* c, int chunk) {
  if (!is_kv(c->signal)) return 0;
  return plane_sums_bytes(c, chunk) + prange_bytes(c, chunk);
}

int check_cfg(const epikv_cfg* c) {
  if (!c) return EPIKV_EINVAL_NULL;
  if (c->signal < EPIKV_SIGNAL_HS || c->signal > EPIKV_SIGNAL_LAGKV_KEY) return EPIKV_EINVAL_PARAM;
  if (c->smoothing < EPIKV_SMOOTH_Z || c->smoothing > EPIKV_SMOOTH_EMA) return EPIKV_EINVAL_PARAM;
  if (!(c->ema_alpha >= 0.f && c->ema_alpha <= 1.f)) return EPIKV_EINVAL_PARAM;
  if (c->window < 1 || c->window > EPIKV_MAX_WINDOW) return EPIKV_EINVAL_PARAM;
  if (!(c->eps >= 0.f) || !isfinite(c->eps)) return EPIKV_EINVAL_PARAM;
  if (c->budget < 1) return EPIKV_EINVAL_PARAM;
  if (c->recent < -1) return EPIKV_EINVAL_PARAM;
  if (c->batch < 1 || c->batch > 65535) return EPIKV_EINVAL_SHAPE;
  if (c->page_size < 1 || c->page_size > 1024) return EPIKV_EINVAL_SHAPE;
  if (c->n_layers < 1 || c->n_layers > 1024) return EPIKV_EINVAL_SHAPE;
  if (c->n_kv_heads < 1) return EPIKV_EINVAL_SHAPE;
  if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256) return EPIKV_EINVAL_SHAPE;
  const int hd = c->n_kv_heads * c->head_dim;
  if (hd > 2048) return EPIKV_EINVAL_SHAPE;
  const int row_vec = hd / 8;
  // One row of one plane is streamed by one wavefront (at most 4 16-byte
  // columns per lane): H*d <= 2048 guarantees it.
  if (is_kv(c->signal) && (kScoreThreads % row_vec) != 0) return EPIKV_EINVAL_SHAPE;
  if (c->signal == EPIKV_SIGNAL_HS) {
    if (c->n_band_a < 1 || c->n_band_b < 0 || n_band(c) > EPIKV_MAX_BAND) return EPIKV_EINVAL_SHAPE;
    if (c->hidden < 8 || c->hidden > 16384 || (c->hidden % 8) != 0) return EPIKV_EINVAL_SHAPE;
  }
  return EPIKV_OK;
}

int check_pool(const epikv_pool* p) {
  if (!p || !p->base) return EPIKV_EINVAL_NULL;
  if (p->n_pages < 1 || p->n_pages > INT32_MAX) return EPIKV_EINVAL_SHAPE;
  if (p->stride_layer < 0 || p->stride_kv < 0 || p->stride_page < 0) return EPIKV_EINVAL_SHAPE;
  if (!aligned16(p->base) || (p->stride_layer % 16) || (p->stride_kv % 16) || (p->stride_page % 16))
    return EPIKV_EALIGN;
  return EPIKV_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

int launched(hipError_t e) { return e == hipSuccess ? EPIKV_OK : EPIKV_ELAUNCH; }

// ---------------------------------------------------------------------------
// Per-stage validation + argument building
// ---------------------------------------------------------------------------
// The state pair: both present, aligned, and not overlapping (a step reads
// the whole input state after writing parts of the output).
int check_state_pair(const epikv_cfg* c, const void* state_in, void* state_out) {
  if (!state_in || !state_out) return EPIKV_EINVAL_NULL;
  if (!aligned16(state_in) || !aligned16(state_out)) return EPIKV_EALIGN;
  const size_t sb = state_layout(c).total;
  if (overlap(state_in, sb, state_out, sb)) return EPIKV_EALIAS;
  return EPIKV_OK;
}

// The band-layer hidden states of a chunk: one aligned pointer per band
// layer, rows of D elements at ld_tok, sequences at ld_seq.
int check_hidden(const epikv_cfg* c, int32_t chunk, const void* const* hidden, int64_t ld_tok,
                 int64_t ld_seq) {
  if (!hidden) return EPIKV_EINVAL_NULL;
  for (int l = 0; l < n_band(c); ++l) {
    if (!hidden[l]) return EPIKV_EINVAL_NULL;
    if (!aligned16(hidden[l])) return EPIKV_EALIGN;
  }
  if (ld_tok < 0 || ld_seq < 0) return EPIKV_EINVAL_SHAPE;
  if (chunk > 1 && ld_tok < c->hidden) return EPIKV_EINVAL_SHAPE;
  if ((ld_tok % 8) || (ld_seq % 8)) return EPIKV_EALIGN;
  return EPIKV_OK;
}

int check_score(const epikv_cfg* c, int32_t chunk, const void* const* hidden, int64_t ld_tok,
                int64_t ld_seq, const epikv_pool* pool, const int32_t* page_table, int64_t ld_pt,
                const int32_t* n_cached, const void* state_in, void* state_out, float* sig,
                void* ws, size_t ws_bytes, bool check_ws) {
  int st = check_cfg(c);
  if (st) return st;
  if (!state_in || !state_out || !sig) return EPIKV_EINVAL_NULL;
  if (chunk < 1) return EPIKV_EINVAL_SHAPE;
  st = check_state_pair(c, state_in, state_out);
  if (st) return st;
  if (c->signal == EPIKV_SIGNAL_HS) {
    st = check_hidden(c, chunk, hidden, ld_tok, ld_seq);
    if (st) return st;
  } else {
    st = check_pool(pool);
    if (st) return st;
    if (!page_table || !n_cached) return EPIKV_EINVAL_NULL;
    if (ld_pt < 1) return EPIKV_EINVAL_SHAPE;
    if (check_ws) {
      if (!ws || ws_bytes < sig_bytes(c, chunk) + partial_bytes(c, chunk)) return EPIKV_EWORKSPACE;
      if (!aligned16(ws)) return EPIKV_EALIGN;
    }
  }
  return EPIKV_OK;
}

ScoreHsArgs hs_args(const epikv_cfg* c, int32_t chunk, const void* const* hidden, int64_t ld_tok,
                    int64_t ld_seq, const void* state_in, void* state_out, float* sig) {
  const Layout L = state_layout(c);
  ScoreHsArgs a;
  memset(&a, 0, sizeof(a));
  for (int l = 0; l < n_band(c); ++l) a.hidden[l] = (const uint16_t*)hidden[l];
  a.ld_tok = ld_tok;
  a.ld_seq = ld_seq;
  a.B = c->batch;
  a.C = chunk;
  a.D = c->hidden;
  a.n_band = n_band(c);
  a.seg_len = kScoreSeg;
  a.n_tok_in = (const int32_t*)state_in;
  a.h_prev_in = (const uint16_t*)((const char*)state_in + L.off[2]);
  a.h_prev_out = (uint16_t*)((char*)state_out + L.off[2]);
  a.sig = sig;
  return a;
}

void lag_args(const epikv_cfg* c, int32_t chunk, const epikv_pool* pool, const int32_t* pt,
              int64_t ld_pt, const int32_t* n_cached, const void* state_in, void* state_out,
              float* sig, float* partial, ScoreLagArgs* a, LagReduceArgs* r) {
  const Layout L = state_layout(c);
  a->base = (const char*)pool->base;
  a->s_layer = pool->stride_layer;
  a->s_kv = pool->stride_kv;
  a->s_page = pool->stride_page;
  a->n_pages = pool->n_pages;
  a->pt = pt;
  a->ld_pt = ld_pt;
  a->n_cached = n_cached;
  a->B = c->batch;
  a->C = chunk;
  a->L = c->n_layers;
  a->H = c->n_kv_heads;
  a->d = c->head_dim;
  a->page_size = c->page_size;
  a->page_shift = -1;
  for (int sh = 0; sh < 31; ++sh)
    if ((1 << sh) == c->page_size) a->page_shift = sh;
  const bool use_k = c->signal != EPIKV_SIGNAL_KV_VAL;
  const bool use_v = c->signal == EPIKV_SIGNAL_LAGKV || c->signal == EPIKV_SIGNAL_KV_VAL;
  a->lag = uses_range(c->signal);
  a->n_planes = lag_planes(c);
  a->two = use_k && use_v;
  a->kv0 = use_k ? 0 : 1;
  a->eps = c->eps;
  a->n_tok_in = (const int32_t*)state_in;
  a->range_in = (const float*)((const char*)state_in + L.off[3]);
  a->range_out = (float*)((char*)state_out + L.off[3]);
  a->partial = partial;
  a->splits = lag_splits(c, chunk);
  a->prange = prange_bytes(c, chunk) ? (float*)((char*)partial + plane_sums_bytes(c, chunk))
                                     : nullptr;
  r->partial = partial;
  r->sig = sig;
  r->B = c->batch;
  r->C = chunk;
  r->L = c->n_layers;
  r->n_sums = a->n_planes * lagkv_segments(c->n_kv_heads, c->head_dim, a->lag);
  r->inv_count = 1.0f / (float)(c->n_layers * c->n_kv_heads);
  r->lag = a->lag;
  r->use_k = use_k;
  r->use_v = use_v;
  r->splits = a->splits;
  r->n_chan = c->n_layers * 2 * c->n_kv_heads * c->head_dim;
  r->prange = a->prange;
  r->range_out = a->range_out;
}

int run_score(const epikv_cfg* c, int32_t chunk, const void* const* hidden, int64_t ld_tok,
              int64_t ld_seq, const epikv_pool* pool, const int32_t* pt, int64_t ld_pt,
              const int32_t* n_cached, const void* state_in, void* state_out, float* sig,
              float* partial, hipStream_t s) {
  if (c->signal == EPIKV_SIGNAL_HS)
    return launched(launch_score_hs(hs_args(c, chunk, hidden, ld_tok, ld_seq, state_in, state_out, sig), s));
  ScoreLagArgs a;
  LagReduceArgs r;
  lag_args(c, chunk, pool, pt, ld_pt, n_cached, state_in, state_out, sig, partial, &a, &r);
  return launched(launch_score_lagkv(a, r, s));
}

int check_score_tokens(const epikv_cfg* c, int32_t chunk, const void* const* hidden,
                       int64_t ld_tok, int64_t ld_seq, const int32_t* n_cached,
                       const void* state_in, void* state_out, float* scores, int64_t ld_s) {
  int st = check_cfg(c);
  if (st) return st;
  if (c->signal != EPIKV_SIGNAL_HS) return EPIKV_EINVAL_PARAM;
  if (chunk < 1 || chunk > kZscoreTile || c->hidden > kTokMaxRow) return EPIKV_EINVAL_SHAPE;
  if (!n_cached || !scores || !state_in || !state_out) return EPIKV_EINVAL_NULL;
  if (ld_s < chunk) return EPIKV_EINVAL_SHAPE;
  st = check_state_pair(c, state_in, state_out);
  if (st) return st;
  return check_hidden(c, chunk, hidden, ld_tok, ld_seq);
}

ScoreTokArgs score_tokens_args(const epikv_cfg* c, int32_t chunk, const void* const* hidden,
                               int64_t ld_tok, int64_t ld_seq, const int32_t* n_cached,
                               const void* state_in, void* state_out, float* scores,
                               int64_t ld_s) {
  const Layout L = state_layout(c);
  ScoreTokArgs a;
  memset(&a, 0, sizeof(a));
  for (int l = 0; l < n_band(c); ++l) a.hidden[l] = (const uint16_t*)hidden[l];
  a.ld_tok = ld_tok;
  a.ld_seq = ld_seq;
  a.B = c->batch;
  a.C = chunk;
  a.D = c->hidden;
  a.n_band = n_band(c);
  a.n_a = c->n_band_a;
  a.n_b = c->n_band_b;
  a.w = c->window;
  a.mode = c->smoothing;
  a.eps = c->eps;
  a.alpha = c->ema_alpha;
  a.n_cached = n_cached;
  a.n_tok_in = (const int32_t*)state_in;
  a.ring_in = (const float*)((const char*)state_in + L.off[1]);
  a.h_prev_in = (const uint16_t*)((const char*)state_in + L.off[2]);
  a.ema_in = (const float*)((const char*)state_in + L.off[4]);
  a.n_tok_out = (int32_t*)state_out;
  a.ring_out = (float*)((char*)state_out + L.off[1]);
  a.h_prev_out = (uint16_t*)((char*)state_out + L.off[2]);
  a.ema_out = (float*)((char*)state_out + L.off[4]);
  a.scores = scores;
  a.ld_s = ld_s;
  return a;
}

int check_zscore(const epikv_cfg* c, int32_t chunk, const float* sig, const int32_t* n_cached,
                 const void* state_in, void* state_out, float* scores, int64_t ld_s) {
  int st = check_cfg(c);
  if (st) return st;
  if (!sig || !n_cached || !state_in || !state_out || !scores) return EPIKV_EINVAL_NULL;
  if (chunk < 1) return EPIKV_EINVAL_SHAPE;
  if (ld_s < chunk) return EPIKV_EINVAL_SHAPE;
  if (!aligned16(state_in) || !aligned16(state_out)) return EPIKV_EALIGN;
  const size_t sb = state_layout(c).total;
  if (overlap(state_in, sb, state_out, sb)) return EPIKV_EALIAS;
  return EPIKV_OK;
}

ZscoreArgs zscore_args(const epikv_cfg* c, int32_t chunk, const float* sig, const int32_t* n_cached,
                       const void* state_in, void* state_out, float* scores, int64_t ld_s,
                       float* smoothed) {
  const Layout L = state_layout(c);
  ZscoreArgs a;
  a.sig = sig;
  a.B = c->batch;
  a.C = chunk;
  a.n_sig = n_sig(c);
  a.n_a = c->signal == EPIKV_SIGNAL_HS ? c->n_band_a : 1;
  a.n_b = c->signal == EPIKV_SIGNAL_HS ? c->n_band_b : 0;
  a.w = c->window;
  a.mode = c->smoothing;
  a.hs = c->signal == EPIKV_SIGNAL_HS ? 1 : 0;
  a.eps = c->eps;
  a.n_cached = n_cached;
  a.n_tok_in = (const int32_t*)state_in;
  a.ring_in = (const float*)((const char*)state_in + L.off[1]);
  a.n_tok_out = (int32_t*)state_out;
  a.ring_out = (float*)((char*)state_out + L.off[1]);
  a.ema_in = (const float*)((const char*)state_in + L.off[4]);
  a.ema_out = (float*)((char*)state_out + L.off[4]);
  a.alpha = c->ema_alpha;
  a.scores = scores;
  a.ld_s = ld_s;
  a.smoothed = smoothed;
  return a;
}

int check_select(const epikv_cfg* c, const float* scores, int64_t ld_s, const int32_t* n_cached,
                 const int32_t* n_prefix, int32_t* keep_idx, int32_t* n_keep, int32_t* seq_status) {
  int st = check_cfg(c);
  if (st) return st;
  if (!scores || !n_cached || !n_prefix || !keep_idx || !n_keep || !seq_status) return EPIKV_EINVAL_NULL;
  if (ld_s < 1 || ld_s > INT32_MAX) return EPIKV_EINVAL_SHAPE;
  return EPIKV_OK;
}

// The split selection's scratch must not overlap what the selection reads
// or writes.
int check_select_scratch(const epikv_cfg* c, const float* scores, int64_t ld_s,
                         const int32_t* n_cached, const int32_t* n_prefix,
                         const int32_t* keep_idx, const int32_t* n_keep,
                         const int32_t* seq_status, const void* ws) {
  const size_t n = select_scratch_bytes(c->batch);
  if (n == 0) return EPIKV_OK;
  const size_t B = (size_t)c->batch;
  if (overlap(ws, n, scores, B * (size_t)ld_s * 4) || overlap(ws, n, n_cached, B * 4) ||
      overlap(ws, n, n_prefix, B * 4) || overlap(ws, n, keep_idx, B * (size_t)c->budget * 4) ||
      overlap(ws, n, n_keep, B * 4) || overlap(ws, n, seq_status, B * 4))
    return EPIKV_EALIAS;
  return EPIKV_OK;
}

SelectArgs select_args(const epikv_cfg* c, const float* scores, int64_t ld_s, const int32_t* n_cached,
                       const int32_t* n_prefix, int32_t* keep_idx, int32_t* n_keep,
                       int32_t* seq_status, int min_n) {
  SelectArgs a;
  a.scores = scores;
  a.ld_s = ld_s;
  a.n_cached = n_cached;
  a.n_prefix = n_prefix;
  a.B = c->batch;
  a.K = c->budget;
  a.R = recent_of(c);
  a.min_n = min_n;
  a.keep_idx = keep_idx;
  a.n_keep = n_keep;
  a.seq_status = seq_status;
  return a;
}

int check_compact(const epikv_cfg* c, const epikv_pool* src, const int32_t* src_pt, int64_t ld_src_pt,
                  const epikv_pool* dst, const int32_t* dst_pt, int64_t ld_dst_pt,
                  const int32_t* keep_idx, const int32_t* n_keep, const float* src_scores,
                  float* dst_scores, const int32_t* src_pos, int32_t* dst_pos, int64_t ld_s,
                  const void* ws, size_t ws_bytes) {
  int st = check_cfg(c);
  if (st) return st;
  if (!ws || ws_bytes < compact_ws_bytes(c)) return EPIKV_EWORKSPACE;
  if (!aligned16(ws)) return EPIKV_EALIGN;
  st = check_pool(src);
  if (st) return st;
  st = check_pool(dst);
  if (st) return st;
  if (!src_pt || !dst_pt || !keep_idx || !n_keep) return EPIKV_EINVAL_NULL;
  if ((src_scores == nullptr) != (dst_scores == nullptr)) return EPIKV_EINVAL_NULL;
  if ((src_pos == nullptr) != (dst_pos == nullptr)) return EPIKV_EINVAL_NULL;
  if (ld_src_pt < 1 || ld_dst_pt < pages_for(c->budget, c->page_size)) return EPIKV_EINVAL_SHAPE;
  if ((dst_scores || dst_pos) && ld_s < 1) return EPIKV_EINVAL_SHAPE;
  const size_t bytes = 4 * (size_t)c->batch * (size_t)(ld_s > 0 ? ld_s : 0);
  if (dst_scores && overlap(src_scores, bytes, dst_scores, bytes)) return EPIKV_EALIAS;
  if (dst_pos && overlap(src_pos, bytes, dst_pos, bytes)) return EPIKV_EALIAS;
  return EPIKV_OK;
}

CompactArgs compact_args(const epikv_cfg* c, const epikv_pool* src, const int32_t* src_pt,
                         int64_t ld_src_pt, const epikv_pool* dst, const int32_t* dst_pt,
                         int64_t ld_dst_pt, const int32_t* keep_idx, const int32_t* n_keep,
                         const float* src_scores, float* dst_scores, const int32_t* src_pos,
                         int32_t* dst_pos, int64_t ld_s, int32_t* seq_status, void* ws) {
  CompactArgs a;
  a.src = (const char*)src->base;
  a.s_layer = src->stride_layer;
  a.s_kv = src->stride_kv;
  a.s_page = src->stride_page;
  a.s_npages = src->n_pages;
  a.dst = (char*)dst->base;
  a.d_layer = dst->stride_layer;
  a.d_kv = dst->stride_kv;
  a.d_page = dst->stride_page;
  a.d_npages = dst->n_pages;
  a.src_pt = src_pt;
  a.ld_src_pt = ld_src_pt;
  a.dst_pt = dst_pt;
  a.ld_dst_pt = ld_dst_pt;
  a.keep_idx = keep_idx;
  a.n_keep = n_keep;
  a.src_scores = src_scores;
  a.dst_scores = dst_scores;
  a.src_pos = src_pos;
  a.dst_pos = dst_pos;
  a.ld_s = ld_s;
  a.seq_status = seq_status;
  a.offsets = (int64_t*)ws;
  a.rank = (int32_t*)((char*)ws + compact_records_bytes(c) + align_up(8 * (size_t)c->batch));
  a.B = c->batch;
  a.K = c->budget;
  a.page_size = c->page_size;
  a.row_bytes = row_bytes(c);
  a.n_lk = 2 * c->n_layers;
  a.n_pg = budget_pages(c);
  a.units = 0;
  return a;
}

int check_compact_inplace(const epikv_cfg* c, const epikv_pool* pool, const int32_t* pt,
                          int64_t ld_pt, const int32_t* keep_idx, const int32_t* n_keep,
                          const float* scores, const int32_t* pos, int64_t ld_s, const void* ws,
                          size_t ws_bytes) {
  int st = check_cfg(c);
  if (st) return st;
  if (!ws || ws_bytes < compact_ws_bytes(c)) return EPIKV_EWORKSPACE;
  if (!aligned16(ws)) return EPIKV_EALIGN;
  st = check_pool(pool);
  if (st) return st;
  if (!pt || !keep_idx || !n_keep) return EPIKV_EINVAL_NULL;
  if (ld_pt < 1) return EPIKV_EINVAL_SHAPE;
  if ((scores || pos) && (ld_s < 1 || ld_s > INT32_MAX)) return EPIKV_EINVAL_SHAPE;
  const size_t bytes = 4 * (size_t)c->batch * (size_t)(ld_s > 0 ? ld_s : 0);
  if (scores && pos && overlap(scores, bytes, pos, bytes)) return EPIKV_EALIAS;
  return EPIKV_OK;
}

InplaceArgs inplace_args(const epikv_cfg* c, const epikv_pool* pool, const int32_t* pt,
                         int64_t ld_pt, const int32_t* keep_idx, const int32_t* n_keep,
                         float* scores, int32_t* pos, int64_t ld_s, int32_t* seq_status,
                         void* ws) {
  InplaceArgs a;
  a.pool = (char*)pool->base;
  a.s_layer = pool->stride_layer;
  a.s_kv = pool->stride_kv;
  a.s_page = pool->stride_page;
  a.n_pages = pool->n_pages;
  a.pt = pt;
  a.ld_pt = ld_pt;
  a.keep_idx = keep_idx;
  a.n_keep = n_keep;
  a.scores = scores;
  a.pos = pos;
  a.ld_s = ld_s;
  a.seq_status = seq_status;
  a.offsets = (int64_t*)ws;
  a.info = (int32_t*)((char*)ws + compact_records_bytes(c));
  a.remap = 0;
  a.pt_out = nullptr;
  a.remap_ws = (int32_t*)((char*)ws + compact_records_bytes(c) + align_up(8 * (size_t)c->batch));
  a.n_pg = budget_pages(c);
  a.B = c->batch;
  a.K = c->budget;
  a.page_size = c->page_size;
  a.row_bytes = row_bytes(c);
  a.n_lk = 2 * c->n_layers;
  // A wavefront per (sequence, plane, column slice): the widest slice --
  // 1 KiB or 256 B, that is 64 or 16 lanes per row -- that still gives
  // enough independent walks to keep HBM busy (each walk has one tile in
  // flight), with tiles of 16 and 32 rows.  Short of that (a few sequences)
  // the walks stay 256 B wide and take 64-row tiles instead: narrower
  // slices would give more walks, but 64-byte pieces of rows use HBM poorly
  // (measured 2.7 TB/s at 64 B against 4.5 TB/s at 256 B for one
  // sequence).  Rows narrower than 256 B use 64-byte slices.
  const int row_vec = a.row_bytes / 16;
  auto walks = [&](int lpr) { return (int64_t)a.B * a.n_lk * ((row_vec + lpr - 1) / lpr); };
  if (row_vec >= 64 && walks(64) >= kInplaceUnitsWanted) {
    a.lanes_per_row = 64;
    a.tile_ni = 16;
  } else if (row_vec >= 16) {
    a.lanes_per_row = 16;
    a.tile_ni = walks(16) >= kInplaceUnitsWanted ? 8 : 16;
  } else {
    a.lanes_per_row = 4;
    a.tile_ni = walks(4) >= kInplaceUnitsWanted ? 4 : 16;
  }
  a.n_slices = (row_vec + a.lanes_per_row - 1) / a.lanes_per_row;
  return a;
}

// The page table that epikv_compact_remap rewrites must not overlap what
// the device reads while it is being rewritten.
int check_remap_table(const epikv_cfg* c, const int32_t* pt, int64_t ld_pt, const int32_t* keep_idx,
                      const int32_t* n_keep, const void* ws, size_t ws_bytes) {
  const size_t pt_bytes = 4 * (size_t)c->batch * (size_t)ld_pt;
  if (overlap(pt, pt_bytes, keep_idx, 4 * (size_t)c->batch * (size_t)c->budget) ||
      overlap(pt, pt_bytes, n_keep, 4 * (size_t)c->batch) || overlap(pt, pt_bytes, ws, ws_bytes))
    return EPIKV_EALIAS;
  return EPIKV_OK;
}

InplaceArgs remap_args(InplaceArgs a, int32_t* pt) {
  a.remap = 1;
  a.pt_out = pt;
  return a;
}

__global__ void k_fill(FillArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = i; k < a.n_words; k += stride) a.p[k] = a.value;
}

}  // namespace

hipError_t launch_fill(const FillArgs& a, hipStream_t s) {
  int64_t blocks = (a.n_words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace epikv

using namespace epikv;

// ---------------------------------------------------------------------------
// Exported entry points
// ---------------------------------------------------------------------------
EPIKV_EXPORT int epikv_default_cfg(epikv_cfg* cfg) {
  if (!cfg) return EPIKV_EINVAL_NULL;
  cfg->batch = 1;
  cfg->hidden = 4096;
  cfg->n_layers = 32;
  cfg->n_kv_heads = 8;
  cfg->head_dim = 128;
  cfg->page_size = 16;
  cfg->n_band_a = 7;
  cfg->n_band_b = 8;
  cfg->window = 64;
  cfg->eps = 1e-6f;
  cfg->signal = EPIKV_SIGNAL_HS;
  cfg->smoothing = EPIKV_SMOOTH_Z;
  cfg->budget = 4096;
  cfg->recent = -1;
  cfg->ema_alpha = 0.9f;
  return EPIKV_OK;
}

EPIKV_EXPORT const char* epikv_strerror(int status) {
  switch (status) {
    case EPIKV_OK: return "ok";
    case EPIKV_EINVAL_NULL: return "a required pointer is NULL";
    case EPIKV_EINVAL_SHAPE: return "a size is outside the supported range";
    case EPIKV_EINVAL_PARAM: return "invalid parameter (budget, window, eps or enum)";
    case EPIKV_EALIGN: return "pointer, stride or leading dimension misaligned";
    case EPIKV_EWORKSPACE: return "workspace missing or too small";
    case EPIKV_EALIAS: return "an output overlaps an input it must not overlap";
    case EPIKV_ELAUNCH: return "kernel launch failed";
    default: return "unknown status";
  }
}

EPIKV_EXPORT int epikv_check_cfg(const epikv_cfg* cfg) { return check_cfg(cfg); }

EPIKV_EXPORT size_t epikv_state_bytes(const epikv_cfg* cfg) {
  if (check_cfg(cfg)) return 0;
  return state_layout(cfg).total;
}

EPIKV_EXPORT int epikv_state_layout(const epikv_cfg* cfg, size_t offsets[5]) {
  const int st = check_cfg(cfg);
  if (st) return st;
  if (!offsets) return EPIKV_EINVAL_NULL;
  const Layout L = state_layout(cfg);
  for (int i = 0; i < kSections; ++i) offsets[i] = L.off[i];
  return EPIKV_OK;
}

EPIKV_EXPORT size_t epikv_workspace_bytes(const epikv_cfg* cfg, int32_t chunk) {
  if (check_cfg(cfg) || chunk < 0) return 0;
  const size_t fixed = select_scratch_bytes(cfg->batch) + compact_ws_bytes(cfg);
  if (chunk == 0) return fixed;  // a step without scoring
  return fixed + sig_bytes(cfg, chunk) + partial_bytes(cfg, chunk);
}

EPIKV_EXPORT size_t epikv_compact_workspace_bytes(const epikv_cfg* cfg) {
  if (check_cfg(cfg)) return 0;
  return compact_ws_bytes(cfg);
}

EPIKV_EXPORT int epikv_state_init(const epikv_cfg* cfg, void* state, hipStream_t stream) {
  const int st = check_cfg(cfg);
  if (st) return st;
  if (!state) return EPIKV_EINVAL_NULL;
  if (!aligned16(state)) return EPIKV_EALIGN;
  FillArgs f;
  f.p = (uint32_t*)state;
  f.n_words = (int64_t)(state_layout(cfg).total / 4);
  f.value = 0u;
  return launched(launch_fill(f, stream));
}

EPIKV_EXPORT int epikv_score(const epikv_cfg* cfg, int32_t chunk, const void* const* hidden,
                             int64_t ld_tok, int64_t ld_seq, const epikv_pool* pool,
                             const int32_t* page_table, int64_t ld_pt, const int32_t* n_cached,
                             const void* state_in, void* state_out, float* sig, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  const int st = check_score(cfg, chunk, hidden, ld_tok, ld_seq, pool, page_table, ld_pt, n_cached,
                             state_in, state_out, sig, workspace, workspace_bytes, true);
  if (st) return st;
  // Standalone: the Lag-KV partial sums use the start of the workspace.
  return run_score(cfg, chunk, hidden, ld_tok, ld_seq, pool, page_table, ld_pt, n_cached, state_in,
                   state_out, sig, (float*)workspace, stream);
}

EPIKV_EXPORT int epikv_zscore(const epikv_cfg* cfg, int32_t chunk, const float* sig,
                              const int32_t* n_cached, const void* state_in, void* state_out,
                              float* scores, int64_t ld_s, float* smoothed, hipStream_t stream) {
  const int st = check_zscore(cfg, chunk, sig, n_cached, state_in, state_out, scores, ld_s);
  if (st) return st;
  return launched(launch_zscore(
      zscore_args(cfg, chunk, sig, n_cached, state_in, state_out, scores, ld_s, smoothed), stream));
}

EPIKV_EXPORT int epikv_score_tokens(const epikv_cfg* cfg, int32_t chunk, const void* const* hidden,
                                    int64_t ld_tok, int64_t ld_seq, const int32_t* n_cached,
                                    const void* state_in, void* state_out, float* scores,
                                    int64_t ld_s, hipStream_t stream) {
  const int st = check_score_tokens(cfg, chunk, hidden, ld_tok, ld_seq, n_cached, state_in,
                                    state_out, scores, ld_s);
  if (st) return st;
  return launched(launch_score_tokens(score_tokens_args(cfg, chunk, hidden, ld_tok, ld_seq, n_cached,
                                                        state_in, state_out, scores, ld_s),
                                      stream));
}

EPIKV_EXPORT int epikv_select(const epikv_cfg* cfg, const float* scores, int64_t ld_s,
                              const int32_t* n_cached, const int32_t* n_prefix, int32_t* keep_idx,
                              int32_t* n_keep, int32_t* seq_status, hipStream_t stream) {
  const int st = check_select(cfg, scores, ld_s, n_cached, n_prefix, keep_idx, n_keep, seq_status);
  if (st) return st;
  return launched(launch_select(
      select_args(cfg, scores, ld_s, n_cached, n_prefix, keep_idx, n_keep, seq_status, 0), stream));
}

EPIKV_EXPORT size_t epikv_select_workspace_bytes(const epikv_cfg* cfg) {
  if (check_cfg(cfg)) return 0;
  return select_scratch_bytes(cfg->batch);
}

EPIKV_EXPORT int epikv_select_ws(const epikv_cfg* cfg, const float* scores, int64_t ld_s,
                                 const int32_t* n_cached, const int32_t* n_prefix,
                                 int32_t* keep_idx, int32_t* n_keep, int32_t* seq_status,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = check_select(cfg, scores, ld_s, n_cached, n_prefix, keep_idx, n_keep, seq_status);
  if (st) return st;
  const size_t need = select_scratch_bytes(cfg->batch);
  if (need > 0) {
    if (!workspace || workspace_bytes < need) return EPIKV_EWORKSPACE;
    if (!aligned16(workspace)) return EPIKV_EALIGN;
    st = check_select_scratch(cfg, scores, ld_s, n_cached, n_prefix, keep_idx, n_keep, seq_status,
                              workspace);
    if (st) return st;
  }
  const SelectArgs a =
      select_args(cfg, scores, ld_s, n_cached, n_prefix, keep_idx, n_keep, seq_status, 0);
  return launched(need > 0 ? launch_select_groups(a, workspace, stream) : launch_select(a, stream));
}

EPIKV_EXPORT int epikv_compact(const epikv_cfg* cfg, const epikv_pool* src, const int32_t* src_pt,
                               int64_t ld_src_pt, const epikv_pool* dst, const int32_t* dst_pt,
                               int64_t ld_dst_pt, const int32_t* keep_idx, const int32_t* n_keep,
                               const float* src_scores, float* dst_scores, const int32_t* src_pos,
                               int32_t* dst_pos, int64_t ld_s, int32_t* seq_status,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const int st = check_compact(cfg, src, src_pt, ld_src_pt, dst, dst_pt, ld_dst_pt, keep_idx, n_keep,
                               src_scores, dst_scores, src_pos, dst_pos, ld_s, workspace,
                               workspace_bytes);
  if (st) return st;
  return launched(launch_compact(compact_args(cfg, src, src_pt, ld_src_pt, dst, dst_pt, ld_dst_pt,
                                              keep_idx, n_keep, src_scores, dst_scores, src_pos,
                                              dst_pos, ld_s, seq_status, workspace),
                                 stream));
}

EPIKV_EXPORT int epikv_compact_inplace(const epikv_cfg* cfg, const epikv_pool* pool,
                                       const int32_t* page_table, int64_t ld_pt,
                                       const int32_t* keep_idx, const int32_t* n_keep,
                                       float* scores, int32_t* pos, int64_t ld_s,
                                       int32_t* seq_status, void* workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
  const int st = check_compact_inplace(cfg, pool, page_table, ld_pt, keep_idx, n_keep, scores, pos,
                                       ld_s, workspace, workspace_bytes);
  if (st) return st;
  return launched(launch_compact_inplace(inplace_args(cfg, pool, page_table, ld_pt, keep_idx, n_keep,
                                                      scores, pos, ld_s, seq_status, workspace),
                                         stream));
}

EPIKV_EXPORT int epikv_compact_remap(const epikv_cfg* cfg, const epikv_pool* pool,
                                     int32_t* page_table, int64_t ld_pt, const int32_t* keep_idx,
                                     const int32_t* n_keep, float* scores, int32_t* pos,
                                     int64_t ld_s, int32_t* seq_status, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  int st = check_compact_inplace(cfg, pool, page_table, ld_pt, keep_idx, n_keep, scores, pos, ld_s,
                                 workspace, workspace_bytes);
  if (st) return st;
  st = check_remap_table(cfg, page_table, ld_pt, keep_idx, n_keep, workspace, workspace_bytes);
  if (st) return st;
  return launched(launch_compact_inplace(
      remap_args(inplace_args(cfg, pool, page_table, ld_pt, keep_idx, n_keep, scores, pos, ld_s,
                              seq_status, workspace),
                 page_table),
      stream));
}

EPIKV_EXPORT int epikv_evict_step(const epikv_cfg* cfg, const epikv_step_io* io, hipStream_t stream) {
  if (!io) return EPIKV_EINVAL_NULL;
  int st = check_cfg(cfg);
  if (st) return st;
  if (io->chunk < 0) return EPIKV_EINVAL_SHAPE;
  // chunk 0: the chunk's scores are already frozen (scored token by token
  // with epikv_score_tokens), so the step is selection + rebuild only
  const bool scoring = io->chunk > 0;
  if (!io->workspace || io->workspace_bytes < epikv_workspace_bytes(cfg, io->chunk))
    return EPIKV_EWORKSPACE;
  if (!aligned16(io->workspace)) return EPIKV_EALIGN;
  // Workspace: the selection's scratch first (at a place that does not
  // depend on the chunk, since it is kept from one call to the next), then
  // the signal, the Lag-KV partial sums and the compaction's scratch.
  void* ws_select = io->workspace;
  const size_t sel_bytes = select_scratch_bytes(cfg->batch);
  char* ws = (char*)io->workspace + sel_bytes;
  const size_t ws_rest = io->workspace_bytes - sel_bytes;
  if (scoring) {
    st = check_score(cfg, io->chunk, io->hidden, io->ld_tok, io->ld_seq, &io->src, io->src_pt,
                     io->ld_src_pt, io->n_cached, io->state_in, io->state_out, (float*)ws, ws,
                     ws_rest, false);
    if (st) return st;
    st = check_zscore(cfg, io->chunk, (const float*)ws, io->n_cached, io->state_in,
                      io->state_out, io->scores, io->ld_s);
    if (st) return st;
  }
  st = check_select(cfg, io->scores, io->ld_s, io->n_cached, io->n_prefix, io->keep_idx, io->n_keep,
                    io->seq_status);
  if (st) return st;
  char* ws_offsets =
      scoring ? ws + sig_bytes(cfg, io->chunk) + partial_bytes(cfg, io->chunk) : ws;
  // The scores are compacted only when the caller asks for them (out of
  // place); in place they always follow their rows.
  const float* src_scores = io->dst_scores ? io->scores : nullptr;
  if (io->in_place < 0 || io->in_place > EPIKV_COMPACT_REMAP) return EPIKV_EINVAL_PARAM;
  if (io->in_place) {
    if (io->dst_scores && io->dst_scores != io->scores) return EPIKV_EALIAS;
    if (io->src_pos != io->dst_pos) return EPIKV_EALIAS;
    st = check_compact_inplace(cfg, &io->src, io->src_pt, io->ld_src_pt, io->keep_idx, io->n_keep,
                               io->scores, io->dst_pos, io->ld_s, ws_offsets,
                               compact_ws_bytes(cfg));
    if (!st && io->in_place == EPIKV_COMPACT_REMAP)
      st = check_remap_table(cfg, io->src_pt, io->ld_src_pt, io->keep_idx, io->n_keep,
                             io->workspace, io->workspace_bytes);
  } else {
    st = check_compact(cfg, &io->src, io->src_pt, io->ld_src_pt, &io->dst, io->dst_pt,
                       io->ld_dst_pt, io->keep_idx, io->n_keep, src_scores, io->dst_scores,
                       io->src_pos, io->dst_pos, io->ld_s, ws_offsets, compact_ws_bytes(cfg));
  }
  if (st) return st;
  st = check_select_scratch(cfg, io->scores, io->ld_s, io->n_cached, io->n_prefix, io->keep_idx,
                            io->n_keep, io->seq_status, ws_select);
  if (st) return st;
  const size_t ws_state = state_layout(cfg).total;
  if (scoring && (overlap(io->workspace, io->workspace_bytes, io->state_in, ws_state) ||
                  overlap(io->workspace, io->workspace_bytes, io->state_out, ws_state)))
    return EPIKV_EALIAS;

  float* sig = (float*)ws;
  float* partial = (float*)(ws + sig_bytes(cfg, io->chunk));
  const SelectArgs sel = select_args(cfg, io->scores, io->ld_s, io->n_cached, io->n_prefix,
                                     io->keep_idx, io->n_keep, io->seq_status, io->chunk);
  const ZscoreArgs zs = zscore_args(cfg, io->chunk, sig, io->n_cached, io->state_in, io->state_out,
                                    io->scores, io->ld_s, nullptr);
  bool selected = false;  // the select stage is on the stream
  if (!scoring) {
    st = launched(launch_select_groups(sel, ws_select, stream));
    if (st) return st;
    selected = true;
  } else if (cfg->signal == EPIKV_SIGNAL_HS) {
    const ScoreHsArgs hs =
        hs_args(cfg, io->chunk, io->hidden, io->ld_tok, io->ld_seq, io->state_in, io->state_out, sig);
    if (select_score_fusable(sel, hs)) {
      // The chunk lies inside the recency window: selection needs only the
      // older, frozen scores, so it runs beside the scoring, then the
      // chunk's scores are smoothed and written.
      st = launched(launch_select_score(sel, hs, stream));
      if (st) return st;
      st = launched(launch_zscore(zs, stream));
      if (st) return st;
      selected = true;
    }
  }
  if (!selected) {
    st = run_score(cfg, io->chunk, io->hidden, io->ld_tok, io->ld_seq, &io->src, io->src_pt,
                   io->ld_src_pt, io->n_cached, io->state_in, io->state_out, sig, partial, stream);
    if (st) return st;
    st = launched(launch_zscore(zs, stream));
    if (st) return st;
    st = launched(launch_select_groups(sel, ws_select, stream));
    if (st) return st;
  }
  if (io->in_place) {
    InplaceArgs a = inplace_args(cfg, &io->src, io->src_pt, io->ld_src_pt, io->keep_idx, io->n_keep,
                                 io->scores, io->dst_pos, io->ld_s, io->seq_status, ws_offsets);
    // (with page remapping the caller's table is documented as rewritten)
    if (io->in_place == EPIKV_COMPACT_REMAP) a = remap_args(a, const_cast<int32_t*>(io->src_pt));
    return launched(launch_compact_inplace(a, stream));
  }
  return launched(launch_compact(
      compact_args(cfg, &io->src, io->src_pt, io->ld_src_pt, &io->dst, io->dst_pt, io->ld_dst_pt,
                   io->keep_idx, io->n_keep, src_scores, io->dst_scores,
                   io->src_pos, io->dst_pos, io->ld_s, io->seq_status, ws_offsets),
      stream));
}
