"""Plain, slow CPU oracle of the EpiKV eviction step (float64 NumPy).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library and imports
nothing from it.

Source: "Epiphany-Aware KV Cache Eviction Without the Attention Matrix"
(Kolawole & Smith, arXiv 2606.26472).  Every function names the passage it
follows.  Where the paper is silent the reading taken is stated in the
function's docstring; all such readings are listed together in the
module-level constant READINGS below.

Conventions
-----------
* bf16 inputs arrive as their 16-bit patterns (uint16) and are widened
  exactly: a bf16 value is the upper half of an IEEE binary32 word.
* All arithmetic is float64.
* A "sample" is one value of a per-token signal (g_l(t) for the hidden-state
  family, q(t) for Lag-KV).  A token with no predecessor has no hidden-state
  sample (reading R7).
"""
from __future__ import annotations

import numpy as np

# Readings of passages the paper leaves open (R-numbers are referred to by
# the docstrings below).
READINGS = {
    "R1": "Band score is the mean z over Band A layers minus the mean z over "
          "Band B layers; with A={10}, B={21} this is z_10 - z_21 (Sec. 3.2 "
          "Eq. 3 text, Table 1, Fig. 1).",
    "R2": "Window w = 64 trailing samples (Sec. 3.2, App. E).",
    "R3": "The window includes the current sample t (Sec. 3.2: only positions "
          "<= t are used).",
    "R4": "sigma is the population standard deviation (ddof = 0).",
    "R5": "eps = 1e-6, added to sigma (Eq. 3).",
    "R6": "Warm-up: the window holds the samples available so far; a single "
          "sample gives sigma = 0 and z = 0.",
    "R7": "A token with no predecessor hidden state has no sample: its "
          "smoothed value is 0 and it enters no window.",
    "R9": "Scores are frozen when the token is generated (Sec. 3.3) for every "
          "signal.",
    "R10": "Recency R = min(128, floor(K/4)) (App. D); N <= K keeps all; "
           "N > K with P + R >= K is a budget error (sequence untouched).",
    "R11": "Ranking is by score descending, ties by lower position; -0 == +0; "
           "NaN ranks below every number, NaNs tie and break by position.",
    "R13": "The rebuilt cache is order preserving (App. H) and written out of "
           "place.",
    "R18": "In-place rebuild (the move-minimising form): the retained rows "
           "are packed to the front of the sequence's own pages in order; "
           "slots past the retained count keep whatever they held.",
    "R19": "Page remapping in the in-place rebuild: a destination page "
           "whose slots receive, in order, every row of one later source "
           "page takes that page in the page table instead of a copy; the "
           "pages this frees are handed, in ascending order, to the source "
           "positions that gave theirs away (ascending), so the sequence "
           "keeps the same set of pages.",
    "R17": "EMA smoothing (App. E, alpha = 0.9): y(t) = alpha * y(t-1) + "
           "(1 - alpha) * x(t), starting at the stream's first sample "
           "(y = x); tokens without a sample leave y unchanged and get 0.",
    "R14": "Lag-KV: each channel of a token's key and value is min-max "
           "normalised with the previous chunk's per-(layer, K|V, head, "
           "channel) range plus eps; the population variance over the head "
           "dimension is taken for K and for V and summed; the sum is "
           "averaged over layers and KV heads; the per-token result is "
           "smoothed with the w-sample trailing mean (Sec. 3.3, Table 1, "
           "App. D 'top variance').  The first chunk of a stream, having no "
           "previous chunk, uses its own range.",
}

EPS_DEFAULT = 1e-6
WINDOW_DEFAULT = 64


# ---------------------------------------------------------------------------
# Number formats
# ---------------------------------------------------------------------------
def bf16_to_float64(bits) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) exactly to float64.

    bf16 is the upper 16 bits of an IEEE binary32 word, so the value is the
    binary32 number whose high half is `bits` and whose low half is zero.
    """
    u16 = np.asarray(bits, dtype=np.uint16)
    u32 = u16.astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Sec. 3.2, Eq. 1: hidden-state change
# ---------------------------------------------------------------------------
def residual_delta(h, h_before=None):
    """g_l(t) = || h_l(t) - h_l(t-1) ||_2 for every token of `h` (Eq. 1).

    h        : float64 [T][D], the hidden states of consecutive tokens at one
               layer.
    h_before : float64 [D] hidden state of the token just before h[0], or
               None when h[0] starts the stream.
    Returns (g [T] float64, has_sample [T] bool).  Without a predecessor the
    first token has no sample (R7) and g is reported as 0 there.
    """
    h = np.asarray(h, dtype=np.float64)
    T = h.shape[0]
    g = np.zeros(T, dtype=np.float64)
    has = np.ones(T, dtype=bool)
    for t in range(T):
        if t == 0:
            if h_before is None:
                has[0] = False
                continue
            prev = np.asarray(h_before, dtype=np.float64)
        else:
            prev = h[t - 1]
        d = h[t] - prev
        g[t] = np.sqrt(np.sum(d * d))
    return g, has


# ---------------------------------------------------------------------------
# Sec. 3.2, Eqs. 2-3: causal trailing-window smoothing
# ---------------------------------------------------------------------------
def trailing_window(x, i, w):
    """The causal trailing window of sample i: x[max(0, i-w+1) .. i]
    (Sec. 3.2: only positions <= t; R2, R3, R6)."""
    return x[max(0, i - w + 1):i + 1]


def rolling_mean(x, w=WINDOW_DEFAULT):
    """Trailing-window mean bar-g(t) of Eq. 2 for every sample of x."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.size, dtype=np.float64)
    for i in range(x.size):
        win = trailing_window(x, i, w)
        out[i] = np.sum(win) / win.size
    return out


def rolling_zscore(x, w=WINDOW_DEFAULT, eps=EPS_DEFAULT):
    """z(t) = (x(t) - mu(t)) / (sigma(t) + eps), Eq. 3, for every sample.

    mu and sigma are the mean and population standard deviation (R4) of the
    trailing window of at most w samples ending at t inclusive (R2, R3, R6).
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.size, dtype=np.float64)
    for i in range(x.size):
        win = trailing_window(x, i, w)
        mu = np.sum(win) / win.size
        sigma = np.sqrt(np.sum((win - mu) ** 2) / win.size)
        out[i] = (x[i] - mu) / (sigma + eps)
    return out


SMOOTH_Z = "z"        # Eq. 3 (EpiKV)
SMOOTH_MEAN = "mean"  # Eq. 2 (HS-variance, KV family)
SMOOTH_RAW = "raw"    # unsmoothed signal (App. E, "raw")
SMOOTH_EMA = "ema"    # exponential moving average (App. E, alpha = 0.9)
EMA_ALPHA = 0.9


def ema(x, alpha=EMA_ALPHA, y_before=None):
    """Exponential moving average of a sample sequence (App. E, R17):
    y(t) = alpha * y(t-1) + (1 - alpha) * x(t).  y_before is the average
    just before x[0] (None: the sequence starts the stream, y(0) = x(0))."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.size, dtype=np.float64)
    y = y_before
    for i in range(x.size):
        y = x[i] if y is None else alpha * y + (1.0 - alpha) * x[i]
        out[i] = y
    return out


def smooth(samples, mode, w=WINDOW_DEFAULT, eps=EPS_DEFAULT):
    """Apply the smoothing `mode` to a chronological sample sequence."""
    if mode == SMOOTH_Z:
        return rolling_zscore(samples, w, eps)
    if mode == SMOOTH_MEAN:
        return rolling_mean(samples, w)
    if mode == SMOOTH_RAW:
        return np.asarray(samples, dtype=np.float64).copy()
    if mode == SMOOTH_EMA:
        return ema(samples)
    raise ValueError(f"unknown smoothing mode {mode!r}")


def smooth_stream(prior, new, has_sample, mode, w=WINDOW_DEFAULT,
                  eps=EPS_DEFAULT, ema_before=None):
    """Smoothed value of each new token of one signal row.

    prior      : earlier samples of the stream, chronological (only the last
                 w-1 can enter a window of a new token).
    new        : per-token signal of the new tokens.
    has_sample : which new tokens carry a sample (R7); the others get 0.
    ema_before : EMA mode only: the running average after the prior samples
                 (default: computed from `prior`).
    """
    new = np.asarray(new, dtype=np.float64)
    has_sample = np.asarray(has_sample, dtype=bool)
    prior = np.asarray(prior, dtype=np.float64)
    if mode == SMOOTH_EMA:
        if ema_before is None and prior.size:
            ema_before = ema(prior)[-1]
        sm = ema(new[has_sample], y_before=ema_before)
    else:
        seq = np.concatenate([prior, new[has_sample]])
        sm = smooth(seq, mode, w, eps)[prior.size:]
    out = np.zeros(new.size, dtype=np.float64)
    out[has_sample] = sm
    return out


def band_score(smoothed, n_a, n_b):
    """s(t) = mean over Band A of the smoothed signal minus mean over Band B.

    smoothed : [n_a + n_b][T], Band A rows first (R1; Fig. 1 draws
    s = z_A - z_B, Eq. 3's text z_10 - z_21 is the case A={10}, B={21}).
    With n_b = 0 the score is the Band A mean alone.
    """
    smoothed = np.asarray(smoothed, dtype=np.float64)
    s = np.mean(smoothed[:n_a], axis=0)
    if n_b > 0:
        s = s - np.mean(smoothed[n_a:n_a + n_b], axis=0)
    return s


def hs_chunk_scores(hidden, h_before, prior, n_a, n_b, mode=SMOOTH_Z,
                    w=WINDOW_DEFAULT, eps=EPS_DEFAULT):
    """Frozen scores of a chunk of new tokens from band-layer hidden states.

    hidden   : float64 [n_band][C][D], Band A layers then Band B layers.
    h_before : float64 [n_band][D] (hidden state of the token before the
               chunk) or None at the start of a stream.
    prior    : list of n_band arrays: earlier samples of each layer.
    Returns (s [C], g [n_band][C], smoothed [n_band][C], has_sample [C]).
    Eq. 1 per layer, Eq. 3 (or Eq. 2) per layer, then the band combination.
    """
    n_band = n_a + n_b
    C = hidden.shape[1]
    g = np.zeros((n_band, C))
    sm = np.zeros((n_band, C))
    has = None
    for l in range(n_band):
        hb = None if h_before is None else h_before[l]
        g[l], has = residual_delta(hidden[l], hb)
        sm[l] = smooth_stream(prior[l], g[l], has, mode, w, eps)
    return band_score(sm, n_a, n_b), g, sm, has


# ---------------------------------------------------------------------------
# Sec. 3.3: Lag-KV signal
# ---------------------------------------------------------------------------
def chunk_range(k, v):
    """Per-channel minimum and maximum over the tokens of a chunk.

    k, v : float64 [T][L][H][d].  Returns (mn, mx), each [L][2][H][d] with
    index 0 = keys and 1 = values (Sec. 3.3: the previous chunk's
    per-channel range).
    """
    mn = np.stack([k.min(axis=0), v.min(axis=0)], axis=1)
    mx = np.stack([k.max(axis=0), v.max(axis=0)], axis=1)
    return mn, mx


def lagkv_signal(k, v, mn, mx, eps=EPS_DEFAULT):
    """Per-token Lag-KV signal q(t) (Sec. 3.3, Table 1, R14).

    k, v   : float64 [T][L][H][d], keys and values of the new tokens.
    mn, mx : float64 [L][2][H][d], the range of the previous chunk.
    Each channel is normalised, x~ = (x - mn) / (mx - mn + eps); the
    population variance over d is taken per (token, layer, head) for keys and
    for values; q(t) is the mean over (layer, head) of the two variances'
    sum.
    """
    kt = (k - mn[None, :, 0]) / (mx[None, :, 0] - mn[None, :, 0] + eps)
    vt = (v - mn[None, :, 1]) / (mx[None, :, 1] - mn[None, :, 1] + eps)
    var_k = np.var(kt, axis=-1)   # population variance over head dim
    var_v = np.var(vt, axis=-1)
    return np.mean(var_k + var_v, axis=(1, 2))


def kv_variance_signal(k, v, use_k=True, use_v=True, rng=None,
                       eps=EPS_DEFAULT):
    """Per-token signal of the KV-vector family (Sec. 3.3, Table 1).

    For each used tensor (keys, values) the population variance over the
    head dimension is taken per (token, layer, head) -- of the raw vectors
    for KV-key / KV-val, of the vectors min-max normalised by `rng`
    (= (mn, mx) of the previous chunk) for the lag-normalised variants; the
    variances of the used tensors are summed and averaged over (layer,
    head).  Lag-KV = keys + values normalised; lag-kv-key = keys only
    (Tables B1-B4).
    """
    q = np.zeros(k.shape[0])
    for use, x, kv in ((use_k, k, 0), (use_v, v, 1)):
        if not use:
            continue
        if rng is not None:
            mn, mx = rng
            x = (x - mn[None, :, kv]) / (mx[None, :, kv] - mn[None, :, kv] + eps)
        q = q + np.mean(np.var(x, axis=-1), axis=(1, 2))
    return q


def kv_chunk_scores(k, v, use_k, use_v, lag, prev_range, prior,
                    mode=SMOOTH_MEAN, w=WINDOW_DEFAULT, eps=EPS_DEFAULT):
    """Frozen scores of one chunk for any KV-vector signal; with lag=True the
    previous chunk's range normalises (the first chunk uses its own, R14).
    Returns (s, q, this chunk's (mn, mx))."""
    own = chunk_range(k, v)
    rng = None
    if lag:
        rng = own if prev_range is None else prev_range
    q = kv_variance_signal(k, v, use_k, use_v, rng, eps)
    s = smooth_stream(prior, q, np.ones(q.size, dtype=bool), mode, w, eps)
    return s, q, own


def lagkv_chunk_scores(k, v, prev_range, prior, mode=SMOOTH_MEAN,
                       w=WINDOW_DEFAULT, eps=EPS_DEFAULT):
    """Frozen Lag-KV scores of one chunk of new tokens.

    prev_range : (mn, mx) of the previous chunk, or None for the first chunk
                 of a stream, which then uses its own range (R14).
    prior      : earlier q samples of the stream.
    Returns (s [T], q [T], this chunk's (mn, mx)).
    """
    own = chunk_range(k, v)
    mn, mx = own if prev_range is None else prev_range
    q = lagkv_signal(k, v, mn, mx, eps)
    s = smooth_stream(prior, q, np.ones(q.size, dtype=bool), mode, w, eps)
    return s, q, own


# ---------------------------------------------------------------------------
# Sec. 3.1, Sec. 3.3, App. D: which positions survive
# ---------------------------------------------------------------------------
BUDGET_ERROR = "budget"


def default_recent(K):
    """Recency window R = min(128, K/4) (App. D), K/4 rounded down."""
    return min(128, K // 4)


def ranking_key(score, pos):
    """Sort key realising R11: higher score first, lower position first among
    equals; every NaN after every number."""
    x = float(score)
    if np.isnan(x):
        return (1, 0.0, pos)
    return (0, -x, pos)


def select_keep(scores, n_prefix, K, recent=None):
    """Retained positions of one sequence after an eviction step.

    scores   : frozen per-position scores s of the N cached tokens.
    n_prefix : number P of prefill (prompt) positions, all retained.
    K        : the budget.
    recent   : recency window R (default min(128, K/4)).
    Returns the ascending int64 array of retained positions, or BUDGET_ERROR.

    The rule (Sec. 3.1: keep the K highest-scoring positions; Sec. 3.3 and
    App. D: prefill and a trailing recency window are always kept and the
    score fills the rest, so exactly K survive):
      * N <= K: nothing is evicted;
      * N > K, P + R >= K: no room for scored tokens -> budget error (R10);
      * else keep [0, P), [N - R, N) and the K - P - R best positions of
        [P, N - R) under R11.
    """
    N = len(scores)
    R = default_recent(K) if recent is None else recent
    if N <= K:
        return np.arange(N, dtype=np.int64)
    if n_prefix + R >= K:
        return BUDGET_ERROR
    M = K - n_prefix - R
    eligible = list(range(n_prefix, N - R))
    ranked = sorted(eligible, key=lambda i: ranking_key(scores[i], i))
    kept = set(range(n_prefix)) | set(range(N - R, N)) | set(ranked[:M])
    return np.array(sorted(kept), dtype=np.int64)


# ---------------------------------------------------------------------------
# App. H: rebuilding the cache from the retained positions
# ---------------------------------------------------------------------------
def compact_rows(rows, keep):
    """Order-preserving rebuild: out[j] = rows[keep[j]] for every j (App. H,
    R13).  `rows` may carry any trailing shape; copying is exact."""
    rows = np.asarray(rows)
    return rows[np.asarray(keep, dtype=np.int64)].copy()


def first_hole(keep):
    """First slot j whose retained position differs from j (len(keep) when
    the retained set is a leading run).  Slots before it need no move."""
    keep = np.asarray(keep, dtype=np.int64)
    moved = np.nonzero(keep != np.arange(keep.size))[0]
    return int(moved[0]) if moved.size else int(keep.size)


def compact_rows_inplace(rows, keep):
    """In-place order-preserving rebuild (App. H, R18): slot j < len(keep)
    receives the row that position keep[j] held; every later slot keeps its
    old row.  `rows` holds the sequence's rows before the rebuild (leading
    axis = position); the result is a new array."""
    rows = np.asarray(rows)
    keep = np.asarray(keep, dtype=np.int64)
    out = rows.copy()
    out[:keep.size] = rows[keep]
    return out


def remap_pairs(keep, page_size):
    """Whole-page retention (R19): the destination pages m (of the full
    pages of the rebuilt sequence) whose page_size slots receive, in order,
    all rows of one source page p, with p > m.  Ascending list of (m, p).
    A page with p == m is already in place (the leading run)."""
    keep = np.asarray(keep, dtype=np.int64)
    ps = int(page_size)
    pairs = []
    for m in range(keep.size // ps):
        run = keep[m * ps:(m + 1) * ps]
        p, r = divmod(int(run[0]), ps)
        if r == 0 and p > m and np.array_equal(run, np.arange(p * ps, (p + 1) * ps)):
            pairs.append((m, p))
    return pairs


def page_table_after_remap(pt_row, keep, page_size):
    """The sequence's page-table row after an in-place rebuild with page
    remapping (R19): pair destination m takes the page of its source p; the
    pages of destinations that are not themselves sources are released and
    go, k-th to k-th in ascending order, to the sources that are not
    themselves destinations.  Every other entry is unchanged, so the row is
    a permutation of the old one."""
    pairs = remap_pairs(keep, page_size)
    dests = {m for m, _ in pairs}
    srcs = {p for _, p in pairs}
    old = np.asarray(pt_row)
    new = old.copy()
    for m, p in pairs:
        new[m] = old[p]
    released = [m for m, _ in pairs if m not in srcs]
    losing = [p for _, p in pairs if p not in dests]
    assert len(released) == len(losing)
    for m, p in zip(released, losing):
        new[p] = old[m]
    return new


def compact_pages_remap(pool, pt_row, keep, page_size):
    """In-place rebuild of one sequence with page remapping (App. H, R18,
    R19).  pool: physical pages [n_pages][page_size][...]; pt_row: the
    sequence's page table.  Returns (pool after, page-table row after).
    Through the new row, slot j < len(keep) reads the row that position
    keep[j] held through the old row.  Slots of a remapped destination page
    are not written (its page already holds them); every other slot j <
    len(keep) is written with its row; nothing else changes."""
    ps = int(page_size)
    keep = np.asarray(keep, dtype=np.int64)
    dests = {m for m, _ in remap_pairs(keep, ps)}
    new_pt = page_table_after_remap(pt_row, keep, ps)
    pool = np.asarray(pool)
    out = pool.copy()
    for j, i in enumerate(keep):
        d = j // ps
        if d in dests:
            continue
        out[new_pt[d], j % ps] = pool[pt_row[i // ps], i % ps]
    return out, new_pt
