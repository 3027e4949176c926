"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than its own formula: a
closed form, a brute-force enumeration, an invariant the paper states, a
textbook special case or a value the paper prints.  Each is chosen so that a
plausible slip (a dropped term, a window off by one, a wrong variance
estimator, a sign flipped, a tie broken the wrong way) fails it.
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy.stats import spearmanr

import oracle as O
import synth

W = 64
EPS = 1e-6


# ---------------------------------------------------------------------------
# bf16 widening (format definition)
# ---------------------------------------------------------------------------
def test_bf16_widening_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x4049,
                     0x0001, 0x3F81], dtype=np.uint16)
    v = O.bf16_to_float64(bits)
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == math.inf and v[3] == -math.inf
    assert v[4] == 0.0 and math.copysign(1.0, v[5]) == -1.0
    assert v[6] == 3.140625                      # 0x4049 = 1.5703125 * 2
    assert v[7] == 2.0 ** -133                   # smallest bf16 subnormal
    assert v[8] == 1.0 + 2.0 ** -7               # one ulp above 1 in bf16
    assert np.isnan(O.bf16_to_float64(np.array([0x7FC0], np.uint16)))[0]


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    g = synth.rng(11)
    x = (g.standard_normal(20000) * 10.0 ** g.integers(-30, 30, 20000)
         ).astype(np.float32)
    x[:4] = [np.inf, -np.inf, 0.0, -0.0]
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(ours, ref.view(np.uint16))
    # round trip through the oracle's widening is the identity on bf16 values
    back = O.bf16_to_float64(ours).astype(np.float32)
    assert np.array_equal(synth.f32_to_bf16_bits(back), ours)


# ---------------------------------------------------------------------------
# Eq. 1: g_l(t) = || h_l(t) - h_l(t-1) ||_2
# ---------------------------------------------------------------------------
def test_residual_delta_axis_steps():
    D = 16
    h = np.zeros((4, D))
    h[1, 3] = 2.5          # step along one axis
    h[2, 3] = 2.5
    h[2, 7] = -4.0         # second step along another axis
    h[3] = h[2]            # no change
    g, has = O.residual_delta(h, np.zeros(D))
    assert has.all()
    assert g.tolist() == [0.0, 2.5, 4.0, 0.0]


def test_residual_delta_pythagorean_triples():
    h = np.zeros((4, 3))
    h[1] = [3.0, 4.0, 0.0]          # |(3,4,0)| = 5
    h[2] = [4.0, 6.0, 2.0]          # |(1,2,2)| = 3
    h[3] = [6.0, 9.0, 8.0]          # |(2,3,6)| = 7
    g, _ = O.residual_delta(h, np.zeros(3))
    assert g.tolist() == [0.0, 5.0, 3.0, 7.0]


def test_residual_delta_is_norm_of_difference_not_difference_of_norms():
    x = np.array([1.0, 2.0, 2.0])   # |x| = 3
    h = np.stack([x, -x])
    g, _ = O.residual_delta(h, x)   # first row equals its predecessor
    assert g.tolist() == [0.0, 6.0]


def test_residual_delta_stream_start_has_no_sample():
    h = np.ones((3, 5))
    g, has = O.residual_delta(h, None)
    assert has.tolist() == [False, True, True]
    assert g[1] == 0.0


# ---------------------------------------------------------------------------
# Eq. 3: rolling z-score over a trailing window of w = 64 samples
# ---------------------------------------------------------------------------
def test_zscore_linear_ramp_closed_form():
    # For x = a + c t with c > 0 every full window gives
    # z = sqrt(3 (w-1) / (w+1)) (inclusive window, population sigma).
    # An exclusive window or ddof=1 give 1.7593 / 1.6918 instead.
    for a, c in [(0.0, 1.0), (1e3, 0.25), (-7.0, 3.0)]:
        x = a + c * np.arange(300, dtype=np.float64)
        z = O.rolling_zscore(x, W, EPS)
        zc = math.sqrt(3.0 * (W - 1) / (W + 1))
        sigma = c * math.sqrt((W * W - 1) / 12.0)
        assert np.allclose(z[W - 1:], zc * sigma / (sigma + EPS),
                           rtol=1e-12, atol=0)
        assert abs(zc - 1.705196) < 1e-6


def test_zscore_isolated_spike_closed_form():
    # w-1 zeros then a value x: mu = x/w, sigma = x sqrt(w-1)/w, so
    # z = sqrt(w-1) (= 7.937 at w = 64) for any x > 0.
    for x in [1.0, 5.0, 1e4]:
        s = np.zeros(W)
        s[-1] = x
        z = O.rolling_zscore(s, W, EPS)[-1]
        sigma = x * math.sqrt(W - 1) / W
        assert z == pytest.approx((x - x / W) / (sigma + EPS), rel=1e-13)
        assert z == pytest.approx(math.sqrt(W - 1), rel=1e-5)


def test_zscore_window_length_is_exactly_w():
    g = synth.rng(5)
    x = g.standard_normal(400)
    base = O.rolling_zscore(x, W, EPS)
    t = 300
    y = x.copy()
    y[t - W] += 100.0          # just outside the window of t
    assert O.rolling_zscore(y, W, EPS)[t] == base[t]
    y = x.copy()
    y[t - W + 1] += 100.0      # oldest sample inside the window of t
    assert O.rolling_zscore(y, W, EPS)[t] != base[t]


def test_zscore_warmup():
    z = O.rolling_zscore(np.array([4.0, 10.0, 10.0]), W, EPS)
    assert z[0] == 0.0                                  # single sample
    assert z[1] == pytest.approx(3.0 / (3.0 + EPS), rel=1e-14)  # two samples
    # three samples {4, 10, 10}: mu = 8, sigma = sqrt(8), z = 2 / sqrt(8)
    assert z[2] == pytest.approx(2.0 / (math.sqrt(8.0) + EPS), rel=1e-14)


def test_zscore_constant_stream_is_zero():
    assert np.all(O.rolling_zscore(np.full(200, 3.25), W, EPS) == 0.0)


def test_zscore_affine_invariance():
    g = synth.rng(6)
    x = np.abs(g.standard_normal(500)) + 2.0
    # eps = 0 so that the invariance is exact; the first sample (0/0) is
    # left out.
    z = O.rolling_zscore(x, W, 0.0)[1:]
    for alpha, beta in [(3.0, 0.0), (0.01, 50.0), (250.0, -7.0)]:
        assert np.allclose(O.rolling_zscore(alpha * x + beta, W, 0.0)[1:], z,
                           atol=1e-9)
    assert np.allclose(O.rolling_zscore(-2.0 * x + 1.0, W, 0.0)[1:], -z,
                       atol=1e-9)


def test_zscore_removes_positional_drift():
    # Sec. 3.2: the raw signal tracks position; the causal z-score removes
    # the trend.  Band A drifts down and Band B up (opposite signs).
    g = synth.rng(7)
    T = 4000
    t = np.arange(T, dtype=np.float64)
    a = g.standard_normal(T) + 10.0 - 0.004 * t
    b = g.standard_normal(T) + 10.0 + 0.004 * t
    raw = a - b
    z = O.rolling_zscore(a, W, EPS) - O.rolling_zscore(b, W, EPS)
    assert abs(spearmanr(raw[W:], t[W:])[0]) > 0.8
    assert abs(spearmanr(z[W:], t[W:])[0]) < 0.05


def test_zscore_is_causal_and_chunking_invariant():
    g = synth.rng(8)
    x = g.standard_normal(600)
    full = O.rolling_zscore(x, W, EPS)
    # appending future samples changes no earlier value
    assert np.array_equal(O.rolling_zscore(x[:400], W, EPS), full[:400])
    # processing in chunks with only the last w-1 samples carried over
    out = []
    prior = np.zeros(0)
    for lo in range(0, 600, 128):
        new = x[lo:lo + 128]
        out.append(O.smooth_stream(prior, new, np.ones(new.size, bool),
                                   O.SMOOTH_Z, W, EPS))
        prior = np.concatenate([prior, new])[-(W - 1):]
    assert np.array_equal(np.concatenate(out), full)


def test_rolling_mean_ramp_closed_form():
    x = 2.0 + 0.5 * np.arange(200, dtype=np.float64)
    m = O.rolling_mean(x, W)
    t = np.arange(W - 1, 200)
    assert np.allclose(m[W - 1:], 2.0 + 0.5 * (t - (W - 1) / 2.0),
                       rtol=1e-14)
    assert m[0] == 2.0 and m[1] == 2.25


def test_ema_closed_forms():
    # step response: from y = 0, a unit step gives y(n) = 1 - alpha^(n+1)
    a = O.EMA_ALPHA
    y = O.ema(np.ones(50), a, y_before=0.0)
    n = np.arange(50)
    assert np.allclose(y, 1.0 - a ** (n + 1), rtol=1e-14, atol=0)
    # a constant stream started fresh stays constant
    assert np.all(O.ema(np.full(30, 2.5)) == 2.5)
    # impulse response decays geometrically with ratio alpha
    x = np.zeros(20)
    x[0] = 1.0
    y = O.ema(x, a, y_before=0.0)
    assert np.allclose(y, (1 - a) * a ** np.arange(20), rtol=1e-14)
    # carrying the average across chunks equals one pass
    x = synth.rng(21).standard_normal(300)
    full = O.ema(x)
    part = O.ema(x[120:], y_before=O.ema(x[:120])[-1])
    assert np.allclose(part, full[120:], rtol=1e-13)


def test_smooth_stream_skips_tokens_without_sample():
    new = np.array([123.0, 1.0, 3.0])
    out = O.smooth_stream(np.zeros(0), new, np.array([False, True, True]),
                          O.SMOOTH_MEAN, W, EPS)
    assert out.tolist() == [0.0, 1.0, 2.0]


def test_smooth_stream_raw_is_the_signal_itself():
    # App. E's unsmoothed baseline: each token's own sample, whatever came
    # before it; tokens without a sample get 0
    new = np.array([3.5, -2.0, 7.0, 0.25])
    has = np.array([True, False, True, True])
    for prior in (np.zeros(0), synth.rng(30).standard_normal(100)):
        out = O.smooth_stream(prior, new, has, O.SMOOTH_RAW, W, EPS)
        assert out.tolist() == [3.5, 0.0, 7.0, 0.25]


def test_smooth_stream_ema_hand_values_and_carry():
    # App. E: y(t) = 0.9 y(t-1) + 0.1 x(t), the stream's first sample
    # starting the average
    out = O.smooth_stream(np.zeros(0), np.array([4.0, 0.0, 10.0]),
                          np.ones(3, bool), O.SMOOTH_EMA, W, EPS)
    assert np.allclose(out, [4.0, 3.6, 4.24], rtol=1e-15, atol=0)
    # the same stream cut after two samples: the average carries over,
    # from the earlier samples or given explicitly
    cut = O.smooth_stream(np.array([4.0, 0.0]), np.array([10.0]),
                          np.ones(1, bool), O.SMOOTH_EMA, W, EPS)
    assert np.allclose(cut, [4.24], rtol=1e-15, atol=0)
    given = O.smooth_stream(np.zeros(0), np.array([2.0]), np.ones(1, bool),
                            O.SMOOTH_EMA, W, EPS, ema_before=1.0)
    assert np.allclose(given, [1.1], rtol=1e-15, atol=0)
    # a token without a sample neither moves the average nor gets a value
    skip = O.smooth_stream(np.zeros(0), np.array([10.0, 99.0, 0.0]),
                           np.array([True, False, True]), O.SMOOTH_EMA, W,
                           EPS, ema_before=0.0)
    assert np.allclose(skip, [1.0, 0.0, 0.9], rtol=1e-15, atol=0)


def test_smooth_stream_mean_in_chunks_equals_one_pass():
    # Eq. 2's trailing mean only looks back w-1 samples, so carrying the
    # last w-1 samples between chunks reproduces the one-pass values
    x = synth.rng(31).standard_normal(300)
    full = O.rolling_mean(x, W)
    out = []
    prior = np.zeros(0)
    for lo in range(0, 300, 50):
        new = x[lo:lo + 50]
        out.append(O.smooth_stream(prior, new, np.ones(new.size, bool),
                                   O.SMOOTH_MEAN, W, EPS))
        prior = np.concatenate([prior, new])[-(W - 1):]
    assert np.array_equal(np.concatenate(out), full)


# ---------------------------------------------------------------------------
# Band combination (Fig. 1, Eq. 3 text)
# ---------------------------------------------------------------------------
def test_band_score_reduces_to_z10_minus_z21():
    g = synth.rng(9)
    z = g.standard_normal((2, 50))
    assert np.array_equal(O.band_score(z, 1, 1), z[0] - z[1])


def test_band_score_signs():
    base = np.zeros((15, 1))
    up_a = base.copy()
    up_a[3] = 1.0          # a Band A layer rises
    up_b = base.copy()
    up_b[10] = 1.0         # a Band B layer rises
    assert O.band_score(up_a, 7, 8)[0] == pytest.approx(1.0 / 7.0)
    assert O.band_score(up_b, 7, 8)[0] == pytest.approx(-1.0 / 8.0)
    assert O.band_score(up_a, 15, 0)[0] == pytest.approx(1.0 / 15.0)


def test_hs_chunk_scores_spike_on_band_a_raises_score():
    # A token whose Band A hidden state jumps is scored above its
    # neighbours; the same jump on Band B pushes it below (Sec. 3.2).
    g = synth.rng(10)
    n_a, n_b, T, D = 2, 2, 200, 32
    hid = g.standard_normal((n_a + n_b, T, D))
    prior = [np.zeros(0)] * 4
    spike = 150
    ha = hid.copy()
    ha[:n_a, spike] *= 6.0
    s_a, *_ = O.hs_chunk_scores(ha, None, prior, n_a, n_b)
    assert np.argmax(s_a[W:]) + W == spike
    hb = hid.copy()
    hb[n_a:, spike] *= 6.0
    s_b, *_ = O.hs_chunk_scores(hb, None, prior, n_a, n_b)
    assert np.argmin(s_b[W:]) + W == spike


# ---------------------------------------------------------------------------
# Band constants against the paper's per-layer table (App. A)
# ---------------------------------------------------------------------------
def _rho_table():
    path = os.path.join(os.path.dirname(__file__), "golden",
                        "perlayer_rho.txt")
    rows = [l.split() for l in open(path) if l.strip() and l[0] != "#"]
    return {int(r[0]): [float(v) for v in r[1:]] for r in rows}


def test_band_layers_have_the_sign_the_table_prints():
    rho = _rho_table()
    assert len(rho) == 32
    for l in synth.BAND_A:
        assert all(v > 0 for v in rho[l]), l
    for l in synth.BAND_B:
        assert all(v < 0 for v in rho[l]), l
    # the layers just outside each band break its sign in some column
    for l in (6, 14, 26):
        assert not all(v > 0 for v in rho[l]) or not all(v < 0 for v in rho[l])
    assert any(v < 0 for v in rho[6]) and any(v < 0 for v in rho[14])
    assert any(v > 0 for v in rho[26])
    # the last layer flips sign across columns and is not used
    assert any(v > 0 for v in rho[31]) and any(v < 0 for v in rho[31])
    # the single-layer preset 10/21 sits inside the bands
    assert 10 in synth.BAND_A and 21 in synth.BAND_B


# ---------------------------------------------------------------------------
# Sec. 3.3: Lag-KV signal
# ---------------------------------------------------------------------------
def _lag_shapes(g, T=6, L=2, H=2, d=8):
    return (g.standard_normal((T, L, H, d)), g.standard_normal((T, L, H, d)))


def test_chunk_range_brute_force():
    g = synth.rng(12)
    k, v = _lag_shapes(g)
    mn, mx = O.chunk_range(k, v)
    T, L, H, d = k.shape
    for l in range(L):
        for h in range(H):
            for c in range(d):
                col_k = [k[t, l, h, c] for t in range(T)]
                col_v = [v[t, l, h, c] for t in range(T)]
                assert mn[l, 0, h, c] == min(col_k)
                assert mx[l, 0, h, c] == max(col_k)
                assert mn[l, 1, h, c] == min(col_v)
                assert mx[l, 1, h, c] == max(col_v)


def test_lagkv_previous_chunk_maps_into_unit_interval():
    g = synth.rng(13)
    k, v = _lag_shapes(g)
    mn, mx = O.chunk_range(k, v)
    kt = (k - mn[None, :, 0]) / (mx[None, :, 0] - mn[None, :, 0] + EPS)
    assert kt.min() >= 0.0 and kt.max() < 1.0


def test_lagkv_alternating_extremes_closed_form():
    # A token whose channels alternate between the previous chunk's min and
    # max normalises to 0,1,0,1,...: population variance 1/4 (times
    # (r/(r+eps))^2), for K and V, so q = 1/2.
    L, H, d = 2, 3, 8
    mn = np.full((L, 2, H, d), -1.0)
    mx = np.full((L, 2, H, d), 3.0)
    tok = np.where(np.arange(d) % 2 == 0, -1.0, 3.0)
    k = np.broadcast_to(tok, (1, L, H, d)).copy()
    q = O.lagkv_signal(k, k.copy(), mn, mx, EPS)
    r = 4.0 / (4.0 + EPS)
    assert q[0] == pytest.approx(2 * 0.25 * r * r, rel=1e-14)
    # a token at the middle of every range has zero variance
    q0 = O.lagkv_signal(np.ones((1, L, H, d)), np.ones((1, L, H, d)), mn, mx)
    assert q0[0] == 0.0


def test_lagkv_invariant_to_per_channel_affine_maps():
    # Sec. 3.3: the lag normalisation removes domain-level magnitude shifts.
    g = synth.rng(14)
    T, L, H, d = 5, 2, 2, 8
    prev_k, prev_v = _lag_shapes(g, T, L, H, d)
    k, v = _lag_shapes(g, T, L, H, d)
    s_k = np.exp(g.standard_normal((L, H, d)))
    o_k = g.standard_normal((L, H, d)) * 10
    s_v = np.exp(g.standard_normal((L, H, d)))
    o_v = g.standard_normal((L, H, d)) * 10
    rng0 = O.chunk_range(prev_k, prev_v)
    rng1 = O.chunk_range(prev_k * s_k + o_k, prev_v * s_v + o_v)
    q0 = O.lagkv_signal(k, v, *rng0, eps=0.0)
    q1 = O.lagkv_signal(k * s_k + o_k, v * s_v + o_v, *rng1, eps=0.0)
    assert np.allclose(q0, q1, rtol=1e-10)


def test_lagkv_first_chunk_uses_own_range():
    g = synth.rng(15)
    k, v = _lag_shapes(g)
    s, q, own = O.lagkv_chunk_scores(k, v, None, np.zeros(0))
    assert np.array_equal(q, O.lagkv_signal(k, v, *O.chunk_range(k, v)))
    # the smoothed score of the first token is its own signal (one sample)
    assert s[0] == q[0]


def _channel_grid(L, H, d):
    """Per-(layer, K|V, head, channel) low ends and widths, dyadic so that
    lo + r, lo + r/2 and lo + r/4 are exact; keys and values differ, so a
    range taken from the wrong tensor, layer or head breaks the closed
    forms below."""
    l, kv, h, c = np.meshgrid(np.arange(L), np.arange(2), np.arange(H),
                              np.arange(d), indexing="ij")
    lo = 0.25 * c - l + 3.0 * kv - h
    r = 1.0 + l + 2.0 * kv + 0.5 * h + 0.125 * c
    return lo, r


def _alternating(lo, r, even, odd):
    """One token per (even, odd) pair: channel c of every (layer, K|V, head)
    sits at lo + even*r for even c and lo + odd*r for odd c.  Returns keys
    and values [1][L][H][d]."""
    d = lo.shape[-1]
    frac = np.where(np.arange(d) % 2 == 0, even, odd)
    tok = lo + frac * r                      # [L][2][H][d]
    return tok[None, :, 0], tok[None, :, 1]


def _chunk(lo, r, *pairs):
    ks, vs = zip(*(_alternating(lo, r, a, b) for a, b in pairs))
    return np.concatenate(ks), np.concatenate(vs)


@pytest.mark.parametrize("use_v", [True, False])
def test_lag_signal_uses_the_previous_chunks_range(use_v):
    """Sec. 3.3 / Table 1 ("lag-norm."): a chunk is normalised by the range
    of the chunk before it, not by its own.  Three chained chunks, eps = 0,
    every channel with its own range:
      chunk 1: tokens alternating lo / lo+r and lo+r / lo -> own range
               [lo, lo+r], values 0 / 1, variance 1/4 per tensor;
      chunk 2: lo / lo+r/2 and back, under chunk 1's range -> 0 / 1/2,
               variance 1/16 (its own range would give 1/4);
      chunk 3: lo+r/4 / lo+r/2 and back, under chunk 2's range
               [lo, lo+r/2] -> 1/2 / 1, variance 1/16 (chunk 1's range
               would give 1/64, its own range 1/4).
    Lag-KV sums the key and value variances, lag-kv-key has the key's only;
    averaging over layers and heads keeps the per-head value."""
    L, H, d = 2, 3, 8
    lo, r = _channel_grid(L, H, d)
    chunks = [_chunk(lo, r, (0.0, 1.0), (1.0, 0.0)),
              _chunk(lo, r, (0.0, 0.5), (0.5, 0.0)),
              _chunk(lo, r, (0.25, 0.5), (0.5, 0.25))]
    n_t = 2.0 if use_v else 1.0
    want_q = [n_t / 4, n_t / 16, n_t / 16]
    prev, prior = None, np.zeros(0)
    qs = []
    for j, (k, v) in enumerate(chunks):
        s, q, own = O.kv_chunk_scores(k, v, True, use_v, True, prev, prior,
                                      O.SMOOTH_MEAN, W, 0.0)
        assert np.array_equal(q, [want_q[j]] * 2), (j, q)
        if use_v:
            s2, q2, own2 = O.lagkv_chunk_scores(k, v, prev, prior,
                                                O.SMOOTH_MEAN, W, 0.0)
            assert np.array_equal(q2, q) and np.array_equal(s2, s)
            assert all(np.array_equal(a, b) for a, b in zip(own, own2))
        # the range handed on is this chunk's own, per channel
        mn, mx = own
        for t in range(2):
            assert np.all(mn[:, 0] <= k[t]) and np.all(k[t] <= mx[:, 0])
            assert np.all(mn[:, 1] <= v[t]) and np.all(v[t] <= mx[:, 1])
        assert np.array_equal(mn[:, 0], np.minimum(k[0], k[1]))
        assert np.array_equal(mx[:, 1], np.maximum(v[0], v[1]))
        qs.extend(q)
        # trailing-window mean (Eq. 2) of every sample so far
        for i in range(2):
            seen = qs[:2 * j + i + 1]
            assert s[i] == pytest.approx(sum(seen) / len(seen), rel=1e-14)
        prev, prior = own, np.concatenate([prior, q])
    # The same chunks scored by their own ranges (what a missing lag would
    # compute) differ from chunk 2 on.
    for j in (1, 2):
        k, v = chunks[j]
        own_q = O.kv_chunk_scores(k, v, True, use_v, True, None, np.zeros(0),
                                  O.SMOOTH_MEAN, W, 0.0)[1]
        assert np.array_equal(own_q, [n_t / 4] * 2)
    # and chunk 3 under chunk 1's range (a range not handed on) differs too
    k, v = chunks[2]
    stale = O.chunk_range(*chunks[0])
    stale_q = O.kv_chunk_scores(k, v, True, use_v, True, stale, np.zeros(0),
                                O.SMOOTH_MEAN, W, 0.0)[1]
    assert np.array_equal(stale_q, [n_t / 64] * 2)


@pytest.mark.parametrize("use_v", [True, False])
def test_lag_signal_previous_range_with_eps_closed_form(use_v):
    """A token alternating between the previous chunk's per-channel minimum
    and maximum (width r = 4 in every channel, low ends all different):
    0, r/(r+eps), ... -> variance (r/(r+eps))^2 / 4 per tensor, so Lag-KV
    q = (r/(r+eps))^2 / 2 and lag-kv-key q = (r/(r+eps))^2 / 4.  Scored by
    its own (degenerate) range the same token gives 0."""
    L, H, d = 2, 2, 8
    lo, _ = _channel_grid(L, H, d)
    r = np.full(lo.shape, 4.0)
    prev = _chunk(lo, r, (0.0, 1.0), (1.0, 0.0))
    k, v = _chunk(lo, r, (0.0, 1.0))
    rr = (4.0 / (4.0 + EPS)) ** 2
    want = rr / 2 if use_v else rr / 4
    q = O.kv_chunk_scores(k, v, True, use_v, True, O.chunk_range(*prev),
                          np.zeros(0), O.SMOOTH_MEAN, W, EPS)[1]
    assert q[0] == pytest.approx(want, rel=1e-14)
    q_own = O.kv_chunk_scores(k, v, True, use_v, True, None, np.zeros(0),
                              O.SMOOTH_MEAN, W, EPS)[1]
    assert q_own[0] == 0.0
    if use_v:
        q2 = O.lagkv_chunk_scores(k, v, O.chunk_range(*prev), np.zeros(0),
                                  O.SMOOTH_MEAN, W, EPS)[1]
        assert q2[0] == pytest.approx(want, rel=1e-14)
        assert O.lagkv_chunk_scores(k, v, None, np.zeros(0),
                                    O.SMOOTH_MEAN, W, EPS)[1][0] == 0.0


@pytest.mark.parametrize("use_k,use_v", [(True, False), (False, True),
                                         (True, True)])
def test_raw_kv_signals_ignore_any_range(use_k, use_v):
    """KV-key / KV-val (and both) are variances of the raw vectors (Sec. 3.3,
    Table 1): keys alternating +-2 and values +-1/2 give 4, 1/4 and 17/4
    whatever range is passed, and the range handed on is still the
    chunk's own."""
    L, H, d = 3, 2, 8
    sign = np.where(np.arange(d) % 2 == 0, 1.0, -1.0)
    k = np.broadcast_to(2.0 * sign, (2, L, H, d)).copy()
    v = np.broadcast_to(0.5 * sign, (2, L, H, d)).copy()
    want = (4.0 if use_k else 0.0) + (0.25 if use_v else 0.0)
    odd_range = (np.full((L, 2, H, d), -7.0), np.full((L, 2, H, d), 9.0))
    for rng in (None, odd_range):
        s, q, own = O.kv_chunk_scores(k, v, use_k, use_v, False, rng,
                                      np.zeros(0), O.SMOOTH_MEAN, W, EPS)
        assert np.array_equal(q, [want, want])
        assert np.array_equal(own[0][:, 0], np.minimum(k[0], k[1]))


def test_kv_variance_closed_forms():
    # Channels alternating +a / -a have population variance a^2 in every
    # head, whatever the layer: KV-key gives a_k^2, KV-val a_v^2, both
    # together their sum; the lag-normalised key-only signal of a token at
    # the previous chunk's extremes gives 1/4 (times the eps factor).
    L, H, d = 3, 2, 8
    sign = np.where(np.arange(d) % 2 == 0, 1.0, -1.0)
    k = np.broadcast_to(2.0 * sign, (1, L, H, d)).copy()
    v = np.broadcast_to(0.5 * sign, (1, L, H, d)).copy()
    assert O.kv_variance_signal(k, v, True, False)[0] == 4.0
    assert O.kv_variance_signal(k, v, False, True)[0] == 0.25
    assert O.kv_variance_signal(k, v, True, True)[0] == 4.25
    mn = np.full((L, 2, H, d), -2.0)
    mx = np.full((L, 2, H, d), 2.0)
    r = 4.0 / (4.0 + EPS)
    q = O.kv_variance_signal(k, v, True, False, (mn, mx))[0]
    assert q == pytest.approx(0.25 * r * r, rel=1e-14)
    # the lag-normalised key + value signal is the Lag-KV signal
    g = synth.rng(19)
    k2, v2 = _lag_shapes(g)
    rng2 = O.chunk_range(*_lag_shapes(g))
    assert np.allclose(O.kv_variance_signal(k2, v2, True, True, rng2),
                       O.lagkv_signal(k2, v2, *rng2), rtol=1e-14)


def test_kv_variance_raw_is_not_scale_invariant_but_lag_is():
    # KV-key tracks magnitude (scaling the keys by c scales q by c^2); the
    # lag-normalised variant removes it (Sec. 3.3).
    g = synth.rng(20)
    prev_k, prev_v = _lag_shapes(g)
    k, v = _lag_shapes(g)
    q1 = O.kv_variance_signal(k, v, True, False)
    q3 = O.kv_variance_signal(3 * k, v, True, False)
    assert np.allclose(q3, 9 * q1, rtol=1e-12)
    r1 = O.chunk_range(prev_k, prev_v)
    r3 = O.chunk_range(3 * prev_k, prev_v)
    assert np.allclose(O.kv_variance_signal(3 * k, v, True, False, r3, 0.0),
                       O.kv_variance_signal(k, v, True, False, r1, 0.0),
                       rtol=1e-12)


# ---------------------------------------------------------------------------
# Which positions survive (Sec. 3.1, Sec. 3.3, App. D)
# ---------------------------------------------------------------------------
def _dominates(scores, i, j):
    """Position i outranks position j: higher score, or equal score and lower
    position; NaN below everything (written independently of the oracle's
    sort key)."""
    si, sj = float(scores[i]), float(scores[j])
    if math.isnan(si) and math.isnan(sj):
        return i < j
    if math.isnan(sj):
        return True
    if math.isnan(si):
        return False
    if si != sj:
        return si > sj
    return i < j


def _brute_force_keep(scores, P, K, R):
    N = len(scores)
    if N <= K:
        return list(range(N))
    protected = set(range(P)) | set(range(N - R, N))
    elig = [i for i in range(P, N - R)]
    M = K - P - R
    found = []
    for sub in itertools.combinations(elig, M):
        rest = [j for j in elig if j not in sub]
        if all(_dominates(scores, i, j) for i in sub for j in rest):
            found.append(sorted(protected | set(sub)))
    assert len(found) == 1      # the retained set is unique
    return found[0]


def test_select_matches_brute_force_small():
    g = synth.rng(16)
    cases = 0
    for N in range(1, 13):
        for K in range(1, 13):
            for P in range(0, 4):
                R = K // 4
                if N > K and P + R >= K:
                    assert O.select_keep(np.zeros(N), P, K, R) == \
                        O.BUDGET_ERROR
                    continue
                # coarse values force many exact ties
                s = np.round(g.standard_normal(N) * 2) / 2
                if N > 3:
                    s[g.integers(0, N)] = np.nan
                    s[g.integers(0, N)] = -0.0
                got = O.select_keep(s, P, K, R)
                assert got.tolist() == _brute_force_keep(s, P, K, R)
                cases += 1
    assert cases > 300


def test_select_properties_large():
    g = synth.rng(17)
    for N, K, P in [(5000, 1024, 0), (5000, 1024, 37), (20000, 4096, 0)]:
        s = synth.old_scores(g, N, ties=True)
        keep = O.select_keep(s, P, K)
        R = O.default_recent(K)
        assert keep.size == K
        assert np.all(np.diff(keep) > 0)
        assert set(range(P)) <= set(keep.tolist())
        assert set(range(N - R, N)) <= set(keep.tolist())
        # every evicted eligible position is outranked by every kept one
        kept_e = [i for i in keep if P <= i < N - R]
        evicted = np.setdiff1d(np.arange(P, N - R), keep)
        worst_kept = max(kept_e, key=lambda i: O.ranking_key(s[i], i))
        best_evicted = min(evicted, key=lambda i: O.ranking_key(s[i], i))
        assert _dominates(s, worst_kept, best_evicted)


def test_select_ties_keep_lower_positions():
    s = np.zeros(10)
    keep = O.select_keep(s, 0, 6, 1)        # M = 5 of positions 0..8
    assert keep.tolist() == [0, 1, 2, 3, 4, 9]


def test_select_negative_zero_equals_zero_and_nan_is_lowest():
    s = np.array([-0.0, 0.0, np.nan, -np.inf, 0.0, 5.0, 1.0])
    keep = O.select_keep(s, 0, 5, 1)       # M = 4 of positions 0..5
    assert keep.tolist() == [0, 1, 4, 5, 6]
    keep = O.select_keep(s, 0, 6, 1)       # M = 5: -inf beats NaN
    assert keep.tolist() == [0, 1, 3, 4, 5, 6]


def test_select_no_eviction_and_budget_error():
    assert O.select_keep(np.arange(8.0), 0, 8).tolist() == list(range(8))
    assert O.select_keep(np.arange(3.0), 0, 8).tolist() == [0, 1, 2]
    assert O.select_keep(np.arange(9.0), 6, 8) == O.BUDGET_ERROR   # 6+2>=8


def test_default_recent():
    assert O.default_recent(256) == 64
    assert O.default_recent(4096) == 128
    assert O.default_recent(8192) == 128
    assert O.default_recent(100) == 25
    assert O.default_recent(3) == 0


# ---------------------------------------------------------------------------
# App. H: order-preserving rebuild
# ---------------------------------------------------------------------------
def test_compact_rows_bytewise():
    g = synth.rng(18)
    rows = synth.random_bits16(g, (50, 4, 16))
    rows[7, 0, 0] = 0x7FC1               # a NaN payload must survive
    keep = np.array([0, 3, 7, 8, 20, 49])
    out = O.compact_rows(rows, keep)
    assert out.shape == (6, 4, 16)
    for j, i in enumerate(keep):
        assert out[j].tobytes() == rows[i].tobytes()
    assert out[2, 0, 0] == 0x7FC1


# ---------------------------------------------------------------------------
# App. H, in place (R18): pack the retained rows to the front of the
# sequence's own pages
# ---------------------------------------------------------------------------
def _sequential_move(rows, keep):
    """Independent check: move one row at a time, lowest slot first, in one
    buffer, asserting that no source row is read after it was overwritten."""
    buf = [r.copy() for r in rows]
    written = np.zeros(len(rows), bool)
    for j, i in enumerate(keep):
        assert not written[i] or i == j, "source overwritten before its read"
        buf[j] = buf[i].copy()
        written[j] = True
    return np.stack(buf)


def test_inplace_rebuild_matches_sequential_move():
    g = synth.rng(19)
    for trial in range(200):
        N = int(g.integers(1, 60))
        rows = synth.random_bits16(g, (N, 3, 4))
        if trial % 2:   # the real producer: the selection rule on scores
            K = int(g.integers(1, N + 1))
            P = int(g.integers(0, K))
            keep = O.select_keep(g.standard_normal(N), P, K,
                                 int(g.integers(0, K - P + 1)))
            if isinstance(keep, str):
                continue
        else:           # any ascending subset
            keep = np.sort(g.choice(N, int(g.integers(0, N + 1)),
                                    replace=False))
        out = O.compact_rows_inplace(rows, keep)
        assert out.tobytes() == _sequential_move(rows, keep).tobytes()
        n = len(keep)
        assert out[:n].tobytes() == O.compact_rows(rows, keep).tobytes()
        assert out[n:].tobytes() == rows[n:].tobytes()       # tail untouched
        h = O.first_hole(keep)
        assert out[:h].tobytes() == rows[:h].tobytes()       # leading run kept


def test_inplace_rebuild_needs_ascending_order():
    # moving the highest slot first overwrites a row before it is read, so
    # the in-place form is only correct walked from the front
    rows = np.arange(3, dtype=np.uint16)[:, None] * np.ones((1, 2), np.uint16)
    keep = np.array([1, 2])
    buf = rows.copy()
    for j in reversed(range(keep.size)):
        buf[j] = buf[keep[j]]
    assert buf[0, 0] == 2                                    # wrong row
    assert O.compact_rows_inplace(rows, keep)[0, 0] == 1     # the rebuild


def test_first_hole():
    assert O.first_hole(np.arange(5)) == 5
    assert O.first_hole(np.array([0, 1, 3, 4])) == 2
    assert O.first_hole(np.array([2, 3])) == 0
    assert O.first_hole(np.array([], dtype=np.int64)) == 0
    # protected prefill is never moved: the first hole is at or past P
    g = synth.rng(20)
    for _ in range(50):
        keep = O.select_keep(g.standard_normal(300), 40, 100, 25)
        assert O.first_hole(keep) >= 40


# ---------------------------------------------------------------------------
# The workloads' KV shape against the paper's capacity figures (Sec. 4.4,
# App. I): 224 concurrent 32,768-token requests at a 2048-token budget
# against 14 without eviction, projected for an 80 GB GPU from the per-token
# cache size.
# ---------------------------------------------------------------------------
def test_kv_bytes_per_token_matches_capacity_figures():
    w = synth.workload("ragged_batch32")
    b = w.kv_bytes_per_token
    assert b == 2 * 32 * 8 * 128 * 2 == 128 * 1024
    # usable cache memory M implied by each figure: floor(M / bytes) = count
    lo1, hi1 = 14 * 32768 * b, 15 * 32768 * b
    lo2, hi2 = 224 * 2048 * b, 225 * 2048 * b
    lo, hi = max(lo1, lo2), min(hi1, hi2)
    assert lo < hi                           # both figures agree
    # ... on about 60 GB: an 80 GB GPU less the ~16 GB of bf16 weights of an
    # 8B-parameter model and some headroom
    assert 55e9 < lo and hi < 64e9
    # half the per-token size (4 KV heads) would leave only ~30 GB of cache
    assert 224 * 2048 * (b // 2) < 31e9


# ---------------------------------------------------------------------------
# App. H, in place with page remapping (R19): a destination page that
# receives one later source page whole, in order, takes that page instead of
# a copy
# ---------------------------------------------------------------------------
def _paged_case(g, N, ps, extra=3):
    """A sequence of N tokens in ceil(N/ps) scattered physical pages of a
    pool that also holds pages nobody owns."""
    n_pg = -(-N // ps)
    n_phys = n_pg + extra
    pt = g.permutation(n_phys)[:n_pg].astype(np.int64)
    pool = synth.random_bits16(g, (n_phys, ps, 3))
    return pool, pt


def _walk_through_tables(pool, old_pt, new_pt, keep, ps, skip_pages):
    """Independent check of the in-place walk: slots in ascending order, each
    row read through the old table and written through the new one, in one
    buffer, asserting that no row is read after it was overwritten."""
    buf = pool.copy()
    written = set()
    for j, i in enumerate(keep):
        d = j // ps
        if d in skip_pages:
            continue
        src = (int(old_pt[i // ps]), int(i % ps))
        dst = (int(new_pt[d]), j % ps)
        assert src not in written or src == dst, "row overwritten before read"
        buf[dst] = buf[src].copy()
        written.add(dst)
    return buf, written


def test_remap_evicting_an_aligned_block_only_rotates_the_table():
    # evicting e whole pages starting at page a moves every later page e
    # places forward: the rebuild is a rotation of the table, no row copied
    g = synth.rng(21)
    for ps, n, a, e in [(4, 4, 1, 1), (4, 8, 2, 3), (16, 10, 0, 2),
                        (1, 9, 3, 2), (3, 7, 6, 1)]:
        N = n * ps
        pool, pt = _paged_case(g, N, ps)
        keep = np.array([i for i in range(N)
                         if not a * ps <= i < (a + e) * ps])
        new_pool, new_pt = O.compact_pages_remap(pool, pt, keep, ps)
        expect = np.concatenate([pt[:a], pt[a + e:], pt[a:a + e]])
        assert new_pt.tolist() == expect.tolist()
        assert new_pool.tobytes() == pool.tobytes()       # nothing written
        assert O.remap_pairs(keep, ps) == [(m, m + e) for m in range(a, n - e)]


def test_remap_hand_example():
    # 4-token pages, page table [10, 11, 12, 13]; positions 4..7 evicted:
    # slots 4..7 take page 12 and slots 8..11 page 13, the page that held
    # positions 4..7 (11) goes to the position page 13 left
    pt = np.array([10, 11, 12, 13])
    keep = np.array([0, 1, 2, 3, 8, 9, 10, 11, 12, 13, 14, 15])
    assert O.remap_pairs(keep, 4) == [(1, 2), (2, 3)]
    assert O.page_table_after_remap(pt, keep, 4).tolist() == [10, 12, 13, 11]
    # one more token evicted inside page 3: page 1 still takes page 2 whole,
    # slots 8..10 are copied from positions 12, 13, 15 into page 11
    keep = np.array([0, 1, 2, 3, 8, 9, 10, 11, 12, 13, 15])
    assert O.remap_pairs(keep, 4) == [(1, 2)]
    assert O.page_table_after_remap(pt, keep, 4).tolist() == [10, 12, 11, 13]


def test_remap_with_no_whole_page_equals_plain_inplace():
    # a shift that is not a multiple of the page size leaves no whole page:
    # the table is unchanged and the pool is the plain in-place rebuild
    g = synth.rng(22)
    ps, N = 4, 40
    pool, pt = _paged_case(g, N, ps)
    keep = np.array([i for i in range(N) if i not in (5, 17, 30)])
    assert O.remap_pairs(keep, ps) == []
    new_pool, new_pt = O.compact_pages_remap(pool, pt, keep, ps)
    assert new_pt.tolist() == pt.tolist()
    rows = pool[pt].reshape(N, 3)
    moved = O.compact_rows_inplace(rows, keep)
    assert new_pool[pt].reshape(N, 3).tobytes() == moved.tobytes()


def test_remap_brute_force_small():
    # every ascending retained set of up to 9 tokens, page sizes 1..4
    g = synth.rng(23)
    import itertools
    n_cases = n_pairs = 0
    for ps in (1, 2, 3, 4):
        for N in range(0, 10):
            pool, pt = _paged_case(g, N, ps)
            for r in range(N + 1):
                for keep in itertools.combinations(range(N), r):
                    keep = np.array(keep, dtype=np.int64)
                    new_pool, new_pt = O.compact_pages_remap(pool, pt, keep, ps)
                    pairs = O.remap_pairs(keep, ps)
                    n_cases += 1
                    n_pairs += len(pairs)
                    # the row is a permutation of the old one
                    assert sorted(new_pt.tolist()) == sorted(pt.tolist())
                    # logical content: slot j holds the row of keep[j]
                    for j, i in enumerate(keep):
                        got = new_pool[new_pt[j // ps], j % ps]
                        assert got.tobytes() == pool[pt[i // ps], i % ps].tobytes()
                    # walked in ascending slot order inside one buffer, no
                    # row is overwritten before it is read, and the result is
                    # the oracle's
                    skip = {m for m, _ in pairs}
                    buf, written = _walk_through_tables(pool, pt, new_pt, keep,
                                                        ps, skip)
                    assert buf.tobytes() == new_pool.tobytes()
                    # only slots of the sequence's own pages are written, and
                    # none of a remapped page; pages nobody owns are unchanged
                    own = set(pt.tolist())
                    assert all(p in own for p, _ in written)
                    assert not any(new_pt[m] == p for p, _ in written
                                   for m in skip)
                    assert len(written) == len(keep) - ps * len(pairs)
                    other = sorted(set(range(pool.shape[0])) - own)
                    assert new_pool[other].tobytes() == pool[other].tobytes()
    assert n_cases > 2000 and n_pairs > 500


def test_remap_release_order_matters():
    # handing the released pages over in descending order would overwrite a
    # row before it is read: the ascending order of R19 is what makes the
    # front-to-back walk safe
    # (with fewer than two released pages the order cannot differ: search
    # the 2-token-page cases for one with two)
    ps = 2
    g = synth.rng(24)
    found = False
    import itertools
    for N in range(6, 13):
        pool, pt = _paged_case(g, N, ps, extra=0)
        for r in range(N + 1):
            for keep in itertools.combinations(range(N), r):
                keep = np.array(keep)
                pairs = O.remap_pairs(keep, ps)
                dests = {m for m, _ in pairs}
                srcs = {p for _, p in pairs}
                rel = [m for m, _ in pairs if m not in srcs]
                lose = [p for _, p in pairs if p not in dests]
                if len(rel) < 2:
                    continue
                wrong = pt.copy()
                for m, p in pairs:
                    wrong[m] = pt[p]
                for m, p in zip(rel, reversed(lose)):
                    wrong[p] = pt[m]
                try:
                    _walk_through_tables(pool, pt, wrong, keep, ps, dests)
                except AssertionError:
                    found = True
                    break
            if found:
                break
        if found:
            break
    assert found
