"""Seeded synthetic inputs for the EpiKV eviction step.

This module only draws inputs: random hidden states, ragged lengths, page
tables, frozen scores of older tokens, and the like.  It contains none of the
method's arithmetic (no differences, norms, windows, rankings or copies of
the method), so the oracle and the HIP library can both be fed from it
without sharing any computation.

Random numbers come from NumPy's Philox-4x32-10 counter-based generator
(Salmon et al., "Parallel random numbers: as easy as 1, 2, 3", SC'11).
Every workload is derived from BASE_SEED plus a workload index.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np

BASE_SEED = 260626472


def rng(seed: int) -> np.random.Generator:
    """A Philox-4x32-10 stream for `seed`."""
    return np.random.Generator(np.random.Philox(int(seed)))


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even) and
    return the 16-bit patterns.  Integer arithmetic on the binary32 word:
    add 0x7FFF plus the lowest kept bit, then drop the low half.  NaNs map to
    a quiet NaN of the same sign."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32)
    nan = np.isnan(f)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u.astype(np.uint64) + np.uint64(0x7FFF) + lsb) >> np.uint64(16))
    out = r.astype(np.uint16)
    if nan.any():
        sign = (u[nan] >> np.uint32(16)) & np.uint32(0x8000)
        out[nan] = (sign | np.uint32(0x7FC0)).astype(np.uint16)
    return out


# ---------------------------------------------------------------------------
# Workloads: shapes of a 32-layer, 4096-wide, 8 KV-head x 128 decoder
# ---------------------------------------------------------------------------
BAND_A = tuple(range(7, 14))    # layers 7..13
BAND_B = tuple(range(18, 26))   # layers 18..25


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                 # seed offset
    B: int                     # sequences
    chunk: int                 # new tokens per step (C = eviction cadence E)
    budget: int                # K
    n_min: int                 # cached tokens N_b at the step (incl. chunk)
    n_max: int
    signal: str = "hs"         # "hs" | "lagkv"
    hidden: int = 4096
    n_layers: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    page_size: int = 16
    window: int = 64
    band_a: tuple = BAND_A
    band_b: tuple = BAND_B
    n_prefix: int = 0
    amplitude: str = "lognormal_spikes"   # | "drift"
    drift: float = 0.0
    spike_rate: float = 0.01
    spike_gain: float = 8.0
    trace_len: int = 0         # multi-step replays: total tokens generated
    notes: str = ""

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def n_band(self) -> int:
        return len(self.band_a) + len(self.band_b)

    @property
    def row_bytes(self) -> int:
        """Bytes of one token's K (or V) row at one layer (all KV heads)."""
        return self.n_kv_heads * self.head_dim * 2

    @property
    def kv_bytes_per_token(self) -> int:
        return 2 * self.n_layers * self.row_bytes

    def band_layers(self):
        return list(self.band_a) + list(self.band_b)


WORKLOADS = {
    # small replay: one sequence, 1024 tokens, evict every 64 to K=256
    "drift_replay": Workload("drift_replay", 1, B=1, chunk=64, budget=256, n_min=320, n_max=320,
                   amplitude="drift", drift=0.001, trace_len=1024,
                   notes="drift replay"),
    # one 16k trace, lognormal deltas + 1% 8x spikes, evict every 128 to 4096
    "spike_replay": Workload("spike_replay", 2, B=1, chunk=128, budget=4096, n_min=4224,
                   n_max=4224, trace_len=16384, notes="spike replay"),
    # headline: 32 ragged sequences 8k..32k, one batched step, K=4096
    "ragged_batch32": Workload("ragged_batch32", 3, B=32, chunk=128, budget=4096, n_min=8192,
                   n_max=32768, notes="batched ragged step"),
    # Lag-KV: 8 sequences of 32k, chunk 256, K=8192
    "lagkv_batch8": Workload("lagkv_batch8", 4, B=8, chunk=256, budget=8192, n_min=32768,
                   n_max=32768, signal="lagkv", notes="lag-kv step"),
    # one-shot scoring of a 65,536-token prefill, K=8192
    "prefill_64k": Workload("prefill_64k", 5, B=1, chunk=65536, budget=8192, n_min=65536,
                   n_max=65536, amplitude="drift_spikes", drift=0.0005,
                   notes="one-shot prefill"),
}


def workload(name: str, **overrides) -> Workload:
    w = WORKLOADS[name]
    return replace(w, **overrides) if overrides else w


# ---------------------------------------------------------------------------
# Draws
# ---------------------------------------------------------------------------
def ragged_lengths(w: Workload, g: np.random.Generator) -> np.ndarray:
    """Cached-token counts N_b, uniform on [n_min, n_max] (inclusive)."""
    return g.integers(w.n_min, w.n_max + 1, size=w.B).astype(np.int64)


def amplitudes(w: Workload, g: np.random.Generator, t0: int, T: int,
               spikes=None) -> np.ndarray:
    """Per-token scale a_l(t) of the band-layer hidden states for tokens
    t0 .. t0+T-1 of one sequence; shape [n_band][T] float32.

    drift            : a_l(t) = (1 + 0.05 l) + dir_l * drift * t, clipped at
                       0.05, with dir = -1 on Band A and +1 on Band B (the
                       direction of the positional trend the paper reports).
    lognormal_spikes : a_l(t) = (1 + 0.05 l) * m, m ~ LogNormal(0, 0.5) iid;
                       on a spike token (rate spike_rate, shared by the
                       layers) Band A amplitudes are multiplied by spike_gain.
    drift_spikes     : the drift model plus the Band A spikes.
    """
    layers = np.array(w.band_layers(), dtype=np.float64)
    base = 1.0 + 0.05 * layers
    t = np.arange(t0, t0 + T, dtype=np.float64)
    na = len(w.band_a)
    direction = np.where(np.arange(w.n_band) < na, -1.0, 1.0)
    if spikes is None:
        spikes = g.random(T) < w.spike_rate
    if w.amplitude == "drift":
        a = base[:, None] + direction[:, None] * w.drift * t[None, :]
        a = np.maximum(a, 0.05)
    elif w.amplitude == "lognormal_spikes":
        m = g.lognormal(0.0, 0.5, size=(w.n_band, T))
        a = base[:, None] * m
        a[:na, spikes] *= w.spike_gain
    elif w.amplitude == "drift_spikes":
        a = base[:, None] + direction[:, None] * w.drift * t[None, :]
        a = np.maximum(a, 0.05)
        a[:na, spikes] *= w.spike_gain
    else:
        raise ValueError(w.amplitude)
    return a.astype(np.float32)


def hidden_rows(a: np.ndarray, D: int, g: np.random.Generator) -> np.ndarray:
    """bf16 bit patterns of hidden-state rows h = a * xi, xi ~ N(0, I_D).

    a : [T] float32 scales.  Returns uint16 [T][D]."""
    xi = g.standard_normal((a.size, D), dtype=np.float32)
    xi *= a[:, None]
    return f32_to_bf16_bits(xi)


def hidden_chunk(w: Workload, g: np.random.Generator, t0, T: int,
                 with_before: bool = True):
    """Hidden states of the band layers for T tokens of every sequence.

    t0 : start token index per sequence (int or [B]).
    Returns (hidden uint16 [n_band][B][T][D], before uint16 [n_band][B][D] or
    None, spikes bool [B][T]).  `before` is the row of the token preceding
    the chunk.
    """
    t0 = np.broadcast_to(np.asarray(t0, dtype=np.int64), (w.B,))
    D = w.hidden
    hid = np.empty((w.n_band, w.B, T, D), dtype=np.uint16)
    before = np.empty((w.n_band, w.B, D), dtype=np.uint16) if with_before \
        else None
    spikes = np.zeros((w.B, T), dtype=bool)
    for b in range(w.B):
        tb = int(t0[b])
        first = tb - 1 if with_before else tb
        n = T + (1 if with_before else 0)
        sp = g.random(n) < w.spike_rate
        a = amplitudes(w, g, first, n, spikes=sp)
        spikes[b] = sp[-T:]
        for l in range(w.n_band):
            rows = hidden_rows(a[l], D, g)
            if with_before:
                before[l, b] = rows[0]
                hid[l, b] = rows[1:]
            else:
                hid[l, b] = rows
    return hid, before, spikes


def prior_samples(w: Workload, g: np.random.Generator, count: int):
    """Earlier per-layer signal samples (the trailing-window history of a
    stream that is already running), drawn at the level a hidden-state
    change of these amplitudes has: sqrt(D * (a1^2 + a2^2)).  Shape
    [B][n_band][count] float32."""
    out = np.empty((w.B, w.n_band, count), dtype=np.float32)
    for b in range(w.B):
        a1 = amplitudes(w, g, 0, count)
        a2 = amplitudes(w, g, 0, count)
        out[b] = np.sqrt(w.hidden * (a1.astype(np.float64) ** 2
                                     + a2.astype(np.float64) ** 2))
    return out


def old_scores(g: np.random.Generator, n: int, ties: bool = False):
    """Frozen fp32 scores of tokens scored by earlier steps: N(0, 0.5^2) with
    1% of them raised by 3.  With ties=True the values are put on a coarse
    grid (multiples of 1/8) so that many exact ties occur."""
    s = g.normal(0.0, 0.5, size=n)
    s[g.random(n) < 0.01] += 3.0
    if ties:
        s = np.round(s * 8.0) / 8.0
    return s.astype(np.float32)


def page_tables(lengths, page_size: int, g: np.random.Generator,
                n_pages_total: int | None = None, ld: int | None = None):
    """Scattered page assignment for sequences of the given lengths.

    Pages of all sequences are a random permutation of 0 .. n_pages-1, so a
    sequence's pages are not contiguous in the pool.  Returns
    (table int32 [B][ld] padded with -1, n_pages_total)."""
    lengths = np.asarray(lengths, dtype=np.int64)
    need = (lengths + page_size - 1) // page_size
    total = int(need.sum())
    if n_pages_total is None:
        n_pages_total = total
    assert n_pages_total >= total
    perm = g.permutation(n_pages_total)[:total]
    if ld is None:
        ld = int(need.max()) if need.size else 1
    table = np.full((lengths.size, ld), -1, dtype=np.int32)
    o = 0
    for b, k in enumerate(need):
        table[b, :k] = perm[o:o + k]
        o += k
    return table, n_pages_total


def contiguous_page_tables(lengths, page_size: int, first: int = 0,
                           ld: int | None = None):
    """Each sequence gets one contiguous run of pages, sequences one after
    another (the allocation of a freshly rebuilt cache).  Returns
    (table int32 [B][ld] padded with -1, n_pages_total)."""
    lengths = np.asarray(lengths, dtype=np.int64)
    need = (lengths + page_size - 1) // page_size
    if ld is None:
        ld = int(need.max()) if need.size else 1
    table = np.full((lengths.size, ld), -1, dtype=np.int32)
    o = first
    for b, k in enumerate(need):
        table[b, :k] = np.arange(o, o + k)
        o += k
    return table, int(o)


def kv_rows(g: np.random.Generator, shape, scale=None) -> np.ndarray:
    """bf16 patterns of N(0,1) values (optionally times a broadcastable
    per-channel scale)."""
    x = g.standard_normal(shape, dtype=np.float32)
    if scale is not None:
        x *= np.asarray(scale, dtype=np.float32)
    return f32_to_bf16_bits(x)


def lagkv_channel_scale(w: Workload, g: np.random.Generator, chunk_idx: int):
    """Per-(layer, K|V, head, channel) magnitude of chunk `chunk_idx` for the
    Lag-KV workload: a fixed log-normal channel profile times a slow drift
    (1 + 0.05 * chunk) and a per-chunk jitter, shape [L][2][H][d]."""
    prof = rng(w.seed * 7 + 1).lognormal(
        0.0, 0.5, size=(w.n_layers, 2, w.n_kv_heads, w.head_dim))
    jitter = g.lognormal(0.0, 0.1, size=prof.shape)
    return (prof * (1.0 + 0.05 * chunk_idx) * jitter).astype(np.float32)


def random_bits16(g: np.random.Generator, shape) -> np.ndarray:
    """Uniform 16-bit patterns (every bf16 value, NaNs included): uniform
    64-bit integers cut into four 16-bit words."""
    n = int(np.prod(shape))
    raw = g.integers(0, np.iinfo(np.uint64).max, size=(n + 3) // 4,
                     dtype=np.uint64, endpoint=True)
    return raw.view(np.uint16)[:n].reshape(shape)
