"""Benchmark of the EpiKV eviction step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload ragged_batch32] [--no-cpu-baseline]

One step = epikv_evict_step over one batch: score the new chunk of every
sequence from its band-layer hidden states, z-score it, select the survivors
and compact the paged KV cache (all 32 layers, K and V, 8 KV heads x 128).
Inputs are seeded synthetic data resident in HBM before the timed region.
Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = ("eviction steps/sec + achieved HBM GB/s (score+select+compact), "
          "B=32, K=4096")
HBM_PEAK_GBPS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# Workload setup (device-resident)
# ---------------------------------------------------------------------------
class Setup:
    pass


# KV-vector signals of the Lag-KV workload: (C-ABI signal, keys, values,
# lag-normalised)
KV_SIGNALS = {"lagkv": ("SIGNAL_LAGKV", True, True, True),
              "kv_key": ("SIGNAL_KV_KEY", True, False, False),
              "kv_val": ("SIGNAL_KV_VAL", False, True, False),
              "lagkv_key": ("SIGNAL_LAGKV_KEY", True, False, True)}


def workload_kind(w: synth.Workload) -> str:
    """hs: a batch evicting after a chunk of new tokens; lagkv: the same
    with the Lag-KV signal; prefill: one trace scored in one shot; replay:
    one sequence at the steady state of a decode loop (timed hot and after
    a cache scrub)."""
    if w.signal == "lagkv":
        return "lagkv"
    if w.chunk == w.n_max:
        return "prefill"
    return "hs" if w.B > 1 else "replay"


def algorithmic_bytes(w: synth.Workload, lengths, n_keep, signal="lagkv"):
    """Bytes the step must move at least once (reads + writes), per stage.

    score   : hidden-state signal: the chunk's band-layer rows, h_prev read +
              write, signal write; KV-vector signals: the chunk's K and/or V
              rows at every layer, for the lag-normalised ones the previous
              and new per-channel ranges of the used tensors, the per-plane
              partial sums written and read, signal write
    zscore  : signal read, carried ring read + write, scores write
    select  : every cached score read once, keep_idx written
    compact : per kept token, its K and V rows at every layer read and
              written (2 * L * H * d * 2 bytes each way), plus its score and
              position read and written
    """
    B, C, nb, D = w.B, w.chunk, w.n_band, w.hidden
    row = w.kv_bytes_per_token
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    out = {}
    if w.signal == "lagkv":
        n_sig = 1
        _, use_k, use_v, lag = KV_SIGNALS[signal]
        used = (int(use_k) + int(use_v)) / 2
        rng_bytes = 2 * B * L * 2 * H * d * 4
        out["score"] = int(B * C * row * used + 2 * rng_bytes * used * lag
                           + 2 * B * 2 * L * C * 4 + B * C * 4)
    else:
        n_sig = nb
        out["score"] = B * nb * (C * D * 2 + 2 * D * 2 + C * 4)
    out["zscore"] = B * n_sig * (C * 4 + 2 * (w.window - 1) * 4) + B * C * 4
    out["select"] = int(np.sum(lengths)) * 4 + int(np.sum(n_keep)) * 4
    out["compact"] = int(np.sum(n_keep)) * (2 * row + 2 * 8)
    out["step"] = sum(out.values())
    return out


def setup_hs(w: synth.Workload, E, log_every=True):
    """Build the headline (hidden-state signal) workload on the GPU."""
    import torch
    S = Setup()
    g = synth.rng(w.seed)
    lengths = synth.ragged_lengths(w, g)
    S.lengths = lengths
    B, C, D, nb = w.B, w.chunk, w.hidden, w.n_band
    L, H, d, page = w.n_layers, w.n_kv_heads, w.head_dim, w.page_size
    K = w.budget
    t0 = time.time()
    hid, before, _ = synth.hidden_chunk(w, g, lengths - C, C)
    ring = synth.prior_samples(w, g, w.window - 1)
    log(f"[setup] hidden states drawn in {time.time() - t0:.1f}s")
    S.hidden_host = hid
    S.before_host = before
    S.ring_host = ring
    ld_s = int(lengths.max())
    S.ld_s = ld_s
    scores = np.zeros((B, ld_s), dtype=np.float32)
    S.old_scores = []
    for b in range(B):
        s = synth.old_scores(g, int(lengths[b]) - C)
        scores[b, :s.size] = s
        S.old_scores.append(s)
    # The cache being evicted has its pages scattered over the pool (a random
    # permutation: the fragmented state of a long-running allocator); the
    # rebuilt cache gets one contiguous run of ceil(K/16) pages per sequence.
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    S.src_pt_host, S.dst_pt_host = src_pt, dst_pt

    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_kv_heads=H,
                        head_dim=d, page_size=page,
                        n_band_a=len(w.band_a), n_band_b=len(w.band_b),
                        window=w.window, budget=K)
    S.cfg = cfg
    dev = torch.device("cuda")
    S.hidden = torch.from_numpy(hid.view(np.int16)).to(dev)   # [nb][B][C][D]
    S.hidden_ptrs = [S.hidden[l] for l in range(nb)]
    st = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st)
    sec["n_tok"][:] = torch.from_numpy((lengths - C).astype(np.int32))
    sec["ring"][:] = torch.from_numpy(ring)
    sec["h_prev"][:] = torch.from_numpy(before.transpose(1, 0, 2).copy()
                                        .view(np.int16))
    S.state_in = st.to(dev)
    S.state_out = torch.zeros_like(S.state_in)
    S.scores = torch.from_numpy(scores).to(dev)
    S.dst_scores = torch.zeros_like(S.scores)
    pos = np.tile(np.arange(ld_s, dtype=np.int32), (B, 1))
    S.src_pos = torch.from_numpy(pos).to(dev)
    S.dst_pos = torch.zeros_like(S.src_pos)
    S.n_cached = torch.from_numpy(lengths.astype(np.int32)).to(dev)
    S.n_prefix = torch.zeros(B, dtype=torch.int32, device=dev)
    S.src_pt = torch.from_numpy(src_pt).to(dev)
    S.dst_pt = torch.from_numpy(dst_pt).to(dev)
    S.keep_idx = torch.zeros((B, K), dtype=torch.int32, device=dev)
    S.n_keep = torch.zeros(B, dtype=torch.int32, device=dev)
    S.status = torch.zeros(B, dtype=torch.int32, device=dev)
    S.ws_bytes = E.workspace_bytes(cfg, C)
    S.ws = torch.zeros(S.ws_bytes, dtype=torch.uint8, device=dev)
    S.cws_bytes = E.compact_workspace_bytes(cfg)
    S.cws = torch.zeros(S.cws_bytes, dtype=torch.uint8, device=dev)
    S.sel_ws_bytes = E.select_workspace_bytes(cfg)
    S.sel_ws = torch.zeros(max(S.sel_ws_bytes, 16), dtype=torch.uint8,
                           device=dev)

    t0 = time.time()
    row = H * d
    S.src_pool = torch.empty((L, 2, n_src, page, row), dtype=torch.int16,
                             device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    flat = S.src_pool.view(-1)
    step = 1 << 30
    for o in range(0, flat.numel(), step):
        n = min(step, flat.numel() - o)
        flat[o:o + n].random_(-32768, 32768, generator=gen)
    S.dst_pool = torch.zeros((L, 2, n_dst, page, row), dtype=torch.int16,
                             device=dev)
    torch.cuda.synchronize()
    log(f"[setup] pools: src {S.src_pool.numel() * 2 / 1e9:.1f} GB, "
        f"dst {S.dst_pool.numel() * 2 / 1e9:.1f} GB filled in "
        f"{time.time() - t0:.1f}s")
    S.src = E.pool_of(S.src_pool.view(L, 2, n_src, page, H, d))
    S.dst = E.pool_of(S.dst_pool.view(L, 2, n_dst, page, H, d))
    S.io = E.make_step_io(
        C, S.hidden_ptrs, D, C * D, S.n_cached, S.n_prefix, S.src, S.src_pt,
        src_pt.shape[1], S.dst, S.dst_pt, dst_pt.shape[1], S.scores, ld_s,
        S.state_in, S.state_out, S.keep_idx, S.n_keep, S.status, S.ws,
        S.ws_bytes, dst_scores=S.dst_scores, src_pos=S.src_pos,
        dst_pos=S.dst_pos)
    # (a buffer of its own: the step keeps the selection's scratch at the
    # start of its workspace from one call to the next)
    S.sig = torch.zeros((E.n_sig(cfg), B, C), device=dev)
    S.score_call = lambda: E.epikv_score(
        cfg, C, S.hidden_ptrs, D, C * D, state_in=S.state_in,
        state_out=S.state_out, sig=S.sig)
    return S


def _step_buffers(S, E, cfg, w, lengths, src_pt, dst_pt, n_src, n_dst, dev):
    """Scores, positions, selection outputs, workspaces and the two pools'
    descriptors shared by every workload."""
    import torch
    B, K, C = w.B, w.budget, w.chunk
    S.n_cached = torch.from_numpy(lengths.astype(np.int32)).to(dev)
    S.n_prefix = torch.zeros(B, dtype=torch.int32, device=dev)
    S.src_pt = torch.from_numpy(src_pt).to(dev)
    S.dst_pt = torch.from_numpy(dst_pt).to(dev)
    S.keep_idx = torch.zeros((B, K), dtype=torch.int32, device=dev)
    S.n_keep = torch.zeros(B, dtype=torch.int32, device=dev)
    S.status = torch.zeros(B, dtype=torch.int32, device=dev)
    S.dst_scores = torch.zeros_like(S.scores)
    pos = np.tile(np.arange(S.ld_s, dtype=np.int32), (B, 1))
    S.src_pos = torch.from_numpy(pos).to(dev)
    S.dst_pos = torch.zeros_like(S.src_pos)
    S.ws_bytes = E.workspace_bytes(cfg, C)
    S.ws = torch.zeros(S.ws_bytes, dtype=torch.uint8, device=dev)
    S.cws_bytes = E.compact_workspace_bytes(cfg)
    S.cws = torch.zeros(S.cws_bytes, dtype=torch.uint8, device=dev)
    S.sel_ws_bytes = E.select_workspace_bytes(cfg)
    S.sel_ws = torch.zeros(max(S.sel_ws_bytes, 16), dtype=torch.uint8,
                           device=dev)
    L, H, d, page = w.n_layers, w.n_kv_heads, w.head_dim, w.page_size
    S.src = E.pool_of(S.src_pool.view(L, 2, n_src, page, H, d))
    S.dst = E.pool_of(S.dst_pool.view(L, 2, n_dst, page, H, d))


def setup_lag(w: synth.Workload, E, signal="lagkv"):
    """The Lag-KV batch: B sequences of n_max cached tokens whose previous
    chunk has been scored (so the step normalises by that chunk's range),
    scored with one of the KV-vector signals."""
    import torch
    S = Setup()
    g = synth.rng(w.seed)
    B, C, K, page = w.B, w.chunk, w.budget, w.page_size
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    N = w.n_max
    lengths = np.full(B, N)
    S.lengths = lengths
    dev = torch.device("cuda")
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    t0 = time.time()
    S.src_pool = torch.empty((L, 2, n_src, page, H * d), dtype=torch.int16,
                             device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    for l in range(L):               # N(0, 1) keys and values, as bf16
        S.src_pool[l].view(torch.bfloat16).normal_(generator=gen)
    S.dst_pool = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                             device=dev)
    torch.cuda.synchronize()
    log(f"[setup] pools: src {S.src_pool.numel() * 2 / 1e9:.1f} GB, "
        f"dst {S.dst_pool.numel() * 2 / 1e9:.1f} GB filled in "
        f"{time.time() - t0:.1f}s")
    cfg = E.default_cfg(batch=B, n_layers=L, n_kv_heads=H, head_dim=d,
                        page_size=page,
                        signal=getattr(E, KV_SIGNALS[signal][0]),
                        smoothing=E.SMOOTH_MEAN, window=w.window, budget=K)
    S.cfg = cfg
    S.ld_s = N
    sc = np.zeros((B, N), np.float32)
    for b in range(B):
        sc[b, :N - 2 * C] = synth.old_scores(g, N - 2 * C)
    S.scores = torch.from_numpy(sc).to(dev)
    _step_buffers(S, E, cfg, w, lengths, src_pt, dst_pt, n_src, n_dst, dev)
    S.src_pt_host, S.dst_pt_host = src_pt, dst_pt
    # score the previous chunk from a fresh stream: its state is the input
    st0 = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device=dev)
    E.epikv_state_init(cfg, st0)
    S.state_in = torch.zeros_like(st0)
    S.state_out = torch.zeros_like(st0)
    S.sig = torch.zeros((1, B, C), device=dev)
    n_prev = torch.full((B,), N - C, dtype=torch.int32, device=dev)
    E.epikv_score(cfg, C, pool=S.src, page_table=S.src_pt,
                  ld_pt=src_pt.shape[1], n_cached=n_prev, state_in=st0,
                  state_out=S.state_in, sig=S.sig, workspace=S.ws,
                  workspace_bytes_=S.ws_bytes)
    E.epikv_zscore(cfg, C, S.sig, n_prev, st0, S.state_in, S.scores, N)
    torch.cuda.synchronize()
    S.sws = torch.zeros(S.ws_bytes, dtype=torch.uint8, device=dev)
    S.score_call = lambda: E.epikv_score(
        cfg, C, pool=S.src, page_table=S.src_pt, ld_pt=src_pt.shape[1],
        n_cached=S.n_cached, state_in=S.state_in, state_out=S.state_out,
        sig=S.sig, workspace=S.sws, workspace_bytes_=S.ws_bytes)
    S.io = E.make_step_io(
        C, None, 0, 0, S.n_cached, S.n_prefix, S.src, S.src_pt,
        src_pt.shape[1], S.dst, S.dst_pt, dst_pt.shape[1], S.scores, N,
        S.state_in, S.state_out, S.keep_idx, S.n_keep, S.status, S.ws,
        S.ws_bytes, dst_scores=S.dst_scores, src_pos=S.src_pos,
        dst_pos=S.dst_pos)
    return S


def setup_prefill(w: synth.Workload, E):
    """One sequence whose whole prefill is scored in one shot, then evicted
    to K (hidden states drawn on the device: h = a(t) * xi)."""
    import torch
    S = Setup()
    g = synth.rng(w.seed)
    T, K, page, D = w.chunk, w.budget, w.page_size, w.hidden
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    nb = w.n_band
    dev = torch.device("cuda")
    lengths = np.array([T])
    S.lengths = lengths
    t0 = time.time()
    a = torch.from_numpy(synth.amplitudes(w, g, 0, T)).to(dev)
    S.hidden = torch.empty((nb, 1, T, D), dtype=torch.int16, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    for l in range(nb):
        x = torch.empty((T, D), dtype=torch.float32, device=dev)
        x.normal_(generator=gen)
        S.hidden[l, 0] = (x * a[l][:, None]).to(torch.bfloat16).view(
            torch.int16)
        del x
    S.hidden_ptrs = [S.hidden[l] for l in range(nb)]
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.array([K]), page)
    S.src_pool = torch.empty((L, 2, n_src, page, H * d), dtype=torch.int16,
                             device=dev)
    S.src_pool.view(-1).random_(-32768, 32768, generator=gen)
    S.dst_pool = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                             device=dev)
    torch.cuda.synchronize()
    log(f"[setup] hidden {S.hidden.numel() * 2 / 1e9:.1f} GB, pool "
        f"{S.src_pool.numel() * 2 / 1e9:.1f} GB in {time.time() - t0:.1f}s")
    cfg = E.default_cfg(batch=1, hidden=D, n_layers=L, n_kv_heads=H,
                        head_dim=d, page_size=page, n_band_a=len(w.band_a),
                        n_band_b=len(w.band_b), window=w.window, budget=K)
    S.cfg = cfg
    S.ld_s = T
    S.scores = torch.zeros((1, T), device=dev)
    _step_buffers(S, E, cfg, w, lengths, src_pt, dst_pt, n_src, n_dst, dev)
    S.state_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8,
                             device=dev)
    E.epikv_state_init(cfg, S.state_in)
    S.state_out = torch.zeros_like(S.state_in)
    # (a buffer of its own: the step keeps the selection's scratch at the
    # start of its workspace from one call to the next)
    S.sig = torch.zeros((nb, 1, T), device=dev)
    S.score_call = lambda: E.epikv_score(
        cfg, T, S.hidden_ptrs, D, T * D, state_in=S.state_in,
        state_out=S.state_out, sig=S.sig)
    S.io = E.make_step_io(
        T, S.hidden_ptrs, D, T * D, S.n_cached, S.n_prefix, S.src, S.src_pt,
        src_pt.shape[1], S.dst, S.dst_pt, dst_pt.shape[1], S.scores, T,
        S.state_in, S.state_out, S.keep_idx, S.n_keep, S.status, S.ws,
        S.ws_bytes, dst_scores=S.dst_scores, src_pos=S.src_pos,
        dst_pos=S.dst_pos)
    return S


def run_stages(E, S, w, events=None):
    """The four stages as separate C-ABI calls, events between them."""
    C = w.chunk
    if events:
        events[0].record()
    S.score_call()
    if events:
        events[1].record()
    E.epikv_zscore(S.cfg, C, S.sig, S.n_cached, S.state_in, S.state_out,
                   S.scores, S.ld_s)
    if events:
        events[2].record()
    E.epikv_select_ws(S.cfg, S.scores, S.ld_s, S.n_cached, S.n_prefix,
                      S.keep_idx, S.n_keep, S.status, S.sel_ws,
                      S.sel_ws_bytes)
    if events:
        events[3].record()
    E.epikv_compact(S.cfg, S.src, S.src_pt, S.src_pt.shape[1], S.dst,
                    S.dst_pt, S.dst_pt.shape[1], S.keep_idx, S.n_keep,
                    S.scores, S.dst_scores, S.src_pos, S.dst_pos, S.ld_s,
                    S.status, S.cws, S.cws_bytes)
    if events:
        events[4].record()


# ---------------------------------------------------------------------------
# In-place rebuild (epikv_compact_inplace) against the out-of-place one
# ---------------------------------------------------------------------------
def _time_calls(fn, reps, warm=3):
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record()
    for i in range(reps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    return float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))


def _time_graph(fn, reps):
    """Device time per call of `fn` with the host out of the loop: `reps`
    calls captured in one HIP graph, replayed between two events."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(3):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(reps):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    graph.replay()
    ev[1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / reps


def first_holes(keep, n_keep):
    """Per sequence, the first slot whose retained position is not the slot
    itself (n_keep when the kept set is a leading run): the in-place rebuild
    moves exactly the slots from there to n_keep."""
    out = []
    for b in range(keep.shape[0]):
        k = keep[b, :n_keep[b]]
        bad = np.nonzero(k != np.arange(k.size))[0]
        out.append(int(bad[0]) if bad.size else int(k.size))
    return np.array(out)


def whole_pages(keep, n_keep, page):
    """Destination pages that take a whole source page (page remapping):
    full pages whose slots hold one later, aligned source page in order."""
    total = 0
    for b in range(keep.shape[0]):
        n = int(n_keep[b]) // page * page
        if n <= 0:
            continue
        runs = keep[b, :n].reshape(-1, page).astype(np.int64)
        first = runs[:, 0]
        ok = ((first % page == 0) & (first > np.arange(runs.shape[0]) * page)
              & (runs[:, -1] - first == page - 1))
        total += int(ok.sum())
    return total


def compare_compactions(E, cfg, w, src, src_pt, dst, dst_pt, keep, n_keep,
                        scores, dscores, ld_s, status, cws, reps):
    """Time epikv_compact (into contiguous and into randomly placed
    destination pages), epikv_compact_inplace and epikv_compact_remap on the
    same kept sets.
    The in-place call rewrites the source pool: its later repetitions move
    the same slots (the cost depends on the kept sets, not the bytes)."""
    kh, nk = keep.cpu().numpy(), n_keep.cpu().numpy()
    holes = first_holes(kh, nk)
    row = w.kv_bytes_per_token
    kept = int(nk.sum())
    moved = int((nk - holes).sum())
    ms_out = _time_calls(lambda: E.epikv_compact(
        cfg, src, src_pt, src_pt.shape[1], dst, dst_pt, dst_pt.shape[1],
        keep, n_keep, scores, dscores, None, None, ld_s, status, cws,
        cws.numel()), reps)
    # the same rebuild into the same destination pages placed at random
    # (the fragmented pool of a long-running allocator)
    import torch
    perm = torch.from_numpy(synth.rng(w.seed + 13).permutation(
        int(dst.n_pages)).astype(np.int32)).to(dst_pt.device)
    dst_pt_scat = perm[dst_pt.long()].contiguous()
    ms_scat = _time_calls(lambda: E.epikv_compact(
        cfg, src, src_pt, src_pt.shape[1], dst, dst_pt_scat,
        dst_pt_scat.shape[1], keep, n_keep, scores, dscores, None, None,
        ld_s, status, cws, cws.numel()), reps)
    ms_in = _time_calls(lambda: E.epikv_compact_inplace(
        cfg, src, src_pt, src_pt.shape[1], keep, n_keep, scores, None, ld_s,
        status, cws, cws.numel()), reps)
    # page remapping rewrites the table: each call permutes a copy again,
    # with the same pages remapped and the same rows moved every time
    pt_copy = src_pt.clone()
    ms_remap = _time_calls(lambda: E.epikv_compact_remap(
        cfg, src, pt_copy, src_pt.shape[1], keep, n_keep, scores, None, ld_s,
        status, cws, cws.numel()), reps)
    pages = whole_pages(kh, nk, w.page_size)
    moved_remap = moved - pages * w.page_size
    out_bytes = kept * (2 * row + 8)
    in_bytes = moved * (2 * row + 8)
    return {"rows_kept": kept, "rows_moved_in_place": moved,
            "pages_remapped": pages, "rows_moved_remap": moved_remap,
            "ms_out_of_place": round(ms_out, 4),
            "ms_out_of_place_scattered_pages": round(ms_scat, 4),
            "ms_in_place": round(ms_in, 4),
            "ms_remap": round(ms_remap, 4),
            "gbps_out_of_place": round(out_bytes / ms_out / 1e6, 1),
            "gbps_out_of_place_scattered_pages": round(out_bytes / ms_scat / 1e6, 1),
            "gbps_in_place": round(in_bytes / ms_in / 1e6, 1),
            "gbps_remap": round(moved_remap * (2 * row) / ms_remap / 1e6, 1)}


def inplace_report(E, S, w, reps):
    import torch
    dev = torch.device("cuda")
    out = []
    # 1. the headline batch (select already ran in the correctness guard)
    r = compare_compactions(E, S.cfg, w, S.src, S.src_pt, S.dst, S.dst_pt,
                            S.keep_idx, S.n_keep, S.scores, S.dst_scores,
                            S.ld_s, S.status, S.cws, reps)
    r["workload"] = (f"{w.name}: B={w.B}, N in [{w.n_min},{w.n_max}] -> "
                     f"K={w.budget}, no protected prefill")
    out.append(r)
    log(f"[inplace] {r}")
    del S.src_pool, S.dst_pool, S.src, S.dst
    torch.cuda.empty_cache()
    # 2. steady-state decode eviction: every sequence at K + C, back to K
    B, K, C, page = w.B, w.budget, w.chunk, w.page_size
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    g = synth.rng(w.seed + 7)
    lengths = np.full(B, K + C)
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    src_pool = torch.empty((L, 2, n_src, page, H * d), dtype=torch.int16,
                           device=dev)
    src_pool.view(-1)[: 1 << 30].random_(-32768, 32768)
    dst_pool = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                           device=dev)
    src = E.pool_of(src_pool.view(L, 2, n_src, page, H, d))
    dst = E.pool_of(dst_pool.view(L, 2, n_dst, page, H, d))
    sc = np.stack([synth.old_scores(g, K + C) for _ in range(B)])
    scores = torch.from_numpy(sc).to(dev)
    dscores = torch.zeros_like(scores)
    spt = torch.from_numpy(src_pt).to(dev)
    dpt = torch.from_numpy(dst_pt).to(dev)
    n_cached = torch.from_numpy(lengths.astype(np.int32)).to(dev)
    for P in (0, 1024):
        n_prefix = torch.full((B,), P, dtype=torch.int32, device=dev)
        E.epikv_select(S.cfg, scores, K + C, n_cached, n_prefix, S.keep_idx,
                       S.n_keep, S.status)
        r = compare_compactions(E, S.cfg, w, src, spt, dst, dpt, S.keep_idx,
                                S.n_keep, scores, dscores, K + C, S.status,
                                S.cws, reps)
        r["workload"] = (f"steady-state decode eviction: B={B}, N={K + C} "
                         f"-> K={K}, protected prefill P={P}")
        out.append(r)
        log(f"[inplace] {r}")
    # 3. the best case of page remapping: the evicted tokens fill whole
    # aligned pages (here the lowest scores are C/page whole pages)
    for b in range(B):
        pages = g.choice((K - C) // page, size=C // page, replace=False)
        for a in pages:
            sc[b, a * page:(a + 1) * page] -= 1000.0
    scores.copy_(torch.from_numpy(sc))
    n_prefix = torch.zeros((B,), dtype=torch.int32, device=dev)
    E.epikv_select(S.cfg, scores, K + C, n_cached, n_prefix, S.keep_idx,
                   S.n_keep, S.status)
    r = compare_compactions(E, S.cfg, w, src, spt, dst, dpt, S.keep_idx,
                            S.n_keep, scores, dscores, K + C, S.status,
                            S.cws, reps)
    r["workload"] = (f"steady-state decode eviction, evicted tokens in whole "
                     f"pages: B={B}, N={K + C} -> K={K}")
    out.append(r)
    log(f"[inplace] {r}")
    return out


# ---------------------------------------------------------------------------
# Online scoring: one fused launch per decode token vs the two separate calls
# ---------------------------------------------------------------------------
def online_report(E, w, reps):
    import torch
    dev = torch.device("cuda")
    B, D, nb = w.B, w.hidden, w.n_band
    g = synth.rng(w.seed + 11)
    out = []
    for C in (1, 2, 4, 16, 64):
        cfg = E.default_cfg(batch=B, hidden=D, n_band_a=len(w.band_a),
                            n_band_b=len(w.band_b), window=w.window)
        hid = torch.from_numpy(synth.f32_to_bf16_bits(
            g.standard_normal((nb, B, C, D), dtype=np.float32)).view(
                np.int16)).to(dev)
        hidden = [hid[l] for l in range(nb)]
        st = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
        sec = E.state_sections(cfg, st)
        sec["n_tok"][:] = 5000
        sec["ring"][:] = torch.from_numpy(
            (50 + g.standard_normal(tuple(sec["ring"].shape))).astype(
                np.float32))
        st_in = st.to(dev)
        st_out = torch.zeros_like(st_in)
        ld_s = 8192
        scores = torch.zeros((B, ld_s), device=dev)
        n_cached = torch.full((B,), 5000 + C, dtype=torch.int32, device=dev)
        sig = torch.zeros((nb, B, C), device=dev)

        def two():
            E.epikv_score(cfg, C, hidden, D, C * D, state_in=st_in,
                          state_out=st_out, sig=sig)
            E.epikv_zscore(cfg, C, sig, n_cached, st_in, st_out, scores, ld_s)

        def fused():
            E.epikv_score_tokens(cfg, C, hidden, D, C * D, n_cached, st_in,
                                 st_out, scores, ld_s)

        ms2 = _time_graph(two, reps)
        ms1 = _time_graph(fused, reps)
        by = B * nb * (C + 2) * D * 2          # rows + h_prev in/out
        r = {"tokens_per_call": C, "B": B, "us_fused": round(ms1 * 1e3, 2),
             "us_two_calls": round(ms2 * 1e3, 2),
             "gbps_fused": round(by / ms1 / 1e6, 1)}
        log(f"[online] {r}")
        out.append(r)
    return out


def online_step_report(E, w, reps):
    """The headline batch's eviction step when the chunk's tokens were
    already scored one by one (epikv_evict_step with chunk 0: select and
    rebuild only) against the step that scores the chunk itself."""
    S = setup_hs(w, E)
    ms_scoring = _time_calls(lambda: E.epikv_evict_step(S.cfg, S.io), reps)
    import torch
    ws_n = E.workspace_bytes(S.cfg, 0)
    ws0 = torch.zeros(ws_n, dtype=torch.uint8, device=S.scores.device)
    io0 = E.make_step_io(
        0, None, 0, 0, S.n_cached, S.n_prefix, S.src, S.src_pt,
        S.src_pt.shape[1], S.dst, S.dst_pt, S.dst_pt.shape[1], S.scores,
        S.ld_s, None, None, S.keep_idx, S.n_keep, S.status, ws0, ws_n,
        dst_scores=S.dst_scores, src_pos=S.src_pos, dst_pos=S.dst_pos)
    ms_online = _time_calls(lambda: E.epikv_evict_step(S.cfg, io0), reps)
    r = {"workload": f"{w.name}: B={w.B}, C={w.chunk}, K={w.budget}",
         "ms_step_scoring_the_chunk": round(ms_scoring, 4),
         "ms_step_chunk_scored_online": round(ms_online, 4)}
    log(f"[online] {r}")
    return r


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the same workload
# ---------------------------------------------------------------------------
def cpu_baseline(w: synth.Workload, S, budget_s: float = 12.0):
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(1)
    except Exception:
        limiter = None
    g = synth.rng(w.seed + 1000)
    C, nb = w.chunk, w.n_band
    na = len(w.band_a)
    spent = 0.0
    done = 0
    row_elems = w.n_kv_heads * w.head_dim
    # source rows: random bits as on the GPU, a 2048-token block tiled to the
    # longest sampled length (the oracle's work does not depend on content)
    block = synth.random_bits16(g, (2048, w.n_layers, 2, row_elems))
    n_max = int(S.lengths.max())
    all_rows = np.concatenate([block] * ((n_max + 2047) // 2048))[:n_max]
    del block
    while done < w.B and spent < budget_s:
        b = done
        N = int(S.lengths[b])
        rows = all_rows[:N]
        hid = O.bf16_to_float64(S.hidden_host[:, b])        # [nb][C][D]
        before = O.bf16_to_float64(S.before_host[:, b])     # [nb][D]
        prior = [S.ring_host[b, l].astype(np.float64) for l in range(nb)]
        scores = np.concatenate([S.old_scores[b].astype(np.float64),
                                 np.zeros(C)])
        t0 = time.perf_counter()
        s_new, *_ = O.hs_chunk_scores(hid, before, prior, na, nb - na,
                                      O.SMOOTH_Z, w.window, 1e-6)
        scores[N - C:] = s_new
        keep = O.select_keep(scores, 0, w.budget)
        kept = O.compact_rows(rows, keep)
        spent += time.perf_counter() - t0
        done += 1
        del kept
    if limiter is not None:
        limiter.unregister()
    per_step = spent / done * w.B
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": 1,
            "host_cores": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{done} of {w.B} sequences of the same step (score, "
                      f"select, compact of all 32 layers) timed on one core; "
                      f"scaled to the full batch ({spent:.1f}s measured)"}


def _oracle_rows(g, w, n):
    """Source rows for the oracle's rebuild: random bits as on the GPU, a
    2048-token block tiled to n tokens (the copy does not depend on them)."""
    block = synth.random_bits16(
        g, (2048, w.n_layers, 2, w.n_kv_heads * w.head_dim))
    return np.concatenate([block] * ((n + 2047) // 2048))[:n]


def cpu_baseline_lag(w: synth.Workload, S, budget_s: float = 12.0,
                     signal="lagkv"):
    """The oracle on sequences of the Lag-KV step: the new chunk's variance
    signal (normalised against the previous chunk's range for the lag
    variants), the trailing mean, the selection over all N tokens, the
    rebuild."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(1)
    except Exception:
        limiter = None
    g = synth.rng(w.seed + 1000)
    C, N, L, H, d = w.chunk, w.n_max, w.n_layers, w.n_kv_heads, w.head_dim
    rows = _oracle_rows(g, w, N)
    prev = O.bf16_to_float64(synth.kv_rows(g, (C, L, 2, H, d)))
    new = O.bf16_to_float64(synth.kv_rows(g, (C, L, 2, H, d)))
    _, use_k, use_v, lag = KV_SIGNALS[signal]
    _, q_prev, rng_prev = O.kv_chunk_scores(prev[:, :, 0], prev[:, :, 1],
                                            use_k, use_v, lag, None,
                                            np.zeros(0))
    old = S.scores.cpu().numpy().astype(np.float64)
    spent, done = 0.0, 0
    while done < w.B and spent < budget_s:
        scores = old[done, :N].copy()
        t0 = time.perf_counter()
        s_new, _, _ = O.kv_chunk_scores(new[:, :, 0], new[:, :, 1], use_k,
                                        use_v, lag, rng_prev,
                                        q_prev[-(w.window - 1):])
        scores[N - C:] = s_new
        keep = O.select_keep(scores, 0, w.budget)
        kept = O.compact_rows(rows, keep)
        spent += time.perf_counter() - t0
        done += 1
        del kept
    if limiter is not None:
        limiter.unregister()
    per_step = spent / done * w.B
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": 1,
            "host_cores": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{done} of {w.B} sequences of the same step "
                      f"({signal} score of the {C}-token chunk, select, "
                      f"compact of all "
                      f"{L} layers) timed on one core; scaled to the full "
                      f"batch ({spent:.1f}s measured)"}


def cpu_baseline_prefill(w: synth.Workload, S, sample_tokens: int = 2048):
    """The oracle on the one-shot prefill: Eq. 1 + Eq. 3 + band combination
    over a block of the trace (scaled to the whole trace), then the
    selection over all T tokens and the rebuild of K rows."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(1)
    except Exception:
        limiter = None
    g = synth.rng(w.seed + 1000)
    T, nb, na = w.chunk, w.n_band, len(w.band_a)
    hid = O.bf16_to_float64(S.hidden[:, 0, :sample_tokens].cpu().numpy()
                            .view(np.uint16))
    # rows of the source cache: a 2048-token block of random bits, row i of
    # the trace read from row i % 2048 (the copy's work is the same)
    block = synth.random_bits16(
        g, (2048, w.n_layers, 2, w.n_kv_heads * w.head_dim))
    scores = S.scores.cpu().numpy()[0].astype(np.float64)
    t0 = time.perf_counter()
    O.hs_chunk_scores(hid, None, [np.zeros(0)] * nb, na, nb - na)
    t_score = (time.perf_counter() - t0) * T / sample_tokens
    t0 = time.perf_counter()
    keep = O.select_keep(scores, 0, w.budget)
    kept = O.compact_rows(block, keep % 2048)
    t_rest = time.perf_counter() - t0
    del kept
    if limiter is not None:
        limiter.unregister()
    per_step = t_score + t_rest
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": 1,
            "host_cores": os.cpu_count(),
            "kind": "oracle",
            "sample": f"scores of the first {sample_tokens} of {T} tokens "
                      f"timed and scaled to the trace, plus the selection "
                      f"over all {T} and the rebuild of {w.budget} rows, on "
                      f"one core ({t_score + t_rest:.1f}s estimated)"}


def _copy_probe_lib():
    """The streaming-copy probe (libcopyprobe.so, built beside libepikv.so):
    plain device copies in several launch shapes."""
    import ctypes
    path = os.path.join(ROOT, "paper_2606_26472_amd", "libcopyprobe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run "
                           "python -m paper_2606_26472_amd.build")
    lib = ctypes.CDLL(path)
    lib.copy_probe.restype = ctypes.c_int
    lib.copy_probe.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    lib.copy_probe_variants.restype = ctypes.c_int
    lib.copy_probe_name.restype = ctypes.c_char_p
    lib.copy_probe_name.argtypes = [ctypes.c_int]
    return lib


def copy_ceiling(n_bytes: int = 4 << 30, reps: int = 5):
    """Practical streaming ceiling of this GPU: the fastest of the copy
    probe's launch shapes copying one contiguous n_bytes buffer (read +
    write bytes / time, HIP events on the launch stream), and torch's own
    copy for reference.  Returns (best GB/s, its ms, its shape, every
    shape's GB/s)."""
    import torch
    lib = _copy_probe_lib()
    a = torch.empty(n_bytes // 2, dtype=torch.int16, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    def timed(fn):
        fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            fn()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        return float(np.mean([ev[i].elapsed_time(ev[i + 1])
                              for i in range(reps)]))

    shapes = {}
    for v in range(lib.copy_probe_variants()):
        def run(v=v):
            rc = lib.copy_probe(a.data_ptr(), b.data_ptr(), n_bytes, v, sh)
            if rc != 0:
                raise RuntimeError(f"copy probe shape {v} failed: {rc}")
        ms = timed(run)
        shapes[lib.copy_probe_name(v).decode()] = (
            round(2 * n_bytes / (ms * 1e-3) / 1e9, 1), ms)
    ms_torch = timed(lambda: b.copy_(a))
    del a, b
    best = max(shapes, key=lambda k: shapes[k][0])
    gbps = {k: v[0] for k, v in shapes.items()}
    gbps["torch copy_"] = round(2 * n_bytes / (ms_torch * 1e-3) / 1e9, 1)
    return shapes[best][0], shapes[best][1], best, gbps


COMPACT_SOURCES = ("paper_2606_26472_amd/csrc/compact.hip",)


def compact_source_hash() -> str:
    """Hash of the source that defines the compaction kernels and their
    launch shape."""
    h = hashlib.sha256()
    for rel in COMPACT_SOURCES:
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    return h.hexdigest()


def traffic_from_profiles():
    """HBM bytes per epikv_compact call from the committed counter summary,
    if it was taken on the current kernel sources (else None), and where
    the figure comes from."""
    rel = os.path.join("profiles", "compact_ragged_batch32_traffic.json")
    path = os.path.join(ROOT, rel)
    if not os.path.exists(path):
        return None, None
    try:
        rec = json.load(open(path))
        if rec.get("kernel_sha256") != compact_source_hash():
            return None, None
        return rec.get("bytes_per_launch"), (
            f"{rel}: FETCH_SIZE + WRITE_SIZE counters of an earlier run on "
            f"the same compaction source (sha256 "
            f"{rec['kernel_sha256'][:16]}), not measured in this run")
    except Exception:
        return None, None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="ragged_batch32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stages-only", action="store_true",
                    help="only the per-stage loop (for profiling)")
    ap.add_argument("--online", action="store_true",
                    help="time the fused per-token scorer against the two "
                         "separate calls (one JSON line of its own)")
    ap.add_argument("--signal", default="lagkv", choices=sorted(KV_SIGNALS),
                    help="KV-vector signal of the lagkv_batch8 workload")
    ap.add_argument("--inplace", action="store_true",
                    help="compare the in-place and out-of-place rebuilds "
                         "(one JSON line of its own) instead of the step")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not "
              "supported (the eviction step is per-sequence and shards over "
              "sequences without communication)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_26472_amd import epikv as E
    E.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = synth.workload(args.workload)
    kind = workload_kind(w)
    if (args.online or args.inplace) and kind != "hs":
        print("--online and --inplace run on the hidden-state batch only",
              file=sys.stderr)
        sys.exit(2)
    log(f"[bench] workload {w.name}: B={w.B} K={w.budget} C={w.chunk}")
    if args.online:
        rows = online_report(E, w, max(args.steps, 100))
        steps = online_step_report(E, w, max(args.steps // 5, 10))
        print(json.dumps({
            "metric": "online scoring: microseconds per scoring call "
                      "(hidden-state signal, 15 band layers x 4096)",
            "unit": "us", "n_gpus": 1, "data": "synthetic",
            "results": rows, "eviction_step": steps}), flush=True)
        return
    if args.signal != "lagkv" and kind != "lagkv":
        print("--signal applies to the lagkv_batch8 workload", file=sys.stderr)
        sys.exit(2)
    if kind == "lagkv":
        S = setup_lag(w, E, args.signal)
    else:
        S = {"hs": setup_hs, "replay": setup_hs,
             "prefill": setup_prefill}[kind](w, E)

    # correctness guard: one step, every sequence must be OK with K kept
    E.epikv_evict_step(S.cfg, S.io)
    torch.cuda.synchronize()
    st = S.status.cpu().numpy()
    nk = S.n_keep.cpu().numpy()
    assert np.all(st == 0) and np.all(nk == np.minimum(S.lengths, w.budget)), \
        (st, nk)
    ab = algorithmic_bytes(w, S.lengths, nk, args.signal)
    if args.inplace:
        rows = inplace_report(E, S, w, args.steps)
        print(json.dumps({
            "metric": "in-place vs out-of-place cache rebuild (GB/s of the "
                      "bytes each must move)",
            "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "data": "synthetic", "results": rows}), flush=True)
        return

    stream = torch.cuda.current_stream()
    if not args.stages_only:
        for _ in range(args.warmup):
            E.epikv_evict_step(S.cfg, S.io)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            E.epikv_evict_step(S.cfg, S.io)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_step = wall / args.steps * 1e3
        log(f"[bench] evict_step: {ms_step:.3f} ms/step")
    scrubbed_ms = None
    if kind == "replay" and not args.stages_only:
        # the same step with the caches flushed first: a 512 MiB write
        # between steps, the step alone between two events
        scrub = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
              for _ in range(args.steps)]
        for i in range(args.steps):
            scrub.fill_(float(i))
            ev[i][0].record()
            E.epikv_evict_step(S.cfg, S.io)
            ev[i][1].record()
        torch.cuda.synchronize()
        scrubbed_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        log(f"[bench] evict_step after a cache scrub: {scrubbed_ms:.4f} ms")
        del scrub
    # per-stage durations with events on the launch stream
    n_ev = args.steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)]
           for _ in range(n_ev)]
    for _ in range(args.warmup):
        run_stages(E, S, w)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(n_ev):
        run_stages(E, S, w, evs[i])
    torch.cuda.synchronize()
    stage_wall = (time.perf_counter() - t0) / n_ev * 1e3
    names = ["score", "zscore", "select", "compact"]
    stage_ms = {n: float(np.mean([e[k].elapsed_time(e[k + 1]) for e in evs]))
                for k, n in enumerate(names)}
    log("[bench] stages (ms): " + ", ".join(f"{k}={v:.4f}"
                                          for k, v in stage_ms.items()))
    if args.stages_only:
        ms_step = stage_wall
    copy_gbps, copy_ms, copy_shape, copy_all = copy_ceiling()
    log(f"[bench] streaming copy of 4 GiB: best {copy_ms:.3f} ms = "
        f"{copy_gbps:.0f} GB/s ({copy_shape}); all shapes: {copy_all}")
    step_gbps = ab["step"] / (ms_step * 1e-3) / 1e9
    # the roofline is the dominant kernel's: the rebuild, or the scoring of
    # a one-shot prefill
    dom = "compact" if stage_ms["compact"] >= stage_ms["score"] else "score"
    dom_gbps = ab[dom] / (stage_ms[dom] * 1e-3) / 1e9
    dom_name = {"compact": "epikv_compact (k_compact_order + "
                           "k_compact_resolve + k_compact)",
                "score": ("epikv_score (k_score_lagkv + k_lag_reduce)"
                          if kind == "lagkv" else
                          "epikv_score (k_score_hs_wave)")}[dom]
    traffic, traffic_src = (traffic_from_profiles()
                            if (w.name, dom) == ("ragged_batch32", "compact")
                            else (None, None))

    descr = {
        "hs": f"{w.name}: batched eviction step, B={w.B} ragged N in "
              f"[{w.n_min},{w.n_max}], K={w.budget}, C={w.chunk} new tokens, "
              f"{w.n_layers} layers x {w.n_kv_heads} KV heads x {w.head_dim} "
              f"bf16 paged ({w.page_size}-token pages), HS bands 7-13/18-25, "
              f"z-score w={w.window}",
        "lagkv": f"{w.name}: batched {args.signal} eviction step, "
                 f"B={w.B}, N={w.n_max}, K={w.budget}, chunk of {w.chunk} "
                 f"new tokens"
                 + (" normalised by the previous chunk's range"
                    if KV_SIGNALS[args.signal][3] else "")
                 + f", {w.n_layers} layers x {w.n_kv_heads} KV heads x "
                 f"{w.head_dim} bf16 paged, trailing mean w={w.window}",
        "replay": f"{w.name}: one sequence at its steady state, "
                  f"N={w.n_max} -> K={w.budget} after a {w.chunk}-token "
                  f"chunk, {w.n_layers} layers x {w.n_kv_heads} KV heads x "
                  f"{w.head_dim} bf16 paged, HS bands 7-13/18-25",
        "prefill": f"{w.name}: one {w.chunk}-token prefill scored in one "
                   f"shot (HS bands 7-13/18-25, z-score w={w.window}) and "
                   f"evicted to K={w.budget}, {w.n_layers} layers x "
                   f"{w.n_kv_heads} KV heads x {w.head_dim} bf16 paged",
    }[kind]
    result = {
        "metric": METRIC if w.name == "ragged_batch32" else
        f"eviction steps/sec + achieved HBM GB/s (score+select+compact), "
        f"B={w.B}, K={w.budget}",
        "value": round(1e3 / ms_step, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "achieved_hbm_gbps": round(step_gbps, 1),
        "config": {
            "workload": descr,
            "B": w.B, "K": w.budget, "chunk": w.chunk,
            "n_cached": [int(x) for x in S.lengths],
            "algorithmic_bytes": ab,
            "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
            **({"ms_per_step_cache_scrubbed": round(scrubbed_ms, 4)}
               if scrubbed_ms is not None else {}),
        },
        "roofline": {
            "kernel": dom_name,
            "bound": "hbm",
            "achieved": round(dom_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "traffic_source": traffic_src,
            "device_copy_gbps": round(copy_gbps, 1),
            "device_copy_shape": copy_shape,
            "frac_of_device_copy": round(dom_gbps / copy_gbps, 4),
        },
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample ...")
        if kind == "lagkv":
            result["cpu_baseline"] = cpu_baseline_lag(w, S,
                                                      signal=args.signal)
        else:
            result["cpu_baseline"] = {"hs": cpu_baseline,
                                      "replay": cpu_baseline,
                                      "prefill": cpu_baseline_prefill}[kind](
                                          w, S)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
