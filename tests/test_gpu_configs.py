"""Parity of the Lag-KV batch and the one-shot long prefill at full size.

Both run epikv_evict_step at the workload's real shape.  The oracle checks
every score the step writes (the new chunks' for Lag-KV, all 65,536 of the
prefill, computed in float64 from the same bf16 rows), the retained set
exactly against the oracle's ranking of the GPU's fp32 scores and against
the oracle's own float64 ranking up to near-ties at the cut, and every row of
the rebuilt cache bit for bit (compared on the device).
"""
import numpy as np
import pytest

import oracle as O
import synth
from harness import (NEAR_ZERO, POSITIVE, TOL, dev, host, idx,
                     rebuilt_rows_equal, rel_err, tie_exempt_compare)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def _sync():
    import torch
    torch.cuda.synchronize()


def test_lagkv_batch_full_size(E):
    import torch
    w = synth.workload("lagkv_batch8")
    print("lagkv batch 8 x 32768, chunk 256, K=8192", flush=True)
    g = synth.rng(w.seed)
    B, C, K, page = w.B, w.chunk, w.budget, w.page_size
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    N = w.n_max
    HD = H * d
    src_pt, n_src = synth.page_tables(np.full(B, N), page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    pool = torch.empty((L, 2, n_src, page, HD), dtype=torch.bfloat16,
                       device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)
    for l in range(L):
        pool[l].normal_(generator=gen)
    # the last two chunks (the previous and the new one) with per-channel
    # magnitude drift, drawn on the host so the oracle sees the same rows
    chunks = []
    for j, lo in enumerate((N - 2 * C, N - C)):
        rows = np.stack([synth.kv_rows(g, (C, L, 2, H, d),
                                       synth.lagkv_channel_scale(w, g, j))
                         for _ in range(B)])               # [B][C][L][2][H][d]
        chunks.append(rows)
        for b in range(B):
            p = np.arange(lo, lo + C)
            pool.view(torch.int16)[:, :, idx(src_pt[b, p // page]),
                                   idx(p % page), :] = dev(
                rows[b].reshape(C, L, 2, HD).transpose(1, 2, 0, 3))
    cfg = E.default_cfg(batch=B, n_layers=L, signal=E.SIGNAL_LAGKV,
                        smoothing=E.SMOOTH_MEAN, budget=K)
    st = [torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
          for _ in range(3)]
    E.epikv_state_init(cfg, st[0])
    ld_s = N
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :N - 2 * C] = synth.old_scores(g, N - 2 * C)
    old = sc[:, :N - 2 * C].astype(np.float64)
    scores = dev(sc)
    ws_n = E.workspace_bytes(cfg, C)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    P = E.pool_of(pool.view(L, 2, n_src, page, H, d))
    spt = dev(src_pt)
    # the previous chunk: score and smooth it (fresh stream: own range)
    sig = torch.zeros((1, B, C), device="cuda")
    n_prev = dev(np.full(B, N - C, np.int32))
    E.epikv_score(cfg, C, pool=P, page_table=spt, ld_pt=src_pt.shape[1],
                  n_cached=n_prev, state_in=st[0], state_out=st[1], sig=sig,
                  workspace=ws, workspace_bytes_=ws_n)
    E.epikv_zscore(cfg, C, sig, n_prev, st[0], st[1], scores, ld_s)
    # the eviction step on the new chunk
    dst = torch.zeros((L, 2, n_dst, page, HD), dtype=torch.int16,
                      device="cuda")
    keep = torch.zeros((B, K), dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    io = E.make_step_io(
        C, None, 0, 0, dev(np.full(B, N, np.int32)),
        torch.zeros(B, dtype=torch.int32, device="cuda"), P, spt,
        src_pt.shape[1], E.pool_of(dst.view(L, 2, n_dst, page, H, d)),
        dev(dst_pt), dst_pt.shape[1], scores, ld_s, st[1], st[2], keep,
        n_keep, status, ws, ws_n)
    E.epikv_evict_step(cfg, io)
    _sync()
    assert np.all(host(status) == 0) and np.all(host(n_keep) == K)
    gs = host(scores)
    kh = host(keep)
    R = O.default_recent(K)
    for b in range(B):
        k1 = O.bf16_to_float64(chunks[0][b].reshape(C, L, 2, H, d))
        k2 = O.bf16_to_float64(chunks[1][b].reshape(C, L, 2, H, d))
        s1, q1, r1 = O.lagkv_chunk_scores(k1[:, :, 0], k1[:, :, 1], None,
                                          np.zeros(0), O.SMOOTH_MEAN)
        s2, q2, _ = O.lagkv_chunk_scores(k2[:, :, 0], k2[:, :, 1], r1,
                                         q1[-63:], O.SMOOTH_MEAN)
        # Lag-KV scores are trailing means of variances: strictly positive
        assert rel_err(gs[b, N - 2 * C:N - C], s1, POSITIVE) <= TOL, b
        assert rel_err(gs[b, N - C:], s2, POSITIVE) <= TOL, b
        ref = O.select_keep(gs[b, :N], 0, K, R)
        assert np.array_equal(kh[b], ref), b
        # the oracle's own float64 ranking, near-ties at the cut exempted
        s64 = np.concatenate([old[b], s1, s2])
        tie_exempt_compare(kh[b], O.select_keep(s64, 0, K, R), s64, 0, N, K,
                           R)
        assert rebuilt_rows_equal(pool, src_pt[b], dst, dst_pt[b], kh[b],
                                  page), b


def test_prefill_one_shot_full_size(E):
    import torch
    w = synth.workload("prefill_64k")
    print("prefill 65536 tokens one shot, K=8192", flush=True)
    g = synth.rng(w.seed)
    T, K, page, D = w.chunk, w.budget, w.page_size, w.hidden
    L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
    na, nb = len(w.band_a), len(w.band_b)
    a = synth.amplitudes(w, g, 0, T)                       # [n_band][T]
    # hidden states h = a * xi drawn on the device, rounded to bf16
    hid = torch.empty((w.n_band, 1, T, D), dtype=torch.bfloat16,
                      device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)
    a_dev = torch.from_numpy(a).cuda()
    for l in range(w.n_band):
        x = torch.empty((T, D), dtype=torch.float32, device="cuda")
        x.normal_(generator=gen)
        hid[l, 0] = (x * a_dev[l][:, None]).to(torch.bfloat16)
        del x
    src_pt, n_src = synth.page_tables(np.array([T]), page, g)
    dst_pt, n_dst = synth.contiguous_page_tables(np.array([K]), page)
    pool = torch.empty((L, 2, n_src, page, H * d), dtype=torch.int16,
                       device="cuda")
    pool.view(-1).random_(-32768, 32768, generator=gen)
    dstp = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                       device="cuda")
    cfg = E.default_cfg(batch=1, budget=K)
    st = [torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
          for _ in range(2)]
    E.epikv_state_init(cfg, st[0])
    scores = torch.zeros((1, T), device="cuda")
    keep = torch.zeros((1, K), dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(1, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws_n = E.workspace_bytes(cfg, T)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    hidv = hid.view(torch.int16)
    io = E.make_step_io(
        T, [hidv[l] for l in range(w.n_band)], D, T * D,
        dev(np.array([T], np.int32)), torch.zeros(1, dtype=torch.int32,
                                                  device="cuda"),
        E.pool_of(pool.view(L, 2, n_src, page, H, d)), dev(src_pt),
        src_pt.shape[1], E.pool_of(dstp.view(L, 2, n_dst, page, H, d)),
        dev(dst_pt), dst_pt.shape[1], scores, T, st[0], st[1], keep, n_keep,
        status, ws, ws_n)
    E.epikv_evict_step(cfg, io)
    _sync()
    assert host(status)[0] == 0 and host(n_keep)[0] == K
    gs = host(scores)[0]
    # every token's float64 score: Eq. 1 over each band layer's rows in
    # blocks (the last row of a block is the next block's predecessor), then
    # the trailing-window z-score of the whole stream and the band
    # combination
    blk = 4096
    sm = np.zeros((w.n_band, T))
    for l in range(w.n_band):
        gl = np.zeros(T)
        has = np.zeros(T, dtype=bool)
        before = None
        for lo in range(0, T, blk):
            rows = O.bf16_to_float64(host(hidv[l, 0, lo:lo + blk]))
            gl[lo:lo + blk], has[lo:lo + blk] = O.residual_delta(rows, before)
            before = rows[-1]
        sm[l] = O.smooth_stream(np.zeros(0), gl, has, O.SMOOTH_Z)
        print(f"  oracle band layer {l} done", flush=True)
    s64 = O.band_score(sm, na, nb)
    # band difference of z-scores: can sit at 0
    assert rel_err(gs, s64, NEAR_ZERO) <= TOL
    R = O.default_recent(K)
    ref = O.select_keep(gs, 0, K, R)
    kh = host(keep)[0]
    assert np.array_equal(kh, ref)
    swaps = tie_exempt_compare(kh, O.select_keep(s64, 0, K, R), s64, 0, T, K,
                               R)
    print(f"  prefill: {swaps} near-tie swaps against the float64 ranking",
          flush=True)
    assert rebuilt_rows_equal(pool, src_pt[0], dstp, dst_pt[0], kh, page)
