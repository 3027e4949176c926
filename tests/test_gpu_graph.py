"""epikv_evict_step under HIP graph capture.

The step enqueues only kernels (no memset, no allocation, no host
synchronisation), so a caller can capture it once and replay it.  Every
replay -- with unrelated eager work and synchronisations between replays --
must reproduce the eager step bit for bit.
"""
import numpy as np
import pytest

import synth
from harness import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


@pytest.mark.parametrize("signal", ["hs", "lagkv"])
def test_graph_replays_match_eager(E, signal):
    import torch
    print(f"graph capture {signal}", flush=True)
    g = synth.rng(800)
    B, C, K, page, L, H, d, D = 3, 64, 256, 16, 4, 8, 128, 512
    na, nb = 2, 2
    lengths = np.array([700, 300, 200])
    ld_s = int(lengths.max())
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g)
    pool = synth.random_bits16(g, (L, 2, n_src, page, H * d))
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    if signal == "hs":
        cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_band_a=na,
                            n_band_b=nb, budget=K)
        hid = dev(synth.f32_to_bf16_bits(
            g.standard_normal((na + nb, B, C, D)).astype(np.float32)))
        hidden = [hid[l] for l in range(na + nb)]
    else:
        cfg = E.default_cfg(batch=B, n_layers=L, signal=E.SIGNAL_LAGKV,
                            smoothing=E.SMOOTH_MEAN, budget=K)
        hidden = None
    st_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
    E.epikv_state_init(cfg, st_in)
    torch.cuda.synchronize()
    sec = E.state_sections(cfg, st_in)
    sec["n_tok"][:] = torch.from_numpy((lengths - C).astype(np.int32)).cuda()
    sec["ring"][:] = torch.from_numpy(
        (5.0 + g.standard_normal(tuple(sec["ring"].shape))).astype(
            np.float32)).cuda()
    st_out = torch.zeros_like(st_in)
    src = dev(pool)
    dst = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                      device="cuda")
    scores = dev(sc)
    dsc = torch.zeros_like(scores)
    keep = torch.zeros((B, K), dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    ws_n = E.workspace_bytes(cfg, C)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    io = E.make_step_io(
        C, hidden, D, C * D, dev(lengths.astype(np.int32)),
        torch.zeros(B, dtype=torch.int32, device="cuda"),
        E.pool_of(src.view(L, 2, n_src, page, H, d)), dev(src_pt),
        src_pt.shape[1], E.pool_of(dst.view(L, 2, n_dst, page, H, d)),
        dev(dst_pt), dst_pt.shape[1], scores, ld_s, st_in, st_out, keep,
        n_keep, status, ws, ws_n, dst_scores=dsc)
    outs = (scores, dsc, keep, n_keep, status, st_out, dst)

    def snapshot():
        torch.cuda.synchronize()
        return [host(t).copy() for t in outs]

    def clobber():
        for t in outs:
            t.view(torch.uint8).fill_(0x5B)

    # every run starts from the same bytes in the outputs (the step leaves
    # slots past n_keep and the state's padding untouched)
    clobber()
    scores.copy_(dev(sc))
    E.epikv_evict_step(cfg, io)
    eager = snapshot()
    # capture on a side stream (warm it up first, as graph capture requires)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        E.epikv_evict_step(cfg, io)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        E.epikv_evict_step(cfg, io)
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        clobber()
        # the scores of the older tokens are inputs: restore them
        scores.copy_(dev(sc))
        graph.replay()
        got = snapshot()
        for a, b in zip(got, eager):
            assert a.tobytes() == b.tobytes(), rep    # bytewise: NaN-safe
        junk = junk * 1.0001 + 1.0              # unrelated eager work
        torch.cuda.synchronize()


@pytest.mark.parametrize("mode", ["in_place", "remap"])
def test_graph_in_place_step_and_token_scorer(E, mode):
    """The in-place step (plain, or with page remapping) and the fused
    per-token scorer under capture: each replay starts from the same inputs
    (the pool, page table, scores and positions the in-place step rewrites
    are restored first) and must match eager."""
    import torch
    print(f"graph capture in place ({mode}) + score_tokens", flush=True)
    g = synth.rng(801)
    B, C, K, page, L, H, d, D = 3, 16, 96, 16, 2, 8, 128, 256
    na, nb = 2, 2
    lengths = np.array([400, 150, 90])
    ld_s = int(lengths.max())
    pt, n_pages = synth.page_tables(lengths, page, g)
    pool0 = dev(synth.random_bits16(g, (L, 2, n_pages, page, H * d)))
    sc0 = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc0[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    sc0 = dev(sc0)
    pos0 = dev(np.tile(np.arange(ld_s, dtype=np.int32), (B, 1)))
    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_band_a=na,
                        n_band_b=nb, budget=K)
    hid = dev(synth.f32_to_bf16_bits(
        g.standard_normal((na + nb, B, C, D)).astype(np.float32)))
    hidden = [hid[l] for l in range(na + nb)]
    st_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
    E.epikv_state_init(cfg, st_in)
    torch.cuda.synchronize()
    sec = E.state_sections(cfg, st_in)
    sec["n_tok"][:] = torch.from_numpy((lengths - C).astype(np.int32)).cuda()
    st_out = torch.zeros_like(st_in)
    st_tok = torch.zeros_like(st_in)
    pool, scores, pos = pool0.clone(), sc0.clone(), pos0.clone()
    tok_scores = torch.zeros_like(scores)
    keep = torch.zeros((B, K), dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    ws_n = E.workspace_bytes(cfg, C)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    n_cached = dev(lengths.astype(np.int32))
    pt0 = dev(pt)
    pt_d = pt0.clone()
    io = E.make_step_io(
        C, hidden, D, C * D, n_cached,
        torch.zeros(B, dtype=torch.int32, device="cuda"),
        E.pool_of(pool.view(L, 2, n_pages, page, H, d)), pt_d, pt.shape[1],
        E.Pool(), None, 0, scores, ld_s, st_in, st_out, keep, n_keep, status,
        ws, ws_n, src_pos=pos, dst_pos=pos,
        in_place=E.COMPACT_IN_PLACE if mode == "in_place" else E.COMPACT_REMAP)

    def work():
        E.epikv_evict_step(cfg, io)
        E.epikv_score_tokens(cfg, C, hidden, D, C * D, n_cached, st_in,
                             st_tok, tok_scores, ld_s)

    outs = (pool, scores, pos, keep, n_keep, status, st_out, st_tok,
            tok_scores, pt_d)

    def reset():
        for t in outs:
            t.view(torch.uint8).fill_(0x5B)
        pool.copy_(pool0)
        scores.copy_(sc0)
        pos.copy_(pos0)
        pt_d.copy_(pt0)

    def snapshot():
        torch.cuda.synchronize()
        return [host(t).copy() for t in outs]

    reset()
    work()
    eager = snapshot()
    assert np.all(eager[5] == 0)
    if mode == "remap":                  # the table changed
        assert not np.array_equal(eager[9], pt)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        reset()
        work()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        work()
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        reset()
        graph.replay()
        got = snapshot()
        for a, b in zip(got, eager):
            assert a.tobytes() == b.tobytes(), rep
        junk = junk * 1.0001 + 1.0
        torch.cuda.synchronize()


def _small_step(E, seed, B=3, C=16, K=96, L=2, H=8, d=128, D=256, page=16):
    """Inputs and output buffers of one small eviction step (HS signal)."""
    import torch
    g = synth.rng(seed)
    na, nb = 2, 2
    lengths = np.array([400, 150, 200][:B])
    ld_s = int(lengths.max())
    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_band_a=na,
                        n_band_b=nb, budget=K)
    hid = dev(synth.f32_to_bf16_bits(
        (g.standard_normal((na + nb, B, C, D)) * 2).astype(np.float32)))
    sc0 = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc0[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    st_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
    E.epikv_state_init(cfg, st_in)
    torch.cuda.synchronize()
    sec = E.state_sections(cfg, st_in)
    sec["n_tok"][:] = torch.from_numpy((lengths - C).astype(np.int32)).cuda()
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g)
    src = dev(synth.random_bits16(g, (L, 2, n_src, page, H * d)))
    out = dict(
        scores=dev(sc0), dst=torch.zeros((L, 2, n_dst, page, H * d),
                                         dtype=torch.int16, device="cuda"),
        st_out=torch.zeros_like(st_in),
        keep=torch.zeros((B, K), dtype=torch.int32, device="cuda"),
        nk=torch.zeros(B, dtype=torch.int32, device="cuda"),
        status=torch.zeros(B, dtype=torch.int32, device="cuda"))
    ws_n = E.workspace_bytes(cfg, C)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    io = E.make_step_io(
        C, [hid[l] for l in range(na + nb)], D, C * D,
        dev(lengths.astype(np.int32)), dev(np.zeros(B, np.int32)),
        E.pool_of(src.view(L, 2, n_src, page, H, d)), dev(src_pt),
        src_pt.shape[1], E.pool_of(out["dst"].view(L, 2, n_dst, page, H, d)),
        dev(dst_pt), dst_pt.shape[1], out["scores"], ld_s, st_in,
        out["st_out"], out["keep"], out["nk"], out["status"], ws, ws_n)
    io._keep_src = (src, hid, sc0)
    return cfg, io, out, sc0


def test_two_steps_on_two_streams_at_once(E):
    """The library keeps no global state: two eviction steps with their own
    buffers, enqueued on two streams without any synchronisation between
    them, give bit for bit what each gives alone."""
    import torch
    print("two streams", flush=True)
    runs = [_small_step(E, 1201), _small_step(E, 1202)]

    def reset():
        for cfg, io, out, sc0 in runs:
            for k, t in out.items():
                if k == "scores":
                    t.copy_(torch.from_numpy(sc0).cuda())
                else:
                    t.zero_()
        torch.cuda.synchronize()

    def snap():
        torch.cuda.synchronize()
        return [[host(t).copy() for t in out.values()] for _, _, out, _ in runs]

    reset()
    for cfg, io, _, _ in runs:               # one after the other
        E.epikv_evict_step(cfg, io)
    alone = snap()
    assert all(np.all(a[5] == 0) for a in alone)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        reset()
        for (cfg, io, _, _), s in zip(runs, streams):
            with torch.cuda.stream(s):
                E.epikv_evict_step(cfg, io)
        got = snap()
        for a, b in zip(got, alone):
            for x, y in zip(a, b):
                assert x.tobytes() == y.tobytes(), rep
