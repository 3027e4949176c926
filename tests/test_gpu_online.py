"""Online scoring: each token scored when it is generated (Sec. 3.3).

A decoder calls epikv_score + epikv_zscore with chunk = 1 after every token
and evicts with epikv_select + epikv_compact every E tokens.  The frozen
scores must not depend on how the stream was cut into calls: one token at a
time, 64 at a time and the whole stream at once give bit-identical scores
and carried state (the per-token arithmetic and the reduction orders do not
depend on the chunking), and all of them match the oracle.
"""
import numpy as np
import pytest

import oracle as O
import synth
from harness import NEAR_ZERO, TOL, dev, host, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def _score_stream(E, cfg, hid, chunks, fused=False, state0=None):
    """Score a [n_band][B][T][D] stream cut into the given chunk sizes, with
    epikv_score + epikv_zscore or (fused) epikv_score_tokens; returns
    (scores [B][T], final state bytes)."""
    import torch
    nb, B, T, D = hid.shape
    hd = dev(hid)
    st = [torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
          for _ in range(2)]
    if state0 is None:
        E.epikv_state_init(cfg, st[0])
    else:
        st[0].copy_(state0)
    scores = torch.zeros((B, T), device="cuda")
    t0 = 0
    for C in chunks:
        # rows t0..t0+C-1 of every sequence: [nb][B][T][D] with ld_seq = T*D
        hidden = [hd[l, :, t0:] for l in range(nb)]
        n_cached = dev(np.full(B, t0 + C, np.int32))
        if fused:
            E.epikv_score_tokens(cfg, C, hidden, D, T * D, n_cached, st[0],
                                 st[1], scores, T)
        else:
            sig = torch.zeros((nb, B, C), device="cuda")
            E.epikv_score(cfg, C, hidden, D, T * D, state_in=st[0],
                          state_out=st[1], sig=sig)
            E.epikv_zscore(cfg, C, sig, n_cached, st[0], st[1], scores, T)
        st = [st[1], st[0]]
        t0 += C
    assert t0 == T
    torch.cuda.synchronize()
    return host(scores), host(st[0])


@pytest.mark.parametrize("mode", ["z", "mean"])
def test_chunking_invariance_bitwise(E, mode):
    print(f"online chunking invariance {mode}", flush=True)
    g = synth.rng(900)
    B, T, D = 2, 256, 4096
    w = synth.workload("drift_replay", B=B)
    na, nb = len(w.band_a), len(w.band_b)
    hid = np.stack([np.stack([synth.hidden_rows(
        synth.amplitudes(w, g, 0, T)[l], D, g) for b in range(B)])
        for l in range(w.n_band)])                       # [nb][B][T][D]
    smode = E.SMOOTH_Z if mode == "z" else E.SMOOTH_MEAN
    cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb,
                        smoothing=smode)
    runs = {"token by token": [1] * T, "64 at a time": [64] * 4,
            "ragged": [1, 2, 61, 64, 100, 28], "one shot": [T]}
    out = {k: _score_stream(E, cfg, hid, c) for k, c in runs.items()}
    ref_s, ref_st = out["one shot"]
    for k, (s, st) in out.items():
        assert s.tobytes() == ref_s.tobytes(), k
        assert st.tobytes() == ref_st.tobytes(), k
    omode = O.SMOOTH_Z if mode == "z" else O.SMOOTH_MEAN
    for b in range(B):
        sm = []
        for l in range(w.n_band):
            gl, has = O.residual_delta(O.bf16_to_float64(hid[l, b]), None)
            sm.append(O.smooth_stream(np.zeros(0), gl, has, omode))
        s64 = O.band_score(np.array(sm), na, nb)
        assert rel_err(ref_s[b], s64, NEAR_ZERO) <= TOL


def test_ema_online_matches_one_shot(E):
    # the EMA scan's rounding depends on the tile boundaries, so chunkings
    # agree to fp32 accuracy rather than bitwise
    print("online EMA", flush=True)
    g = synth.rng(901)
    B, T, D = 2, 200, 1024
    w = synth.workload("drift_replay", B=B, hidden=D)
    na, nb = len(w.band_a), len(w.band_b)
    hid = np.stack([np.stack([synth.hidden_rows(
        synth.amplitudes(w, g, 0, T)[l], D, g) for b in range(B)])
        for l in range(w.n_band)])
    cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb,
                        smoothing=E.SMOOTH_EMA)
    s1, _ = _score_stream(E, cfg, hid, [1] * T)
    s2, _ = _score_stream(E, cfg, hid, [T])
    assert np.max(np.abs(s1 - s2) / np.maximum(1.0, np.abs(s2))) <= 1e-5
    for b in range(B):
        sm = []
        for l in range(w.n_band):
            gl, has = O.residual_delta(O.bf16_to_float64(hid[l, b]), None)
            sm.append(O.smooth_stream(np.zeros(0), gl, has, O.SMOOTH_EMA))
        s64 = O.band_score(np.array(sm), na, nb)
        assert rel_err(s1[b], s64, NEAR_ZERO) <= TOL


def _oracle_stream(hid, na, nb, mode, window):
    """Float64 frozen scores of every token of [n_band][B][T][D] streams
    scored from their start (Eq. 1, then the smoothing `mode` per band
    layer, then the band combination)."""
    omode = {"z": O.SMOOTH_Z, "mean": O.SMOOTH_MEAN, "raw": O.SMOOTH_RAW,
             "ema": O.SMOOTH_EMA}[mode]
    n_band, B, T, _ = hid.shape
    out = np.zeros((B, T))
    for b in range(B):
        sm = []
        for l in range(n_band):
            gl, has = O.residual_delta(O.bf16_to_float64(hid[l, b]), None)
            sm.append(O.smooth_stream(np.zeros(0), gl, has, omode, window))
        out[b] = O.band_score(np.array(sm), na, nb)
    return out


@pytest.mark.parametrize("mode", ["z", "mean", "raw", "ema"])
@pytest.mark.parametrize("D", [1000, 4096])
def test_score_tokens_equals_two_calls(E, mode, D):
    """epikv_score_tokens (one launch per call) against epikv_score +
    epikv_zscore on the same chunking: scores and carried state bitwise,
    from a fresh stream and from a carried state (window 64 and 5); and its
    scores against the oracle's float64 scores of the same stream (Sec. 3.3:
    a token's score is frozen when it is generated, so scoring a stream
    call by call must give the scores of the whole stream)."""
    import torch
    print(f"fused per-token scoring {mode} D={D}", flush=True)
    g = synth.rng(903 + D)
    B, T = 3, 150
    w = synth.workload("drift_replay", B=B, hidden=D)
    na, nb = len(w.band_a), len(w.band_b)
    hid = np.stack([np.stack([synth.hidden_rows(
        synth.amplitudes(w, g, 0, T)[l], D, g) for b in range(B)])
        for l in range(w.n_band)])
    smode = {"z": E.SMOOTH_Z, "mean": E.SMOOTH_MEAN, "raw": E.SMOOTH_RAW,
             "ema": E.SMOOTH_EMA}[mode]
    for window in (64, 5):
        cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb,
                            smoothing=smode, window=window)
        ref = _oracle_stream(hid, na, nb, mode, window)
        # a carried state: the stream's first 40 tokens scored beforehand
        _, st40 = _score_stream(E, cfg, hid[:, :, :40], [40])
        for chunks in ([1] * 12 + [7, 64, 1, 2, 64], [64, 64, 22]):
            a = _score_stream(E, cfg, hid, chunks)
            f = _score_stream(E, cfg, hid, chunks, fused=True)
            assert a[0].tobytes() == f[0].tobytes(), (window, chunks)
            assert a[1].tobytes() == f[1].tobytes(), (window, chunks)
            # band differences: can sit at 0
            assert rel_err(f[0], ref, NEAR_ZERO) <= TOL, (window, chunks)
        rest = hid[:, :, 40:]
        a = _score_stream(E, cfg, rest, [1] * 20 + [30, 60],
                          state0=torch.from_numpy(st40).cuda())
        f = _score_stream(E, cfg, rest, [1] * 20 + [30, 60], fused=True,
                          state0=torch.from_numpy(st40).cuda())
        assert a[0].tobytes() == f[0].tobytes()
        assert a[1].tobytes() == f[1].tobytes()
        # resumed from the carried state (ring, h_prev, EMA average): the
        # scores of tokens 40.. of the uninterrupted stream
        assert rel_err(f[0], ref[:, 40:], NEAR_ZERO) <= TOL, window


def test_state_checkpoint_and_resume(E):
    """Checkpoint = a copy of the state buffer to the host.  Scoring a stream
    in two halves, with the state saved after the first and restored into a
    fresh device buffer, gives the scores and final state of the
    uninterrupted run bit for bit."""
    import torch
    print("state checkpoint / resume", flush=True)
    g = synth.rng(904)
    B, T, D = 2, 200, 1024
    w = synth.workload("drift_replay", B=B, hidden=D)
    na, nb = len(w.band_a), len(w.band_b)
    hid = np.stack([np.stack([synth.hidden_rows(
        synth.amplitudes(w, g, 0, T)[l], D, g) for b in range(B)])
        for l in range(w.n_band)])
    cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb)
    chunks = [16] * 12 + [8]
    full_s, full_st = _score_stream(E, cfg, hid, chunks)
    split = 7 * 16
    s1, st1 = _score_stream(E, cfg, hid[:, :, :split], [16] * 7)
    saved = np.array(st1, copy=True)              # the checkpoint (host bytes)
    s2, st2 = _score_stream(E, cfg, hid[:, :, split:], [16] * 5 + [8],
                            state0=torch.from_numpy(saved).cuda())
    assert st2.tobytes() == full_st.tobytes()
    assert s1.tobytes() == full_s[:, :split].tobytes()
    assert s2.tobytes() == full_s[:, split:].tobytes()


def test_online_step_equals_the_scoring_step(E):
    """The online regime end to end: the C new tokens scored one call each
    with epikv_score_tokens, then epikv_evict_step with chunk 0 (select and
    rebuild only), give bit for bit the scores, kept sets, rebuilt cache and
    scorer state of one epikv_evict_step that scores the same C tokens."""
    import torch
    print("online step vs scoring step", flush=True)
    g = synth.rng(910)
    B, C, K, page, L, H, d, D = 3, 16, 96, 16, 2, 8, 128, 256
    na, nb = 2, 2
    lengths = np.array([400, 150, 90])           # include the C new tokens
    ld_s = int(lengths.max())
    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_band_a=na,
                        n_band_b=nb, budget=K)
    hid = dev(synth.f32_to_bf16_bits(
        (g.standard_normal((na + nb, B, C, D)) * 2).astype(np.float32)))
    sc0 = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc0[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    st = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st)
    sec["n_tok"][:] = torch.from_numpy((lengths - C + 30).astype(np.int32))
    sec["ring"][:] = torch.from_numpy(
        (20 + g.standard_normal(tuple(sec["ring"].shape))).astype(np.float32))
    sec["h_prev"][:] = torch.from_numpy(synth.f32_to_bf16_bits(
        g.standard_normal(tuple(sec["h_prev"].shape)).astype(np.float32)
    ).view(np.int16))
    st0 = st.cuda()
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g)
    src = dev(synth.random_bits16(g, (L, 2, n_src, page, H * d)))
    S = E.pool_of(src.view(L, 2, n_src, page, H, d))
    n_cached = dev(lengths.astype(np.int32))
    n_prefix = dev(np.zeros(B, np.int32))
    hidden = [hid[l] for l in range(na + nb)]

    def run(online):
        scores = dev(sc0)
        dst = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                          device="cuda")
        dsc = torch.full((B, ld_s), -7.0, device="cuda")
        keep = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
        nk = torch.zeros(B, dtype=torch.int32, device="cuda")
        status = torch.zeros(B, dtype=torch.int32, device="cuda")
        s_in, s_out = st0.clone(), torch.zeros_like(st0)
        chunk = C
        if online:
            for t in range(C):
                E.epikv_score_tokens(
                    cfg, 1, [h[:, t:] for h in hidden], D, C * D,
                    dev((lengths - C + t + 1).astype(np.int32)), s_in, s_out,
                    scores, ld_s)
                s_in, s_out = s_out, s_in
            chunk, state = 0, s_in
        ws_n = E.workspace_bytes(cfg, chunk)
        ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
        io = E.make_step_io(
            chunk, None if online else hidden, D, C * D, n_cached, n_prefix,
            S, dev(src_pt), src_pt.shape[1],
            E.pool_of(dst.view(L, 2, n_dst, page, H, d)), dev(dst_pt),
            dst_pt.shape[1], scores, ld_s, None if online else s_in,
            None if online else s_out, keep, nk, status, ws, ws_n,
            dst_scores=dsc)
        E.epikv_evict_step(cfg, io)
        if not online:
            state = s_out
        torch.cuda.synchronize()
        return [host(t).copy() for t in (scores, dst, dsc, keep, nk, status,
                                         state)]

    a = run(online=False)
    b = run(online=True)
    assert np.all(a[5] == 0) and np.all(a[4] == np.minimum(lengths, K))
    for x, y, what in zip(a, b, ["scores", "cache", "compacted scores",
                                 "keep_idx", "n_keep", "status", "state"]):
        assert x.tobytes() == y.tobytes(), what


def _random_online_cases(n, seed=20261207):
    g = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        T = int(g.integers(1, 200))
        cuts = []
        left = T
        while left:
            c = int(min(left, g.choice([1, 1, 2, 3, 17, 63, 64])))
            cuts.append(c)
            left -= c
        out.append(dict(B=int(g.integers(1, 6)),
                        D=int(g.choice([8, 64, 1000, 2048, 4096])),
                        window=int(g.choice([1, 2, 5, 64, 128])),
                        mode=str(g.choice(["z", "mean", "raw", "ema"])),
                        na=int(g.integers(1, 9)), nb=int(g.integers(0, 9)),
                        chunks=cuts, seed=int(g.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _random_online_cases(12),
                         ids=lambda c: f"{c['mode']}-D{c['D']}-w{c['window']}")
def test_score_tokens_random(E, case):
    """Seeded mixes of batch, hidden width, window, smoothing, band sizes and
    a random cut of the stream into calls of 1..64 tokens: the fused scorer
    bitwise equal to the two separate calls, and both equal to the oracle's
    float64 scores of the whole stream."""
    print(f"fused per-token scoring, random: {case}", flush=True)
    g = np.random.default_rng(case["seed"])
    B, D, T = case["B"], case["D"], sum(case["chunks"])
    na, nb = case["na"], case["nb"]
    scale = np.exp(g.normal(0.0, 0.5, size=(na + nb, 1, T, 1)))
    hid = synth.f32_to_bf16_bits(
        (g.standard_normal((na + nb, B, T, D)) * scale).astype(np.float32))
    smode = {"z": E.SMOOTH_Z, "mean": E.SMOOTH_MEAN, "raw": E.SMOOTH_RAW,
             "ema": E.SMOOTH_EMA}[case["mode"]]
    cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb,
                        smoothing=smode, window=case["window"])
    assert E.check_cfg(cfg) == 0
    a = _score_stream(E, cfg, hid, case["chunks"])
    f = _score_stream(E, cfg, hid, case["chunks"], fused=True)
    assert a[0].tobytes() == f[0].tobytes()
    assert a[1].tobytes() == f[1].tobytes()
    ref = _oracle_stream(hid, na, nb, case["mode"], case["window"])
    tol = TOL if case["mode"] != "ema" else 1e-3
    assert rel_err(f[0], ref, NEAR_ZERO) <= tol
