"""Kernel-level parity of the HIP path against the CPU oracle.

Each stage is fed the same seeded inputs as the oracle (for select and
compact: the oracle's own scores and indices) and compared element by
element: g, z and scores within 1e-3 relative (the tolerance of the
eviction-step target), indices and copied bytes exactly.
"""
import numpy as np
import pytest

import oracle as O
import synth
from harness import (NEAR_ZERO, POSITIVE, TOL, dev, gather_logical, host,
                     rel_err)

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


# ---------------------------------------------------------------------------
# score (HS): Eq. 1
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("D,C,fresh,pad", [
    (4096, 100, False, 0), (4096, 100, True, 0), (4096, 1, False, 0),
    (1000, 33, True, 0), (8192, 40, False, 64), (16384, 5, False, 0),
    (4096, 64, False, 128)])
def test_score_hs_matches_oracle(E, D, C, fresh, pad):
    import torch
    print(f"score_hs D={D} C={C} fresh={fresh} pad={pad}", flush=True)
    g = synth.rng(100 + D + C)
    B, na, nb = 3, 2, 2
    nband = na + nb
    ld_tok = D + pad
    hid = np.zeros((nband, B, C, ld_tok), dtype=np.uint16)
    hid[..., :D] = synth.f32_to_bf16_bits(
        g.standard_normal((nband, B, C, D)).astype(np.float32)
        * (1 + np.arange(C, dtype=np.float32)[None, None, :, None] % 3))
    before = synth.f32_to_bf16_bits(
        g.standard_normal((B, nband, D)).astype(np.float32))
    if C > 2:
        hid[1, 2, 2, :D] = hid[1, 2, 1, :D]      # an exact zero change
    cfg = E.default_cfg(batch=B, hidden=D, n_band_a=na, n_band_b=nb)
    st_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st_in)
    sec["n_tok"][:] = 0 if fresh else 500
    sec["h_prev"][:] = torch.from_numpy(before.view(np.int16))
    st_in = st_in.cuda()
    st_out = torch.zeros_like(st_in)
    hd = dev(hid)
    hidden = [hd[l] for l in range(nband)]
    sig = torch.full((nband, B, C), -7.0, device="cuda")
    E.epikv_score(cfg, C, hidden, ld_tok, C * ld_tok, state_in=st_in,
                  state_out=st_out, sig=sig)
    _sync()
    got = host(sig)
    for l in range(nband):
        for b in range(B):
            hb = None if fresh else O.bf16_to_float64(before[b, l])
            ref, has = O.residual_delta(O.bf16_to_float64(hid[l, b, :, :D]),
                                        hb)
            assert rel_err(got[l, b], ref, POSITIVE) <= TOL, (l, b)
            assert np.all(got[l, b][~has] == 0.0)
    out = E.state_sections(cfg, st_out.cpu())
    assert np.array_equal(out["h_prev"].numpy().view(np.uint16),
                          hid[:, :, C - 1, :D].transpose(1, 0, 2))


# ---------------------------------------------------------------------------
# zscore: Eqs. 2-3 and the band combination
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["z", "mean", "raw", "ema"])
@pytest.mark.parametrize("C", [1, 7, 600])
def test_zscore_matches_oracle(E, mode, C):
    import torch
    print(f"zscore mode={mode} C={C}", flush=True)
    g = synth.rng(200 + C)
    B, na, nb, w = 4, 3, 2, 64
    nsig = na + nb
    smode = {"z": E.SMOOTH_Z, "mean": E.SMOOTH_MEAN, "raw": E.SMOOTH_RAW,
             "ema": E.SMOOTH_EMA}[mode]
    omode = {"z": O.SMOOTH_Z, "mean": O.SMOOTH_MEAN, "raw": O.SMOOTH_RAW,
             "ema": O.SMOOTH_EMA}[mode]
    cfg = E.default_cfg(batch=B, n_band_a=na, n_band_b=nb, smoothing=smode)
    n_tok = np.array([0, 10, 1000, 64], dtype=np.int32)
    # signal at the level of a 4096-wide hidden-state change: mean ~90x the
    # spread, the regime where one-pass variance would lose digits
    sig = (90.0 + g.standard_normal((nsig, B, C))).astype(np.float32)
    ring = np.zeros((B, nsig, w - 1), dtype=np.float32)
    priors = []
    for b in range(B):
        cnt = min(w - 1, max(int(n_tok[b]) - 1, 0))
        pb = (90.0 + g.standard_normal((nsig, cnt))).astype(np.float32)
        if cnt:
            ring[b, :, w - 1 - cnt:] = pb
        priors.append(pb)
    ld_s = 2000
    n_cached = np.array([C, C + 5, 1500, ld_s], dtype=np.int32)
    # carried running averages (EMA): any value for streams with a sample
    ema_in = (90.0 + g.standard_normal((B, nsig))).astype(np.float32)
    ema_in[0] = 0.0                       # fresh stream: nothing carried
    st_in = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st_in)
    sec["n_tok"][:] = torch.from_numpy(n_tok)
    sec["ring"][:] = torch.from_numpy(ring)
    sec["ema"][:] = torch.from_numpy(ema_in)
    st_in = st_in.cuda()
    st_out = torch.zeros_like(st_in)
    scores = torch.full((B, ld_s), 123.0, device="cuda")
    sm = torch.zeros((nsig, B, C), device="cuda")
    E.epikv_zscore(cfg, C, dev(sig), dev(n_cached), st_in, st_out, scores,
                   ld_s, smoothed=sm)
    _sync()
    got_s = host(scores)
    got_sm = host(sm)
    out = E.state_sections(cfg, st_out.cpu())
    worst = 0.0
    for b in range(B):
        has = np.ones(C, dtype=bool)
        if n_tok[b] == 0:
            has[0] = False
        rows = []
        prior_samples = max(int(n_tok[b]) - 1, 0)
        for l in range(nsig):
            eb = float(ema_in[b, l]) if prior_samples > 0 else None
            r = O.smooth_stream(priors[b][l], sig[l, b], has, omode, w, 1e-6,
                                ema_before=eb)
            rows.append(r)
            # a z-score can sit at 0; the signal and its mean, raw and
            # EMA smoothing are ~90
            row_floor = NEAR_ZERO if mode == "z" else POSITIVE
            worst = max(worst, rel_err(got_sm[l, b], r, row_floor))
            # carried window: the last min(w-1, samples) samples
            seq = np.concatenate([priors[b][l], sig[l, b][has]])
            k = min(w - 1, seq.size)
            exp = np.zeros(w - 1, dtype=np.float32)
            if k:
                exp[w - 1 - k:] = seq[-k:]
            assert np.array_equal(out["ring"][b, l].numpy(), exp), (b, l)
        s_ref = O.band_score(np.array(rows), na, nb)
        N = n_cached[b]
        # band difference: can sit at 0 in every mode
        worst = max(worst, rel_err(got_s[b, N - C:N], s_ref, NEAR_ZERO))
        # nothing outside the chunk's slots is written
        assert np.all(got_s[b, :N - C] == 123.0)
        assert np.all(got_s[b, N:] == 123.0)
        if mode == "ema":
            # the carried average after the chunk
            seq_y = O.smooth_stream(priors[b][0], sig[0, b], has, omode,
                                    ema_before=float(ema_in[b, 0])
                                    if prior_samples > 0 else None)
            last = seq_y[has][-1] if has.any() else (
                ema_in[b, 0] if prior_samples > 0 else None)
            if last is not None:
                assert rel_err([float(out["ema"][b, 0])], [last]) <= TOL
        else:
            assert np.array_equal(out["ema"][b].numpy(), ema_in[b])
    assert worst <= TOL, worst
    assert np.array_equal(out["n_tok"].numpy(), n_tok + C)


# ---------------------------------------------------------------------------
# select: Sec. 3.1, Sec. 3.3, App. D
# ---------------------------------------------------------------------------
def _select(E, entry, cfg, scores, ld_s, n_cached, n_prefix, keep, n_keep,
            status):
    """epikv_select, or epikv_select_ws (one sequence split over several
    workgroups when the batch is small) with a workspace of garbage."""
    import torch
    if entry == "select":
        E.epikv_select(cfg, scores, ld_s, n_cached, n_prefix, keep, n_keep,
                       status)
        return
    n = E.select_workspace_bytes(cfg)
    ws = torch.randint(-2**31, 2**31 - 1, (max(n, 16) // 4,),
                       dtype=torch.int32, device="cuda")
    E.epikv_select_ws(cfg, scores, ld_s, n_cached, n_prefix, keep, n_keep,
                      status, ws, n)


@pytest.mark.parametrize("entry", ["select", "select_ws"])
@pytest.mark.parametrize("ld_s", [65536, 80000, 3000])
def test_select_matches_oracle_bit_exact(E, ld_s, entry):
    import torch
    print(f"{entry} ld_s={ld_s}", flush=True)
    g = synth.rng(300 + ld_s)
    K = 1024
    # ld_s picks the kernel variant: keys in registers (<= 64 Ki positions)
    # or re-read from memory in every sweep (longer rows)
    Ns = [0, 37, 1024, 1025, 1500, 5000, 32768, 65536, 70000, 4000, 2048,
          ld_s, ld_s + 1, 2049]
    Ps = [0, 0, 3, 0, 17, 100, 0, 64, 0, 1000, 896, 5, 0, 0]
    B = len(Ns)
    sc = np.zeros((B, ld_s), dtype=np.float32)
    for b in range(B):
        s = synth.old_scores(g, ld_s, ties=(b % 2 == 0))
        s[g.integers(0, ld_s, 20)] = np.nan
        s[g.integers(0, ld_s, 20)] = -0.0
        s[g.integers(0, ld_s, 20)] = 0.0
        s[g.integers(0, ld_s, 5)] = -np.inf
        sc[b] = s
    cfg = E.default_cfg(batch=B, budget=K)
    keep = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.full((B,), 9, dtype=torch.int32, device="cuda")
    _select(E, entry, cfg, dev(sc), ld_s, dev(np.array(Ns, np.int32)),
            dev(np.array(Ps, np.int32)), keep, n_keep, status)
    _sync()
    keep, n_keep, status = host(keep), host(n_keep), host(status)
    R = O.default_recent(K)
    for b in range(B):
        N, P = Ns[b], Ps[b]
        if N > ld_s:
            assert status[b] == E.SEQ_RANGE and n_keep[b] == -1
            continue
        ref = O.select_keep(sc[b, :N], P, K, R)
        if isinstance(ref, str):
            assert status[b] == E.SEQ_BUDGET and n_keep[b] == -1, b
            continue
        assert status[b] == E.SEQ_OK, b
        assert n_keep[b] == ref.size, b
        assert np.array_equal(keep[b, :ref.size], ref), b
        assert np.all(keep[b, ref.size:] == -5)


@pytest.mark.parametrize("entry", ["select", "select_ws"])
@pytest.mark.parametrize("N", [3000, 65536])
def test_select_all_equal_scores_keeps_lowest_positions(E, N, entry):
    # every eligible key ties: the kept ones are the lowest positions, also
    # when the positions are split over several workgroups
    import torch
    B, K = 2, 256
    sc = np.zeros((B, N), dtype=np.float32)
    sc[1] = np.nan
    cfg = E.default_cfg(batch=B, budget=K)
    keep = torch.zeros((B, K), dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    st = torch.full((B,), 9, dtype=torch.int32, device="cuda")
    _select(E, entry, cfg, dev(sc), N, dev(np.full(B, N, np.int32)),
            dev(np.zeros(B, np.int32)), keep, n_keep, st)
    _sync()
    R = 64
    exp = np.concatenate([np.arange(K - R), np.arange(N - R, N)])
    assert np.array_equal(host(st), [E.SEQ_OK] * B)
    assert np.array_equal(host(n_keep), [K] * B)
    for b in range(B):
        assert np.array_equal(host(keep)[b], exp)


@pytest.mark.parametrize("B,ld_s,K", [(1, 65536, 8192), (1, 3000, 1024),
                                      (32, 32896, 4096), (4, 80000, 8192),
                                      (1, 70000, 300), (128, 2048, 256)])
def test_select_split_matches_oracle_bit_exact(E, B, ld_s, K):
    """epikv_select_ws at the batch shapes that split a sequence: a single
    long prefill (64 workgroups of one key per thread), the decode batch of
    32 ragged sequences (5 workgroups of 8), a ragged tail, slices past N,
    and the biggest batch that still splits."""
    import torch
    print(f"select_ws B={B} ld_s={ld_s} K={K}", flush=True)
    g = synth.rng(900 + B + ld_s + K)
    Ns = g.integers(max(K + 1, ld_s // 4), ld_s + 1, B)
    Ns[0] = ld_s
    if B > 2:
        Ns[1] = K          # keep all
        Ns[2] = ld_s // 3  # short row: trailing workgroups see no position
    Ps = g.integers(0, max(1, K // 8), B)
    sc = np.zeros((B, ld_s), dtype=np.float32)
    for b in range(B):
        s = synth.old_scores(g, ld_s, ties=(b % 2 == 0))
        s[g.integers(0, ld_s, 20)] = np.nan
        s[g.integers(0, ld_s, 20)] = -0.0
        s[g.integers(0, ld_s, 5)] = -np.inf
        sc[b] = s
    cfg = E.default_cfg(batch=B, budget=K)
    keep = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.full((B,), 9, dtype=torch.int32, device="cuda")
    d_sc, d_n, d_p = (dev(sc), dev(Ns.astype(np.int32)),
                      dev(Ps.astype(np.int32)))
    _select(E, "select_ws", cfg, d_sc, ld_s, d_n, d_p, keep, n_keep, status)
    _sync()
    # a second call on the same (now dirty) workspace gives the same result
    keep2 = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
    n2 = torch.zeros(B, dtype=torch.int32, device="cuda")
    st2 = torch.full((B,), 9, dtype=torch.int32, device="cuda")
    n = E.select_workspace_bytes(cfg)
    ws = torch.empty(n // 4, dtype=torch.int32, device="cuda")
    for kk, nn, ss in ((keep, n_keep, status), (keep2, n2, st2)):
        kk.fill_(-5)
        E.epikv_select_ws(cfg, d_sc, ld_s, d_n, d_p, kk, nn, ss, ws, n)
    _sync()
    assert torch.equal(keep, keep2) and torch.equal(n_keep, n2) \
        and torch.equal(status, st2)
    R = O.default_recent(K)

    def check(keep, n_keep, status, sc, Ns, Ps):
        keep, n_keep, status = host(keep), host(n_keep), host(status)
        for b in range(B):
            ref = O.select_keep(sc[b, :Ns[b]], int(Ps[b]), K, R)
            assert status[b] == E.SEQ_OK, b
            assert n_keep[b] == ref.size, b
            assert np.array_equal(keep[b, :ref.size], ref), b
            assert np.all(keep[b, ref.size:] == -5)

    check(keep, n_keep, status, sc, Ns, Ps)
    # The workspace carries the cleared scratch from call to call: further
    # calls on it with other scores, lengths and prefixes, and with a
    # shorter row (a different split), are exact too.
    for rep in range(3):
        ld2 = ld_s if rep < 2 else max(K + 1, ld_s // 2)
        sc2 = np.stack([synth.old_scores(g, ld2, ties=(rep == 1))
                        for _ in range(B)])
        Ns2 = g.integers(min(ld2, K + 1), ld2 + 1, B)
        Ps2 = g.integers(0, max(1, K // 8), B)
        kk = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
        E.epikv_select_ws(cfg, dev(sc2), ld2, dev(Ns2.astype(np.int32)),
                          dev(Ps2.astype(np.int32)), kk, n2, st2, ws, n)
        _sync()
        check(kk, n2, st2, sc2, Ns2, Ps2)


# ---------------------------------------------------------------------------
# compact: App. H
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dst_layout", ["scattered", "ascending"])
@pytest.mark.parametrize("page", [16, 8])
def test_compact_matches_oracle_bytes(E, page, dst_layout):
    """Scattered destination pages are written in page-id order through a
    bitmap rank; ascending ones (runs of pages, sequences in order, with
    unused pages of short and refused sequences among them) through the
    prefix counts.  Either order gives the same bytes."""
    import torch
    print(f"compact page={page} dst={dst_layout}", flush=True)
    g = synth.rng(400 + page)
    L, H, d, K = 4, 8, 128, 256
    Ns = np.array([37, 300, 1000, 777, 256], dtype=np.int64)
    Ps = np.array([0, 5, 0, 300, 0])
    B = Ns.size
    src_pt, n_src = synth.page_tables(Ns, page, g, n_pages_total=None)
    n_src += 7
    pool = synth.random_bits16(g, (L, 2, n_src, page, H * d))
    pool[0, 0, src_pt[1, 0], 3, 5] = 0x7FC1          # NaN payload
    dpp = (K + page - 1) // page
    if dst_layout == "scattered":
        dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g,
                                          n_pages_total=B * dpp + 3)
    else:
        dst_pt, n_dst = synth.contiguous_page_tables(np.full(B, K), page,
                                                     first=2)
        n_dst += 3
    SENT = 0x5A5A
    ld_s = int(Ns.max())
    sc = np.zeros((B, ld_s), dtype=np.float32)
    pos = np.full((B, ld_s), -1, dtype=np.int32)
    keep = np.full((B, K), -1, dtype=np.int32)
    n_keep = np.zeros(B, dtype=np.int32)
    for b in range(B):
        sc[b, :Ns[b]] = synth.old_scores(g, int(Ns[b]), ties=True)
        pos[b, :Ns[b]] = 100000 * b + np.arange(Ns[b])
        k = O.select_keep(sc[b, :Ns[b]], int(Ps[b]), K)
        if isinstance(k, str):
            n_keep[b] = -1
            continue
        n_keep[b] = k.size
        keep[b, :k.size] = k
    assert n_keep[3] == -1
    src_t = dev(pool)
    dst_t = torch.full((L, 2, n_dst, page, H * d), SENT, dtype=torch.int16,
                       device="cuda")
    cfg = E.default_cfg(batch=B, n_layers=L, budget=K, page_size=page)
    dsc = torch.full((B, ld_s), -9.0, device="cuda")
    dpos = torch.full((B, ld_s), -9, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    cws_n = E.compact_workspace_bytes(cfg)
    cws = torch.zeros(cws_n, dtype=torch.uint8, device="cuda")
    E.epikv_compact(cfg, E.pool_of(src_t.view(L, 2, n_src, page, H, d)),
                    dev(src_pt), src_pt.shape[1],
                    E.pool_of(dst_t.view(L, 2, n_dst, page, H, d)),
                    dev(dst_pt), dst_pt.shape[1], dev(keep), dev(n_keep),
                    dev(sc), dsc, dev(pos), dpos, ld_s, status, cws, cws_n)
    _sync()
    dst = host(dst_t)
    dsc, dpos = host(dsc), host(dpos)
    assert np.all(host(status) == 0)
    for b in range(B):
        if n_keep[b] < 0:
            assert np.all(dst[:, :, dst_pt[b, :dpp]] == SENT)
            assert np.all(dsc[b] == -9.0)
            continue
        n = int(n_keep[b])
        src_rows = gather_logical(pool, src_pt[b], int(Ns[b]))
        exp = O.compact_rows(src_rows.transpose(2, 0, 1, 3), keep[b, :n])
        got = gather_logical(dst, dst_pt[b], dpp * page)
        assert np.array_equal(got[:, :, :n].transpose(2, 0, 1, 3), exp), b
        assert np.all(got[:, :, n:] == SENT), b          # guard slots
        assert np.array_equal(dsc[b, :n], sc[b, keep[b, :n]])
        assert np.array_equal(dpos[b, :n], pos[b, keep[b, :n]])
        assert np.all(dsc[b, n:] == -9.0)


# ---------------------------------------------------------------------------
# score (Lag-KV): Sec. 3.3
# ---------------------------------------------------------------------------
KV_SIGNALS = {  # name: (use keys, use values, lag-normalised)
    "lagkv": (True, True, True), "kv_key": (True, False, False),
    "kv_val": (False, True, False), "lagkv_key": (True, False, True)}


@pytest.mark.parametrize("C", [64, 37, 200, 1, 300, 1000])
@pytest.mark.parametrize("signal", list(KV_SIGNALS))
def test_kv_signals_match_oracle(E, signal, C):
    """Chunk lengths that split a plane's rows between several workgroups
    evenly (64), unevenly (37, 200) and not at all (1); 300 and 1000 rows
    with the workgroup's row offsets in an LDS table (300) or computed per
    block of 64 rows from the page table (1000, past that table's size),
    and a first chunk whose rows the first share walks alone."""
    _run_kv(E, signal, C)


@pytest.mark.parametrize("H,d", [(1, 64), (2, 128), (4, 128), (2, 256),
                                 (16, 128), (8, 256)])
@pytest.mark.parametrize("signal", ["lagkv", "kv_val", "lagkv_key"])
def test_kv_signals_head_shapes(E, signal, H, d):
    """Rows of 64 to 2048 channels: several narrow rows per wavefront
    (64, 256 channels), one wavefront per row (512) and rows split into 2
    or 4 wavefront segments (1024, 2048), heads of 64 to 256 channels."""
    _run_kv(E, signal, 37, H=H, d=d)


@pytest.mark.parametrize("signal", ["lagkv", "kv_key"])
def test_kv_signal_nan_propagates_as_in_the_oracle(E, signal):
    """A NaN key channel of one token: its variance is NaN, the trailing
    mean carries it through the window, and (lag-normalised) the chunk's
    range of that channel is NaN, so the next chunk's signal is NaN too --
    the plain minimum / maximum over the chunk the oracle takes."""
    _run_kv(E, signal, 64, nan=True)


@pytest.mark.parametrize("signal,L", [("lagkv", 65), ("lagkv_key", 129)])
def test_kv_signals_many_planes(E, signal, L):
    """More than 256 (used plane, sequence) pairs: the lag-normalised
    signals then take 8-wavefront workgroups, two per CU (fewer pairs take
    16-wavefront ones, one per CU)."""
    _run_kv(E, signal, 37, L=L)


def _run_kv(E, signal, C, nan=False, H=8, d=128, L=4, B=2, page=16):
    import torch
    print(f"kv signal {signal} C={C} nan={nan} H={H} d={d} L={L} B={B} "
          f"page={page}", flush=True)
    use_k, use_v, lag = KV_SIGNALS[signal]
    sig_id = {"lagkv": E.SIGNAL_LAGKV, "kv_key": E.SIGNAL_KV_KEY,
              "kv_val": E.SIGNAL_KV_VAL, "lagkv_key": E.SIGNAL_LAGKV_KEY}[signal]
    g = synth.rng(500)
    w = 64
    n_chunks = 3
    T = C * n_chunks
    Ns = T + 16 * np.arange(B)       # sequence b has 16 b older tokens first
    pt, n_pages = synth.page_tables(Ns, page, g)
    pool = np.zeros((L, 2, n_pages, page, H * d), dtype=np.uint16)
    tok = []   # logical rows per sequence [N][L][2][H*d]
    wl = synth.workload("lagkv_batch8", B=B, n_layers=L, n_kv_heads=H,
                        head_dim=d)
    for b in range(B):
        chunks = [synth.kv_rows(g, (C, L, 2, H, d),
                                synth.lagkv_channel_scale(wl, g, j))
                  for j in range(n_chunks)]
        rows = np.concatenate(chunks).reshape(T, L, 2, H * d)
        if Ns[b] > T:
            rows = np.concatenate([synth.kv_rows(g, (Ns[b] - T, L, 2, H * d)),
                                   rows])
        if nan and b == 0:
            rows[5, 1, 0, 7] = 0x7FC0        # token 5, layer 1, key channel 7
        tok.append(rows)
        pos = np.arange(Ns[b])
        pool[:, :, pt[b, pos // page], pos % page] = rows.transpose(1, 2, 0, 3)
    cfg = E.default_cfg(batch=B, n_layers=L, n_kv_heads=H, head_dim=d,
                        page_size=page, signal=sig_id,
                        smoothing=E.SMOOTH_MEAN, budget=4096)
    st = [torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
          for _ in range(2)]
    E.epikv_state_init(cfg, st[0])
    ws_n = E.workspace_bytes(cfg, C)
    # the workspace's contents are the caller's (here: bytes 0x7F, floats of
    # 3.4e38, as a stale partial range would leave them): nothing the call
    # reads may come from them
    ws = torch.full((ws_n,), 0x7F, dtype=torch.uint8, device="cuda")
    pool_t = dev(pool)
    P = E.pool_of(pool_t.view(L, 2, n_pages, page, H, d))
    ld_s = int(Ns.max())
    scores = torch.zeros((B, ld_s), device="cuda")
    prev_range = [None] * B
    prior = [np.zeros(0)] * B
    for j in range(n_chunks):
        n_cached = (Ns - T + (j + 1) * C).astype(np.int32)
        sig = torch.zeros((1, B, C), device="cuda")
        E.epikv_score(cfg, C, pool=P, page_table=dev(pt), ld_pt=pt.shape[1],
                      n_cached=dev(n_cached), state_in=st[0],
                      state_out=st[1], sig=sig, workspace=ws,
                      workspace_bytes_=ws_n)
        E.epikv_zscore(cfg, C, sig, dev(n_cached), st[0], st[1], scores, ld_s)
        _sync()
        got_q = host(sig)[0]
        got_s = host(scores)
        secs = E.state_sections(cfg, st[1].cpu())
        for b in range(B):
            lo = n_cached[b] - C
            rows = O.bf16_to_float64(tok[b][lo:lo + C])   # [C][L][2][HD]
            k = rows[:, :, 0].reshape(C, L, H, d)
            v = rows[:, :, 1].reshape(C, L, H, d)
            s_ref, q_ref, own = O.kv_chunk_scores(
                k, v, use_k, use_v, lag, prev_range[b], prior[b],
                O.SMOOTH_MEAN, w, cfg.eps)
            # q and its trailing mean are variances: strictly positive
            assert rel_err(got_q[b], q_ref, POSITIVE) <= TOL, (j, b)
            assert rel_err(got_s[b, lo:lo + C], s_ref, POSITIVE) <= TOL, (j, b)
            if lag:
                mn, mx = own
                rng_out = secs["range"].numpy()
                if use_k:
                    assert np.array_equal(rng_out[0, b][:, 0],
                                          mn[:, 0].astype(np.float32), equal_nan=True)
                    assert np.array_equal(rng_out[1, b][:, 0],
                                          mx[:, 0].astype(np.float32), equal_nan=True)
                if use_v:
                    assert np.array_equal(rng_out[0, b][:, 1],
                                          mn[:, 1].astype(np.float32), equal_nan=True)
                    assert np.array_equal(rng_out[1, b][:, 1],
                                          mx[:, 1].astype(np.float32), equal_nan=True)
            prev_range[b] = own
            prior[b] = np.concatenate([prior[b], q_ref])[-(w - 1):]
            if nan and b == 0 and j == 0:
                assert np.isnan(got_s[b, lo:lo + C]).any()
        st = [st[1], st[0]]


def _random_kv_cases(n, seed=20261203):
    """Seeded mixes of signal, chunk length, head shape (H*d / 8 dividing
    256), layers, sequences and page size for the KV-vector scorers."""
    g = np.random.default_rng(seed)
    shapes = [(1, 64), (2, 64), (1, 128), (4, 64), (2, 128), (8, 64),
              (4, 128), (2, 256), (8, 128), (16, 64), (4, 256), (8, 256),
              (16, 128)]
    out = []
    for _ in range(n):
        H, d = shapes[g.integers(len(shapes))]
        out.append(dict(signal=str(g.choice(list(KV_SIGNALS))),
                        C=int(g.choice([1, 2, 9, 63, 64, 65, 130, 257, 520])),
                        H=H, d=d, L=int(g.integers(1, 7)),
                        B=int(g.integers(1, 6)),
                        page=int(g.choice([1, 3, 16, 64]))))
    return out


RANDOM_KV = _random_kv_cases(16)


@pytest.mark.parametrize("i", range(len(RANDOM_KV)))
def test_kv_signals_random_shapes(E, i):
    """Every KV-vector signal over three chained chunks (the first from a
    fresh stream) against the oracle, on random mixes of shapes."""
    _run_kv(E, **RANDOM_KV[i])


def _random_select_shapes(n, seed=20261206):
    """Seeded (B, row length, K) for the split selection: rows longer than
    K, B * row length within 2 M positions (the oracle sorts in Python)."""
    g = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        K = int(g.choice([1, 7, 64, 300, 1024, 4096, 8192, 16384]))
        B = int(g.choice([1, 2, 3, 5, 8, 17, 32, 64, 128]))
        ld_s = int(g.integers(K + 1, K + 1 + 100000))
        if B * ld_s <= 2_000_000:
            out.append((B, ld_s, K))
    return out


@pytest.mark.parametrize("B,ld_s,K", _random_select_shapes(10))
def test_select_split_random_shapes(E, B, ld_s, K):
    test_select_split_matches_oracle_bit_exact(E, B, ld_s, K)


def test_select_split_ignores_stale_workspace(E):
    """epikv_select_ws accepts any workspace contents: here every word but
    each sequence's clear-marker is overwritten with garbage between two
    calls (what another layout's data can leave), and the second call must
    still be exact."""
    import torch
    B, ld_s, K = 3, 40000, 1024
    g = synth.rng(911)
    Ns = g.integers(K + 1, ld_s + 1, B)
    Ps = g.integers(0, K // 8, B)
    sc = np.stack([synth.old_scores(g, ld_s, ties=True) for _ in range(B)])
    cfg = E.default_cfg(batch=B, budget=K)
    n = E.select_workspace_bytes(cfg)
    assert n > 0
    ws = torch.zeros(n // 4, dtype=torch.int32, device="cuda")
    d_sc, d_n, d_p = dev(sc), dev(Ns.astype(np.int32)), dev(Ps.astype(np.int32))
    R = O.default_recent(K)
    for rep in range(2):
        keep = torch.full((B, K), -5, dtype=torch.int32, device="cuda")
        nk = torch.zeros(B, dtype=torch.int32, device="cuda")
        st = torch.full((B,), 9, dtype=torch.int32, device="cuda")
        E.epikv_select_ws(cfg, d_sc, ld_s, d_n, d_p, keep, nk, st, ws, n)
        _sync()
        kh, nh, sh = host(keep), host(nk), host(st)
        for b in range(B):
            ref = O.select_keep(sc[b, :Ns[b]], int(Ps[b]), K, R)
            assert sh[b] == E.SEQ_OK and nh[b] == ref.size, (rep, b)
            assert np.array_equal(kh[b, :ref.size], ref), (rep, b)
        # garbage everywhere except the first two words of every block
        words = ws.cpu().numpy()
        marks = words.copy()
        words[:] = 0x11111111
        seq_words = 6208                 # words per sequence block (24832 bytes)
        for b in range(B):
            words[b * seq_words:b * seq_words + 2] = marks[b * seq_words:b * seq_words + 2]
        ws.copy_(torch.from_numpy(words))
