"""Edge cases of epikv_evict_step against the oracle.

Each case builds a small batch, runs the whole step on the GPU and checks:
new-chunk scores within 1e-3 (NaN where the oracle has NaN), the retained
set exactly equal to the oracle's ranking of the GPU's fp32 scores (or the
same status), and the rebuilt rows bit-exact.
"""
import zlib

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


CASES = {
    # name: dict of overrides
    "K1": dict(K=1, lengths=[40, 1, 2]),
    "recent0": dict(K=64, recent=0, lengths=[200, 65, 64]),
    "recent_ge_K": dict(K=32, recent=40, lengths=[100, 32, 10]),
    "window1": dict(window=1, lengths=[300, 130]),
    "window256": dict(window=256, C=300, lengths=[700, 320]),
    "N_eq_K_and_K1": dict(K=96, lengths=[96, 97, 95]),
    "one_eligible": dict(K=64, prefix=[47, 0], lengths=[80, 80]),
    "page1": dict(page=1, lengths=[150, 90]),
    "page1024": dict(page=1024, lengths=[2500, 600]),
    "hd64_h1": dict(H=1, d=64, lengths=[300, 200]),
    "hd256_h8": dict(H=8, d=256, lengths=[300, 200]),
    "hd128_h3": dict(H=3, d=128, lengths=[300, 200]),
    "band_b_empty": dict(nb=0, lengths=[300, 200]),
    "nan_hidden": dict(nan=True, lengths=[300, 200]),
    "single_layer_preset": dict(na=1, nb=1, lengths=[400, 150]),
    "max_bands": dict(na=16, nb=16, lengths=[300, 200]),
    # 1500 short sequences: grids sized by the batch, per-sequence loops
    "many_sequences": dict(K=64, C=16, H=1, d=64,
                           lengths=list(20 + (np.arange(1500) * 37) % 180)),
}


def _run_case(E, name, K=64, recent=-1, window=64, C=32, page=16, H=8, d=128,
              L=2, D=256, na=2, nb=2, prefix=None, lengths=(300,),
              nan=False, mode="z"):
    import torch
    g = synth.rng(zlib.crc32(name.encode()))
    lengths = np.asarray(lengths, np.int64)
    B = lengths.size
    prefix = np.zeros(B, np.int32) if prefix is None else \
        np.asarray(prefix, np.int32)
    nband = na + nb
    HD = H * d
    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_kv_heads=H,
                        head_dim=d, page_size=page, n_band_a=na, n_band_b=nb,
                        window=window, budget=K, recent=recent,
                        smoothing={"z": E.SMOOTH_Z, "mean": E.SMOOTH_MEAN,
                                   "raw": E.SMOOTH_RAW}[mode])
    assert E.check_cfg(cfg) == 0
    R = recent if recent >= 0 else O.default_recent(K)
    Cc = min(C, int(lengths.min()))                 # chunk fits every N
    hid = synth.f32_to_bf16_bits(
        (g.standard_normal((nband, B, Cc, D)) * 3).astype(np.float32))
    before = synth.f32_to_bf16_bits(
        g.standard_normal((B, nband, D)).astype(np.float32))
    if nan:
        hid[0, 0, 5, 17] = 0x7FC0                     # NaN in Band A row
        hid[nband - 1, 1, 9, 3] = 0x7FC0              # NaN in the last row
    ring = (50.0 + g.standard_normal((B, nband, window - 1))).astype(
        np.float32)
    n_tok = (lengths - Cc + 70).astype(np.int32)      # long-running streams
    ld_s = int(lengths.max())
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - Cc] = synth.old_scores(g, int(lengths[b]) - Cc,
                                                   ties=True)
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g)
    pool = synth.random_bits16(g, (L, 2, n_src, page, HD))
    st = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st)
    sec["n_tok"][:] = torch.from_numpy(n_tok)
    sec["ring"][:] = torch.from_numpy(ring)
    sec["h_prev"][:] = torch.from_numpy(before.view(np.int16))
    st_in = st.cuda()
    st_out = torch.zeros_like(st_in)
    hd = dev(hid)
    src = dev(pool)
    SENT = 0x2D2D
    dst = torch.full((L, 2, n_dst, page, HD), SENT, dtype=torch.int16,
                     device="cuda")
    scores = dev(sc)
    keep = torch.full((B, K), -3, dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    ws_n = E.workspace_bytes(cfg, Cc)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    io = E.make_step_io(
        Cc, [hd[l] for l in range(nband)], D, Cc * D,
        dev(lengths.astype(np.int32)), dev(prefix),
        E.pool_of(src.view(L, 2, n_src, page, H, d)), dev(src_pt),
        src_pt.shape[1], E.pool_of(dst.view(L, 2, n_dst, page, H, d)),
        dev(dst_pt), dst_pt.shape[1], scores, ld_s, st_in, st_out, keep,
        n_keep, status, ws, ws_n)
    E.epikv_evict_step(cfg, io)
    torch.cuda.synchronize()
    gs, kh, nk, sth = host(scores), host(keep), host(n_keep), host(status)
    dsth = host(dst)
    for b in range(B):
        N = int(lengths[b])
        # the stream has n_tok - 1 earlier samples; the ring holds the last
        # min(w - 1, that many), right-aligned
        cnt = min(window - 1, int(n_tok[b]) - 1)
        prior = [ring[b, l, window - 1 - cnt:].astype(np.float64)
                 for l in range(nband)]
        s_new, *_ = O.hs_chunk_scores(
            O.bf16_to_float64(hid[:, b]), O.bf16_to_float64(before[b]),
            prior, na, nb, {"z": O.SMOOTH_Z, "mean": O.SMOOTH_MEAN,
                            "raw": O.SMOOTH_RAW}[mode], window)
        # band differences of z-scores (can sit at 0); NaN where the
        # oracle has NaN
        assert rel_err(gs[b, N - Cc:N], s_new, NEAR_ZERO) <= TOL, (name, b)
        ref = O.select_keep(gs[b, :N], int(prefix[b]), K, R)
        if isinstance(ref, str):
            assert sth[b] == E.SEQ_BUDGET and nk[b] == -1, (name, b)
            assert np.all(kh[b] == -3)
            continue
        assert sth[b] == E.SEQ_OK and nk[b] == ref.size, (name, b)
        assert np.array_equal(kh[b, :ref.size], ref), (name, b)
        n = ref.size
        pos = np.arange(N)
        rows = pool[:, :, src_pt[b, pos // page], pos % page]
        exp = O.compact_rows(rows.transpose(2, 0, 1, 3), ref)
        j = np.arange(n)
        out = dsth[:, :, dst_pt[b, j // page], j % page].transpose(2, 0, 1, 3)
        assert np.array_equal(out, exp), (name, b)
        # slots past n_keep stay untouched
        jj = np.arange(n, dst_pt.shape[1] * page)
        jj = jj[dst_pt[b, jj // page] >= 0]
        if jj.size:
            assert np.all(dsth[:, :, dst_pt[b, jj // page], jj % page] == SENT)


@pytest.mark.parametrize("name", list(CASES))
def test_edge_case(E, name):
    print(f"edge case {name}", flush=True)
    _run_case(E, name, **CASES[name])


def _random_cases(n, seed=20261202):
    """Seeded mixes of the step's dimensions (budget, recency window,
    window length, chunk, page size, head shape, layers, hidden width, band
    sizes, prefill, smoothing, ragged lengths), each checked like the cases
    above: scores, kept sets and every rebuilt byte."""
    g = np.random.default_rng(seed)
    out = {}
    for i in range(n):
        B = int(g.integers(1, 6))
        H, d = [(1, 64), (8, 128), (3, 128), (2, 256), (4, 64)][g.integers(5)]
        K = int(g.choice([1, 16, 64, 100, 256]))
        lengths = g.integers(1, 700, size=B)
        recent = int(g.choice([-1, -1, 0, int(g.integers(0, K + 1))]))
        R = recent if recent >= 0 else O.default_recent(K)
        prefix = [int(g.integers(0, max(1, min(n_, K - R)))) for n_ in lengths]
        out[f"random{i}"] = dict(
            K=K, recent=recent, window=int(g.choice([1, 5, 64, 100])),
            C=int(g.choice([1, 7, 32, 64, 129])),
            page=int(g.choice([1, 3, 16, 64])), H=H, d=d,
            L=int(g.integers(1, 4)), D=int(g.choice([8, 256, 1000, 4096])),
            na=int(g.integers(1, 5)), nb=int(g.integers(0, 5)),
            prefix=prefix, lengths=[int(x) for x in lengths],
            mode=str(g.choice(["z", "mean", "raw"])))
    return out


RANDOM_CASES = _random_cases(16)


@pytest.mark.parametrize("name", list(RANDOM_CASES))
def test_random_step_case(E, name):
    print(f"random step case {name}: {RANDOM_CASES[name]}", flush=True)
    _run_case(E, name, **RANDOM_CASES[name])
