"""In-place rebuild of the cache against the oracle.

epikv_compact_inplace (and epikv_evict_step with in_place set) packs each
sequence's retained rows to the front of its own pages.  After the call
every byte of the pool must equal the oracle's in-place rebuild of every
sequence (compact_rows_inplace): moved rows bit-exact, the leading run
before the first hole and every slot past n_keep unchanged, pages no
sequence owns unchanged.  Scores and positions follow their rows.
"""
import zlib

import numpy as np
import pytest

import oracle as O
import synth
from harness import (NEAR_ZERO, TOL, dev, gather_logical, host, rel_err,
                     remap_expected, scatter_logical)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def _expected(pool, pt, keeps, lengths):
    """Apply the oracle's in-place rebuild to every sequence of a host pool
    [L][2][n_pages][page][H*d]."""
    exp = pool.copy()
    for b, keep in enumerate(keeps):
        if keep is None:
            continue
        N = int(lengths[b])
        rows = gather_logical(exp, pt[b], N).transpose(2, 0, 1, 3)
        moved = O.compact_rows_inplace(rows, keep)
        scatter_logical(exp, pt[b], 0, moved.transpose(1, 2, 0, 3))
    return exp


CASES = {
    # name: overrides of _run
    # column slices of 1 KiB and 256 B (the library picks the widest that
    # still gives 2048 independent walks, with 16- and 32-row tiles), 256 B
    # with 64-row tiles when there are fewer walks, and 64 B for rows under
    # 256 B (64- and 256-row tiles)
    "narrow_slices": dict(lengths=[300, 90, 500], K=64),
    "mid_slices": dict(lengths=[300, 90, 500, 120, 260, 64, 65, 200], K=64,
                       L=16),
    "wide_slices": dict(lengths=list(range(64, 320, 8)), K=48, L=16),
    "row128_many": dict(lengths=list(range(64, 320, 8)), K=48, L=16, H=1,
                        d=64),
    "page1": dict(lengths=[150, 90], K=40, page=1),
    "page3": dict(lengths=[150, 91, 400], K=40, page=3),
    "page1024": dict(lengths=[2500, 600], K=300, page=1024),
    "hd64_h1": dict(lengths=[300, 200], K=64, H=1, d=64),
    "hd256_h8": dict(lengths=[300, 200], K=64, H=8, d=256),
    "hd128_h3": dict(lengths=[300, 200], K=64, H=3, d=128),
    "no_hole": dict(lengths=[50, 400], K=64),
    "prefix_shared": dict(lengths=[400, 300], K=96, prefix=[40, 40],
                          share_pages=2),
    "bad_input": dict(lengths=[300, 300, 300, 300, 300], K=64, corrupt=True),
    "side_arrays_off": dict(lengths=[300, 90], K=64, side=False),
}


def _run(E, name, lengths, K, L=2, H=8, d=128, page=16, prefix=None,
         share_pages=0, corrupt=False, side=True):
    import torch
    g = synth.rng(zlib.crc32(name.encode()))
    lengths = np.asarray(lengths, np.int64)
    B = lengths.size
    prefix = np.zeros(B, np.int64) if prefix is None else np.asarray(prefix)
    R = O.default_recent(K)
    cfg = E.default_cfg(batch=B, n_layers=L, n_kv_heads=H, head_dim=d,
                        page_size=page, budget=K)
    assert E.check_cfg(cfg) == 0
    # scattered pages plus a few that no sequence owns
    pt, used = synth.page_tables(lengths, page, g)
    n_pages = used + 3
    if share_pages:                 # sequence 1 reuses sequence 0's first pages
        pt[1, :share_pages] = pt[0, :share_pages]
    pool = synth.random_bits16(g, (L, 2, n_pages, page, H * d))
    ld_s = int(lengths.max())
    sc = np.zeros((B, ld_s), np.float32)
    pos = g.integers(0, 1 << 30, size=(B, ld_s), dtype=np.int32)
    keep_idx = np.full((B, K), -3, np.int32)
    n_keep = np.zeros(B, np.int32)
    keeps = []
    for b in range(B):
        N = int(lengths[b])
        sc[b, :N] = synth.old_scores(g, N, ties=True)
        keep = O.select_keep(sc[b, :N], int(prefix[b]), K, R)
        assert not isinstance(keep, str)
        keep_idx[b, :keep.size] = keep
        n_keep[b] = keep.size
        keeps.append(keep)
    status = np.zeros(B, np.int32)
    want_status = np.zeros(B, np.int32)
    if corrupt:
        # 0: not ascending; 1: refused by the selection (n_keep = -1);
        # 2: nothing kept; 3: reaches a page the table does not hold
        keep_idx[0, [5, 6]] = keep_idx[0, [6, 5]]
        n_keep[1] = -1
        n_keep[2] = 0
        keep_idx[3, keeps[3].size - 1] = pt.shape[1] * page + 7
        for b in (0, 3):
            want_status[b] = E.SEQ_RANGE
        for b in (0, 1, 2, 3):
            keeps[b] = None
    exp_pool = _expected(pool, pt, keeps, lengths)
    exp_sc, exp_pos = sc.copy(), pos.copy()
    for b, keep in enumerate(keeps):
        if keep is not None:
            exp_sc[b] = O.compact_rows_inplace(sc[b], keep)
            exp_pos[b] = O.compact_rows_inplace(pos[b], keep)

    pool_d = dev(pool)
    sc_d, pos_d = dev(sc), dev(pos)
    st_d = dev(status)
    ws_n = E.compact_workspace_bytes(cfg)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    E.epikv_compact_inplace(
        cfg, E.pool_of(pool_d.view(L, 2, n_pages, page, H, d)), dev(pt),
        pt.shape[1], dev(keep_idx), dev(n_keep),
        sc_d if side else None, pos_d if side else None, ld_s, st_d, ws, ws_n)
    torch.cuda.synchronize()
    got = host(pool_d)
    assert np.array_equal(host(st_d), want_status), name
    for b, keep in enumerate(keeps):
        if keep is None:
            continue
        h = O.first_hole(keep)
        print(f"  seq {b}: N={lengths[b]} kept={keep.size} first hole={h}")
    assert got.tobytes() == exp_pool.tobytes(), name
    if side:
        assert host(sc_d).tobytes() == exp_sc.tobytes(), name
        assert np.array_equal(host(pos_d), exp_pos), name
    else:
        assert host(sc_d).tobytes() == sc.tobytes()
        assert np.array_equal(host(pos_d), pos)


@pytest.mark.parametrize("name", list(CASES))
def test_inplace_case(E, name):
    print(f"in-place case {name}", flush=True)
    _run(E, name, **CASES[name])


def test_inplace_twice_in_a_row(E):
    """A second rebuild on the packed cache (the steady state: K + E rows
    down to K again) -- the workspace is reused and nothing leaks from the
    first call."""
    import torch
    print("in-place twice", flush=True)
    g = synth.rng(77)
    B, K, E_, L, H, d, page = 3, 96, 32, 2, 8, 128, 16
    R = O.default_recent(K)
    lengths = np.array([K + E_, K + E_, K + 5])
    pt, used = synth.page_tables(lengths, page, g)
    pool = synth.random_bits16(g, (L, 2, used, page, H * d))
    cfg = E.default_cfg(batch=B, n_layers=L, page_size=page, budget=K)
    ws_n = E.compact_workspace_bytes(cfg)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    pool_d = dev(pool)
    desc = E.pool_of(pool_d.view(L, 2, used, page, H, d))
    exp = pool.copy()
    cur_len = lengths.copy()
    for rep in range(2):
        keeps = []
        keep_idx = np.full((B, K), -1, np.int32)
        for b in range(B):
            N = int(cur_len[b])
            keep = O.select_keep(g.standard_normal(N), 0, K, R)
            keep_idx[b, :keep.size] = keep
            keeps.append(keep)
        n_keep = np.array([k.size for k in keeps], np.int32)
        exp = _expected(exp, pt, keeps, cur_len)
        E.epikv_compact_inplace(cfg, desc, dev(pt), pt.shape[1],
                                dev(keep_idx), dev(n_keep), None, None, 0,
                                None, ws, ws_n)
        torch.cuda.synchronize()
        assert host(pool_d).tobytes() == exp.tobytes(), rep
        # next step: the packed rows plus a few new tokens (already there)
        cur_len = np.minimum(n_keep + 20, lengths)


@pytest.mark.parametrize("mode", ["in_place", "remap"])
def test_inplace_step_small(E, mode):
    """epikv_evict_step with in_place set (plain, or with page remapping):
    the chunk's scores as the oracle computes them, the selection of the
    GPU's fp32 scores, and the pool, the page table and the scores rebuilt
    in place."""
    import torch
    print(f"in-place evict_step ({mode})", flush=True)
    g = synth.rng(78)
    lengths = np.array([400, 150, 64])
    B, C, K, page, L, H, d, D, na, nb = 3, 32, 96, 16, 2, 8, 128, 256, 2, 2
    nband, w = na + nb, 64
    R = O.default_recent(K)
    cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, page_size=page,
                        n_band_a=na, n_band_b=nb, budget=K)
    hid = synth.f32_to_bf16_bits(
        (g.standard_normal((nband, B, C, D)) * 3).astype(np.float32))
    before = synth.f32_to_bf16_bits(
        g.standard_normal((B, nband, D)).astype(np.float32))
    ring = (50.0 + g.standard_normal((B, nband, w - 1))).astype(np.float32)
    n_tok = (lengths - C + 70).astype(np.int32)
    ld_s = int(lengths.max())
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    pt, used = synth.page_tables(lengths, page, g)
    pool = synth.random_bits16(g, (L, 2, used, page, H * d))
    pos = g.integers(0, 1 << 30, size=(B, ld_s), dtype=np.int32)
    st = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8)
    sec = E.state_sections(cfg, st)
    sec["n_tok"][:] = torch.from_numpy(n_tok)
    sec["ring"][:] = torch.from_numpy(ring)
    sec["h_prev"][:] = torch.from_numpy(before.view(np.int16))
    st_in = st.cuda()
    st_out = torch.zeros_like(st_in)
    hd = dev(hid)
    pool_d = dev(pool)
    scores, pos_d = dev(sc), dev(pos)
    keep = torch.full((B, K), -3, dtype=torch.int32, device="cuda")
    n_keep = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(B, dtype=torch.int32, device="cuda")
    ws_n = E.workspace_bytes(cfg, C)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    desc = E.pool_of(pool_d.view(L, 2, used, page, H, d))
    pt_d = dev(pt)
    io = E.make_step_io(
        C, [hd[l] for l in range(nband)], D, C * D,
        dev(lengths.astype(np.int32)), torch.zeros(B, dtype=torch.int32,
                                                   device="cuda"),
        desc, pt_d, pt.shape[1], E.Pool(), None, 0, scores, ld_s, st_in,
        st_out, keep, n_keep, status, ws, ws_n, src_pos=pos_d,
        dst_pos=pos_d, in_place=E.COMPACT_IN_PLACE if mode == "in_place"
        else E.COMPACT_REMAP)
    # the chunk's fp32 scores as the step computes them: the same kernels
    # called one by one on the same inputs (deterministic, so bitwise equal)
    sig = torch.zeros((nband, B, C), device="cuda")
    st_tmp = torch.zeros_like(st_in)
    chunk_sc = scores.clone()
    E.epikv_score(cfg, C, [hd[l] for l in range(nband)], D, C * D,
                  state_in=st_in, state_out=st_tmp, sig=sig)
    E.epikv_zscore(cfg, C, sig, dev(lengths.astype(np.int32)), st_in, st_tmp,
                   chunk_sc, ld_s)
    E.epikv_evict_step(cfg, io)
    torch.cuda.synchronize()
    kh, nk, sth = host(keep), host(n_keep), host(status)
    full = host(chunk_sc)
    assert np.all(sth == 0)
    keeps = []
    exp_sc, exp_pos = full.copy(), pos.copy()
    for b in range(B):
        N = int(lengths[b])
        cnt = min(w - 1, int(n_tok[b]) - 1)
        prior = [ring[b, l, w - 1 - cnt:].astype(np.float64)
                 for l in range(nband)]
        s_new, *_ = O.hs_chunk_scores(
            O.bf16_to_float64(hid[:, b]), O.bf16_to_float64(before[b]),
            prior, na, nb, O.SMOOTH_Z, w)
        # band differences of z-scores: can sit at 0
        assert rel_err(full[b, N - C:N], s_new, NEAR_ZERO) <= TOL, b
        ref = O.select_keep(full[b, :N], 0, K, R)
        assert nk[b] == ref.size and np.array_equal(kh[b, :ref.size], ref), b
        keeps.append(ref)
        exp_sc[b] = O.compact_rows_inplace(full[b], ref)
        exp_pos[b] = O.compact_rows_inplace(pos[b], ref)
    assert host(scores).tobytes() == exp_sc.tobytes()
    assert np.array_equal(host(pos_d), exp_pos)
    if mode == "in_place":
        exp_pool, exp_pt = _expected(pool, pt, keeps, lengths), pt
    else:
        exp_pool, exp_pt = remap_expected(pool, pt, keeps, page)
        print(f"  remapped pages: {[len(O.remap_pairs(k, page)) for k in keeps]}")
    assert np.array_equal(host(pt_d), exp_pt)
    assert host(pool_d).tobytes() == exp_pool.tobytes()


@pytest.mark.parametrize("mode", ["in_place", "remap"])
def test_inplace_full_size_matches_out_of_place(E, mode):
    """The 32-sequence batch (N 8k..32k, K = 4096, 32 layers): the step run
    out of place, then in place (plain, or with page remapping) on the same
    inputs.  Every sequence's scores and positions, and sampled rows of
    every layer and K/V, agree; in place, sampled slots past n_keep keep
    their bytes; with remapping the page table is the oracle's."""
    import torch
    import bench
    print(f"in-place full size ({mode})", flush=True)
    w = synth.workload("ragged_batch32")
    S = bench.setup_hs(w, E)
    K, page = w.budget, w.page_size
    E.epikv_evict_step(S.cfg, S.io)
    torch.cuda.synchronize()
    keep = host(S.keep_idx).copy()
    assert np.all(host(S.status) == 0) and np.all(host(S.n_keep) == K)
    g = synth.rng(902)
    pick = {b: np.sort(g.choice(K, 32, replace=False)) for b in range(w.B)}
    tail = {b: np.sort(g.choice(np.arange(K, int(S.lengths[b])), 16,
                                replace=False)) for b in range(w.B)}

    def rows(pool, pt, b, idx):
        return host(pool[:, :, torch.from_numpy(
            pt[b, idx // page].astype(np.int64)).cuda(),
            torch.from_numpy((idx % page).astype(np.int64)).cuda(), :])

    tail_before = {b: rows(S.src_pool, S.src_pt_host, b, tail[b])
                   for b in range(w.B)}
    io = E.make_step_io(
        w.chunk, S.hidden_ptrs, w.hidden, w.chunk * w.hidden, S.n_cached,
        S.n_prefix, S.src, S.src_pt, S.src_pt_host.shape[1], E.Pool(), None,
        0, S.scores, S.ld_s, S.state_in, S.state_out, S.keep_idx, S.n_keep,
        S.status, S.ws, S.ws_bytes, src_pos=S.src_pos, dst_pos=S.src_pos,
        in_place=E.COMPACT_IN_PLACE if mode == "in_place" else E.COMPACT_REMAP)
    E.epikv_evict_step(S.cfg, io)
    torch.cuda.synchronize()
    assert np.array_equal(host(S.keep_idx), keep)
    assert np.all(host(S.status) == 0)
    assert host(S.scores)[:, :K].tobytes() == host(S.dst_scores)[:, :K].tobytes()
    assert np.array_equal(host(S.src_pos)[:, :K], host(S.dst_pos)[:, :K])
    new_pt = host(S.src_pt)
    moved = pages = 0
    for b in range(w.B):
        moved += K - O.first_hole(keep[b])
        if mode == "remap":
            n = int(np.count_nonzero(S.src_pt_host[b] >= 0))
            exp = O.page_table_after_remap(S.src_pt_host[b, :n], keep[b], page)
            assert np.array_equal(new_pt[b, :n], exp), b
            pages += len(O.remap_pairs(keep[b], page))
        else:
            assert np.array_equal(new_pt, S.src_pt_host)
            assert np.array_equal(rows(S.src_pool, S.src_pt_host, b, tail[b]),
                                  tail_before[b]), b
        assert np.array_equal(rows(S.src_pool, new_pt, b, pick[b]),
                              rows(S.dst_pool, S.dst_pt_host, b, pick[b])), b
    print(f"  rows moved: {moved} of {w.B * K}; pages remapped: {pages}")


def test_inplace_step_lagkv_matches_out_of_place(E):
    """The Lag-KV step reads the chunk's K/V rows from the pool it then
    rebuilds: in place it must give the scores, selection and rows of the
    out-of-place step on the same inputs."""
    import torch
    print("in-place Lag-KV step", flush=True)
    g = synth.rng(79)
    B, C, K, page, L, H, d = 3, 64, 96, 16, 4, 8, 128
    lengths = np.array([400, 150, 80])
    ld_s = int(lengths.max())
    pt, used = synth.page_tables(lengths, page, g)
    dpt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    pool = synth.kv_rows(g, (L, 2, used, page, H, d)).reshape(
        L, 2, used, page, H * d)
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    cfg = E.default_cfg(batch=B, n_layers=L, signal=E.SIGNAL_LAGKV,
                        smoothing=E.SMOOTH_MEAN, budget=K)
    st0 = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
    E.epikv_state_init(cfg, st0)
    ws_n = E.workspace_bytes(cfg, C)

    def run(in_place):
        src = dev(pool)
        dst = torch.zeros((L, 2, n_dst, page, H * d), dtype=torch.int16,
                          device="cuda")
        scores = dev(sc)
        dsc = torch.zeros_like(scores)
        keep = torch.zeros((B, K), dtype=torch.int32, device="cuda")
        nk = torch.zeros(B, dtype=torch.int32, device="cuda")
        status = torch.zeros(B, dtype=torch.int32, device="cuda")
        st_out = torch.zeros_like(st0)
        ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
        io = E.make_step_io(
            C, None, 0, 0, dev(lengths.astype(np.int32)),
            torch.zeros(B, dtype=torch.int32, device="cuda"),
            E.pool_of(src.view(L, 2, used, page, H, d)), dev(pt), pt.shape[1],
            E.Pool() if in_place else E.pool_of(
                dst.view(L, 2, n_dst, page, H, d)),
            None if in_place else dev(dpt), 0 if in_place else dpt.shape[1],
            scores, ld_s, st0, st_out, keep, nk, status, ws, ws_n,
            dst_scores=None if in_place else dsc, in_place=in_place)
        E.epikv_evict_step(cfg, io)
        torch.cuda.synchronize()
        return (host(src), host(dst), host(scores), host(dsc), host(keep),
                host(nk), host(status), host(st_out))

    src_o, dst_o, sc_o, dsc_o, keep_o, nk_o, stat_o, st_o = run(False)
    src_i, _, sc_i, _, keep_i, nk_i, stat_i, st_i = run(True)
    assert np.all(stat_o == 0) and np.array_equal(stat_i, stat_o)
    assert np.array_equal(nk_i, nk_o) and np.array_equal(keep_i, keep_o)
    assert st_i.tobytes() == st_o.tobytes()
    for b in range(B):
        n = int(nk_o[b])
        # scores: the out-of-place copy, or the sequence's own row if N <= K
        ref = dsc_o[b, :n] if lengths[b] > K else sc_o[b, :n]
        assert sc_i[b, :n].tobytes() == ref.tobytes(), b
        got = gather_logical(src_i, pt[b], n)
        if lengths[b] > K:
            exp = gather_logical(dst_o, dpt[b], n)
        else:
            exp = gather_logical(pool, pt[b], n)
        assert got.tobytes() == exp.tobytes(), b


def _random_cases(n, seed):
    """Seeded mixes of lengths, budget, layers, head shape, page size and
    prefill (kept sets from the selection rule)."""
    g = np.random.default_rng(seed)
    shapes = [(1, 64), (8, 128), (3, 128), (8, 256), (2, 64)]
    out = {}
    for i in range(n):
        B = int(g.integers(1, 7))
        H, d = shapes[g.integers(len(shapes))]
        page = int(g.choice([1, 2, 3, 16, 64]))
        K = int(g.choice([8, 40, 64, 130, 512]))
        lengths = [int(x) for x in g.integers(1, 900, size=B)]
        case = dict(lengths=lengths, K=K, L=int(g.integers(1, 5)), H=H, d=d,
                    page=page)
        if g.random() < 0.5:
            R = min(128, K // 4)
            case["prefix"] = [int(g.integers(0, max(1, min(n_, K - R))))
                              for n_ in lengths]
        out[f"random{i}"] = case
    return out


RANDOM_CASES = _random_cases(12, 20261204)


@pytest.mark.parametrize("name", list(RANDOM_CASES))
def test_random_case(E, name):
    print(f"random case {name}: {RANDOM_CASES[name]}", flush=True)
    _run(E, name, **RANDOM_CASES[name])
