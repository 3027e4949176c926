"""In-place rebuild with whole-page remapping against the oracle.

epikv_compact_remap packs each sequence's retained rows to the front of its
own pages like epikv_compact_inplace, but a destination page that receives
one later source page whole, in order, takes that page in the table instead
of a copy.  After the call the page table must equal the oracle's
(page_table_after_remap) entry for entry, and every byte of the pool the
oracle's compact_pages_remap of every sequence: rows written where the
oracle writes them, nothing else touched.
"""
import zlib

import numpy as np
import pytest

import oracle as O
import synth
from harness import dev, gather_logical, host, remap_expected

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def _keep_sets(kind, lengths, K, page, prefix, g):
    """Retained sets of each kind, ascending, at most K positions."""
    keeps = []
    R = O.default_recent(K)
    for b, N in enumerate(lengths):
        N = int(N)
        P = int(prefix[b])
        if kind == "select":            # the selection rule on random scores
            keep = O.select_keep(synth.old_scores(g, N, ties=True), P, K, R)
        elif kind == "blocks":
            # the lowest scores fill whole aligned pages: the selection then
            # evicts whole pages and every later page can be remapped
            s = g.standard_normal(N)
            n_pg = N // page
            for a in g.choice(max(n_pg - 1, 1), size=min(3, max(n_pg - 1, 1)),
                              replace=False):
                s[a * page:(a + 1) * page] -= 100.0
            keep = O.select_keep(s, P, K, R)
        else:                           # aligned blocks and single tokens
            mask = np.ones(N, bool)
            n_pg = -(-N // page)
            for _ in range(int(g.integers(1, 4))):
                a = int(g.integers(0, n_pg))
                mask[a * page:(a + int(g.integers(1, 3))) * page] = False
            for _ in range(int(g.integers(0, 3))):
                mask[int(g.integers(0, N))] = False
            mask[:P] = True
            keep = np.nonzero(mask)[0][:K]
        assert not isinstance(keep, str)
        keeps.append(np.asarray(keep, np.int64))
    return keeps


CASES = {
    "blocks_p16": dict(kind="blocks", lengths=[400, 300, 520, 130], K=256),
    "mixed_p16": dict(kind="mixed", lengths=[300, 90, 500, 64, 250], K=512),
    "mixed_p4": dict(kind="mixed", lengths=[200, 150, 77], K=512, page=4),
    "mixed_p1": dict(kind="mixed", lengths=[150, 90], K=512, page=1),
    "mixed_p3": dict(kind="mixed", lengths=[200, 151, 77], K=512, page=3),
    "page1_select": dict(kind="select", lengths=[150, 90], K=40, page=1),
    "select_p16": dict(kind="select", lengths=[300, 90, 500, 120], K=64, L=8),
    "blocks_prefix": dict(kind="blocks", lengths=[640, 480], K=256,
                          prefix=[48, 48], share_pages=2),
    "blocks_page1024": dict(kind="mixed", lengths=[5000, 2100], K=8192,
                            page=1024, L=1),
    "blocks_hd64_h1": dict(kind="blocks", lengths=[400, 300], K=128, H=1, d=64),
    "bad_input": dict(kind="mixed", lengths=[300] * 5, K=512, corrupt=True),
}


def _run(E, name, kind, lengths, K, L=2, H=8, d=128, page=16, prefix=None,
         share_pages=0, corrupt=False):
    import torch
    g = synth.rng(zlib.crc32(name.encode()))
    lengths = np.asarray(lengths, np.int64)
    B = lengths.size
    prefix = np.zeros(B, np.int64) if prefix is None else np.asarray(prefix)
    cfg = E.default_cfg(batch=B, n_layers=L, n_kv_heads=H, head_dim=d,
                        page_size=page, budget=K)
    assert E.check_cfg(cfg) == 0
    pt, used = synth.page_tables(lengths, page, g, ld=int(
        (lengths.max() + page - 1) // page) + 2)
    n_pages = used + 3
    if share_pages:                 # sequence 1 reuses sequence 0's first pages
        pt[1, :share_pages] = pt[0, :share_pages]
    pool = synth.random_bits16(g, (L, 2, n_pages, page, H * d))
    ld_s = int(lengths.max())
    sc = g.standard_normal((B, ld_s)).astype(np.float32)
    pos = g.integers(0, 1 << 30, size=(B, ld_s), dtype=np.int32)
    keeps = _keep_sets(kind, lengths, K, page, prefix, g)
    keep_idx = np.full((B, K), -3, np.int32)
    n_keep = np.zeros(B, np.int32)
    for b, keep in enumerate(keeps):
        keep_idx[b, :keep.size] = keep
        n_keep[b] = keep.size
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
    n_pairs = [len(O.remap_pairs(k, page)) if k is not None else 0
               for k in keeps]
    print(f"  remapped pages per sequence: {n_pairs}", flush=True)
    exp_pool, exp_pt = remap_expected(pool, pt, keeps, page)
    exp_sc, exp_pos = sc.copy(), pos.copy()
    for b, keep in enumerate(keeps):
        if keep is not None:
            exp_sc[b] = O.compact_rows_inplace(sc[b], keep)
            exp_pos[b] = O.compact_rows_inplace(pos[b], keep)

    pool_d = dev(pool)
    pt_d = dev(pt)
    sc_d, pos_d = dev(sc), dev(pos)
    st_d = dev(np.zeros(B, np.int32))
    ws_n = E.compact_workspace_bytes(cfg)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    E.epikv_compact_remap(
        cfg, E.pool_of(pool_d.view(L, 2, n_pages, page, H, d)), pt_d,
        pt.shape[1], dev(keep_idx), dev(n_keep), sc_d, pos_d, ld_s, st_d, ws,
        ws_n)
    torch.cuda.synchronize()
    assert np.array_equal(host(st_d), want_status), name
    assert np.array_equal(host(pt_d), exp_pt), name
    assert host(pool_d).tobytes() == exp_pool.tobytes(), name
    assert host(sc_d).tobytes() == exp_sc.tobytes(), name
    assert np.array_equal(host(pos_d), exp_pos), name
    return sum(n_pairs)


@pytest.mark.parametrize("name", list(CASES))
def test_remap_case(E, name):
    print(f"remap case {name}", flush=True)
    n = _run(E, name, **CASES[name])
    if name not in ("select_p16", "bad_input"):
        assert n > 0                      # the case exercises remapping


def test_remap_equals_inplace_logically(E):
    """Read through the tables, the remapped rebuild and the plain in-place
    rebuild hold the same rows (GPU against GPU), steady-state decode kept
    sets (K + 128 -> K) of 32 sequences."""
    import torch
    print("remap vs in place, 32 sequences", flush=True)
    g = synth.rng(4242)
    B, K, C, L, H, d, page = 32, 1024, 128, 2, 8, 128, 16
    lengths = np.full(B, K + C)
    pt, used = synth.page_tables(lengths, page, g)
    pool = synth.random_bits16(g, (L, 2, used, page, H * d))
    keeps = _keep_sets("blocks", lengths, K, page, np.zeros(B), g)[:16] + \
        _keep_sets("select", lengths, K, page, np.zeros(B), g)[16:]
    keep_idx = np.stack([k.astype(np.int32) for k in keeps])
    n_keep = np.full(B, K, np.int32)
    cfg = E.default_cfg(batch=B, n_layers=L, page_size=page, budget=K)
    ws_n = E.compact_workspace_bytes(cfg)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    a_d, b_d = dev(pool), dev(pool)
    pt_r = dev(pt)
    E.epikv_compact_inplace(cfg, E.pool_of(a_d.view(L, 2, used, page, H, d)),
                            dev(pt), pt.shape[1], dev(keep_idx), dev(n_keep),
                            None, None, 0, None, ws, ws_n)
    E.epikv_compact_remap(cfg, E.pool_of(b_d.view(L, 2, used, page, H, d)),
                          pt_r, pt.shape[1], dev(keep_idx), dev(n_keep),
                          None, None, 0, None, ws, ws_n)
    torch.cuda.synchronize()
    a, b_, new_pt = host(a_d), host(b_d), host(pt_r)
    n_pairs = 0
    for s in range(B):
        assert sorted(new_pt[s]) == sorted(pt[s])
        ra = gather_logical(a, pt[s], K)
        rb = gather_logical(b_, new_pt[s], K)
        assert ra.tobytes() == rb.tobytes(), s
        n_pairs += len(O.remap_pairs(keeps[s], page))
    print(f"  remapped pages: {n_pairs}", flush=True)
    assert n_pairs > 16 * 8


def test_remap_twice_in_a_row(E):
    """Two steady-state rebuilds in a row, the second on the table the
    first rewrote, the workspace reused."""
    import torch
    print("remap twice", flush=True)
    g = synth.rng(78)
    B, K, C, L, H, d, page = 3, 96, 32, 2, 8, 128, 16
    lengths = np.array([K + C, K + C, K + 5])
    pt, used = synth.page_tables(lengths, page, g)
    pool = synth.random_bits16(g, (L, 2, used, page, H * d))
    cfg = E.default_cfg(batch=B, n_layers=L, page_size=page, budget=K)
    ws_n = E.compact_workspace_bytes(cfg)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    pool_d, pt_d = dev(pool), dev(pt)
    desc = E.pool_of(pool_d.view(L, 2, used, page, H, d))
    exp, exp_pt = pool.copy(), pt.copy()
    cur = lengths.copy()
    for rep in range(2):
        keeps = _keep_sets("blocks" if rep == 0 else "mixed", cur, K, page,
                           np.zeros(B), g)
        keep_idx = np.full((B, K), -1, np.int32)
        for b, k in enumerate(keeps):
            keep_idx[b, :k.size] = k
        n_keep = np.array([k.size for k in keeps], np.int32)
        exp, exp_pt = remap_expected(exp, exp_pt, keeps, page)
        E.epikv_compact_remap(cfg, desc, pt_d, pt.shape[1], dev(keep_idx),
                              dev(n_keep), None, None, 0, None, ws, ws_n)
        torch.cuda.synchronize()
        assert np.array_equal(host(pt_d), exp_pt), rep
        assert host(pool_d).tobytes() == exp.tobytes(), rep
        cur = np.minimum(n_keep + 20, lengths)


def _random_cases(n, seed):
    """Seeded mixes of lengths, budget, layers, head shape, page size and
    prefill (kept sets from the selection rule, or of each remapping kind)."""
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
                    page=page, kind=str(g.choice(["blocks", "mixed", "select"])))
        if g.random() < 0.5:
            R = min(128, K // 4)
            case["prefix"] = [int(g.integers(0, max(1, min(n_, K - R))))
                              for n_ in lengths]
        out[f"random{i}"] = case
    return out


RANDOM_CASES = _random_cases(12, 20261205)


@pytest.mark.parametrize("name", list(RANDOM_CASES))
def test_random_case(E, name):
    print(f"random case {name}: {RANDOM_CASES[name]}", flush=True)
    _run(E, name, **RANDOM_CASES[name])
