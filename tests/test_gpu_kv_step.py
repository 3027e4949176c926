"""The whole eviction step with a KV-vector signal, against the oracle.

Seeded mixes of signal (Lag-KV, lag-kv-key, KV-key, KV-val), rebuild
(out of place, in place, in place with page remapping), sequences, chunk
length, budget, page size, layers, head shape and prefill, each a fresh
stream: the new tokens' scores against the oracle's (Sec. 3.3, Table 1;
the first chunk of a stream normalised by its own range), the kept sets
bit-exact against the selection rule on the GPU's own scores (App. D), and
every kept row, read back through the page table after the call, equal to
the row the oracle keeps there (App. H).
"""
import numpy as np
import pytest

import oracle as O
import synth
from harness import POSITIVE, TOL, dev, gather_logical, host, rel_err

pytestmark = pytest.mark.gpu

SIGNALS = {"lagkv": (True, True, True), "lagkv_key": (True, False, True),
           "kv_key": (True, False, False), "kv_val": (False, True, False)}


@pytest.fixture(scope="module")
def E():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def _cases(n, seed=20261208):
    g = np.random.default_rng(seed)
    shapes = [(1, 64), (2, 64), (1, 128), (4, 64), (2, 128), (8, 64),
              (4, 128), (2, 256), (8, 128), (4, 256)]
    out = []
    for _ in range(n):
        H, d = shapes[g.integers(len(shapes))]
        C = int(g.choice([1, 5, 32, 64, 100]))
        K = int(g.choice([16, 64, 100, 256]))
        B = int(g.integers(1, 6))
        R = O.default_recent(K)
        lengths = [int(x) for x in g.integers(C, C + 700, size=B)]
        out.append(dict(
            signal=str(g.choice(list(SIGNALS))),
            mode=str(g.choice(["out_of_place", "in_place", "remap"])),
            C=C, K=K, L=int(g.integers(1, 5)), H=H, d=d,
            page=int(g.choice([1, 3, 16, 64])), lengths=lengths,
            prefix=[int(g.integers(0, max(1, min(n_, K - R))))
                    for n_ in lengths],
            seed=int(g.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _cases(16),
                         ids=lambda c: f"{c['signal']}-{c['mode']}")
def test_kv_step_random(E, case):
    import torch
    print(f"KV-signal step: {case}", flush=True)
    g = np.random.default_rng(case["seed"])
    use_k, use_v, lag = SIGNALS[case["signal"]]
    C, K, L, H, d, page = (case[k] for k in ("C", "K", "L", "H", "d", "page"))
    lengths = np.asarray(case["lengths"], np.int64)
    prefix = np.asarray(case["prefix"], np.int32)
    B, HD = lengths.size, H * d
    sig_id = {"lagkv": E.SIGNAL_LAGKV, "lagkv_key": E.SIGNAL_LAGKV_KEY,
              "kv_key": E.SIGNAL_KV_KEY, "kv_val": E.SIGNAL_KV_VAL}
    cfg = E.default_cfg(batch=B, n_layers=L, n_kv_heads=H, head_dim=d,
                        page_size=page, signal=sig_id[case["signal"]],
                        smoothing=E.SMOOTH_MEAN, budget=K)
    assert E.check_cfg(cfg) == 0
    mode = {"out_of_place": E.COMPACT_OUT_OF_PLACE,
            "in_place": E.COMPACT_IN_PLACE, "remap": E.COMPACT_REMAP}[
        case["mode"]]
    pt, used = synth.page_tables(lengths, page, g)
    dpt, n_dst = synth.contiguous_page_tables(np.full(B, K), page)
    pool = synth.kv_rows(g, (L, 2, used, page, HD))
    ld_s = int(lengths.max())
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C,
                                                  ties=True)
    st0 = torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
    E.epikv_state_init(cfg, st0)
    ws_n = E.workspace_bytes(cfg, C)

    def run(m):
        """One step from fresh copies of the inputs in rebuild mode m."""
        oop = m == E.COMPACT_OUT_OF_PLACE
        src, pt_d, scores = dev(pool), dev(pt), dev(sc)
        dst = torch.zeros((L, 2, n_dst, page, HD), dtype=torch.int16,
                          device="cuda")
        dsc = torch.zeros_like(scores)
        keep = torch.full((B, K), -3, dtype=torch.int32, device="cuda")
        nk = torch.zeros(B, dtype=torch.int32, device="cuda")
        status = torch.zeros(B, dtype=torch.int32, device="cuda")
        st_out = torch.zeros_like(st0)
        ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
        io = E.make_step_io(
            C, None, 0, 0, dev(lengths.astype(np.int32)), dev(prefix),
            E.pool_of(src.view(L, 2, used, page, H, d)), pt_d, pt.shape[1],
            E.pool_of(dst.view(L, 2, n_dst, page, H, d)) if oop else E.Pool(),
            dev(dpt) if oop else None, dpt.shape[1] if oop else 0,
            scores, ld_s, st0, st_out, keep, nk, status, ws, ws_n,
            dst_scores=dsc if oop else None, in_place=m)
        E.epikv_evict_step(cfg, io)
        torch.cuda.synchronize()
        return dict(src=host(src), dst=host(dst), pt=host(pt_d),
                    scores=host(scores), dsc=host(dsc), keep=host(keep),
                    nk=host(nk), status=host(status), state=host(st_out))

    o = run(E.COMPACT_OUT_OF_PLACE)
    R = O.default_recent(K)
    for b in range(B):
        N = int(lengths[b])
        rows = gather_logical(pool, pt[b], N)             # [L][2][N][HD]
        new = O.bf16_to_float64(rows[:, :, N - C:N])
        k = new[:, 0].transpose(1, 0, 2).reshape(C, L, H, d)
        v = new[:, 1].transpose(1, 0, 2).reshape(C, L, H, d)
        s_ref, *_ = O.kv_chunk_scores(k, v, use_k, use_v, lag, None,
                                      np.zeros(0), O.SMOOTH_MEAN,
                                      cfg.window, cfg.eps)
        assert rel_err(o["scores"][b, N - C:N], s_ref, POSITIVE) <= TOL, b
        assert np.array_equal(o["scores"][b, :N - C], sc[b, :N - C]), b
        ref = O.select_keep(o["scores"][b, :N], int(prefix[b]), K, R)
        assert o["status"][b] == E.SEQ_OK, b
        assert o["nk"][b] == ref.size, b
        assert np.array_equal(o["keep"][b, :ref.size], ref), b
        if N > K:
            got = gather_logical(o["dst"], dpt[b], ref.size)
            assert np.array_equal(o["dsc"][b, :ref.size],
                                  o["scores"][b, ref]), b
        else:                                   # kept whole, nothing moves
            got = gather_logical(o["src"], pt[b], ref.size)
        assert got.tobytes() == rows[:, :, ref].tobytes(), b

    if mode == E.COMPACT_OUT_OF_PLACE:
        return
    i = run(mode)
    assert np.array_equal(i["status"], o["status"])
    assert np.array_equal(i["nk"], o["nk"]) and np.array_equal(i["keep"], o["keep"])
    assert i["state"].tobytes() == o["state"].tobytes()
    for b in range(B):
        n = int(o["nk"][b])
        ref_sc = o["dsc"][b, :n] if lengths[b] > K else o["scores"][b, :n]
        assert i["scores"][b, :n].tobytes() == ref_sc.tobytes(), b
        ref_rows = gather_logical(pool, pt[b], int(lengths[b]))[
            :, :, o["keep"][b, :n]]
        got = gather_logical(i["src"], i["pt"][b], n)
        assert got.tobytes() == ref_rows.tobytes(), b
