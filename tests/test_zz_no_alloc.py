"""epikv_evict_step_noalloc against epikv_evict_step.

The no-allocation entry point runs the same step with its scratch in the
library's per-GPU array instead of caller workspace.  Each case runs two
steps in a row through the C ABI, the second with a smaller input (fewer
sequences, a shorter chunk, a smaller budget), each on fresh copies of the
inputs, and compares every output of the no-allocation call with the one of
epikv_evict_step on the same inputs, byte for byte: the rebuilt cache,
kept positions, counts and statuses, written and compacted scores and
positions, the carried scorer state (and, page remapping, the rewritten
page table).  The array keeps the first call's contents, so the second call
also shows that nothing read from scratch survives from an earlier call.
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


def _inputs(E, g, signal, B, C, K, n_max):
    """Seeded inputs of one step: (cfg, host arrays)."""
    L, H, d, page, D, na, nb = 3, 8, 128, 16, 1024, 3, 2
    lengths = g.integers(C + 1, n_max + 1, size=B)
    lengths[0] = max(C, K // 2)            # a sequence with N <= K
    ld_s = int(lengths.max())
    if signal == "hs":
        cfg = E.default_cfg(batch=B, hidden=D, n_layers=L, n_band_a=na,
                            n_band_b=nb, budget=K)
    else:
        cfg = E.default_cfg(batch=B, n_layers=L, budget=K,
                            signal=E.SIGNAL_LAGKV, smoothing=E.SMOOTH_MEAN)
    src_pt, n_src = synth.page_tables(lengths, page, g)
    dst_pt, n_dst = synth.page_tables(np.full(B, K), page, g)
    sc = np.zeros((B, ld_s), np.float32)
    for b in range(B):
        sc[b, :lengths[b] - C] = synth.old_scores(g, int(lengths[b]) - C)
    h = dict(
        cfg=cfg, lengths=lengths, ld_s=ld_s, L=L, H=H, d=d, page=page, D=D,
        n_band=na + nb, src_pt=src_pt, dst_pt=dst_pt, n_src=n_src,
        n_dst=n_dst, scores=sc, C=C, K=K, B=B,
        pool=synth.random_bits16(g, (L, 2, n_src, page, H * d)),
        hidden=synth.f32_to_bf16_bits(
            (g.standard_normal((na + nb, B, C, D)) * 2).astype(np.float32)),
        prefix=np.where(np.arange(B) % 3 == 1, 5, 0).astype(np.int32),
        pos=np.tile(np.arange(ld_s, dtype=np.int32), (B, 1)))
    st = np.zeros(E.state_bytes(cfg), np.uint8)
    import torch
    sec = E.state_sections(cfg, torch.from_numpy(st))
    # a carried stream: n_tok > 0, a filled ring and h_prev (HS) or range
    sec["n_tok"][:] = torch.from_numpy((lengths - C).astype(np.int32))
    sec["ring"][:] = torch.from_numpy(
        (30 + g.standard_normal(tuple(sec["ring"].shape))).astype(np.float32))
    if signal == "hs":
        sec["h_prev"][:] = torch.from_numpy(synth.f32_to_bf16_bits(
            g.standard_normal(tuple(sec["h_prev"].shape)).astype(np.float32))
            .view(np.int16))
    else:
        rng = g.standard_normal(tuple(sec["range"].shape)).astype(np.float32)
        rng[1] = rng[0] + 2.0 + np.abs(rng[1])     # max above min
        sec["range"][:] = torch.from_numpy(rng)
    h["state"] = st
    return h


def _run(E, h, noalloc, mode):
    """One step on fresh device copies of the inputs; returns every output
    as host bytes."""
    import torch
    cfg, B, C, K = h["cfg"], h["B"], h["C"], h["K"]
    L, H, d, page, D = h["L"], h["H"], h["d"], h["page"], h["D"]
    src = dev(h["pool"])
    src_pt = dev(h["src_pt"])
    dst = torch.full((L, 2, h["n_dst"], page, H * d), 0x5A5A,
                     dtype=torch.int16, device="cuda")
    scores = dev(h["scores"])
    dsc = torch.full_like(scores, -3.0)
    pos = dev(h["pos"])
    dpos = torch.full_like(pos, -2)
    st_in = dev(h["state"])
    st_out = torch.zeros_like(st_in)
    keep = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    nk = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    status = torch.full((B,), 77, dtype=torch.int32, device="cuda")
    hid = dev(h["hidden"])
    hidden = [hid[l] for l in range(h["n_band"])] \
        if cfg.signal == E.SIGNAL_HS else None
    ws_n = E.workspace_bytes(cfg, C)
    ws = None if noalloc else torch.zeros(ws_n, dtype=torch.uint8,
                                          device="cuda")
    in_place = {"out_of_place": 0, "remap": E.COMPACT_REMAP}[mode]
    io = E.make_step_io(
        C, hidden, D, C * D, dev(h["lengths"].astype(np.int32)),
        dev(h["prefix"]), E.pool_of(src.view(L, 2, h["n_src"], page, H, d)),
        src_pt, h["src_pt"].shape[1],
        E.pool_of(dst.view(L, 2, h["n_dst"], page, H, d)), dev(h["dst_pt"]),
        h["dst_pt"].shape[1], scores, h["ld_s"], st_in, st_out, keep, nk,
        status, ws, 0 if noalloc else ws_n,
        dst_scores=None if in_place else dsc, src_pos=pos,
        dst_pos=pos if in_place else dpos, in_place=in_place)
    if noalloc:
        E.epikv_evict_step_noalloc(cfg, io)
    else:
        E.epikv_evict_step(cfg, io)
    torch.cuda.synchronize()
    out = dict(keep=keep, n_keep=nk, status=status, scores=scores,
               state=st_out, pos=pos, src_pool=src, src_pt=src_pt)
    if not in_place:
        out.update(dst_pool=dst, dst_scores=dsc, dst_pos=dpos)
    return {k: host(v).tobytes() for k, v in out.items()}, host(status)


def test_noalloc_call_sequence_of_changing_shapes(E):
    """Eight calls in a row on the one scratch array, each with another
    layout of it: batch sizes that grow as well as shrink (sequences whose
    selection scratch the previous call used for other data), chunks,
    budgets, signals and rebuild modes; each equal to the step on fresh
    workspace."""
    g = np.random.default_rng(20261209)
    for i in range(8):
        B = int(g.choice([1, 2, 3, 5, 8, 13]))
        C = int(g.choice([1, 16, 64]))
        K = int(g.choice([64, 256, 512]))
        n_max = int(max(C + 2, min(16000 // B, 4000)))
        signal = str(g.choice(["hs", "lagkv"]))
        mode = str(g.choice(["out_of_place", "remap"]))
        print(f"no-alloc call {i}: {signal} {mode} B={B} C={C} K={K} "
              f"n_max={n_max}", flush=True)
        h = _inputs(E, g, signal, B, C, K, n_max)
        ref, st_ref = _run(E, h, False, mode)
        got, _ = _run(E, h, True, mode)
        assert np.all(st_ref == 0), st_ref
        for k in ref:
            assert got[k] == ref[k], (i, k)


@pytest.mark.parametrize("signal,mode", [("hs", "out_of_place"),
                                         ("lagkv", "out_of_place"),
                                         ("hs", "remap")])
def test_noalloc_step_equals_step(E, signal, mode):
    g = synth.rng(4242 + len(signal) + len(mode))
    calls = [dict(B=6, C=64, K=512, n_max=2600),     # then a smaller input:
             dict(B=3, C=16, K=256, n_max=900)]
    for i, shape in enumerate(calls):
        print(f"no-alloc step {signal} {mode} call {i} {shape}", flush=True)
        h = _inputs(E, g, signal, **shape)
        ref, st_ref = _run(E, h, False, mode)
        got, _ = _run(E, h, True, mode)
        assert np.all(st_ref == 0), st_ref
        for k in ref:
            assert got[k] == ref[k], (i, k)


def test_noalloc_refuses_a_step_beyond_its_scratch(E):
    """A step that needs more than EPIKV_NOALLOC_SCRATCH_BYTES of scratch is
    refused on the host (EWORKSPACE) before anything is enqueued."""
    import torch
    B, C, K = 128, 4096, 512
    cfg = E.default_cfg(batch=B, budget=K)
    assert E.workspace_bytes(cfg, C) > (16 << 20)
    io = E.make_step_io(C, None, 0, 0, None, None, E.Pool(), None, 1,
                        E.Pool(), None, 1, None, 1, None, None, None, None,
                        None, None, 0)
    with pytest.raises(E.EpikvError) as ex:
        E.epikv_evict_step_noalloc(cfg, io)
    assert ex.value.status == E.EPIKV_EWORKSPACE
    torch.cuda.synchronize()
