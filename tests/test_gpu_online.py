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


def _score_stream(E, cfg, hid, chunks):
    """Score a [n_band][B][T][D] stream cut into the given chunk sizes;
    returns (scores [B][T], final state bytes)."""
    import torch
    nb, B, T, D = hid.shape
    hd = dev(hid)
    st = [torch.zeros(E.state_bytes(cfg), dtype=torch.uint8, device="cuda")
          for _ in range(2)]
    E.epikv_state_init(cfg, st[0])
    scores = torch.zeros((B, T), device="cuda")
    t0 = 0
    for C in chunks:
        sig = torch.zeros((nb, B, C), device="cuda")
        # rows t0..t0+C-1 of every sequence: [nb][B][T][D] with ld_seq = T*D
        hidden = [hd[l, :, t0:] for l in range(nb)]
        E.epikv_score(cfg, C, hidden, D, T * D, state_in=st[0],
                      state_out=st[1], sig=sig)
        n_cached = dev(np.full(B, t0 + C, np.int32))
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
        err = np.abs(ref_s[b] - s64) / np.maximum(1.0, np.abs(s64))
        assert err.max() <= 1e-3


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
        assert np.max(np.abs(s1[b] - s64) / np.maximum(1.0, np.abs(s64))) \
            <= 1e-3
