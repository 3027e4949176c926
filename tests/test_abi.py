"""The C-ABI library on the CPU: it loads, exports every function the header
declares, and rejects invalid arguments on the host before anything is
enqueued (no call here reaches a kernel launch, so no GPU is needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "epikv.h")


@pytest.fixture(scope="module")
def E():
    from paper_2606_26472_amd import epikv
    epikv.lib()
    return epikv


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(epikv_\w+)\s*\(", text)))


def test_header_declares_the_step_entry_points():
    names = declared_functions()
    for n in ("epikv_score", "epikv_zscore", "epikv_select", "epikv_compact",
              "epikv_evict_step"):
        assert n in names


def test_library_exports_every_declared_function(E):
    L = E.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    assert set(declared_functions()) == set(E.EXPORTED)


def test_only_the_c_abi_is_exported():
    import subprocess
    from paper_2606_26472_amd import epikv
    out = subprocess.run(["nm", "-D", "--defined-only", epikv.LIB_PATH],
                         capture_output=True, text=True).stdout
    syms = {l.split()[-1] for l in out.splitlines() if l.strip()}
    ours = {s for s in syms if s.startswith("epikv_")}
    assert ours == set(declared_functions())
    # no C++ (mangled) symbols leak out of the library
    assert not [s for s in syms if s.startswith("_Z")]


def test_default_cfg_is_the_papers_setting(E):
    c = E.default_cfg()
    assert (c.n_layers, c.hidden, c.n_kv_heads, c.head_dim) == (32, 4096, 8, 128)
    assert (c.n_band_a, c.n_band_b, c.window) == (7, 8, 64)
    assert abs(c.ema_alpha - 0.9) < 1e-7
    assert c.recent == -1 and c.page_size == 16
    assert abs(c.eps - 1e-6) < 1e-12
    assert E.check_cfg(c) == 0


@pytest.mark.parametrize("field,value,code", [
    ("window", 0, -3), ("window", 257, -3), ("eps", -1.0, -3),
    ("eps", float("nan"), -3), ("budget", 0, -3), ("recent", -2, -3),
    ("signal", 5, -3), ("smoothing", 9, -3), ("batch", 0, -2),
    ("hidden", 4100, -2), ("hidden", 0, -2), ("head_dim", 96, -2),
    ("n_kv_heads", 0, -2), ("n_band_a", 0, -2), ("n_band_b", 30, -2),
    ("page_size", 0, -2), ("page_size", 2048, -2), ("n_layers", 0, -2),
    ("ema_alpha", 1.5, -3), ("ema_alpha", -0.1, -3), ("smoothing", 4, -3)])
def test_check_cfg_rejects(E, field, value, code):
    c = E.default_cfg()
    setattr(c, field, value)
    assert E.check_cfg(c) == code
    assert E.state_bytes(c) == 0
    assert E.workspace_bytes(c, 128) == 0


def test_check_cfg_null(E):
    assert E.lib().epikv_check_cfg(None) == E.EPIKV_EINVAL_NULL
    assert E.lib().epikv_default_cfg(None) == E.EPIKV_EINVAL_NULL


def test_state_layout_sizes(E):
    c = E.default_cfg(batch=32)
    off = E.state_layout(c)
    assert len(off) == 5
    assert off[0] == 0 and all(o % 256 == 0 for o in off)
    assert E.state_bytes(c) - off[4] >= 4 * 32 * 15
    assert off[2] - off[1] >= 4 * 32 * 15 * 63
    assert off[3] - off[2] >= 2 * 32 * 15 * 4096
    lag = E.default_cfg(batch=8, signal=E.SIGNAL_LAGKV)
    off = E.state_layout(lag)
    assert off[3] == off[2]                # no h_prev section
    assert off[4] - off[3] >= 4 * 2 * 8 * 32 * 2 * 8 * 128
    assert E.workspace_bytes(c, 128) >= 4 * 15 * 32 * 128
    assert E.workspace_bytes(lag, 256) >= 4 * 8 * 256 + 4 * 8 * 64 * 256
    assert E.workspace_bytes(c, -1) == 0
    # a step that only selects and compacts needs the compaction's scratch
    # and, for batches of up to 128 sequences (the selection may then split
    # a sequence over several workgroups), per sequence a 256-byte head and
    # three 2048-bin histograms plus two words for each of up to 256
    # workgroups
    sel = 32 * (256 + 3 * 2048 * 4) + 256 * 8
    assert E.select_workspace_bytes(c) == sel
    assert E.workspace_bytes(c, 0) == E.compact_workspace_bytes(c) + sel
    big = E.default_cfg(batch=129)
    assert E.workspace_bytes(big, 0) == E.compact_workspace_bytes(big)
    # records, per-sequence info, four page arrays per sequence
    assert E.compact_workspace_bytes(c) == 16 * 32 * 4096 + 256 + 16 * 32 * 256
    assert E.workspace_bytes(c, 128) >= E.compact_workspace_bytes(c) \
        + 4 * 15 * 32 * 128


def test_strerror_covers_every_code(E):
    for code in range(-7, 1):
        assert E.strerror(code) != "unknown status"
    assert E.strerror(-99) == "unknown status"


# Fake device addresses: aligned, never dereferenced (every call below fails
# validation on the host).  On a machine with a GPU these calls are skipped:
# a validation bug there would launch a kernel on addresses that do not
# exist.
A = 1 << 20


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:
        return True


host_only = pytest.mark.skipif(not _no_gpu(),
                               reason="fake-pointer validation runs only "
                                      "without a GPU")


@host_only
def test_score_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, n_band_a=1, n_band_b=1)
    hid = (ctypes.c_void_p * 2)(A, A + 4096)
    f = L.epikv_score
    # null state / sig
    assert f(ctypes.byref(c), 8, hid, 4096, 8 * 4096, None, None, 0, None,
             None, A, A, None, 0, None) == E.EPIKV_EINVAL_NULL
    # chunk < 1
    assert f(ctypes.byref(c), 0, hid, 4096, 8 * 4096, None, None, 0, None,
             A, 2 * A, 3 * A, None, 0, None) == E.EPIKV_EINVAL_SHAPE
    # state_in == state_out
    assert f(ctypes.byref(c), 8, hid, 4096, 8 * 4096, None, None, 0, None,
             A, A, 3 * A, None, 0, None) == E.EPIKV_EALIAS
    # misaligned hidden pointer
    bad = (ctypes.c_void_p * 2)(A, A + 2)
    assert f(ctypes.byref(c), 8, bad, 4096, 8 * 4096, None, None, 0, None,
             A, 8 * A, 3 * A, None, 0, None) == E.EPIKV_EALIGN
    # leading dimension not a multiple of 8
    assert f(ctypes.byref(c), 8, hid, 4100, 8 * 4100, None, None, 0, None,
             A, 8 * A, 3 * A, None, 0, None) == E.EPIKV_EALIGN
    # rows overlapping (ld_tok < D)
    assert f(ctypes.byref(c), 8, hid, 1024, 8 * 4096, None, None, 0, None,
             A, 8 * A, 3 * A, None, 0, None) == E.EPIKV_EINVAL_SHAPE
    # a null band pointer
    nul = (ctypes.c_void_p * 2)(A, None)
    assert f(ctypes.byref(c), 8, nul, 4096, 8 * 4096, None, None, 0, None,
             A, 8 * A, 3 * A, None, 0, None) == E.EPIKV_EINVAL_NULL
    # Lag-KV without a pool, then without workspace
    lag = E.default_cfg(batch=2, signal=E.SIGNAL_LAGKV)
    assert f(ctypes.byref(lag), 8, None, 0, 0, None, A, 4, A, A, 8 * A,
             3 * A, None, 0, None) == E.EPIKV_EINVAL_NULL
    pool = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    assert f(ctypes.byref(lag), 8, None, 0, 0, ctypes.byref(pool), A, 4, A,
             A, 8 * A, 3 * A, None, 0, None) == E.EPIKV_EWORKSPACE
    misal = E.Pool(A, 1 << 30, (1 << 29) + 8, 32768, 100)
    assert f(ctypes.byref(lag), 8, None, 0, 0, ctypes.byref(misal), A, 4, A,
             A, 8 * A, 3 * A, 9 * A, 1 << 20, None) == E.EPIKV_EALIGN
    # a long chunk needs more workspace (per-plane sums of every token)
    assert f(ctypes.byref(lag), 4096, None, 0, 0, ctypes.byref(pool), A, 4,
             A, A, 8 * A, 3 * A, 9 * A, 1 << 20, None) == E.EPIKV_EWORKSPACE


@host_only
def test_zscore_select_compact_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    z = L.epikv_zscore
    assert z(ctypes.byref(c), 8, None, A, A, 8 * A, A, 100, None,
             None) == E.EPIKV_EINVAL_NULL
    assert z(ctypes.byref(c), 8, A, A, A, 8 * A, A, 4, None,
             None) == E.EPIKV_EINVAL_SHAPE            # ld_s < chunk
    assert z(ctypes.byref(c), 8, A, A, A, A + 256, A, 100, None,
             None) == E.EPIKV_EALIAS
    s = L.epikv_select
    assert s(ctypes.byref(c), A, 100, A, A, None, A, A,
             None) == E.EPIKV_EINVAL_NULL
    assert s(ctypes.byref(c), A, 0, A, A, A, A, A,
             None) == E.EPIKV_EINVAL_SHAPE
    # the split selection: workspace missing, too small, misaligned, or
    # overlapping an output (scores at A, the outputs at 2A..)
    sw = L.epikv_select_ws
    nws = E.select_workspace_bytes(c)
    assert nws == 2 * (256 + 3 * 2048 * 4) + 256 * 8
    W = 8 * A
    assert sw(ctypes.byref(c), A, 100, A, A, 2 * A, 3 * A, 4 * A, None, 0,
              None) == E.EPIKV_EWORKSPACE
    assert sw(ctypes.byref(c), A, 100, A, A, 2 * A, 3 * A, 4 * A, W,
              nws - 1, None) == E.EPIKV_EWORKSPACE
    assert sw(ctypes.byref(c), A, 100, A, A, 2 * A, 3 * A, 4 * A, W + 4,
              nws, None) == E.EPIKV_EALIGN
    assert sw(ctypes.byref(c), A, 100, 5 * A, 6 * A, 2 * A, 3 * A, 4 * A,
              2 * A + 256, nws, None) == E.EPIKV_EALIAS
    assert sw(ctypes.byref(c), A, 0, A, A, A, A, A, W, nws,
              None) == E.EPIKV_EINVAL_SHAPE
    assert E.select_workspace_bytes(E.default_cfg(batch=129)) == 0
    cp = L.epikv_compact
    src = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    dst = E.Pool(2 * A, 1 << 30, 1 << 29, 32768, 100)
    bad = E.Pool(None, 0, 0, 0, 0)
    W = 4 * A
    assert cp(ctypes.byref(c), ctypes.byref(bad), A, 4, ctypes.byref(dst), A,
              16, A, A, None, None, None, None, 0, None, W, 1 << 20,
              None) == E.EPIKV_EINVAL_NULL
    # workspace missing, too small, misaligned
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              16, A, A, None, None, None, None, 0, None, None, 0,
              None) == E.EPIKV_EWORKSPACE
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              16, A, A, None, None, None, None, 0, None, W, 64,
              None) == E.EPIKV_EWORKSPACE
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              16, A, A, None, None, None, None, 0, None, W + 8, 1 << 20,
              None) == E.EPIKV_EALIGN
    # destination page table narrower than ceil(K / page_size)
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              15, A, A, None, None, None, None, 0, None, W, 1 << 20,
              None) == E.EPIKV_EINVAL_SHAPE
    # scores given on one side only
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              16, A, A, A, None, None, None, 100, None, W, 1 << 20,
              None) == E.EPIKV_EINVAL_NULL
    # in-place score compaction
    assert cp(ctypes.byref(c), ctypes.byref(src), A, 4, ctypes.byref(dst), A,
              16, A, A, A, A + 64, None, None, 100, None, W, 1 << 20,
              None) == E.EPIKV_EALIAS


@host_only
def test_evict_step_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    io = E.StepIO()
    assert L.epikv_evict_step(ctypes.byref(c), None, None) == \
        E.EPIKV_EINVAL_NULL
    io.chunk = 64
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EWORKSPACE
    io.workspace = A
    io.workspace_bytes = 16
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EWORKSPACE
    io.workspace_bytes = 1 << 20
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL                        # no state
    io.chunk = -1
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_SHAPE
    io.chunk = 0                                   # select + compact only:
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL                        # no state needed, no scores


def _valid_io(E, A):
    """A step description whose pointers are aligned fake addresses."""
    io = E.StepIO()
    io.chunk = 64
    hid = (ctypes.c_void_p * 15)(*[A * (i + 2) for i in range(15)])
    io._keep = hid
    io.hidden = ctypes.cast(hid, ctypes.POINTER(ctypes.c_void_p))
    io.ld_tok, io.ld_seq = 4096, 64 * 4096
    io.n_cached = io.n_prefix = A
    io.src = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    io.dst = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    io.src_pt = io.dst_pt = A
    io.ld_src_pt, io.ld_dst_pt = 64, 16
    io.scores = 64 * A
    io.ld_s = 1024
    io.state_in, io.state_out = 128 * A, 256 * A
    io.keep_idx = io.n_keep = io.seq_status = A
    io.workspace = 512 * A
    io.workspace_bytes = 1 << 30
    return io


@host_only
def test_evict_step_without_scoring_skips_the_scorer_checks(E):
    """chunk = 0: hidden states and scorer state are not used, so a state
    pair that would be refused for a scoring step is not looked at; the
    selection's arguments still are."""
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    io = _valid_io(E, A)
    io.state_out = io.state_in
    io.n_prefix = None
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS                   # scoring step: the state pair
    io.chunk = 0
    io.hidden = None
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL              # no scoring: the missing n_prefix


@host_only
def test_evict_step_scores_copy_is_optional(E):
    """Without dst_scores the step must not demand a score pair; the first
    error it finds in this description is the missing n_prefix."""
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    io = _valid_io(E, A)
    io.n_prefix = None
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL
    io = _valid_io(E, A)
    io.dst_pos = A                       # positions on one side only
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL
    io = _valid_io(E, A)
    io.state_out = io.state_in           # state must not be updated in place
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS
    io = _valid_io(E, A)
    io.workspace = io.state_in           # workspace overlapping the state
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS


@host_only
def test_compact_inplace_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    f = L.epikv_compact_inplace
    pool = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    bad = E.Pool(None, 0, 0, 0, 0)
    W = 4 * A
    n = E.compact_workspace_bytes(c)
    assert n == 16 * 2 * 256 + 256 + 512  # records, info, page arrays
    assert f(ctypes.byref(c), ctypes.byref(bad), A, 4, A, A, None, None, 0,
             None, W, n, None) == E.EPIKV_EINVAL_NULL
    assert f(ctypes.byref(c), ctypes.byref(pool), None, 4, A, A, None, None,
             0, None, W, n, None) == E.EPIKV_EINVAL_NULL
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A, A, None, None, 0,
             None, W, n - 1, None) == E.EPIKV_EWORKSPACE
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A, A, None, None, 0,
             None, W + 8, n, None) == E.EPIKV_EALIGN
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 0, A, A, None, None, 0,
             None, W, n, None) == E.EPIKV_EINVAL_SHAPE      # ld_pt < 1
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A, A, A, None, 0,
             None, W, n, None) == E.EPIKV_EINVAL_SHAPE      # scores, ld_s 0
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A, A, A, A + 64, 100,
             None, W, n, None) == E.EPIKV_EALIAS            # scores on pos


@host_only
def test_compact_remap_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    f = L.epikv_compact_remap
    pool = E.Pool(A, 1 << 30, 1 << 29, 32768, 100)
    W = 4 * A
    n = E.compact_workspace_bytes(c)
    assert f(ctypes.byref(c), ctypes.byref(pool), None, 4, A, A, None, None,
             0, None, W, n, None) == E.EPIKV_EINVAL_NULL
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A, A, None, None, 0,
             None, W, n - 1, None) == E.EPIKV_EWORKSPACE
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 0, A, A, None, None, 0,
             None, W, n, None) == E.EPIKV_EINVAL_SHAPE      # ld_pt < 1
    # the table is rewritten: it may overlap neither keep_idx nor workspace
    assert f(ctypes.byref(c), ctypes.byref(pool), A, 4, A + 16, A, None,
             None, 0, None, W, n, None) == E.EPIKV_EALIAS
    assert f(ctypes.byref(c), ctypes.byref(pool), W + 256, 4, A, A, None,
             None, 0, None, W, n, None) == E.EPIKV_EALIAS
    assert f(ctypes.byref(c), ctypes.byref(pool), 2 * A, 4, A, 2 * A + 8,
             None, None, 0, None, W, n, None) == E.EPIKV_EALIAS  # n_keep


@host_only
def test_evict_step_in_place_validation(E):
    L = E.lib()
    c = E.default_cfg(batch=2, budget=256)
    io = _valid_io(E, A)
    io.in_place = 1
    io.dst_scores = 96 * A               # in place the scores move in place
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS
    io = _valid_io(E, A)
    io.in_place = 1
    io.src_pos, io.dst_pos = 32 * A, 48 * A   # positions must be one array
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS
    io = _valid_io(E, A)
    io.in_place = 3                      # not a compaction mode
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_PARAM
    io = _valid_io(E, A)
    io.in_place = E.COMPACT_REMAP        # the rewritten table on keep_idx
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EALIAS
    io = _valid_io(E, A)
    io.in_place = 1
    io.n_prefix = None                   # the earlier stages still check
    assert L.epikv_evict_step(ctypes.byref(c), ctypes.byref(io), None) == \
        E.EPIKV_EINVAL_NULL


@host_only
def test_score_tokens_validation(E):
    L = E.lib()
    f = L.epikv_score_tokens
    c = E.default_cfg(batch=2, n_band_a=1, n_band_b=1)
    hid = (ctypes.c_void_p * 2)(A, A + 4096)
    ok = (ctypes.byref(c), 1, hid, 4096, 4096, A, 8 * A, 9 * A, 10 * A, 100,
          None)
    lag = E.default_cfg(batch=2, signal=E.SIGNAL_LAGKV)
    assert f(ctypes.byref(lag), *ok[1:]) == E.EPIKV_EINVAL_PARAM
    assert f(ok[0], 65, *ok[2:]) == E.EPIKV_EINVAL_SHAPE        # chunk > 64
    assert f(ok[0], 0, *ok[2:]) == E.EPIKV_EINVAL_SHAPE
    wide = E.default_cfg(batch=2, n_band_a=1, n_band_b=1, hidden=8192)
    assert f(ctypes.byref(wide), *ok[1:]) == E.EPIKV_EINVAL_SHAPE
    assert f(*ok[:8], None, *ok[9:]) == E.EPIKV_EINVAL_NULL      # no scores
    assert f(*ok[:5], None, *ok[6:]) == E.EPIKV_EINVAL_NULL      # no n_cached
    assert f(*ok[:9], 0, None) == E.EPIKV_EINVAL_SHAPE           # ld_s < chunk
    assert f(*ok[:7], 8 * A, *ok[8:]) == E.EPIKV_EALIAS          # state in place
