"""Python binding of libepikv.so (ctypes).

Argument marshalling only: every step of the eviction path runs in the HIP
kernels behind the C ABI declared in include/epikv.h.  torch tensors supply
device memory (``data_ptr``) and the current HIP stream.  The library must be
built (``python -m paper_2606_26472_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# EPIKV_LIB selects another build of the same library (e.g. the host-ASan
# one); a missing file is an error like a missing default build.
LIB_PATH = os.environ.get("EPIKV_LIB") or os.path.join(_HERE, "libepikv.so")

# status codes (include/epikv.h)
EPIKV_OK = 0
EPIKV_EINVAL_NULL = -1
EPIKV_EINVAL_SHAPE = -2
EPIKV_EINVAL_PARAM = -3
EPIKV_EALIGN = -4
EPIKV_EWORKSPACE = -5
EPIKV_EALIAS = -6
EPIKV_ELAUNCH = -7

SEQ_OK = 0
SEQ_BUDGET = 1
SEQ_RANGE = 2
SEQ_SYNC = 3
COMPACT_OUT_OF_PLACE, COMPACT_IN_PLACE, COMPACT_REMAP = 0, 1, 2

SIGNAL_HS = 0
SIGNAL_LAGKV = 1
SIGNAL_KV_KEY = 2
SIGNAL_KV_VAL = 3
SIGNAL_LAGKV_KEY = 4
SMOOTH_Z = 0
SMOOTH_MEAN = 1
SMOOTH_RAW = 2
SMOOTH_EMA = 3
MAX_BAND = 32

EXPORTED = ("epikv_default_cfg", "epikv_strerror", "epikv_check_cfg",
            "epikv_state_bytes", "epikv_state_layout",
            "epikv_workspace_bytes", "epikv_compact_workspace_bytes",
            "epikv_state_init", "epikv_score", "epikv_score_tokens",
            "epikv_zscore", "epikv_select", "epikv_select_workspace_bytes",
            "epikv_select_ws", "epikv_compact",
            "epikv_compact_inplace", "epikv_compact_remap",
            "epikv_evict_step", "epikv_evict_step_noalloc")


class EpikvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} (status {status})")


class Cfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("n_band_a", ctypes.c_int32), ("n_band_b", ctypes.c_int32),
                ("window", ctypes.c_int32), ("eps", ctypes.c_float),
                ("signal", ctypes.c_int32), ("smoothing", ctypes.c_int32),
                ("budget", ctypes.c_int32), ("recent", ctypes.c_int32),
                ("ema_alpha", ctypes.c_float)]


class Pool(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("stride_layer", ctypes.c_int64),
                ("stride_kv", ctypes.c_int64), ("stride_page", ctypes.c_int64),
                ("n_pages", ctypes.c_int64)]


class StepIO(ctypes.Structure):
    _fields_ = [("chunk", ctypes.c_int32),
                ("hidden", ctypes.POINTER(ctypes.c_void_p)),
                ("ld_tok", ctypes.c_int64), ("ld_seq", ctypes.c_int64),
                ("n_cached", ctypes.c_void_p), ("n_prefix", ctypes.c_void_p),
                ("src", Pool), ("src_pt", ctypes.c_void_p),
                ("ld_src_pt", ctypes.c_int64),
                ("dst", Pool), ("dst_pt", ctypes.c_void_p),
                ("ld_dst_pt", ctypes.c_int64),
                ("scores", ctypes.c_void_p), ("dst_scores", ctypes.c_void_p),
                ("src_pos", ctypes.c_void_p), ("dst_pos", ctypes.c_void_p),
                ("ld_s", ctypes.c_int64),
                ("state_in", ctypes.c_void_p), ("state_out", ctypes.c_void_p),
                ("keep_idx", ctypes.c_void_p), ("n_keep", ctypes.c_void_p),
                ("seq_status", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t),
                ("in_place", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libepikv.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build the HIP library first "
            "(python -m paper_2606_26472_amd.build)")
    # The device buffers handed to the library are torch's, and the torch
    # wheel carries its own HIP runtime under the same soname as the
    # system's (libamdhip64.so.7).  Importing torch first makes the library
    # bind to that runtime; opened first, it would bring in the system copy
    # as a second runtime, whose launches fail on torch's allocations.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    cfgp = ctypes.POINTER(Cfg)
    poolp = ctypes.POINTER(Pool)
    sig = {
        "epikv_default_cfg": (ctypes.c_int, [cfgp]),
        "epikv_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "epikv_check_cfg": (ctypes.c_int, [cfgp]),
        "epikv_state_bytes": (sz, [cfgp]),
        "epikv_state_layout": (ctypes.c_int, [cfgp, ctypes.POINTER(sz)]),
        "epikv_workspace_bytes": (sz, [cfgp, i32]),
        "epikv_compact_workspace_bytes": (sz, [cfgp]),
        "epikv_state_init": (ctypes.c_int, [cfgp, P, P]),
        "epikv_score": (ctypes.c_int, [cfgp, i32, ctypes.POINTER(P), i64, i64,
                                       poolp, P, i64, P, P, P, P, P, sz, P]),
        "epikv_zscore": (ctypes.c_int, [cfgp, i32, P, P, P, P, P, i64, P, P]),
        "epikv_score_tokens": (ctypes.c_int, [cfgp, i32, ctypes.POINTER(P), i64,
                                              i64, P, P, P, P, i64, P]),
        "epikv_select": (ctypes.c_int, [cfgp, P, i64, P, P, P, P, P, P]),
        "epikv_select_workspace_bytes": (sz, [cfgp]),
        "epikv_select_ws": (ctypes.c_int, [cfgp, P, i64, P, P, P, P, P, P,
                                           sz, P]),
        "epikv_compact": (ctypes.c_int, [cfgp, poolp, P, i64, poolp, P, i64,
                                         P, P, P, P, P, P, i64, P, P, sz, P]),
        "epikv_compact_inplace": (ctypes.c_int, [cfgp, poolp, P, i64, P, P,
                                                 P, P, i64, P, P, sz, P]),
        "epikv_compact_remap": (ctypes.c_int, [cfgp, poolp, P, i64, P, P,
                                               P, P, i64, P, P, sz, P]),
        "epikv_evict_step": (ctypes.c_int, [cfgp, ctypes.POINTER(StepIO), P]),
        "epikv_evict_step_noalloc": (ctypes.c_int,
                                     [cfgp, ctypes.POINTER(StepIO), P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def strerror(status: int) -> str:
    return lib().epikv_strerror(int(status)).decode()


def _check(status: int, where: str):
    if status != EPIKV_OK:
        raise EpikvError(status, where)


def _ptr(t):
    """Device (or host) address of a tensor, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _ws(t, nbytes):
    """Address of a workspace tensor, refusing one smaller than the size
    that will be declared to the library (it would write past its end)."""
    if t is not None and not isinstance(t, int):
        have = t.numel() * t.element_size()
        if have < int(nbytes):
            raise ValueError(f"workspace tensor holds {have} bytes, "
                             f"{int(nbytes)} declared")
    return _ptr(t)


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# Configuration and sizes
# ---------------------------------------------------------------------------
def default_cfg(**overrides) -> Cfg:
    c = Cfg()
    _check(lib().epikv_default_cfg(ctypes.byref(c)), "epikv_default_cfg")
    for k, v in overrides.items():
        setattr(c, k, v)
    return c


def check_cfg(cfg: Cfg) -> int:
    return lib().epikv_check_cfg(ctypes.byref(cfg))


def state_bytes(cfg: Cfg) -> int:
    return int(lib().epikv_state_bytes(ctypes.byref(cfg)))


def state_layout(cfg: Cfg):
    off = (ctypes.c_size_t * 5)()
    _check(lib().epikv_state_layout(ctypes.byref(cfg), off),
           "epikv_state_layout")
    return [int(x) for x in off]


def workspace_bytes(cfg: Cfg, chunk: int) -> int:
    return int(lib().epikv_workspace_bytes(ctypes.byref(cfg), int(chunk)))


def compact_workspace_bytes(cfg: Cfg) -> int:
    return int(lib().epikv_compact_workspace_bytes(ctypes.byref(cfg)))


def select_workspace_bytes(cfg: Cfg) -> int:
    return int(lib().epikv_select_workspace_bytes(ctypes.byref(cfg)))


def pool_of(t) -> Pool:
    """epikv_pool describing a tensor laid out [L][2][n_pages][page][H][d]."""
    es = t.element_size()
    L, two, n_pages = t.shape[0], t.shape[1], t.shape[2]
    assert two == 2
    s = t.stride()
    return Pool(t.data_ptr(), s[0] * es, s[1] * es, s[2] * es, n_pages)


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def epikv_state_init(cfg: Cfg, state, stream=None):
    _check(lib().epikv_state_init(ctypes.byref(cfg), _ptr(state),
                                  _stream(stream)), "epikv_state_init")


def _hidden_array(hidden):
    if hidden is None:
        return None
    arr = (ctypes.c_void_p * len(hidden))(*[_ptr(h) for h in hidden])
    return arr


def epikv_score(cfg: Cfg, chunk: int, hidden=None, ld_tok=0, ld_seq=0,
                pool: Pool | None = None, page_table=None, ld_pt=0,
                n_cached=None, state_in=None, state_out=None, sig=None,
                workspace=None, workspace_bytes_=0, stream=None):
    arr = _hidden_array(hidden)
    _check(lib().epikv_score(
        ctypes.byref(cfg), int(chunk), arr, int(ld_tok), int(ld_seq),
        ctypes.byref(pool) if pool is not None else None, _ptr(page_table),
        int(ld_pt), _ptr(n_cached), _ptr(state_in), _ptr(state_out),
        _ptr(sig), _ws(workspace, workspace_bytes_), int(workspace_bytes_),
        _stream(stream)),
        "epikv_score")


def epikv_zscore(cfg: Cfg, chunk: int, sig, n_cached, state_in, state_out,
                 scores, ld_s, smoothed=None, stream=None):
    _check(lib().epikv_zscore(
        ctypes.byref(cfg), int(chunk), _ptr(sig), _ptr(n_cached),
        _ptr(state_in), _ptr(state_out), _ptr(scores), int(ld_s),
        _ptr(smoothed), _stream(stream)), "epikv_zscore")


def epikv_score_tokens(cfg: Cfg, chunk: int, hidden, ld_tok, ld_seq, n_cached,
                       state_in, state_out, scores, ld_s, stream=None):
    arr = _hidden_array(hidden)
    _check(lib().epikv_score_tokens(
        ctypes.byref(cfg), int(chunk), arr, int(ld_tok), int(ld_seq),
        _ptr(n_cached), _ptr(state_in), _ptr(state_out), _ptr(scores),
        int(ld_s), _stream(stream)), "epikv_score_tokens")


def epikv_select(cfg: Cfg, scores, ld_s, n_cached, n_prefix, keep_idx,
                 n_keep, seq_status, stream=None):
    _check(lib().epikv_select(
        ctypes.byref(cfg), _ptr(scores), int(ld_s), _ptr(n_cached),
        _ptr(n_prefix), _ptr(keep_idx), _ptr(n_keep), _ptr(seq_status),
        _stream(stream)), "epikv_select")


def epikv_select_ws(cfg: Cfg, scores, ld_s, n_cached, n_prefix, keep_idx,
                    n_keep, seq_status, workspace=None, workspace_bytes_=0,
                    stream=None):
    _check(lib().epikv_select_ws(
        ctypes.byref(cfg), _ptr(scores), int(ld_s), _ptr(n_cached),
        _ptr(n_prefix), _ptr(keep_idx), _ptr(n_keep), _ptr(seq_status),
        _ws(workspace, workspace_bytes_), int(workspace_bytes_),
        _stream(stream)),
        "epikv_select_ws")


def epikv_compact(cfg: Cfg, src: Pool, src_pt, ld_src_pt, dst: Pool, dst_pt,
                  ld_dst_pt, keep_idx, n_keep, src_scores=None,
                  dst_scores=None, src_pos=None, dst_pos=None, ld_s=0,
                  seq_status=None, workspace=None, workspace_bytes_=0,
                  stream=None):
    _check(lib().epikv_compact(
        ctypes.byref(cfg), ctypes.byref(src), _ptr(src_pt), int(ld_src_pt),
        ctypes.byref(dst), _ptr(dst_pt), int(ld_dst_pt), _ptr(keep_idx),
        _ptr(n_keep), _ptr(src_scores), _ptr(dst_scores), _ptr(src_pos),
        _ptr(dst_pos), int(ld_s), _ptr(seq_status),
        _ws(workspace, workspace_bytes_), int(workspace_bytes_),
        _stream(stream)),
        "epikv_compact")


def epikv_compact_inplace(cfg: Cfg, pool: Pool, page_table, ld_pt, keep_idx,
                          n_keep, scores=None, pos=None, ld_s=0,
                          seq_status=None, workspace=None, workspace_bytes_=0,
                          stream=None):
    _check(lib().epikv_compact_inplace(
        ctypes.byref(cfg), ctypes.byref(pool), _ptr(page_table), int(ld_pt),
        _ptr(keep_idx), _ptr(n_keep), _ptr(scores), _ptr(pos), int(ld_s),
        _ptr(seq_status), _ws(workspace, workspace_bytes_), int(workspace_bytes_),
        _stream(stream)), "epikv_compact_inplace")


def epikv_compact_remap(cfg: Cfg, pool: Pool, page_table, ld_pt, keep_idx,
                        n_keep, scores=None, pos=None, ld_s=0,
                        seq_status=None, workspace=None, workspace_bytes_=0,
                        stream=None):
    _check(lib().epikv_compact_remap(
        ctypes.byref(cfg), ctypes.byref(pool), _ptr(page_table), int(ld_pt),
        _ptr(keep_idx), _ptr(n_keep), _ptr(scores), _ptr(pos), int(ld_s),
        _ptr(seq_status), _ws(workspace, workspace_bytes_), int(workspace_bytes_),
        _stream(stream)), "epikv_compact_remap")


def make_step_io(chunk, hidden, ld_tok, ld_seq, n_cached, n_prefix,
                 src: Pool, src_pt, ld_src_pt, dst: Pool, dst_pt, ld_dst_pt,
                 scores, ld_s, state_in, state_out, keep_idx, n_keep,
                 seq_status, workspace, workspace_bytes_, dst_scores=None,
                 src_pos=None, dst_pos=None, in_place=False) -> StepIO:
    """Build the epikv_step_io struct.  The returned object holds references
    to every tensor (and the hidden pointer array) it was built from, so a
    temporary passed here cannot be freed while the struct is in use."""
    io = StepIO()
    io._tensors_keepalive = [n_cached, n_prefix, src_pt, dst_pt, scores,
                             state_in, state_out, keep_idx, n_keep,
                             seq_status, workspace, dst_scores, src_pos,
                             dst_pos, hidden]
    io.chunk = int(chunk)
    arr = _hidden_array(hidden)
    io._hidden_keepalive = arr
    io.hidden = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)) \
        if arr is not None else None
    io.ld_tok, io.ld_seq = int(ld_tok), int(ld_seq)
    io.n_cached, io.n_prefix = _ptr(n_cached), _ptr(n_prefix)
    io.src, io.src_pt, io.ld_src_pt = src, _ptr(src_pt), int(ld_src_pt)
    io.dst, io.dst_pt, io.ld_dst_pt = dst, _ptr(dst_pt), int(ld_dst_pt)
    io.scores, io.dst_scores = _ptr(scores), _ptr(dst_scores)
    io.src_pos, io.dst_pos = _ptr(src_pos), _ptr(dst_pos)
    io.ld_s = int(ld_s)
    io.state_in, io.state_out = _ptr(state_in), _ptr(state_out)
    io.keep_idx, io.n_keep = _ptr(keep_idx), _ptr(n_keep)
    io.seq_status = _ptr(seq_status)
    io.workspace = _ws(workspace, workspace_bytes_)
    io.workspace_bytes = int(workspace_bytes_)
    io.in_place = int(in_place)   # False/True, or a COMPACT_* mode
    return io


def epikv_evict_step(cfg: Cfg, io: StepIO, stream=None):
    _check(lib().epikv_evict_step(ctypes.byref(cfg), ctypes.byref(io),
                                  _stream(stream)), "epikv_evict_step")


def epikv_evict_step_noalloc(cfg: Cfg, io: StepIO, stream=None):
    """epikv_evict_step with the library's per-GPU scratch array
    (io.workspace is ignored)."""
    _check(lib().epikv_evict_step_noalloc(ctypes.byref(cfg), ctypes.byref(io),
                                          _stream(stream)),
           "epikv_evict_step_noalloc")


# ---------------------------------------------------------------------------
# State buffer views (the documented layout of include/epikv.h)
# ---------------------------------------------------------------------------
def n_sig(cfg: Cfg) -> int:
    return cfg.n_band_a + cfg.n_band_b if cfg.signal == SIGNAL_HS else 1


def state_sections(cfg: Cfg, state):
    """Typed views of a uint8 state tensor (CPU or device):
    dict(n_tok [B] int32, ring [B][n_sig][w-1] float32, ema [B][n_sig],
         h_prev [B][n_band][D] int16 (HS), range [2][B][L][2][H][d] float32
         (lag-normalised KV signals))."""
    import torch
    off = state_layout(cfg)
    B, w = cfg.batch, cfg.window
    out = {}
    out["n_tok"] = state[off[0]:off[0] + 4 * B].view(torch.int32)
    nr = B * n_sig(cfg) * (w - 1)
    out["ring"] = state[off[1]:off[1] + 4 * nr].view(torch.float32).view(
        B, n_sig(cfg), w - 1)
    if cfg.signal == SIGNAL_HS:
        nb = cfg.n_band_a + cfg.n_band_b
        nh = B * nb * cfg.hidden
        out["h_prev"] = state[off[2]:off[2] + 2 * nh].view(torch.int16).view(
            B, nb, cfg.hidden)
    elif cfg.signal in (SIGNAL_LAGKV, SIGNAL_LAGKV_KEY):
        shp = (2, B, cfg.n_layers, 2, cfg.n_kv_heads, cfg.head_dim)
        n = 1
        for s in shp:
            n *= s
        out["range"] = state[off[3]:off[3] + 4 * n].view(torch.float32).view(
            *shp)
    ne = B * n_sig(cfg)
    out["ema"] = state[off[4]:off[4] + 4 * ne].view(torch.float32).view(
        B, n_sig(cfg))
    return out
