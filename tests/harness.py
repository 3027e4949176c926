"""Shared helpers of the GPU parity tests: device transfers, paged-pool
bookkeeping on the host, and configuration from a synthetic workload.

Test infrastructure: it may use both the oracle and the HIP binding; the
paging helpers here only move bytes around (the oracle sees logical rows).
"""
from __future__ import annotations

import numpy as np

import synth

DEV = "cuda"

# Agreement with the oracle for floating-point results (the eviction step's
# target: scores within 1e-3 relative).
TOL = 1e-3
# Quantities that are strictly positive -- the hidden-state change g, the
# KV-vector signal q, and the mean / EMA / raw smoothing of such a signal
# on its own (the KV-vector scores) -- are held to a pure relative error.
POSITIVE = 0.0
# Quantities that can sit at or near zero -- z-scores and band differences
# s = mean_A - mean_B -- are held to 1e-3 relative above magnitude 1 and to
# 1e-3 absolute below it.
NEAR_ZERO = 1.0


def torch():
    import torch as t
    return t


def dev(x: np.ndarray):
    """Upload a numpy array (uint16 arrays travel as int16)."""
    T = torch()
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        x = x.view(np.int16)
    return T.from_numpy(x).to(DEV)


def host(t) -> np.ndarray:
    a = t.detach().cpu().numpy()
    if a.dtype == np.int16:
        a = a.view(np.uint16)
    return a


def rel_err(got, ref, floor=POSITIVE) -> float:
    """Largest |got - ref| / max(floor, |ref|) over the elements.  With
    floor 0 a reference of exactly 0 must be matched exactly (else the error
    is infinite).  NaN must sit exactly where the reference has NaN."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if not np.array_equal(np.isnan(got), np.isnan(ref)):
        return float("inf")
    ok = ~np.isnan(ref)
    diff = np.abs(got[ok] - ref[ok])
    den = np.maximum(floor, np.abs(ref[ok]))
    if np.any((den == 0) & (diff != 0)):
        return float("inf")
    err = np.divide(diff, den, out=np.zeros_like(diff), where=den > 0)
    return float(err.max()) if err.size else 0.0


def idx(a):
    """A host index array as a device int64 tensor."""
    T = torch()
    return T.from_numpy(np.asarray(a, dtype=np.int64)).to(DEV)


def rebuilt_rows_equal(src_pool, src_pt_row, dst_pool, dst_pt_row, keep,
                       page, first=0) -> bool:
    """Every rebuilt row j >= first of one sequence, in every layer and K/V
    plane, equals (bit for bit, on the device) the source row of position
    keep[j].  Pools [L][2][n_pages][page][H*d] of 16-bit storage; compared
    as integers, so NaN payloads count."""
    T = torch()
    keep = np.asarray(keep, dtype=np.int64)
    j = np.arange(first, keep.size)
    if j.size == 0:
        return True
    sv = src_pool.view(T.int16)
    dv = dst_pool.view(T.int16)
    src = sv[:, :, idx(src_pt_row[keep[j] // page]), idx(keep[j] % page), :]
    dst = dv[:, :, idx(dst_pt_row[j // page]), idx(j % page), :]
    return bool(T.equal(src, dst))


def cfg_for(E, w: synth.Workload, **kw):
    """epikv_cfg for a workload (keyword overrides win)."""
    c = E.default_cfg(
        batch=w.B, hidden=w.hidden, n_layers=w.n_layers,
        n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, page_size=w.page_size,
        n_band_a=len(w.band_a), n_band_b=len(w.band_b), window=w.window,
        budget=w.budget,
        signal=E.SIGNAL_LAGKV if w.signal == "lagkv" else E.SIGNAL_HS,
        smoothing=E.SMOOTH_MEAN if w.signal == "lagkv" else E.SMOOTH_Z)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def pool_shape(L, n_pages, page, H, d):
    return (L, 2, n_pages, page, H * d)


def gather_logical(pool_np: np.ndarray, pt_row: np.ndarray, n: int):
    """Rows of positions 0..n-1 of one sequence: [L][2][n][H*d] (host)."""
    page = pool_np.shape[3]
    pos = np.arange(n)
    pages = pt_row[pos // page]
    slots = pos % page
    return pool_np[:, :, pages, slots, :]


def scatter_logical(pool_np: np.ndarray, pt_row: np.ndarray, first: int,
                    rows: np.ndarray):
    """Write rows [L][2][n][H*d] into positions first.. of one sequence."""
    page = pool_np.shape[3]
    pos = first + np.arange(rows.shape[2])
    pool_np[:, :, pt_row[pos // page], pos % page, :] = rows


def tie_exempt_compare(keep_gpu, keep_ref, scores_ref, n_prefix, N, K, R,
                       tol=1e-3):
    """Compare retained sets; positions that differ must sit within `tol`
    of the oracle's cut score (the M-th best eligible score).  Returns the
    number of exempted swaps."""
    keep_gpu = np.asarray(keep_gpu)
    keep_ref = np.asarray(keep_ref)
    assert keep_gpu.size == keep_ref.size
    assert np.all(np.diff(keep_gpu) > 0)
    if np.array_equal(keep_gpu, keep_ref):
        return 0
    elig = np.arange(n_prefix, N - R)
    kept_e = np.intersect1d(keep_ref, elig)
    s = np.asarray(scores_ref, dtype=np.float64)
    cut = np.min(s[kept_e])
    diff = np.setxor1d(keep_gpu, keep_ref)
    bound = tol * max(1.0, abs(cut))
    for i in diff:
        assert n_prefix <= i < N - R, f"protected position {i} differs"
        assert abs(s[i] - cut) <= bound, \
            f"position {i}: score {s[i]} vs cut {cut} (not a near tie)"
    return diff.size // 2


def remap_expected(pool_np: np.ndarray, pt: np.ndarray, keeps, page: int):
    """The oracle's in-place rebuild with page remapping of every sequence
    of a host pool [L][2][n_pages][page][H*d], one sequence after the
    other (None in `keeps`: sequence untouched).  Returns (pool, table)."""
    import oracle as O
    phys = pool_np.transpose(2, 3, 0, 1, 4).copy()     # [n_pages][page][...]
    new_pt = pt.copy()
    for b, keep in enumerate(keeps):
        if keep is None:
            continue
        n = int(np.count_nonzero(pt[b] >= 0))
        phys, row = O.compact_pages_remap(phys, pt[b, :n], keep, page)
        new_pt[b, :n] = row
    return phys.transpose(2, 3, 0, 1, 4), new_pt
