"""Mutation audit of the oracle's pins (CPU).

Each entry plants one plausible mistake in a copy of the oracle -- a
dropped or wrong term, a wrong sign, index or estimator, a rule read the
other way -- and runs the pins (test_oracle_pins.py) against the copy.
Every mistake must make at least one pin fail, and the unmodified copy must
pass them all: that is what shows the pins fix the oracle to the paper and
not merely to itself.  The repository's own oracle is never modified.
"""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name: (exact text in oracle/epikv_ref.py, replacement)
MUTATIONS = {
    # Eq. 1: the L2 norm of the change from the previous token
    "eq1_l1_norm": ("        g[t] = np.sqrt(np.sum(d * d))",
                    "        g[t] = np.sum(np.abs(d))"),
    "eq1_change_from_first_token": ("            prev = h[t - 1]",
                                    "            prev = h[0]"),
    # Eq. 3: population sigma, eps added to sigma, window [t-w+1, t]
    "eq3_sample_sigma": (
        "        sigma = np.sqrt(np.sum((win - mu) ** 2) / win.size)",
        "        sigma = np.sqrt(np.sum((win - mu) ** 2) / max(win.size - 1, 1))"),
    "eq3_eps_under_the_root": (
        "        out[i] = (x[i] - mu) / (sigma + eps)",
        "        out[i] = (x[i] - mu) / np.sqrt(sigma ** 2 + eps)"),
    "window_excludes_t": ("    return x[max(0, i - w + 1):i + 1]",
                          "    return x[max(0, i - w):i] if i > 0 else x[:1]"),
    "window_of_w_plus_1": ("    return x[max(0, i - w + 1):i + 1]",
                           "    return x[max(0, i - w):i + 1]"),
    # band combination: mean over Band A minus mean over Band B
    "band_b_added": ("        s = s - np.mean(smoothed[n_a:n_a + n_b], axis=0)",
                     "        s = s + np.mean(smoothed[n_a:n_a + n_b], axis=0)"),
    "band_a_summed": ("    s = np.mean(smoothed[:n_a], axis=0)",
                      "    s = np.sum(smoothed[:n_a], axis=0)"),
    # Sec. 3.3 / Table 1: per-channel range, normalisation, variance
    "range_min_of_v_is_max": (
        "    mn = np.stack([k.min(axis=0), v.min(axis=0)], axis=1)",
        "    mn = np.stack([k.min(axis=0), v.max(axis=0)], axis=1)"),
    "lagkv_wrong_eps": (
        "    kt = (k - mn[None, :, 0]) / (mx[None, :, 0] - mn[None, :, 0] + eps)",
        "    kt = (k - mn[None, :, 0]) / (mx[None, :, 0] - mn[None, :, 0] + 1e-3)"),
    "lagkv_sample_variance": (
        "    var_k = np.var(kt, axis=-1)   # population variance over head dim",
        "    var_k = np.var(kt, axis=-1, ddof=1)"),
    "lagkv_k_v_averaged": ("    return np.mean(var_k + var_v, axis=(1, 2))",
                           "    return np.mean((var_k + var_v) / 2, axis=(1, 2))"),
    "kv_family_drops_values": (
        "        q = q + np.mean(np.var(x, axis=-1), axis=(1, 2))",
        "        q = q + (np.mean(np.var(x, axis=-1), axis=(1, 2)) if kv == 0 else 0)"),
    "kv_family_values_by_key_range": (
        "            x = (x - mn[None, :, kv]) / (mx[None, :, kv] - mn[None, :, kv] + eps)",
        "            x = (x - mn[None, :, 0]) / (mx[None, :, 0] - mn[None, :, 0] + eps)"),
    "lagkv_own_range_always": ("        rng = own if prev_range is None else prev_range",
                               "        rng = own"),
    # App. D: recency window, retention rule, ties, NaN, budget edge
    "recent_k_over_2": ("    return min(128, K // 4)", "    return min(128, K // 2)"),
    "recent_cap_256": ("    return min(128, K // 4)", "    return min(256, K // 4)"),
    "ties_to_higher_position": ("    return (0, -x, pos)", "    return (0, -x, -pos)"),
    "nan_ranked_first": ("        return (1, 0.0, pos)", "        return (-1, 0.0, pos)"),
    "lowest_scores_kept": ("    return (0, -x, pos)", "    return (0, x, pos)"),
    "prefill_not_protected": (
        "    kept = set(range(n_prefix)) | set(range(N - R, N)) | set(ranked[:M])",
        "    kept = set(range(N - R, N)) | set(ranked[:M + n_prefix])"),
    "budget_edge_off_by_one": ("    if n_prefix + R >= K:", "    if n_prefix + R > K:"),
    "evicts_at_n_equal_k": ("    if N <= K:", "    if N < K:"),
    # App. H: rebuilds
    "first_hole_one_late": (
        "    return int(moved[0]) if moved.size else int(keep.size)",
        "    return int(moved[0]) + 1 if moved.size else int(keep.size)"),
    "inplace_clears_the_tail": ("    out = rows.copy()\n    out[:keep.size] = rows[keep]",
                                "    out = np.zeros_like(rows)\n    out[:keep.size] = rows[keep]"),
    # App. H page remapping: which pages qualify, where released pages go
    "remap_unaligned_source_page": (
        "        if r == 0 and p > m and np.array_equal(run, np.arange(p * ps, (p + 1) * ps)):",
        "        if p > m and np.array_equal(run, np.arange(run[0], run[0] + ps)):"),
    "remap_page_already_in_place": (
        "        if r == 0 and p > m and np.array_equal(run, np.arange(p * ps, (p + 1) * ps)):",
        "        if r == 0 and p >= m and np.array_equal(run, np.arange(p * ps, (p + 1) * ps)):"),
    "remap_released_in_reverse": ("    for m, p in zip(released, losing):",
                                  "    for m, p in zip(released[::-1], losing):"),
    # App. E: EMA weighting and start
    "ema_weights_swapped": (
        "        y = x[i] if y is None else alpha * y + (1.0 - alpha) * x[i]",
        "        y = x[i] if y is None else (1.0 - alpha) * y + alpha * x[i]"),
    "ema_starts_from_zero": (
        "        y = x[i] if y is None else alpha * y + (1.0 - alpha) * x[i]",
        "        y = (1.0 - alpha) * x[i] if y is None else alpha * y + (1.0 - alpha) * x[i]"),
    "raw_mode_smoothed": ("        return np.asarray(samples, dtype=np.float64).copy()",
                          "        return rolling_mean(samples, w)"),
    "ema_carry_dropped": ("        sm = ema(new[has_sample], y_before=ema_before)",
                          "        sm = ema(new[has_sample], y_before=None)"),
    # number format: bf16 is the high half of a binary32 word
    "bf16_as_low_half": ("    u32 = u16.astype(np.uint32) << np.uint32(16)",
                         "    u32 = u16.astype(np.uint32)"),
}


def _run_pins(replace):
    """Run the pins against a copy of the oracle with `replace` applied;
    returns (pytest exit code, last line of its report)."""
    with tempfile.TemporaryDirectory() as d:
        for sub in ("oracle", "synth", "tests"):
            shutil.copytree(os.path.join(ROOT, sub), os.path.join(d, sub),
                            ignore=shutil.ignore_patterns("__pycache__"))
        shutil.copy(os.path.join(ROOT, "pytest.ini"), d)
        p = os.path.join(d, "oracle", "epikv_ref.py")
        src = open(p).read()
        if replace is not None:
            a, b = replace
            assert src.count(a) == 1, f"mutation target not found once: {a!r}"
            open(p, "w").write(src.replace(a, b))
        r = subprocess.run(
            [sys.executable, "-m", "pytest", "tests/test_oracle_pins.py", "-q",
             "-x", "-p", "no:cacheprovider"],
            cwd=d, capture_output=True, text=True, timeout=600,
            env={**os.environ, "PYTHONDONTWRITEBYTECODE": "1"})
        lines = [l for l in r.stdout.splitlines() if l.strip()]
        return r.returncode, lines[-1] if lines else r.stderr[-300:]


def test_unmutated_copy_passes_the_pins():
    rc, last = _run_pins(None)
    assert rc == 0, last


def test_every_planted_mistake_fails_a_pin():
    workers = min(8, os.cpu_count() or 1)
    with ThreadPoolExecutor(workers) as ex:
        results = dict(zip(MUTATIONS, ex.map(_run_pins, MUTATIONS.values())))
    # exit code 1 = some pin failed (2 or more would be a broken run)
    missed = {k: last for k, (rc, last) in results.items() if rc != 1}
    assert not missed, f"mistakes no pin catches: {missed}"
