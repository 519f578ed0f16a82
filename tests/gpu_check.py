"""Comparison rules of the GPU-vs-reference parity tests.

Scores: |s_gpu - s_ref| <= tol (2e-3 for 16-bit and e4m3 inputs, 1e-5 for
float32).  Top-k indices: bit-exact, except where the reference's competing
scores lie within tol (then any of the competitors is accepted; indices must
still be distinct).  Levels: bit-exact given the GPU's best score; against the
reference's best, equal unless the reference best is within tol of a
threshold between the two.  Assignment and gather: bit-exact given the GPU's
levels and top-1.
"""
from __future__ import annotations

import sys

import numpy as np

TOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3, "e4m3": 2e-3}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_topk(orc, dtype, q, qs, e, es, gpu_s, gpu_i, ref_s, ref_i, rows=None, q_sq=None, e_sq=None):
    """Tolerance-aware top-k check of the given query rows; returns statistics.

    q/e are host arrays of stored elements; gpu_*/ref_* are [b, k] arrays
    (ref for the selected rows only when `rows` is given).
    """
    tol = TOL[dtype]
    b, k = gpu_i.shape if rows is None else (len(rows), gpu_i.shape[1])
    rows = np.arange(b) if rows is None else np.asarray(rows)
    g_i = gpu_i[rows].astype(np.int64)
    g_s = gpu_s[rows].astype(np.float64)
    assert np.all(g_i >= 0) and np.all(g_i < e.shape[0]), "index out of range"
    for r in range(len(rows)):
        assert len(set(g_i[r].tolist())) == k, f"row {rows[r]}: repeated indices"
    # reference scores of the GPU's own choices
    qi = np.repeat(rows, k)
    s_of_gpu = orc.pair_scores(dtype, q, qs, e, es, qi, g_i.ravel(), q_sq=q_sq, e_sq=e_sq).reshape(len(rows), k)
    err_s = np.abs(g_s - s_of_gpu)
    assert err_s.max() <= tol, f"score error {err_s.max():.3g} > {tol}"
    # rank by rank the GPU's choice scores within tol of the reference's p-th best
    gap = np.abs(s_of_gpu - ref_s)
    assert gap.max() <= tol, f"rank score gap {gap.max():.3g} > {tol}"
    exact = g_i == ref_i
    # GPU's sorted order must be consistent with its own scores
    assert np.all(np.diff(g_s, axis=1) <= 0), "GPU list not sorted by score"
    return {"max_score_err": float(err_s.max()), "index_mismatch": int((~exact).sum()),
            "rows_exact": int(exact.all(axis=1).sum()), "rows": int(len(rows))}


def check_levels(orc, theta, gpu_best, gpu_level, ref_best, tol):
    """GPU level equals the reference level of the GPU's best; against the
    reference's own best it may differ only inside the tolerance band."""
    lv_of_gpu = orc.levels(gpu_best.astype(np.float64), theta)
    assert np.array_equal(gpu_level, lv_of_gpu), "level of the GPU best differs"
    lv_ref = orc.levels(ref_best, theta)
    band = 0
    for i in np.flatnonzero(lv_ref != gpu_level):
        lo, hi = sorted((int(lv_ref[i]), int(gpu_level[i])))
        between = theta[lo:hi].astype(np.float64)
        assert np.any(np.abs(ref_best[i] - between) <= tol), \
            f"query {i}: level {gpu_level[i]} vs reference {lv_ref[i]} outside the band"
        band += 1
    return band
