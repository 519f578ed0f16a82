"""Comparison rules of the GPU-vs-reference parity tests.

Scores: |s_gpu - s_ref| <= tol (2e-3 for 16-bit and e4m3 inputs, 1e-5 for
float32).  Top-k indices: bit-exact, except where the reference's competing
scores lie within tol (then any of the competitors is accepted; indices must
still be distinct).  Strict rule on top of that: wherever the reference's
score at a rank is more than 1e-5 from its neighbours' (the ranks above and
below, and for the last rank the best entry outside the top-k), the entry at
that rank is unique and the GPU's index must equal the reference's (both
sides score the same stored values; float32 accumulation is within ~1e-6 of
float64).  Levels: bit-exact given the GPU's best score; against the
reference's best, equal unless the reference best is within tol of a
threshold between the two.  Assignment and gather: bit-exact given the GPU's
levels and top-1.
"""
from __future__ import annotations

import sys

import numpy as np

TOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3, "e4m3": 2e-3}
STRICT = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_topk(orc, dtype, q, qs, e, es, gpu_s, gpu_i, ref_s, ref_i, rows=None, q_sq=None, e_sq=None):
    """Tolerance-aware top-k check of the given query rows; returns statistics.

    q/e are host arrays of stored elements; gpu_* are [b, k] arrays; ref_* are
    the reference's [rows, k] lists, or [rows, k + 1] (the extra column, the
    best entry outside the top-k, lets the strict rule cover the last rank).
    """
    tol = TOL[dtype]
    k = gpu_i.shape[1]
    nxt = ref_s[:, k].astype(np.float64) if ref_s.shape[1] > k else None
    ref_s, ref_i = ref_s[:, :k], ref_i[:, :k]
    b = gpu_i.shape[0] if rows is None else len(rows)
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
    # strict rule: isolated reference ranks are bit-exact
    rs = ref_s.astype(np.float64)
    above = np.full(rs.shape, np.inf)
    above[:, 1:] = rs[:, :-1] - rs[:, 1:]
    below = np.zeros(rs.shape)
    below[:, :-1] = rs[:, :-1] - rs[:, 1:]
    if nxt is not None:
        below[:, -1] = rs[:, -1] - nxt
    isolated = (above > STRICT) & (below > STRICT)
    bad = isolated & ~exact
    if bad.any():
        r, p = np.argwhere(bad)[0]
        raise AssertionError(f"row {rows[r]} rank {p}: GPU entry {g_i[r, p]} vs reference {ref_i[r, p]} "
                             f"(reference score {rs[r, p]:.9f}, isolated by more than {STRICT})")
    return {"max_score_err": float(err_s.max()), "index_mismatch": int((~exact).sum()),
            "strict_ranks": int(isolated.sum()), "rows_exact": int(exact.all(axis=1).sum()),
            "rows": int(len(rows))}


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
