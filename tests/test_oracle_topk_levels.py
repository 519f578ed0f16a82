"""Pins of the reference's top-k and level selection (CPU only).

Top-k is checked against exact rational ordering on integer-grid vectors
(exhaustive over small grids), against numpy's lexsort on random data, and
by permutation invariance; levels against numpy's searchsorted and exact
boundary cases.
"""
import itertools

import numpy as np
import pytest

from oracle import pyref


def _grid_vectors(d, lo=-2, hi=2):
    vs = [v for v in itertools.product(range(lo, hi + 1), repeat=d) if any(v)]
    return vs


def _check_against_exact(orc, qv, entries, k):
    """Oracle top-k of one query vs exact rational order.

    Exact ties between vectors that are positive multiples of each other give
    equal float64 scores and must come out in index order; other scores
    must follow the exact order wherever they differ by more than 1e-12.
    """
    q = np.array([qv], np.float32)
    e = np.array(entries, np.float32)
    ts, ti = orc.topk("f32", q, None, e, None, k)
    keys = [pyref.cos_key(qv, ev) for ev in entries]
    vals = np.array([pyref.cos_float(kk) for kk in keys])
    exact = pyref.exact_topk(qv, entries, k)
    got = ti[0].tolist()
    assert len(set(got)) == k
    assert np.all(np.abs(ts[0] - vals[got]) <= 1e-15)
    # rank by rank: the chosen index's exact score equals the exact p-th score (up to 1e-12)
    for p in range(k):
        assert abs(vals[got[p]] - vals[exact[p]]) <= 1e-12
    # ties in float64 are ordered by index
    for p in range(k - 1):
        if ts[0, p] == ts[0, p + 1]:
            assert got[p] < got[p + 1]
    # where the exact order is separated, the lists agree exactly
    sep = all(abs(vals[exact[p]] - vals[exact[p + 1]]) > 1e-12 or keys[exact[p]] == keys[exact[p + 1]]
              for p in range(k - 1))
    if sep and (k == len(entries) or abs(vals[exact[k - 1]] - sorted(vals)[::-1][k]) > 1e-12):
        assert got == exact


def test_topk_exhaustive_grid_d2(orc):
    vs = _grid_vectors(2)                       # 24 vectors
    for qv in vs:
        for k in (1, 3, len(vs)):
            _check_against_exact(orc, qv, vs, k)


def test_topk_exhaustive_grid_d3_subsets(orc):
    vs = _grid_vectors(3, -1, 1)                # 26 vectors
    rng = np.random.default_rng(11)
    for qv in vs:
        for _ in range(4):
            n = int(rng.integers(1, 7))
            idx = rng.choice(len(vs), size=n, replace=True)   # duplicates allowed
            entries = [vs[i] for i in idx]
            for k in range(1, n + 1):
                _check_against_exact(orc, qv, entries, k)


def test_topk_matches_lexsort(orc):
    rng = np.random.default_rng(2)
    q = rng.standard_normal((12, 33)).astype(np.float32)
    e = rng.standard_normal((500, 33)).astype(np.float32)
    e[100] = e[7]                   # exact duplicates: equal scores, index order
    e[301] = e[7]
    k = 17
    ts, ti = orc.topk("f32", q, None, e, None, k)
    Q = q.astype(np.float64) / np.linalg.norm(q.astype(np.float64), axis=1, keepdims=True)
    E = e.astype(np.float64) / np.linalg.norm(e.astype(np.float64), axis=1, keepdims=True)
    S = np.clip(Q @ E.T, -1, 1)
    for r in range(12):
        s_or = orc.pair_scores("f32", q, None, e, None, np.full(500, r), np.arange(500))
        assert np.max(np.abs(s_or - S[r])) <= 1e-14
        order = np.lexsort((np.arange(500), -s_or))[:k]
        assert ti[r].tolist() == order.tolist()
        assert np.array_equal(ts[r], s_or[order])


def test_topk_duplicates_all_equal(orc):
    e = np.tile(np.array([[1.0, -2.0, 0.5, 3.0]], np.float32), (9, 1))
    q = np.array([[0.3, 0.1, -1.0, 2.0]], np.float32)
    ts, ti = orc.topk("f32", q, None, e, None, 4)
    assert ti[0].tolist() == [0, 1, 2, 3]
    assert np.all(ts[0] == ts[0, 0])


def test_topk_permutation_invariance(orc):
    rng = np.random.default_rng(4)
    q = rng.standard_normal((5, 20)).astype(np.float32)
    e = rng.standard_normal((200, 20)).astype(np.float32)
    perm = rng.permutation(200)
    ts, ti = orc.topk("f32", q, None, e, None, 8)
    ts2, ti2 = orc.topk("f32", q, None, e[perm], None, 8)
    assert np.array_equal(ts, ts2)
    assert np.array_equal(perm[ti2], ti)        # no equal scores here, so the order is unique


def test_topk_self_match_first(orc):
    rng = np.random.default_rng(9)
    e = rng.standard_normal((64, 16)).astype(np.float32)
    ts, ti = orc.topk("f32", e[10:20], None, e, None, 3)
    assert ti[:, 0].tolist() == list(range(10, 20))
    assert np.all(np.abs(ts[:, 0] - 1.0) <= 5e-16)


def test_topk_rejects_bad_k(orc):
    e = np.ones((3, 4), np.float32)
    with pytest.raises(ValueError):
        orc.topk("f32", e, None, e, None, 4)
    with pytest.raises(ValueError):
        orc.topk("f32", e, None, e, None, 0)


def test_levels_searchsorted_and_boundaries(orc):
    theta = np.array([0.70 + 0.03 * i for i in range(10)], np.float32)
    rng = np.random.default_rng(5)
    best = np.concatenate([rng.uniform(-1, 1, 1000), theta.astype(np.float64),
                           np.nextafter(theta.astype(np.float64), -np.inf), [1.0, -1.0, 0.0]])
    lv = orc.levels(best, theta)
    assert np.array_equal(lv, np.searchsorted(theta.astype(np.float64), best, side="right"))
    # equal to a threshold counts that threshold (inclusive)
    n = 1000
    assert np.array_equal(lv[n:n + 10], np.arange(1, 11))
    assert np.array_equal(lv[n + 10:n + 20], np.arange(0, 10))
    # monotone in the best score
    o = np.argsort(best, kind="stable")
    assert np.all(np.diff(lv[o]) >= 0)


def test_levels_float32_thresholds(orc):
    # thresholds compare as float32 values: 0.9 -> 0.89999997..., 0.8 -> 0.80000001...
    theta = np.array([0.8, 0.9], np.float32)
    lv = orc.levels(np.array([0.9, 0.8999999, 0.79, 0.8, 0.8000001]), theta)
    assert lv.tolist() == [2, 1, 0, 0, 1]
    with pytest.raises(ValueError):
        orc.levels(np.array([0.5]), np.array([0.9, 0.8], np.float32))


def test_levels_exact_against_rationals(orc):
    """Level of the exact best match equals the exact rational comparison."""
    theta = [float(np.float32(t)) for t in (0.5, 0.7071, 0.8, 0.9)]
    vs = _grid_vectors(3, -2, 2)
    rng = np.random.default_rng(12)
    seen = set()
    for trial in range(300):
        qv = vs[int(rng.integers(len(vs)))]
        idx = rng.choice(len(vs), size=5, replace=False)
        # leave out multiples of the query so the best match is not trivially 1
        entries = [vs[i] for i in idx if pyref.cos_key(qv, vs[i]) != 1]
        if not entries:
            continue
        q = np.array([qv], np.float32)
        e = np.array(entries, np.float32)
        ts, ti = orc.topk("f32", q, None, e, None, 1)
        lv = orc.levels(ts[:, 0], np.array(theta, np.float32))[0]
        want = pyref.exact_level(qv, entries[ti[0, 0]], theta)
        assert lv == want
        seen.add(int(lv))
    assert seen == {0, 1, 2, 3, 4}
