"""The library's Route-Plan (apc_route_plan, host only) against the oracle's LP.

The plan is not unique (moves down are free), so the checks compare what is:
the number served and the minimal degradation (the LP optimum, and the
closed form pinned in test_oracle_route_plan), and check that the plan is
feasible and has the documented shape (own level first, first-in-first-out
moves).  Runs on the CPU: the entry point makes no GPU call.
"""
import ctypes

import numpy as np
import pytest

import paper_2502_06798_amd as A
from oracle import oracle

E_ARG, E_TABLE = 1, 3


def _random(rng, Lmax, hmax):
    L = int(rng.integers(0, Lmax + 1))
    K = np.cumsum(rng.integers(1, 9, size=L)).tolist()
    H = rng.integers(0, hmax, size=L + 1).tolist()
    F = rng.integers(0, hmax, size=L + 1).tolist()
    return K, H, F


def _check_plan(K, H, F, X, d):
    X = np.asarray(X, dtype=np.int64)
    assert (X >= 0).all()
    assert (X.sum(axis=1) <= np.array(H)).all() and (X.sum(axis=0) <= np.array(F)).all()
    xo, do, so = oracle.route_plan(H, F, K)
    assert (int(X.sum()), d) == (so, do), (K, H, F, X.tolist())
    assert oracle.plan_cost(X, K) == (do, so)
    L = len(K)
    for i in range(L + 1):                                   # own level first
        assert X[i, i] == min(X[i].sum(), F[i])
    ups = [(i, j) for i in range(L + 1) for j in range(i + 1, L + 1) if X[i, j] > 0]
    for (i, j) in ups:                                       # moves up keep their order
        for (i2, j2) in ups:
            if i < i2:
                assert j <= j2
    downs = [(i, j) for i in range(L + 1) for j in range(i) if X[i, j] > 0]
    for (i, j) in downs:                                     # moves down keep their order
        for (i2, j2) in downs:
            if i < i2:
                assert j <= j2


def test_route_plan_matches_lp_small():
    rng = np.random.default_rng(21)
    for _ in range(500):
        K, H, F = _random(rng, 5, 7)
        X, d = A.apc_route_plan(K, H, F)
        _check_plan(K, H, F, X, d)


def test_route_plan_matches_lp_all_levels_large_counts():
    rng = np.random.default_rng(22)
    for _ in range(40):
        L = 32
        K = np.cumsum(rng.integers(1, 40, size=L)).tolist()
        H = rng.integers(0, 3000, size=L + 1)
        H[rng.random(L + 1) < 0.3] = 0
        F = rng.integers(0, 3000, size=L + 1)
        F[rng.random(L + 1) < 0.3] = 0
        X, d = A.apc_route_plan(K, H.tolist(), F.tolist())
        _check_plan(K, H.tolist(), F.tolist(), X, d)


def test_route_plan_special_cases():
    X, d = A.apc_route_plan([4, 9], [3, 1, 4], [3, 2, 5])
    assert d == 0 and (X == np.diag([3, 1, 4])).all()       # room everywhere: nothing moves
    X, d = A.apc_route_plan([], [5], [3])
    assert X.tolist() == [[3]] and d == 0
    X, d = A.apc_route_plan([2], [0, 0], [0, 0])
    assert X.sum() == 0 and d == 0
    X, d = A.apc_route_plan([4, 9], [2, 1, 0], [0, 0, 5])
    assert d == 2 * 9 + 5 and X[:, 2].sum() == 3
    # sums at the limit
    X, d = A.apc_route_plan([1], [2**31 - 1, 0], [0, 2**31 - 1])
    assert X[0, 1] == 2**31 - 1 and d == 2**31 - 1


def test_route_plan_argument_checks():
    lib = A.load()
    X = np.zeros(64, dtype=np.int32)

    def call(L, K, H, F, out=X):
        arr = lambda v: None if v is None else np.ascontiguousarray(v, dtype=np.int32)
        Ka, Ha, Fa = arr(K), arr(H), arr(F)
        p = lambda a: None if a is None else a.ctypes.data
        return lib.apc_route_plan(L, p(Ka), p(Ha), p(Fa), p(out), None)

    assert call(1, [3], [1, 1], [1, 1]) == 0
    assert call(-1, [], [1], [1]) == E_TABLE
    assert call(33, list(range(1, 34)), [0] * 34, [0] * 34) == E_TABLE
    assert call(2, [3, 3], [1, 1, 1], [1, 1, 1]) == E_TABLE
    assert call(1, [0], [1, 1], [1, 1]) == E_TABLE
    assert call(1, [3], [1, -1], [1, 1]) == E_ARG
    assert call(1, [3], [2**31 - 1, 1], [1, 1]) == E_ARG
    assert call(1, None, [1, 1], [1, 1]) == E_ARG
    assert call(1, [3], [1, 1], [1, 1], out=None) == E_ARG


def test_routed_entries_check_batch_and_plan():
    lib = A.load()
    th = np.array([0.5], dtype=np.float32)
    K = np.array([4], dtype=np.int32)
    il = np.array([0, 1], dtype=np.int32)
    ic = np.array([2, 2], dtype=np.int32)
    fake = ctypes.c_void_p(256)                              # never dereferenced: the checks fail first
    for fn in (lib.apc_assign_routed, lib.apc_assign_planned):
        args = lambda b, plan: (fake, 1, b, 1, th.ctypes.data, K.ctypes.data, 2, il.ctypes.data,
                                ic.ctypes.data, None, plan, fake, fake, fake, fake, fake, None)
        assert fn(*args(16385, fake)) == E_ARG
        assert fn(*args(8, None)) == E_ARG
        assert fn(*args(-1, fake)) == E_ARG
