"""Pins of the reference's Route-Plan (Eq. 1) and routed placement (CPU only).

The LP optimum is checked against exhaustive search over integer plans on tiny
instances, against a closed form (the degradation of any plan telescopes
over the boundaries between consecutive levels, and each boundary must be
crossed upwards by at least the demand below it that the capacity below it
cannot hold), and against feasibility invariants.  The routed placement is
checked against the rounds placement, which it must reproduce when given the
flow that the rounds placement realises, and against the plan it is given.
"""
import itertools

import numpy as np
import pytest

from oracle import oracle


def _cost(x, K):
    """Degradation by the definition: K_j - K_i for every query moved up."""
    Kf = [0] + list(K)
    return sum(x[i][j] * (Kf[j] - Kf[i]) for i in range(len(Kf)) for j in range(len(Kf)) if Kf[j] > Kf[i])


def _closed_form(H, F, K):
    """sum over boundaries m (between levels m and m+1) of (K_{m+1} - K_m) times
    the demand at levels <= m that capacity at levels <= m cannot hold, after
    the min(sum H, sum F) served queries leave out the lowest-level excess."""
    Kf = [0] + list(K)
    U = max(0, sum(H) - sum(F))
    S = G = 0
    d = 0
    for m in range(len(H) - 1):
        S += H[m]
        G += F[m]
        d += (Kf[m + 1] - Kf[m]) * max(0, S - G - U)
    return d


def _rows(h, n):
    """Every way to serve at most h queries of one level over n levels."""
    for parts in itertools.product(range(h + 1), repeat=n):
        if sum(parts) <= h:
            yield parts


def _brute(H, F, K):
    n = len(H)
    best = None
    for x in itertools.product(*[list(_rows(h, n)) for h in H]):
        if any(sum(x[i][j] for i in range(n)) > F[j] for j in range(n)):
            continue
        key = (-sum(map(sum, x)), _cost(x, K))
        best = key if best is None or key < best else best
    return -best[0], best[1]


def _random_case(rng, Lmax=4, hmax=5):
    L = int(rng.integers(1, Lmax + 1))
    K = np.cumsum(rng.integers(1, 7, size=L)).tolist()
    H = rng.integers(0, hmax, size=L + 1).tolist()
    F = rng.integers(0, hmax, size=L + 1).tolist()
    return L, K, H, F


def test_route_plan_exhaustive_tiny():
    rng = np.random.default_rng(5)
    n = 0
    for L in (1, 2):
        for _ in range(60):
            K = np.cumsum(rng.integers(1, 6, size=L)).tolist()
            H = rng.integers(0, 3, size=L + 1).tolist()
            F = rng.integers(0, 3, size=L + 1).tolist()
            x, d, served = oracle.route_plan(H, F, K)
            assert (served, d) == _brute(H, F, K), (H, F, K, x.tolist())
            n += 1
    assert n == 120


def test_route_plan_closed_form_and_feasibility():
    rng = np.random.default_rng(6)
    for _ in range(400):
        L, K, H, F = _random_case(rng, Lmax=6, hmax=9)
        x, d, served = oracle.route_plan(H, F, K)
        assert (x >= 0).all()
        assert (x.sum(axis=1) <= np.array(H)).all() and (x.sum(axis=0) <= np.array(F)).all()
        assert served == min(sum(H), sum(F))
        assert d == _cost(x.tolist(), K) == _closed_form(H, F, K), (H, F, K, x.tolist())


def test_route_plan_special_cases():
    # Capacity at every level covers its own demand: no degradation (moves
    # down are free, so the optimal plan need not be the diagonal).
    assert oracle.route_plan([3, 1, 4], [3, 2, 5], [4, 9])[1:] == (0, 8)
    # Only lower levels have room: moves down are free.
    assert oracle.route_plan([0, 0, 3], [1, 1, 1], [4, 9])[1:] == (0, 3)
    # Only the top level has room: every query pays K_L - K_i.
    x, d, s = oracle.route_plan([2, 1, 0], [0, 0, 5], [4, 9])
    assert (d, s) == (2 * 9 + 1 * 5, 3)
    # Nothing to serve, or nowhere to serve it.
    assert oracle.route_plan([0, 0], [3, 3], [2])[1:] == (0, 0)
    assert oracle.route_plan([4, 2], [0, 0], [2])[1:] == (0, 0)
    # Single level (L = 0).
    x, d, s = oracle.route_plan([5], [3], [])
    assert (d, s) == (0, 3) and x.tolist() == [[3]]


def test_route_plan_beats_the_rounds_placement():
    # Level-2 capacity is taken by level-1 queries in the first redirection
    # round in index order, pushing a level-0 query further up; the plan
    # routes the level-0 queries to the nearest room instead.
    rng = np.random.default_rng(7)
    better = 0
    for _ in range(1500):
        L, K, H, F = _random_case(rng)
        level = np.repeat(np.arange(L + 1), H)
        rng.shuffle(level)
        lev = oracle.assign(level, L, list(range(L + 1)), F)[0]
        flow = np.zeros((L + 1, L + 1), dtype=np.int64)
        for q, j in enumerate(lev):
            if j >= 0:
                flow[level[q], j] += 1
        x, d, served = oracle.route_plan(H, F, K)
        assert flow.sum() == served
        assert _cost(flow.tolist(), K) >= d
        better += _cost(flow.tolist(), K) > d
    assert better > 20


def _flow(level, out_level, L):
    f = np.zeros((L + 1, L + 1), dtype=np.int64)
    for q, j in enumerate(out_level):
        if j >= 0:
            f[level[q], j] += 1
    return f


def test_assign_routed_reproduces_rounds_placement():
    rng = np.random.default_rng(8)
    for _ in range(300):
        L = int(rng.integers(0, 5))
        I = int(rng.integers(1, 8))
        il = rng.integers(0, L + 1, I).tolist()
        ic = rng.integers(0, 5, I).tolist()
        iq = rng.integers(0, 4, I).tolist()
        level = rng.integers(0, L + 1, int(rng.integers(0, 30)))
        want = [a.tolist() for a in oracle.assign(level, L, il, ic, iq)]
        got = [a.tolist() for a in oracle.assign_routed(level, L, _flow(level, want[0], L), il, ic, iq)]
        assert got == want


def test_assign_routed_follows_the_plan():
    rng = np.random.default_rng(9)
    for _ in range(200):
        L, K, H, F = _random_case(rng)
        level = np.repeat(np.arange(L + 1), H)
        rng.shuffle(level)
        # two instances per level sharing its capacity
        il, ic = [], []
        for j, f in enumerate(F):
            il += [j, j]
            ic += [f // 2, f - f // 2]
        x, d, served = oracle.route_plan(H, F, K)
        lev, inst, slot, fill = oracle.assign_routed(level, L, x, il, ic, None)
        assert (_flow(level, lev, L) == x).all()
        assert fill.sum() == served
        # slots are a permutation of 0..fill-1 per instance
        for a in range(len(il)):
            assert sorted(slot[inst == a].tolist()) == list(range(fill[a]))
        # within a level of origin, destinations follow the preference order by query index
        for i in range(L + 1):
            pos = [oracle.preference(i, L).index(j) if j >= 0 else L + 1 for q, j in enumerate(lev) if level[q] == i]
            assert pos == sorted(pos)


def test_assign_routed_quota_beyond_capacity_or_demand():
    level = np.array([1, 1, 1, 0])
    x = np.array([[0, 1], [-2, 3]])                 # level 1 -> 1 three times; negative counts as 0
    lev, inst, slot, fill = oracle.assign_routed(level, 1, x, [0, 1], [4, 2], None)
    assert lev.tolist() == [1, 1, -1, -1]          # level 1 holds two; level 0's only quota goes up, full
    assert fill.tolist() == [0, 2]


def _mutant_lp_charges_down_moves(H, F, K):
    """Planted mistake: degradation charged on moves in both directions."""
    Kf = np.concatenate([[0], np.asarray(K)])
    n = len(H)
    best = None
    for xx in itertools.product(*[list(_rows(h, n)) for h in H]):
        if any(sum(xx[i][j] for i in range(n)) > F[j] for j in range(n)):
            continue
        c = sum(xx[i][j] * abs(int(Kf[j] - Kf[i])) for i in range(n) for j in range(n))
        key = (-sum(map(sum, xx)), c)
        best = key if best is None or key < best else best
    return -best[0], best[1]


def test_planted_mistake_is_caught_by_closed_form():
    rng = np.random.default_rng(10)
    caught = 0
    for _ in range(80):
        K = np.cumsum(rng.integers(1, 6, size=2)).tolist()
        H = rng.integers(0, 3, size=3).tolist()
        F = rng.integers(0, 3, size=3).tolist()
        s, d = _mutant_lp_charges_down_moves(H, F, K)
        caught += d != _closed_form(H, F, K)
    assert caught > 5
