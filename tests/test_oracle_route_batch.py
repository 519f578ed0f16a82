"""Pins of the reference's load-aware route-and-batch (CPU only).

Greedy routing at or above the load threshold is the placement `assign`
already pinned elsewhere; below it, uniform routing at batch size 1 is
pinned by its defining properties: every instance takes at most one query,
the placed count has a closed form, admission rank t of a level lands on the
level's instance with the t-th smallest random key, and over random keys the
chosen instance is uniform.  Planted mistakes in the reading fail the pins.
"""
import numpy as np
import pytest

from oracle import oracle


def _table(rng, L, I, cap_hi=4):
    il = rng.integers(0, L + 1, I).astype(np.int32)
    ic = rng.integers(0, cap_hi + 1, I).astype(np.int32)
    iq = rng.integers(0, 10, I).astype(np.int32)
    return il, ic, iq


def test_switch_at_the_threshold():
    rng = np.random.default_rng(5)
    for _ in range(50):
        L, I, B = int(rng.integers(1, 6)), int(rng.integers(1, 12)), int(rng.integers(1, 40))
        il, ic, iq = _table(rng, L, I)
        lv = rng.integers(0, L + 1, B).astype(np.int32)
        rnd = rng.integers(0, 2**32, I, dtype=np.uint64).astype(np.uint32)
        g = oracle.assign_load_aware(lv, L, il, ic, iq, rnd, load=7, threshold=7)
        assert g[0] == 1
        want = oracle.assign(lv, L, il, ic, iq)
        for a, b in zip(g[1:], want):
            assert np.array_equal(a, b)
        u = oracle.assign_load_aware(lv, L, il, ic, iq, rnd, load=6, threshold=7)
        assert u[0] == 0
        fill = u[4]
        assert np.all(fill <= np.minimum(ic, 1))                 # batch size 1
        # closed form: every query that finds a level with a free instance is
        # placed, so min(B, instances with room) are placed
        assert int((u[1] >= 0).sum()) == min(B, int((ic >= 1).sum()))
        # each placed query sits alone at slot 0 of an instance of its level
        placed = u[1] >= 0
        assert np.all(u[3][placed] == 0)
        assert np.all(il[u[2][placed]] == u[1][placed])
        assert len(set(u[2][placed].tolist())) == int(placed.sum())


def test_rank_t_takes_the_t_th_smallest_key():
    rng = np.random.default_rng(11)
    for _ in range(200):
        m = int(rng.integers(1, 9))
        L = 2
        il = np.full(m, 1, np.int32)                              # m instances at level 1
        ic = rng.integers(1, 5, m).astype(np.int32)
        rnd = rng.permutation(m * 3)[:m].astype(np.uint32)
        B = int(rng.integers(1, m + 1))
        lv = np.full(B, 1, np.int32)
        r = oracle.assign_load_aware(lv, L, il, ic, None, rnd, 0, 1)
        by_key = np.argsort(rnd, kind="stable")
        for t in range(B):                                        # query t is admission rank t
            assert r[1][t] == 1 and r[2][t] == by_key[t] and r[3][t] == 0


def test_ties_in_the_keys_take_the_lower_instance():
    il = np.zeros(4, np.int32)
    ic = np.ones(4, np.int32)
    rnd = np.array([5, 2, 5, 2], np.uint32)
    r = oracle.assign_load_aware(np.zeros(4, np.int32), 0, il, ic, None, rnd, 0, 1)
    assert r[2].tolist() == [1, 3, 0, 2]


def test_uniform_choice_is_uniform_over_random_keys():
    rng = np.random.default_rng(2025)
    m, trials = 5, 5000
    il = np.full(m, 1, np.int32)
    ic = np.full(m, 3, np.int32)
    counts = np.zeros(m, int)
    for _ in range(trials):
        rnd = rng.integers(0, 2**32, m, dtype=np.uint64).astype(np.uint32)
        r = oracle.assign_load_aware(np.array([1], np.int32), 1, il, ic, None, rnd, 0, 1)
        counts[r[2][0]] += 1
    assert np.all(np.abs(counts - trials / m) < 0.1 * trials / m), counts


def _mutant_desc(level, L, il, ic, iq, rnd, load, thr):
    return oracle.assign_load_aware(level, L, il, ic, iq, (~np.asarray(rnd, np.uint32)).astype(np.uint32), load, thr)


def _mutant_full_batch(level, L, il, ic, iq, rnd, load, thr):
    n = len(il)
    order = sorted(range(n), key=lambda i: (int(rnd[i]), i))
    q = np.empty(n, np.int32)
    for pos, i in enumerate(order):
        q[i] = n - pos
    return (0,) + tuple(oracle.assign(level, L, il, ic, q))


@pytest.mark.parametrize("mutant", [_mutant_desc, _mutant_full_batch])
def test_planted_mistakes_are_caught(mutant):
    rng = np.random.default_rng(3)
    caught = False
    for _ in range(50):
        m = int(rng.integers(2, 7))
        il = np.full(m, 1, np.int32)
        ic = rng.integers(2, 5, m).astype(np.int32)
        rnd = rng.permutation(m).astype(np.uint32)
        B = m
        lv = np.full(B, 1, np.int32)
        r = mutant(lv, 2, il, ic, None, rnd, 0, 1)
        by_key = np.argsort(rnd, kind="stable")
        ok = all(r[1][t] == 1 and r[2][t] == by_key[t] and r[3][t] == 0 for t in range(B))
        ok = ok and np.all(r[4] <= 1)
        caught |= not ok
    assert caught
