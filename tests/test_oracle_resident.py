"""Pins of the reference's resident-aware fallback and level histogram (CPU only).

The fallback is checked against an independent formulation (the maximum over
the resident neighbours under the order score desc, entry asc, by
np.lexsort), against the special cases (every entry resident: the top-1;
none: NaN and -1), and against invalid neighbours (-1 entries).  The
histogram is checked against np.bincount.
"""
import numpy as np

from oracle import oracle


def _sorted_lists(rng, b, k, n):
    s = np.round(rng.uniform(-1, 1, (b, k)), 2).astype(np.float32)   # ties on purpose
    idx = np.stack([rng.choice(n, k, replace=False) for _ in range(b)]).astype(np.int64)
    for q in range(b):
        o = np.lexsort((idx[q], -s[q].astype(np.float64)))
        s[q], idx[q] = s[q][o], idx[q][o]
    return s, idx


def test_resident_best_is_best_resident_by_lexsort():
    rng = np.random.default_rng(41)
    n, b, k = 300, 200, 12
    s, idx = _sorted_lists(rng, b, k, n)
    soe = np.where(rng.random(n) < 0.2, rng.integers(0, 50, n), -1)
    soe[rng.integers(0, n, 10)] = 60                              # slots past n_slots are not resident
    got_s, got_i = oracle.resident_best(s, idx, k, soe, 50)
    for q in range(b):
        res = [j for j in range(k) if 0 <= soe[idx[q, j]] < 50]
        if not res:
            assert got_i[q] == -1 and np.isnan(got_s[q])
            continue
        o = np.lexsort((idx[q, res], -s[q, res].astype(np.float64)))
        j = res[o[0]]
        assert got_i[q] == idx[q, j] and got_s[q] == s[q, j]


def test_resident_best_special_cases():
    rng = np.random.default_rng(42)
    s, idx = _sorted_lists(rng, 30, 5, 100)
    gs, gi = oracle.resident_best(s, idx, 5, None, 100)            # all resident: the top-1
    assert np.array_equal(gi, idx[:, 0]) and np.array_equal(gs, s[:, 0])
    gs, gi = oracle.resident_best(s, idx, 5, np.full(100, -1), 10)  # none resident
    assert (gi == -1).all() and np.isnan(gs).all()
    idx2 = idx.copy()
    idx2[:, 0] = -1                                                 # an invalid first neighbour is skipped
    gs, gi = oracle.resident_best(s, idx2, 5, None, 100)
    assert np.array_equal(gi, idx[:, 1])
    gs, gi = oracle.resident_best(s, idx, 1, None, 100)             # k = 1
    assert np.array_equal(gi, idx[:, 0])


def test_level_histogram_is_bincount():
    rng = np.random.default_rng(43)
    for L in (0, 1, 5, 32):
        lv = rng.integers(-1, L + 2, 1000)
        H = oracle.level_histogram(lv, L)
        ok = lv[(lv >= 0) & (lv <= L)]
        assert np.array_equal(H, np.bincount(ok, minlength=L + 1)[: L + 1])
        assert H.sum() == ok.size
