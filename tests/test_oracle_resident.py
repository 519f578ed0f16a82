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


def test_gather_at_level_one_latent_per_entry_is_gather():
    rng = np.random.default_rng(44)
    n, n_slots, lb, b, n_inst, spi = 400, 90, 32, 120, 4, 40
    pool = rng.integers(0, 256, (n_slots, lb), dtype=np.uint8)
    soe = np.full(n, -1, np.int32)
    soe[rng.choice(n, n_slots, replace=False)] = np.arange(n_slots)
    top1 = rng.integers(-1, n, b)
    perm = rng.permutation(n_inst * spi)[:b]
    ol = rng.integers(-1, 4, b).astype(np.int32)
    oi, os_ = (perm // spi).astype(np.int32), (perm % spi).astype(np.int32)
    want = np.zeros((n_inst * spi, lb), np.uint8)
    got = np.zeros_like(want)
    h1 = oracle.gather(top1, ol, oi, os_, soe, n, pool, n_inst, spi, want)
    h2 = oracle.gather_at_level(top1, ol, oi, os_, soe, n, pool, 1, n_inst, spi, got)
    assert np.array_equal(h1, h2) and np.array_equal(want, got) and h1.sum() > 0


def test_gather_at_level_reads_the_level_row():
    # every pool row holds its own (slot, level) code, so the copy names its source
    rng = np.random.default_rng(45)
    n, S, Lp, b, n_inst, spi = 300, 50, 5, 200, 3, 80
    pool = np.zeros((S * Lp, 16), np.uint8)
    for s in range(S):
        for lv in range(1, Lp + 1):
            pool[s * Lp + lv - 1, :2] = (s, lv)
    soe = np.full(n, -1, np.int32)
    ent = rng.choice(n, S, replace=False)
    soe[ent] = np.arange(S)
    top1 = rng.integers(0, n, b)
    top1[: b // 2] = ent[rng.integers(0, S, b // 2)]
    ol = rng.integers(-1, Lp + 2, b).astype(np.int32)
    perm = rng.permutation(n_inst * spi)[:b]
    oi, os_ = (perm // spi).astype(np.int32), (perm % spi).astype(np.int32)
    batch = np.full((n_inst * spi, 16), 255, np.uint8)
    hit = oracle.gather_at_level(top1, ol, oi, os_, soe, n, pool, Lp, n_inst, spi, batch)
    for q in range(b):
        ok = 1 <= ol[q] <= Lp and soe[top1[q]] >= 0
        assert hit[q] == ok
        row = batch[oi[q] * spi + os_[q]]
        if ok:
            assert tuple(row[:2]) == (soe[top1[q]], ol[q])
        else:
            assert (row == 255).all()
