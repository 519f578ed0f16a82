"""Pins of the reference's capacity-constrained assignment and latent gather (CPU only).

The assignment is checked against a hand-worked example, against a second
formulation written level by level (exhaustively on tiny instances), against
a property characterisation and closed forms; planted mistakes in a copy of
the second formulation must be caught by the same checks.  The gather is
checked against numpy indexing.
"""
import itertools
import os

import numpy as np
import pytest

from oracle import pyref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_golden():
    vals = {}
    for line in open(os.path.join(GOLDEN, "assign_worked.txt")):
        if line.startswith("#") or not line.strip():
            continue
        key, *rest = line.split()
        vals[key] = [int(x) for x in rest]
    return vals


def test_assign_hand_worked(orc):
    g = _load_golden()
    L = g["L"][0]
    ol, oi, os_, fill = orc.assign(np.array(g["level"]), L, g["inst_level"], g["inst_cap"],
                                   g["inst_queue"])
    assert ol.tolist() == g["out_level"]
    assert oi.tolist() == g["out_inst"]
    assert os_.tolist() == g["out_slot"]
    assert fill.tolist() == g["inst_fill"]
    # the second formulation agrees with the hand-worked result as well
    r = pyref.assign_by_level(g["level"], L, g["inst_level"], g["inst_cap"], g["inst_queue"])
    assert list(r) == [g["out_level"], g["out_inst"], g["out_slot"], g["inst_fill"]]


def _run_both(orc, level, L, il, ic, iq):
    got = orc.assign(np.array(level, np.int32), L, il, ic, iq)
    got = [a.tolist() for a in got]
    want = pyref.assign_by_level(level, L, il, ic, iq)
    return got, list(want)


def test_assign_exhaustive_tiny(orc):
    """Every level vector and instance table up to B=3, L=2, I=2, cap<=2, queue in {0,1}."""
    n = 0
    for L in (0, 1, 2):
        for I in (0, 1, 2):
            tables = list(itertools.product(range(L + 1), range(3), range(2)))
            for tab in itertools.product(tables, repeat=I):
                il = [t[0] for t in tab]
                ic = [t[1] for t in tab]
                iq = [t[2] for t in tab]
                for B in (0, 1, 2, 3):
                    for level in itertools.product(range(L + 1), repeat=B):
                        got, want = _run_both(orc, list(level), L, il, ic, iq)
                        assert got == want, (L, il, ic, iq, level)
                        n += 1
    assert n > 5000


def test_assign_random_against_second_formulation_and_properties(orc):
    rng = np.random.default_rng(21)
    for trial in range(400):
        L = int(rng.integers(0, 6))
        I = int(rng.integers(0, 9))
        B = int(rng.integers(0, 40))
        il = rng.integers(0, L + 1, I).tolist()
        ic = rng.integers(0, 6, I).tolist()
        iq = rng.integers(0, 4, I).tolist() if trial % 3 else None
        level = rng.integers(0, L + 1, B).tolist()
        got, want = _run_both(orc, level, L, il, ic, iq)
        assert got == want
        errs = pyref.check_assignment(level, L, il, ic, iq, *got)
        assert not errs, errs
        # closed forms
        R = np.zeros(L + 1, int)
        for i in range(I):
            R[il[i]] += ic[i]
        ol = np.array(got[0])
        assert (ol >= 0).sum() == min(B, R.sum())
        demand = np.bincount(np.array(level, int), minlength=L + 1) if B else np.zeros(L + 1, int)
        first = sum((ol == np.array(level)) & (ol >= 0))
        assert first == np.minimum(demand, R).sum()
        if np.all(R >= demand):
            assert np.array_equal(ol, np.array(level))


def test_assign_redirects_down_before_up(orc):
    # level 2 full; levels 1 and 3 both free: the query goes down to 1
    ol, oi, os_, fill = orc.assign(np.array([2, 2]), 3, [2, 1, 3], [1, 5, 5], None)
    assert ol.tolist() == [2, 1]
    # nothing below: up to the closest level above
    ol, *_ = orc.assign(np.array([0, 0]), 3, [0, 2, 1], [1, 5, 5], None)
    assert ol.tolist() == [0, 1]


def test_assign_longest_queue_first(orc):
    ol, oi, os_, fill = orc.assign(np.array([1, 1, 1]), 1, [1, 1, 1], [1, 1, 1], [2, 7, 2])
    assert oi.tolist() == [1, 0, 2]
    assert fill.tolist() == [1, 1, 1]


def test_assign_rejects_bad_tables(orc):
    with pytest.raises(ValueError):
        orc.assign(np.array([0]), 1, [2], [1], None)        # level out of range
    with pytest.raises(ValueError):
        orc.assign(np.array([0]), 1, [0], [-1], None)       # negative capacity
    with pytest.raises(ValueError):
        orc.assign(np.array([3]), 1, [0], [1], None)        # query level out of range


def _mutant_up_first(level, L, il, ic, iq):
    """Planted mistake: redirect upwards before downwards."""
    B, I = len(level), len(il)
    q_ = list(iq) if iq is not None else [0] * I
    seats = {p: [] for p in range(L + 1)}
    for i in sorted(range(I), key=lambda i: (-q_[i], i)):
        seats[il[i]].extend((i, s) for s in range(ic[i]))
    taken = {p: 0 for p in range(L + 1)}
    out = [[-1] * B for _ in range(3)]
    for r in range(L + 1):
        for q in range(B):
            if out[0][q] >= 0:
                continue
            lam = level[q]
            up = list(range(lam, L + 1)) + list(range(lam - 1, -1, -1))
            p = up[r]
            if taken[p] < len(seats[p]):
                out[0][q] = p
                out[1][q], out[2][q] = seats[p][taken[p]]
                taken[p] += 1
    fill = [sum(1 for q in range(B) if out[1][q] == i) for i in range(I)]
    return out[0], out[1], out[2], fill


def _mutant_queue_ignored(level, L, il, ic, iq):
    """Planted mistake: instances in index order, ignoring queue lengths."""
    return pyref.assign_by_level(level, L, il, ic, None)


@pytest.mark.parametrize("mutant", [_mutant_up_first, _mutant_queue_ignored])
def test_planted_mistakes_are_caught(orc, mutant):
    rng = np.random.default_rng(33)
    caught = 0
    for trial in range(200):
        L, I, B = 3, 5, 12
        il = rng.integers(0, L + 1, I).tolist()
        ic = rng.integers(0, 4, I).tolist()
        iq = rng.integers(0, 5, I).tolist()
        level = rng.integers(0, L + 1, B).tolist()
        m = list(mutant(level, L, il, ic, iq))
        good = [a.tolist() for a in orc.assign(np.array(level), L, il, ic, iq)]
        if m != good:
            assert pyref.check_assignment(level, L, il, ic, iq, *m), "mutant passed the checks"
            caught += 1
    assert caught > 20


def test_gather_matches_numpy_indexing(orc):
    rng = np.random.default_rng(8)
    n_entries, n_slots, lb = 50, 20, 48
    pool = rng.integers(0, 256, size=(n_slots, lb), dtype=np.uint8)
    soe = np.full(n_entries, -1, np.int32)
    hot = rng.choice(n_entries, n_slots, replace=False)
    soe[hot] = np.arange(n_slots)
    B, n_inst, spi = 30, 3, 10
    top1 = rng.integers(0, n_entries, B)
    top1[:5] = hot[:5]
    ol = rng.integers(-1, 3, B).astype(np.int32)
    perm = rng.permutation(n_inst * spi)[:B]
    oi = (perm // spi).astype(np.int32)
    os_ = (perm % spi).astype(np.int32)
    oi[ol < 0] = -1
    os_[ol < 0] = -1
    batch = np.zeros((n_inst * spi, lb), np.uint8)
    hit = orc.gather(top1, ol, oi, os_, soe, n_entries, pool, n_inst, spi, batch)
    want = np.zeros_like(batch)
    exp_hit = np.zeros(B, np.int32)
    for q in range(B):
        if ol[q] > 0 and soe[top1[q]] >= 0:
            want[oi[q] * spi + os_[q]] = pool[soe[top1[q]]]
            exp_hit[q] = 1
    assert np.array_equal(hit, exp_hit)
    assert np.array_equal(batch, want)
    assert exp_hit.sum() > 0
    # identity map
    batch2 = np.zeros((n_inst * spi, lb), np.uint8)
    top1b = rng.integers(0, n_slots, B)
    hit2 = orc.gather(top1b, ol, oi, os_, None, n_slots, pool, n_inst, spi, batch2)
    sel = (ol > 0)
    assert np.array_equal(hit2, sel.astype(np.int32))
    assert np.array_equal(batch2[(oi * spi + os_)[sel]], pool[top1b[sel]])
