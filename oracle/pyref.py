"""Small exact twins of the reference, for exhaustive tests on tiny inputs.

TEST INFRASTRUCTURE ONLY.  Written independently of apc_oracle.c (other loop
structure, exact rational arithmetic) so that the tests can pin the float64
reference against it.  Pure Python; meant for inputs of a few elements.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple


def cos_key(q: Sequence[int], e: Sequence[int]) -> Fraction:
    """Exact monotone image of the cosine of two integer vectors.

    sign(<q,e>) * <q,e>^2 / (|q|^2 |e|^2) is a strictly increasing function
    of the cosine, and rational for integer vectors.
    """
    dot = sum(a * b for a, b in zip(q, e))
    nq = sum(a * a for a in q)
    ne = sum(b * b for b in e)
    if nq == 0 or ne == 0:
        raise ValueError("zero vector")
    key = Fraction(dot * dot, nq * ne)
    return key if dot >= 0 else -key


def cos_float(key: Fraction) -> float:
    """Cosine value (float) from the exact key."""
    import math
    v = math.sqrt(abs(key))
    return v if key >= 0 else -v


def exact_topk(q: Sequence[int], entries: Sequence[Sequence[int]], k: int) -> List[int]:
    """Indices of the k best entries by (cosine desc, index asc), exactly."""
    keyed = [(cos_key(q, e), i) for i, e in enumerate(entries)]
    keyed.sort(key=lambda t: (-t[0], t[1]))
    return [i for _, i in keyed[:k]]


def exact_level(q: Sequence[int], e: Sequence[int], theta: Sequence[float]) -> int:
    """Level of a best match given exactly: #{theta_l <= cos(q, e)}, theta as floats."""
    key = cos_key(q, e)
    lv = 0
    for t in theta:
        tf = Fraction(t)                          # exact value of the float
        tkey = tf * tf if tf >= 0 else -(tf * tf)  # same monotone map as cos_key
        if key >= tkey:
            lv += 1
    return lv


def assign_by_level(level: Sequence[int], L: int, inst_level: Sequence[int],
                    inst_cap: Sequence[int], inst_queue=None) -> Tuple[list, list, list, list]:
    """Assignment computed level by level.

    In round r every unassigned query applies to the r-th entry of its
    preference list [lam, lam-1, .., 0, lam+1, .., L].  Applications to
    different levels do not interact within a round, so each level admits
    the lowest-indexed applicants up to its remaining capacity.  Seats of a
    level are the (instance, slot) pairs of its instances in the order
    (queue desc, index asc), handed out in admission order.
    """
    B, I = len(level), len(inst_level)
    queue = list(inst_queue) if inst_queue is not None else [0] * I
    seats = {p: [] for p in range(L + 1)}
    for i in sorted(range(I), key=lambda i: (-queue[i], i)):
        seats[inst_level[i]].extend((i, s) for s in range(inst_cap[i]))
    taken = {p: 0 for p in range(L + 1)}
    out_level = [-1] * B
    out_inst = [-1] * B
    out_slot = [-1] * B
    for r in range(L + 1):
        applicants = {p: [] for p in range(L + 1)}
        for q in range(B):
            if out_level[q] < 0:
                lam = level[q]
                p = lam - r if r <= lam else r
                applicants[p].append(q)
        for p in range(L + 1):
            room = len(seats[p]) - taken[p]
            for q in applicants[p][:max(room, 0)]:
                out_level[q] = p
                out_inst[q], out_slot[q] = seats[p][taken[p]]
                taken[p] += 1
    fill = [0] * I
    for q in range(B):
        if out_inst[q] >= 0:
            fill[out_inst[q]] += 1
    return out_level, out_inst, out_slot, fill


def check_assignment(level, L, inst_level, inst_cap, inst_queue, out_level, out_inst, out_slot,
                     fill) -> List[str]:
    """Properties that characterise the assignment; returns the violated ones.

    * every (instance, slot) is used at most once and within capacity, and an
      instance's slots are 0..fill-1;
    * a query is placed at an instance of its assigned level;
    * no justified waste: every level a query prefers to its assignment is
      full; an unassigned query finds every level full;
    * rounds: at each preference rank, a level admits the lowest-index
      prefix of the queries that reach it at that rank, exactly as many as
      its remaining capacity allows;
    * admissions of a level fill its seats in (rank, index) order.
    """
    errs = []
    B, I = len(level), len(inst_level)
    queue = list(inst_queue) if inst_queue is not None else [0] * I
    R = [0] * (L + 1)
    for i in range(I):
        R[inst_level[i]] += inst_cap[i]
    used = [0] * (L + 1)
    seen = set()
    cnt = [0] * I
    for q in range(B):
        if out_level[q] < 0:
            if out_inst[q] != -1 or out_slot[q] != -1:
                errs.append(f"q{q}: unassigned but has inst/slot")
            continue
        used[out_level[q]] += 1
        i, s = out_inst[q], out_slot[q]
        if not (0 <= i < I) or inst_level[i] != out_level[q]:
            errs.append(f"q{q}: instance {i} not at level {out_level[q]}")
            continue
        if not (0 <= s < inst_cap[i]) or (i, s) in seen:
            errs.append(f"q{q}: bad or repeated slot {(i, s)}")
        seen.add((i, s))
        cnt[i] += 1
    if cnt != list(fill):
        errs.append(f"fill {list(fill)} != counted {cnt}")
    for i in range(I):
        if {s for (j, s) in seen if j == i} != set(range(cnt[i])):
            errs.append(f"instance {i}: slots not contiguous from 0")

    def prefs(lam):
        return [lam - r if r <= lam else r for r in range(L + 1)]

    rank_of = {}
    for q in range(B):
        P = prefs(level[q])
        r_q = P.index(out_level[q]) if out_level[q] >= 0 else L + 1
        rank_of[q] = r_q
        for p in P[:r_q]:
            if used[p] < R[p]:
                errs.append(f"q{q}: level {p} preferred and not full")
    # rank by rank: a level admits the lowest-index prefix of the queries that
    # reach it at that rank, as many as its remaining capacity allows
    admitted_before = [0] * (L + 1)
    for r in range(L + 1):
        for p in range(L + 1):
            appl = [q for q in range(B) if rank_of[q] >= r and prefs(level[q])[r] == p]
            adm = [q for q in appl if rank_of[q] == r]
            if adm != appl[:len(adm)]:
                errs.append(f"round {r} level {p}: admitted {adm} not a prefix of {appl}")
            if len(adm) != min(len(appl), R[p] - admitted_before[p]):
                errs.append(f"round {r} level {p}: admitted {len(adm)} of {len(appl)} "
                            f"with {R[p] - admitted_before[p]} places left")
        for p in range(L + 1):
            admitted_before[p] += sum(1 for q in range(B) if rank_of[q] == r and out_level[q] == p)
    # seat order within a level follows (rank, index)
    order = sorted(range(I), key=lambda i: (-queue[i], i))
    for p in range(L + 1):
        seats = [(i, s) for i in order if inst_level[i] == p for s in range(inst_cap[i])]
        adm = sorted((q for q in range(B) if out_level[q] == p), key=lambda q: (rank_of[q], q))
        got = [(out_inst[q], out_slot[q]) for q in adm]
        if got != seats[:len(adm)]:
            errs.append(f"level {p}: seats {got} not in order {seats[:len(adm)]}")
    return errs
