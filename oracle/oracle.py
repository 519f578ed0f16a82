"""Python binding of the float64 CPU reference (apc_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library.  Shares no code with the
HIP path.  Inputs are host numpy arrays holding the exact stored bytes.
The Route-Plan (Eq. 1) and the placement that follows it are plain Python:
the plan is scipy's LP solver on the transportation problem, the placement a
loop over queries.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "apc_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

DT = {"f32": 0, "f16": 1, "bf16": 2, "e4m3": 3}
OK, E_ARG, E_NONFINITE, E_ZERO_NORM, E_NOMEM = 0, 1, 2, 3, 4


CLANG = "/opt/rocm/lib/llvm/bin/clang"


def build(sanitize_dir: str = "") -> str:
    """Compile the reference with gcc (OpenMP, no HIP).  With sanitize_dir, a
    copy instrumented by AddressSanitizer and UndefinedBehaviorSanitizer
    instead (clang, against its shared sanitizer runtime), written there."""
    if sanitize_dir:
        out = os.path.join(sanitize_dir, "liboracle.so")
        cmd = [CLANG, "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libasan",
               "-o", out, SRC, "-lm"]
        subprocess.run(cmd, check=True)
        return out
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           "-o", LIB, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return LIB


_lib = None


def lib():
    """The reference library: liboracle.so beside this file, or the build
    APC_ORACLE_LIB names (the sanitizer test runs the suite on such a copy)."""
    global _lib
    if _lib is None:
        path = os.environ.get("APC_ORACLE_LIB", "")
        if not path:
            path = LIB
            if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
                build()
        L = ctypes.CDLL(path)
        vp, i64, i32, dp = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        L.oracle_decode.argtypes = [ctypes.c_int, vp, vp, i64, i32, dp]
        L.oracle_row_sqnorms.argtypes = [ctypes.c_int, vp, vp, i64, i32, dp, vp]
        L.oracle_pair_scores.argtypes = [ctypes.c_int, vp, vp, dp, vp, vp, dp, i32, i64, vp, vp, dp]
        L.oracle_topk.argtypes = [ctypes.c_int, vp, vp, dp, i64, vp, vp, dp, i64, i32, i32,
                                  ctypes.c_int, dp, vp]
        L.oracle_levels.argtypes = [dp, i64, i32, vp, vp]
        L.oracle_assign.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp]
        L.oracle_gather.argtypes = [vp, i64, vp, vp, vp, vp, i64, vp, i64, i64, i32, i32, vp, vp]
        L.oracle_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _raw(rows: np.ndarray) -> np.ndarray:
    """Contiguous host array of the stored elements (any 1/2/4-byte view)."""
    return np.ascontiguousarray(rows)


def _check(rc, what):
    if rc != OK:
        raise ValueError(f"{what}: reference returned status {rc}")


def decode(dtype: str, rows: np.ndarray, scale=None) -> np.ndarray:
    rows = _raw(rows)
    n, d = rows.shape
    out = np.empty((n, d), dtype=np.float64)
    sc = None if scale is None else np.ascontiguousarray(scale, dtype=np.float32)
    _check(lib().oracle_decode(DT[dtype], _p(rows), _p(sc), n, d, _p(out)), "decode")
    return out


def row_sqnorms(dtype: str, rows: np.ndarray, scale=None):
    """(squared norms float64[n], status, first bad row)."""
    rows = _raw(rows)
    n, d = rows.shape
    out = np.empty(n, dtype=np.float64)
    bad = np.array([-1], dtype=np.int64)
    sc = None if scale is None else np.ascontiguousarray(scale, dtype=np.float32)
    rc = lib().oracle_row_sqnorms(DT[dtype], _p(rows), _p(sc), n, d, _p(out), _p(bad))
    if rc == E_ARG:
        raise ValueError("row_sqnorms: bad arguments")
    return out, rc, int(bad[0])


def _sq(dtype, rows, scale, sq, what):
    if sq is not None:
        return sq
    sq, rc, _ = row_sqnorms(dtype, rows, scale)
    _check(rc, what)
    return sq


def topk(dtype: str, q: np.ndarray, q_scale, e: np.ndarray, e_scale, k: int,
         threads: int = 0, q_sq=None, e_sq=None):
    """Exact top-k (scores float64[b,k], indices int64[b,k]) of each query row."""
    q, e = _raw(q), _raw(e)
    b, d = q.shape
    n = e.shape[0]
    qs = None if q_scale is None else np.ascontiguousarray(q_scale, dtype=np.float32)
    es = None if e_scale is None else np.ascontiguousarray(e_scale, dtype=np.float32)
    q_sq = _sq(dtype, q, qs, q_sq, "query norms")
    e_sq = _sq(dtype, e, es, e_sq, "entry norms")
    ts = np.empty((b, k), dtype=np.float64)
    ti = np.empty((b, k), dtype=np.int64)
    _check(lib().oracle_topk(DT[dtype], _p(q), _p(qs), _p(q_sq), b, _p(e), _p(es), _p(e_sq),
                             n, d, k, threads, _p(ts), _p(ti)), "topk")
    return ts, ti


def pair_scores(dtype: str, q, q_scale, e, e_scale, qi, ei, q_sq=None, e_sq=None):
    """Scores of the (qi[p], ei[p]) pairs."""
    q, e = _raw(q), _raw(e)
    d = q.shape[1]
    qs = None if q_scale is None else np.ascontiguousarray(q_scale, dtype=np.float32)
    es = None if e_scale is None else np.ascontiguousarray(e_scale, dtype=np.float32)
    q_sq = _sq(dtype, q, qs, q_sq, "query norms")
    e_sq = _sq(dtype, e, es, e_sq, "entry norms")
    qi = np.ascontiguousarray(qi, dtype=np.int64).ravel()
    ei = np.ascontiguousarray(ei, dtype=np.int64).ravel()
    out = np.empty(qi.size, dtype=np.float64)
    _check(lib().oracle_pair_scores(DT[dtype], _p(q), _p(qs), _p(q_sq), _p(e), _p(es),
                                    _p(e_sq), d, qi.size, _p(qi), _p(ei), _p(out)), "pair_scores")
    return out


def levels(best: np.ndarray, theta: np.ndarray) -> np.ndarray:
    best = np.ascontiguousarray(best, dtype=np.float64)
    theta = np.ascontiguousarray(theta, dtype=np.float32)
    out = np.empty(best.size, dtype=np.int32)
    _check(lib().oracle_levels(_p(best), best.size, theta.size, _p(theta), _p(out)), "levels")
    return out


def assign(level: np.ndarray, L: int, inst_level, inst_cap, inst_queue=None):
    """(out_level, out_inst, out_slot, inst_fill), all int32."""
    level = np.ascontiguousarray(level, dtype=np.int32)
    il = np.ascontiguousarray(inst_level, dtype=np.int32)
    ic = np.ascontiguousarray(inst_cap, dtype=np.int32)
    iq = None if inst_queue is None else np.ascontiguousarray(inst_queue, dtype=np.int32)
    b, n = level.size, il.size
    ol, oi, os_ = (np.empty(b, dtype=np.int32) for _ in range(3))
    fill = np.empty(n, dtype=np.int32)
    _check(lib().oracle_assign(_p(level), b, L, n, _p(il), _p(ic), _p(iq),
                               _p(ol), _p(oi), _p(os_), _p(fill)), "assign")
    return ol, oi, os_, fill


# ---- Load-aware route-and-batch (the Query Dispatcher's routing) ------------
# Reading of the Approach's Query Dispatcher paragraph: the dispatcher routes
# by load.  At or above the load threshold it routes greedily: the instances
# of a level are filled longest queue first, each up to its capacity (its
# optimal batch), which is the placement `assign` computes.  Below the
# threshold routing is uniform at batch size 1: every instance of a level
# takes at most one query, and the level's admitted queries go to its
# instances in the order of caller-drawn random keys (ascending, then
# instance index), so that with keys drawn uniformly at random each admitted
# query lands on a uniformly random instance of its level, one per instance.
# Levels and redirections between levels are those of `assign` in both modes.
def assign_load_aware(level, L: int, inst_level, inst_cap, inst_queue, inst_rand, load: int, threshold: int):
    """(routing, out_level, out_inst, out_slot, inst_fill); routing 1 = greedy, 0 = uniform."""
    if load >= threshold:
        return (1,) + tuple(assign(level, L, inst_level, inst_cap, inst_queue))
    il = np.asarray(inst_level, dtype=np.int64)
    ic = np.asarray(inst_cap, dtype=np.int64)
    rnd = np.asarray(inst_rand, dtype=np.uint64)
    n = il.size
    batch1 = np.minimum(ic, 1).astype(np.int32)                 # batch size 1
    order = sorted(range(n), key=lambda i: (int(rnd[i]), i))      # the random order of the instances
    # `assign` fills a level's instances by (queue desc, index asc): queue
    # lengths n, n - 1, ... in the random order make it fill in that order
    queue = np.empty(n, dtype=np.int32)
    for pos, i in enumerate(order):
        queue[i] = n - pos
    return (0,) + tuple(assign(level, L, il.astype(np.int32), batch1, queue))


def gather(top1, out_level, out_inst, out_slot, slot_of_entry, n_entries, pool: np.ndarray,
           n_inst: int, slots_per_inst: int, batch: np.ndarray):
    """Copies into `batch` (uint8 [n_inst*slots_per_inst, latent_bytes]) in place; returns hit."""
    top1 = np.ascontiguousarray(top1, dtype=np.int64)
    b = top1.size
    soe = None if slot_of_entry is None else np.ascontiguousarray(slot_of_entry, dtype=np.int32)
    pool = np.ascontiguousarray(pool, dtype=np.uint8)
    assert batch.flags.c_contiguous and batch.dtype == np.uint8
    hit = np.empty(b, dtype=np.int32)
    ol = np.ascontiguousarray(out_level, dtype=np.int32)
    oi = np.ascontiguousarray(out_inst, dtype=np.int32)
    os_ = np.ascontiguousarray(out_slot, dtype=np.int32)
    _check(lib().oracle_gather(_p(top1), b, _p(ol), _p(oi), _p(os_), _p(soe), n_entries,
                               _p(pool), pool.shape[0], pool.shape[1] if pool.ndim == 2 else 0,
                               n_inst, slots_per_inst, _p(batch), _p(hit)), "gather")
    return hit


def max_threads() -> int:
    return int(lib().oracle_max_threads())


# ---- Route-Plan (the K-to-K' Route Planner, Eq. 1) -------------------------
# Reading of Eq. 1 (its constraint set is not printed): x[i, j] queries of
# optimal level i are served at level j; a query is served at most once and
# level j serves at most F[j]; serving level i at a level with more skipped
# steps (K_j > K_i) degrades it by D = K_j - K_i, serving it at fewer skipped
# steps costs nothing (Eq. 1 sums over K'_j > K_i only).  Queries that no
# capacity can take stay unserved; the cost of leaving one unserved exceeds
# any single move's degradation, so an optimum serves min(sum H, sum F).


def _degradation_matrix(K):
    Kf = np.concatenate([[0], np.asarray(K, dtype=np.int64)])
    n = Kf.size
    return np.array([[max(0, int(Kf[j] - Kf[i])) for j in range(n)] for i in range(n)], dtype=np.int64)


def route_plan(H, F, K):
    """Optimal integer plan x ((L+1) x (L+1), int64), its degradation and the
    number served, by scipy's LP solver (HiGHS dual simplex) on the
    transportation problem above.  H, F: per-level demand and capacity
    (levels 0..L); K: skipped steps of levels 1..L (level 0 skips none).
    A basic optimal solution of a transportation problem with integral
    supplies and capacities is integral; the function checks that it is."""
    from scipy.optimize import linprog
    H = np.asarray(H, dtype=np.int64)
    F = np.asarray(F, dtype=np.int64)
    n = H.size
    cost = _degradation_matrix(K).astype(np.float64)
    unserved = float(cost.max() + 1.0)
    c = np.concatenate([cost.ravel(), np.full(n, unserved)])
    A_eq = np.zeros((n, n * n + n))                  # row i: sum_j x[i, j] + unserved_i = H[i]
    for i in range(n):
        A_eq[i, i * n:(i + 1) * n] = 1.0
        A_eq[i, n * n + i] = 1.0
    A_ub = np.zeros((n, n * n + n))                  # column j: sum_i x[i, j] <= F[j]
    for j in range(n):
        A_ub[j, j:n * n:n] = 1.0
    res = linprog(c, A_ub=A_ub, b_ub=F.astype(np.float64), A_eq=A_eq, b_eq=H.astype(np.float64),
                  bounds=(0, None), method="highs-ds")
    if res.status != 0:
        raise RuntimeError(f"route_plan: LP failed: {res.message}")
    x = res.x[:n * n].reshape(n, n)
    xi = np.rint(x).astype(np.int64)
    if np.abs(x - xi).max() > 1e-6:
        raise RuntimeError("route_plan: the LP vertex is not integral")
    d, served = plan_cost(xi, K)
    return xi, d, served


def plan_cost(x, K):
    """(degradation, number served) of a plan x under the reading above."""
    x = np.asarray(x, dtype=np.int64)
    return int((x * _degradation_matrix(K)).sum()), int(x.sum())


def preference(lam: int, L: int):
    """Redirection order of a query of optimal level lam: its own level, then
    the levels below it, closest first, then the levels above it, closest
    first (the Approach's K-to-K' redirection)."""
    return [lam] + list(range(lam - 1, -1, -1)) + list(range(lam + 1, L + 1))


def assign_routed(level, L: int, x, inst_level, inst_cap, inst_queue=None):
    """Placement that follows a route plan x (negative entries count as 0).
    The queries of optimal level i, in index order, take the levels of their
    preference list in that order, x[i, j] of them for level j; queries past
    sum_j x[i, j] get none.  A level then admits the queries routed to it by
    (position of the level in the query's preference list, query index) while
    it has places; admission rank t lands on the level's instances ordered by
    (queue desc, index asc), each filled to its capacity, slots from 0.
    Given the flow that the rounds placement (assign) realises, this returns
    exactly that placement.  Returns (out_level, out_inst, out_slot,
    inst_fill), int32."""
    level = np.asarray(level, dtype=np.int64)
    x = np.maximum(np.asarray(x, dtype=np.int64), 0)
    b, n_inst = level.size, len(inst_level)
    seen = [0] * (L + 1)
    want = np.full(b, -1, dtype=np.int64)
    rnd = np.full(b, -1, dtype=np.int64)
    for q in range(b):
        i = int(level[q])
        r = seen[i]
        seen[i] += 1
        acc = 0
        for pos, j in enumerate(preference(i, L)):
            acc += int(x[i, j])
            if r < acc:
                want[q], rnd[q] = j, pos
                break
    cap = [0] * (L + 1)
    for a in range(n_inst):
        cap[inst_level[a]] += int(inst_cap[a])
    queue = [0] * n_inst if inst_queue is None else list(inst_queue)
    order = sorted(range(n_inst), key=lambda a: (inst_level[a], -queue[a], a))
    used = [0] * (L + 1)
    out_level = np.full(b, -1, dtype=np.int32)
    out_inst = np.full(b, -1, dtype=np.int32)
    out_slot = np.full(b, -1, dtype=np.int32)
    fill = np.zeros(n_inst, dtype=np.int32)
    for r in range(L + 1):
        for q in range(b):
            if rnd[q] != r:
                continue
            j = int(want[q])
            t = used[j]
            if t >= cap[j]:
                continue
            used[j] += 1
            out_level[q] = j
            for a in order:
                if inst_level[a] != j:
                    continue
                if t < inst_cap[a]:
                    out_inst[q], out_slot[q] = a, t
                    fill[a] += 1
                    break
                t -= inst_cap[a]
    return out_level, out_inst, out_slot, fill


# ---- Resident-aware fallback and the level histogram -----------------------
# A query can only start from a cached state that is resident.  Reading: when
# its nearest entry's latent is not resident, the query falls back to the best
# of its k neighbours whose latent is; the level then follows that
# neighbour's score.  With none resident it gets no score (NaN, level 0).

def resident_best(top_score, top_idx, k: int, slot_of_entry, n_slots: int):
    """For each query row of the (b, >= k) top lists: (score, entry) of the
    first of its k neighbours with a resident latent (slot_of_entry[e] >= 0
    and < n_slots; slot_of_entry None means entry e lives in slot e), else
    (NaN, -1).  The lists are ordered best first, so the first is the best."""
    top_score = np.asarray(top_score, dtype=np.float32)
    top_idx = np.asarray(top_idx, dtype=np.int64)
    b = top_idx.shape[0]
    out_s = np.full(b, np.nan, dtype=np.float32)
    out_i = np.full(b, -1, dtype=np.int32)
    for q in range(b):
        for j in range(k):
            e = int(top_idx[q, j])
            if e < 0:
                continue
            slot = e if slot_of_entry is None else int(slot_of_entry[e])
            if 0 <= slot < n_slots:
                out_s[q], out_i[q] = top_score[q, j], e
                break
    return out_s, out_i


def level_histogram(level, L: int):
    """H[l] = number of queries whose optimal level is l, l = 0..L (values
    outside 0..L are not counted); the per-batch demand of the Optimal-K
    Predictor and of the Route-Plan."""
    H = np.zeros(L + 1, dtype=np.int64)
    for v in np.asarray(level).tolist():
        if 0 <= v <= L:
            H[v] += 1
    return H


# ---- Latents per (entry, level) ---------------------------------------------
# The state after K skipped steps depends on K.  Reading: a resident entry
# holds one latent per level 1..levels_per_slot, stored level-major inside its
# slot (pool row slot * levels_per_slot + level - 1); a query placed at level
# l > 0 copies its entry's latent of level l.  levels_per_slot = 1 keeps one
# latent per entry, used for every level.

def gather_at_level(top1, out_level, out_inst, out_slot, slot_of_entry, n_entries, pool: np.ndarray,
                    levels_per_slot: int, n_inst: int, slots_per_inst: int, batch: np.ndarray):
    """Copies into `batch` in place; returns hit (int32)."""
    pool = np.asarray(pool, dtype=np.uint8)
    n_ent_slots = pool.shape[0] // levels_per_slot
    b = len(top1)
    hit = np.zeros(b, dtype=np.int32)
    for q in range(b):
        lvl, e = int(out_level[q]), int(top1[q])
        if lvl <= 0 or e < 0 or e >= n_entries:
            continue
        if levels_per_slot > 1 and lvl > levels_per_slot:
            continue
        slot = e if slot_of_entry is None else int(slot_of_entry[e])
        if slot < 0 or slot >= n_ent_slots:
            continue
        row = slot * levels_per_slot + (0 if levels_per_slot == 1 else lvl - 1)
        batch[int(out_inst[q]) * slots_per_inst + int(out_slot[q])] = pool[row]
        hit[q] = 1
    return hit


# ---- Merging the top-k lists of cache shards --------------------------------
# With the cache split by rows over several devices, each shard's top-k uses
# its local entry numbers; an entry's global number is its shard's offset plus
# the local one.  The global top-k is the top-k of the union of the shards'
# lists under the total order (score desc, global entry asc), since every
# member of the global top-k is in its own shard's top-k.

def merge_shards(scores, idx, offsets, k: int):
    """scores/idx: (g, b, k_in) lists, best first; offsets: g global offsets.
    Returns (score float32 [b, k], entry int32 [b, k]); slots past the valid
    candidates hold NaN / -1.  Not candidates: entries < 0, NaN scores, and
    global entry numbers of 2^31 - 1 or more (no cache handle holds that many
    entries, and the result is int32)."""
    scores = np.asarray(scores, dtype=np.float32)
    idx = np.asarray(idx, dtype=np.int64)
    g, b, kin = idx.shape
    out_s = np.full((b, k), np.nan, dtype=np.float32)
    out_i = np.full((b, k), -1, dtype=np.int32)
    for q in range(b):
        cand = [(float(scores[s, q, j]), int(idx[s, q, j]) + int(offsets[s]))
                for s in range(g) for j in range(kin)
                if idx[s, q, j] >= 0 and not np.isnan(scores[s, q, j])
                and int(idx[s, q, j]) + int(offsets[s]) < 2**31 - 1]
        cand.sort(key=lambda c: (-c[0], c[1]))
        for j, (sc, e) in enumerate(cand[:k]):
            out_s[q, j], out_i[q, j] = sc, e
    return out_s, out_i


# ---- Storage of float32 rows in a cache type, and row checks ----------------
# The paper keeps prompt embeddings in its cache and fixes no storage type;
# the library's recipe is: binary16 and bfloat16 by rounding each element to
# the nearest representable value (ties to the even one, overflow to +-Inf),
# e4m3fn with one float32 scale per row s = amax / 448 (s = 1 when it is not
# > 0, a row holding NaN included) and the codes of clamp(x / s, -448, 448),
# rounded to the nearest code value with ties to the even code.  Written out
# from the formats' value sets, not from bit tricks.

def e4m3_values() -> np.ndarray:
    """Value of each of the 256 e4m3fn codes (NaN for 0x7f and 0xff): sign,
    4 exponent bits (bias 7), 3 mantissa bits; exponent 0 is subnormal."""
    v = np.empty(256, dtype=np.float64)
    for c in range(256):
        e, m = (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            v[c] = np.nan
            continue
        mag = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
        v[c] = -mag if c & 0x80 else mag
    return v


def _sign_bits(y32: np.ndarray) -> np.ndarray:
    return (y32.view(np.uint32) >> 31).astype(np.uint8)


def round_e4m3(y: np.ndarray) -> np.ndarray:
    """e4m3fn codes of float32 values |y| <= 448 (or NaN): the nearest code
    value, ties to the even code (codes 0..126 grow with their value, and the
    even one of two neighbours has the even mantissa).  NaN gives 0x7f with
    its sign."""
    y32 = np.asarray(y, dtype=np.float32)
    mags = e4m3_values()[:127]                                    # codes 0 .. 126, ascending
    a = np.abs(y32.astype(np.float64))
    if np.any(a[~np.isnan(a)] > 448.0):
        raise ValueError("round_e4m3: |y| > 448")
    hi = np.clip(np.searchsorted(mags, np.nan_to_num(a, nan=0.0), side="left"), 0, 126)
    lo = np.clip(hi - 1, 0, 126)
    dlo, dhi = a - mags[lo], mags[hi] - a
    code = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi))).astype(np.uint8)
    code = np.where(np.isnan(a), 0x7f, code).astype(np.uint8)
    return (code | (_sign_bits(y32) << 7)).astype(np.uint8)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """bfloat16 codes (uint16) of float32 values: of the two bfloat16 values
    around x (its float32 bits with the low 16 cleared, and the next one up in
    magnitude; past the largest finite one stands 2^128, i.e. Inf), the
    nearer, ties to the one with the even code.  NaN gives a quiet NaN of the
    same sign."""
    x32 = np.asarray(x, dtype=np.float32)
    u = x32.view(np.uint32)
    t = u & np.uint32(0xFFFF0000)                                 # toward zero
    up = t + np.uint32(0x10000)                                   # away from zero
    def mag(bits):
        e = (bits >> 23) & 0xFF
        frac = (bits & 0x7FFFFF).astype(np.float64)
        m = np.where(e == 0, frac / 2.0 ** 23 * 2.0 ** -126, (1.0 + frac / 2.0 ** 23) * 2.0 ** (e.astype(np.float64) - 127))
        return np.where(e == 255, 2.0 ** 128, m)                  # the exponent of Inf, as its value would be
    a = np.abs(x32.astype(np.float64))
    dt, du = a - mag(t & 0x7FFFFFFF), mag(up & 0x7FFFFFFF) - a
    pick_up = np.where(du < dt, True, np.where(dt < du, False, ((t >> 16) & 1) == 1))
    out = np.where(pick_up, up >> 16, t >> 16).astype(np.uint32)
    out = np.where(np.isinf(x32), u >> 16, out)                   # +-Inf stays
    out = np.where(np.isnan(x32), (u >> 16) | 0x40, out)
    return out.astype(np.uint16)


def quantize_rows(dtype: str, x: np.ndarray):
    """(stored rows, float32 row scales or None) of float32 rows x."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f16":
        with np.errstate(over="ignore"):
            return x32.astype(np.float16), None
    if dtype == "bf16":
        return round_bf16(x32), None
    if dtype != "e4m3":
        raise ValueError(f"quantize_rows: no such target {dtype}")
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        amax = np.abs(x32).max(axis=1) if x32.shape[1] else np.zeros(x32.shape[0], np.float32)
        s = np.where(np.isnan(x32).any(axis=1), np.float32(np.nan), amax / np.float32(448.0)).astype(np.float32)
        s = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
        y = (x32 / s[:, None]).astype(np.float32)
        y = np.where(np.isnan(y), y, np.clip(y, np.float32(-448.0), np.float32(448.0))).astype(np.float32)
    return round_e4m3(y), s


NONFINITE, ZERO_NORM, BAD_SCALE = 1, 2, 4


def validate_rows(dtype: str, rows: np.ndarray, scale=None) -> np.ndarray:
    """Per-row flags: NONFINITE if an element is not finite or the sum of
    squares reaches 2^128 (it cannot be held in float32); else ZERO_NORM if
    every element is at most 2^-75 in magnitude (each square rounds to zero
    in float32); BAD_SCALE (e4m3) if the row's scale is not finite and > 0.
    For e4m3 the elements are the codes' values (the scale cancels in the
    cosine).  Near the 2^128 boundary a float32 sum may round either way;
    this reads the exact sum."""
    n = np.shape(rows)[0]
    v = decode(dtype, rows, np.ones(n, np.float32) if dtype == "e4m3" else None)
    with np.errstate(over="ignore", invalid="ignore"):
        nonfinite = ~np.isfinite(v).all(axis=1) | ~((v * v).sum(axis=1) < 2.0 ** 128)
    zero = ~nonfinite & (np.abs(np.nan_to_num(v)) <= 2.0 ** -75).all(axis=1)
    flags = np.where(nonfinite, NONFINITE, 0) | np.where(zero, ZERO_NORM, 0)
    if dtype == "e4m3":
        s = np.asarray(scale, dtype=np.float32)
        flags |= np.where(np.isfinite(s) & (s > 0), 0, BAD_SCALE)
    return flags.astype(np.uint8)
