"""Python binding of the float64 CPU reference (apc_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library.  Shares no code with the
HIP path.  Inputs are host numpy arrays holding the exact stored bytes.
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


def build() -> str:
    """Compile the reference with gcc (OpenMP, no HIP)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           "-o", LIB, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB)
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
