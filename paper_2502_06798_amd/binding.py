"""Thin ctypes binding of libapc.so (include/apc.h), argument marshalling only.

Every function has the C name and takes torch tensors where the C call takes
device pointers; host tables are numpy arrays or sequences.  All compute runs
in the HIP library; when the library is missing this module raises instead of
falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libapc.so")

APC_F32, APC_F16, APC_BF16, APC_E4M3 = 0, 1, 2, 3
STATUS = ("APC_OK", "APC_E_ARG", "APC_E_DTYPE", "APC_E_TABLE", "APC_E_NONFINITE",
          "APC_E_ZERO_NORM", "APC_E_WORKSPACE", "APC_E_NOMEM", "APC_E_HIP")
APC_MAX_K, APC_MAX_LEVELS, APC_MAX_INST = 64, 32, 256

DTYPE_OF = {torch.float32: APC_F32, torch.float16: APC_F16, torch.bfloat16: APC_BF16,
            torch.float8_e4m3fn: APC_E4M3}


class ApcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        self.name = STATUS[status] if 0 <= status < len(STATUS) else str(status)
        super().__init__(f"{self.name}: {msg}")


_lib = None


def load() -> ctypes.CDLL:
    """Load libapc.so (or the build APC_LIB names, e.g. one whose host code is
    instrumented by sanitizers); raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("APC_LIB", "") or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          "`python -m paper_2502_06798_amd.build_lib` (hipcc, gfx950)")
    L = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    st = ctypes.c_int
    L.apc_build_cache.argtypes = [ctypes.c_int, i64, i32, vp, vp, vp, i64, i64, vp, vp,
                                  ctypes.POINTER(vp)]
    L.apc_build_cache.restype = st
    L.apc_destroy_cache.argtypes = [vp]
    L.apc_destroy_cache.restype = None
    L.apc_row_factors.argtypes = [ctypes.c_int, i64, i32, vp, vp, vp]
    L.apc_row_factors.restype = st
    L.apc_quantize_rows.argtypes = [ctypes.c_int, i64, i32, vp, vp, vp, vp]
    L.apc_quantize_rows.restype = st
    L.apc_validate_rows.argtypes = [ctypes.c_int, i64, i32, vp, vp, vp, ctypes.POINTER(i64), ctypes.POINTER(i64), vp]
    L.apc_validate_rows.restype = st
    L.apc_cache_row_factors.argtypes = [vp, vp, vp]
    L.apc_cache_row_factors.restype = st
    L.apc_match_workspace.argtypes = [vp, i32, i32, ctypes.POINTER(sz)]
    L.apc_match_workspace.restype = st
    L.apc_match_batch.argtypes = [vp, vp, vp, i32, i32, vp, vp, vp, sz, vp]
    L.apc_match_batch.restype = st
    L.apc_match_batch_static.argtypes = [vp, vp, vp, i32, i32, vp, vp, vp]
    L.apc_match_batch_static.restype = st
    L.apc_assign.argtypes = [vp, i32, i32, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.apc_assign.restype = st
    L.apc_assign_load_aware.argtypes = [vp, i32, i32, i32, vp, vp, i32, vp, vp, vp, vp, i64, i64, vp, vp, vp, vp,
                                        vp, vp, vp]
    L.apc_assign_load_aware.restype = st
    L.apc_route_plan.argtypes = [i32, vp, vp, vp, vp, ctypes.POINTER(i64)]
    L.apc_route_plan.restype = st
    L.apc_assign_routed.argtypes = [vp, i32, i32, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.apc_assign_routed.restype = st
    L.apc_assign_planned.argtypes = [vp, i32, i32, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.apc_assign_planned.restype = st
    L.apc_resident_best.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp, vp]
    L.apc_resident_best.restype = st
    L.apc_level_histogram.argtypes = [vp, i32, i32, vp, vp]
    L.apc_level_histogram.restype = st
    L.apc_gather_latents_at_level.argtypes = [vp, vp, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, vp]
    L.apc_gather_latents_at_level.restype = st
    L.apc_merge_shards.argtypes = [vp, vp, i32, i32, i32, vp, i32, vp, vp, vp]
    L.apc_merge_shards.restype = st
    L.apc_gather_latents.argtypes = [vp, vp, i32, i32, vp, vp, vp, i32, i32, vp, vp, vp]
    L.apc_gather_latents.restype = st
    L.apc_set_kernel_events.argtypes = [vp, vp]
    L.apc_set_kernel_events.restype = st
    L.apc_status_str.argtypes = [ctypes.c_int]
    L.apc_status_str.restype = ctypes.c_char_p
    L.apc_last_error.argtypes = []
    L.apc_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise ApcError(rc, load().apc_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _host(a, dtype) -> Optional[np.ndarray]:
    if a is None:
        return None
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _hp(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def apc_status_str(status: int) -> str:
    return load().apc_status_str(status).decode()


def apc_last_error() -> str:
    return load().apc_last_error().decode()


def apc_set_kernel_events(start, stop):
    """start/stop: raw hipEvent_t handles (ints or c_void_p), or None, None."""
    _check(load().apc_set_kernel_events(start, stop))


class Cache:
    """Handle over a built cache; keeps the borrowed tensors alive."""

    def __init__(self, handle: ctypes.c_void_p, dtype: int, n: int, d: int, keep: tuple):
        self.handle = handle
        self.dtype, self.n, self.d = dtype, n, d
        self._keep = keep

    def close(self):
        if self.handle:
            torch.cuda.synchronize()
            load().apc_destroy_cache(self.handle)
            self.handle = None

    def __del__(self):
        try:
            if self.handle and _lib is not None:
                _lib.apc_destroy_cache(self.handle)
                self.handle = None
        except Exception:
            pass


def apc_build_cache(emb: torch.Tensor, row_scale: Optional[torch.Tensor] = None,
                    latents: Optional[torch.Tensor] = None,
                    slot_of_entry: Optional[torch.Tensor] = None, stream=None) -> Cache:
    """emb: n x d device tensor (float32/float16/bfloat16/float8_e4m3fn);
    latents: n_slots x latent_bytes uint8 device tensor or None."""
    L = load()
    if emb.dim() != 2 or emb.dtype not in DTYPE_OF:
        raise ValueError("emb must be a 2-D float32/float16/bfloat16/float8_e4m3fn tensor")
    n, d = emb.shape
    n_slots, lb = (0, 0) if latents is None else (latents.shape[0], latents[0].numel() * latents.element_size())
    out = ctypes.c_void_p()
    _check(L.apc_build_cache(DTYPE_OF[emb.dtype], n, d, _ptr(emb), _ptr(row_scale), _ptr(latents),
                             n_slots, lb, _ptr(slot_of_entry), _stream(stream), ctypes.byref(out)))
    return Cache(out, DTYPE_OF[emb.dtype], n, d, (emb, row_scale, latents, slot_of_entry))


def apc_destroy_cache(c: Cache):
    c.close()


def apc_row_factors(rows: torch.Tensor, out: torch.Tensor, stream=None):
    n, d = rows.shape
    _check(load().apc_row_factors(DTYPE_OF[rows.dtype], n, d, _ptr(rows), _ptr(out), _stream(stream)))


def apc_quantize_rows(x: torch.Tensor, out: torch.Tensor, row_scale=None, stream=None):
    """float32 rows x into out (f16, bf16 or e4m3fn; row_scale for e4m3fn)."""
    n, d = x.shape
    _check(load().apc_quantize_rows(DTYPE_OF[out.dtype], n, d, _ptr(x), _ptr(out), _ptr(row_scale), _stream(stream)))


def apc_validate_rows(rows: torch.Tensor, row_scale=None, bad=None, stream=None):
    """(bad-row count, lowest bad row or -1); per-row flags into bad (uint8) if given."""
    n, d = rows.shape
    nb, fb = ctypes.c_int64(), ctypes.c_int64()
    _check(load().apc_validate_rows(DTYPE_OF[rows.dtype], n, d, _ptr(rows), _ptr(row_scale), _ptr(bad),
                                    ctypes.byref(nb), ctypes.byref(fb), _stream(stream)))
    return nb.value, fb.value


def apc_cache_row_factors(c: Cache, out: torch.Tensor, stream=None):
    _check(load().apc_cache_row_factors(c.handle, _ptr(out), _stream(stream)))


def apc_match_workspace(c: Cache, b: int, k: int) -> int:
    n = ctypes.c_size_t()
    _check(load().apc_match_workspace(c.handle, b, k, ctypes.byref(n)))
    return n.value


def workspace_tensor(c: Cache, b: int, k: int, device=None) -> torch.Tensor:
    """Device buffer of apc_match_workspace() bytes (torch allocations are 256-byte aligned)."""
    return torch.empty(max(apc_match_workspace(c, b, k), 256), dtype=torch.uint8, device=device or "cuda")


def apc_match_batch(c: Cache, q: torch.Tensor, q_scale: Optional[torch.Tensor], k: int,
                    top_score: torch.Tensor, top_idx: torch.Tensor, ws: torch.Tensor, stream=None):
    b = q.shape[0]
    _check(load().apc_match_batch(c.handle, _ptr(q), _ptr(q_scale), b, k, _ptr(top_score),
                                  _ptr(top_idx), _ptr(ws), ws.numel() * ws.element_size(),
                                  _stream(stream)))


def apc_match_batch_static(c: Cache, q: torch.Tensor, q_scale: Optional[torch.Tensor], k: int,
                           top_score: torch.Tensor, top_idx: torch.Tensor, stream=None):
    """apc_match_batch on the library's static device workspace (allocates nothing)."""
    b = q.shape[0]
    _check(load().apc_match_batch_static(c.handle, _ptr(q), _ptr(q_scale), b, k, _ptr(top_score),
                                         _ptr(top_idx), _stream(stream)))


def apc_assign(top_score: torch.Tensor, ld: int, b: int, theta: Sequence[float], K: Sequence[int],
               inst_level: Sequence[int], inst_cap: Sequence[int], inst_queue: Optional[Sequence[int]],
               opt_level: torch.Tensor, out_level: torch.Tensor, out_inst: torch.Tensor,
               out_slot: torch.Tensor, inst_fill: torch.Tensor, stream=None):
    th = _host(theta, np.float32)
    Kh = _host(K, np.int32)
    il = _host(inst_level, np.int32)
    ic = _host(inst_cap, np.int32)
    iq = _host(inst_queue, np.int32)
    _check(load().apc_assign(_ptr(top_score), ld, b, th.size, _hp(th), _hp(Kh), il.size, _hp(il),
                             _hp(ic), _hp(iq), _ptr(opt_level), _ptr(out_level), _ptr(out_inst),
                             _ptr(out_slot), _ptr(inst_fill), _stream(stream)))


def apc_assign_load_aware(top_score: torch.Tensor, ld: int, b: int, theta: Sequence[float], K: Sequence[int],
                          inst_level: Sequence[int], inst_cap: Sequence[int], inst_queue: Optional[Sequence[int]],
                          inst_rand: Optional[Sequence[int]], load_value: int, load_threshold: int,
                          opt_level: torch.Tensor, out_level: torch.Tensor, out_inst: torch.Tensor,
                          out_slot: torch.Tensor, inst_fill: torch.Tensor, stream=None) -> int:
    """load_value: the caller's load measure (the C call's `load`).  Returns the
    routing used: 1 greedy, 0 uniform."""
    th = _host(theta, np.float32)
    Kh = _host(K, np.int32)
    il = _host(inst_level, np.int32)
    ic = _host(inst_cap, np.int32)
    iq = _host(inst_queue, np.int32)
    ir = _host(inst_rand, np.uint32)
    routing = ctypes.c_int32(-1)
    _check(load().apc_assign_load_aware(_ptr(top_score), ld, b, th.size, _hp(th), _hp(Kh), il.size, _hp(il),
                                        _hp(ic), _hp(iq), _hp(ir), int(load_value), int(load_threshold),
                                        ctypes.byref(routing), _ptr(opt_level), _ptr(out_level), _ptr(out_inst),
                                        _ptr(out_slot), _ptr(inst_fill), _stream(stream)))
    return routing.value


def apc_route_plan(K: Sequence[int], H: Sequence[int], F: Sequence[int]):
    """Host-only Route-Plan: returns (X as an (L+1) x (L+1) int32 array, degradation)."""
    Kh = _host(K, np.int32)
    Hh = _host(H, np.int32)
    Fh = _host(F, np.int32)
    L = Kh.size
    if Hh.size != L + 1 or Fh.size != L + 1:
        raise ValueError("apc_route_plan: H and F need len(K) + 1 entries")
    X = np.zeros((L + 1, L + 1), dtype=np.int32)
    d = ctypes.c_int64(0)
    _check(load().apc_route_plan(L, _hp(Kh), _hp(Hh), _hp(Fh), X.ctypes.data, ctypes.byref(d)))
    return X, int(d.value)


def _assign_plan(fn, top_score, ld, b, theta, K, inst_level, inst_cap, inst_queue, plan, opt_level,
                 out_level, out_inst, out_slot, inst_fill, stream):
    th = _host(theta, np.float32)
    Kh = _host(K, np.int32)
    il = _host(inst_level, np.int32)
    ic = _host(inst_cap, np.int32)
    iq = _host(inst_queue, np.int32)
    _check(fn(_ptr(top_score), ld, b, th.size, _hp(th), _hp(Kh), il.size, _hp(il), _hp(ic), _hp(iq),
              _ptr(plan), _ptr(opt_level), _ptr(out_level), _ptr(out_inst), _ptr(out_slot),
              _ptr(inst_fill), _stream(stream)))


def apc_assign_routed(top_score: torch.Tensor, ld: int, b: int, theta: Sequence[float], K: Sequence[int],
                      inst_level: Sequence[int], inst_cap: Sequence[int], inst_queue: Optional[Sequence[int]],
                      plan: torch.Tensor, opt_level: torch.Tensor, out_level: torch.Tensor,
                      out_inst: torch.Tensor, out_slot: torch.Tensor, inst_fill: torch.Tensor, stream=None):
    _assign_plan(load().apc_assign_routed, top_score, ld, b, theta, K, inst_level, inst_cap, inst_queue,
                 plan, opt_level, out_level, out_inst, out_slot, inst_fill, stream)


def apc_assign_planned(top_score: torch.Tensor, ld: int, b: int, theta: Sequence[float], K: Sequence[int],
                       inst_level: Sequence[int], inst_cap: Sequence[int], inst_queue: Optional[Sequence[int]],
                       plan: torch.Tensor, opt_level: torch.Tensor, out_level: torch.Tensor,
                       out_inst: torch.Tensor, out_slot: torch.Tensor, inst_fill: torch.Tensor, stream=None):
    _assign_plan(load().apc_assign_planned, top_score, ld, b, theta, K, inst_level, inst_cap, inst_queue,
                 plan, opt_level, out_level, out_inst, out_slot, inst_fill, stream)


def apc_resident_best(c: Cache, top_score: torch.Tensor, top_idx: torch.Tensor, ld: int, k: int, b: int,
                      out_score: torch.Tensor, out_idx: torch.Tensor, stream=None):
    _check(load().apc_resident_best(c.handle, _ptr(top_score), _ptr(top_idx), ld, k, b, _ptr(out_score),
                                    _ptr(out_idx), _stream(stream)))


def apc_level_histogram(level: torch.Tensor, b: int, L: int, hist: torch.Tensor, stream=None):
    _check(load().apc_level_histogram(_ptr(level), b, L, _ptr(hist), _stream(stream)))


def apc_gather_latents(c: Cache, top_idx: torch.Tensor, ld: int, b: int, out_level: torch.Tensor,
                       out_inst: torch.Tensor, out_slot: torch.Tensor, n_inst: int,
                       slots_per_inst: int, batch_latents: torch.Tensor, hit: torch.Tensor,
                       stream=None):
    _check(load().apc_gather_latents(c.handle, _ptr(top_idx), ld, b, _ptr(out_level), _ptr(out_inst),
                                     _ptr(out_slot), n_inst, slots_per_inst, _ptr(batch_latents),
                                     _ptr(hit), _stream(stream)))


def apc_gather_latents_at_level(c: Cache, top_idx: torch.Tensor, ld: int, b: int, out_level: torch.Tensor,
                                out_inst: torch.Tensor, out_slot: torch.Tensor, n_inst: int, slots_per_inst: int,
                                levels_per_slot: int, batch_latents: torch.Tensor, hit: torch.Tensor, stream=None):
    _check(load().apc_gather_latents_at_level(c.handle, _ptr(top_idx), ld, b, _ptr(out_level), _ptr(out_inst),
                                              _ptr(out_slot), n_inst, slots_per_inst, levels_per_slot,
                                              _ptr(batch_latents), _ptr(hit), _stream(stream)))


def apc_merge_shards(scores: torch.Tensor, idx: torch.Tensor, g: int, b: int, k_in: int, offsets: Sequence[int],
                     k: int, out_score: torch.Tensor, out_idx: torch.Tensor, stream=None):
    off = _host(offsets, np.int32)
    if off is None or off.size != g:
        raise ValueError("apc_merge_shards: need one offset per shard")
    _check(load().apc_merge_shards(_ptr(scores), _ptr(idx), g, b, k_in, _hp(off), k, _ptr(out_score),
                                   _ptr(out_idx), _stream(stream)))
