"""The C ABI: every declared symbol is exported, and host-side argument checks
return their status before touching the GPU (CPU only: no compute calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apc.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2502_06798_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libapc.so not built")
    return binding.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apc_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("apc_build_cache", "apc_match_batch", "apc_assign", "apc_gather_latents",
                     "apc_destroy_cache", "apc_match_workspace", "apc_last_error", "apc_status_str",
                     "apc_route_plan", "apc_assign_routed", "apc_assign_planned", "apc_resident_best",
                     "apc_level_histogram", "apc_gather_latents_at_level", "apc_merge_shards"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for s in range(9):
        assert lib.apc_status_str(s)
    assert lib.apc_status_str(99) == b"unknown status"


E_ARG, E_DTYPE, E_TABLE = 1, 2, 3
FAKE = ctypes.c_void_p(0x100000)       # never dereferenced: every call below fails its checks first


def _assign(lib, L=2, theta=(0.5, 0.7), K=(5, 10), il=(0, 1), ic=(1, 1), iq=None, b=4, ld=1):
    th = np.array(theta, np.float32)
    Kh = np.array(K, np.int32)
    ilh = np.array(il, np.int32)
    ich = np.array(ic, np.int32)
    iqh = None if iq is None else np.array(iq, np.int32)
    p = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    return lib.apc_assign(FAKE, ld, b, L, p(th), p(Kh), ilh.size, p(ilh), p(ich), p(iqh),
                          FAKE, FAKE, FAKE, FAKE, FAKE, None)


def test_assign_table_checks(lib):
    assert _assign(lib, theta=(0.7, 0.5)) == E_TABLE                    # not increasing
    assert _assign(lib, theta=(0.5, float("nan"))) == E_TABLE
    assert _assign(lib, K=(5, 5)) == E_TABLE
    assert _assign(lib, K=(0, 5)) == E_TABLE
    assert _assign(lib, il=(0, 3)) == E_TABLE                           # level > L
    assert _assign(lib, ic=(1, -1)) == E_TABLE
    assert _assign(lib, il=(0, 1), ic=(2**31 - 1, 1)) == E_TABLE        # total overflows
    assert _assign(lib, L=33, theta=tuple(range(33)), K=tuple(range(1, 34))) == E_TABLE
    assert _assign(lib, il=tuple([0] * 257), ic=tuple([1] * 257)) == E_TABLE
    assert _assign(lib, b=-1) == E_ARG
    assert _assign(lib, ld=0) == E_ARG
    assert b"strictly increasing" in lib.apc_last_error() or True


def test_build_cache_argument_checks(lib):
    out = ctypes.c_void_p()
    b = lambda dt, n, d, emb=FAKE, scale=None, lat=None, ns=0, lb=0, soe=None: lib.apc_build_cache(
        dt, n, d, emb, scale, lat, ns, lb, soe, None, ctypes.byref(out))
    assert b(7, 10, 16) == E_DTYPE
    assert b(1, 10, 12) == E_ARG                       # 24 bytes per row: not a multiple of 16
    assert b(3, 10, 8) == E_ARG                        # e4m3 row of 8 bytes
    assert b(1, 0, 16) == E_ARG                        # empty cache
    assert b(1, 10, 16, emb=ctypes.c_void_p(0x100001)) == E_ARG      # misaligned
    assert b(3, 10, 16) == E_ARG                       # e4m3 without scales
    assert b(1, 10, 16, scale=FAKE) == E_ARG           # scales for a non-e4m3 cache
    assert b(1, 10, 16, lat=FAKE, ns=10, lb=24) == E_ARG          # latent size not 16-aligned
    assert b(1, 10, 16, lat=FAKE, ns=5, lb=32) == E_ARG           # identity map needs n_slots >= n
    assert b(1, 10, 16, soe=FAKE) == E_ARG             # slot map without latents
    assert out.value is None
    assert lib.apc_last_error()


def test_match_and_gather_reject_null_handle(lib):
    assert lib.apc_match_batch(None, FAKE, None, 4, 2, FAKE, FAKE, FAKE, 1 << 20, None) == E_ARG
    n = ctypes.c_size_t()
    assert lib.apc_match_workspace(None, 4, 2, ctypes.byref(n)) == E_ARG
    assert lib.apc_gather_latents(None, FAKE, 1, 4, FAKE, FAKE, FAKE, 1, 1, FAKE, FAKE, None) == E_ARG
    assert lib.apc_row_factors(9, 4, 16, FAKE, FAKE, None) == E_DTYPE
    assert lib.apc_cache_row_factors(None, FAKE, None) == E_ARG
    lib.apc_destroy_cache(None)


def test_merge_shards_argument_checks(lib):
    import ctypes
    import numpy as np
    off = np.zeros(65, dtype=np.int32)
    fake = ctypes.c_void_p(256)                              # never dereferenced: the checks fail first
    call = lambda g, b, kin, k, o=off.ctypes.data: lib.apc_merge_shards(fake, fake, g, b, kin, o, k, fake, fake, None)
    assert call(0, 4, 10, 10) == 1
    assert call(65, 4, 10, 10) == 1
    assert call(2, 4, 0, 10) == 1
    assert call(2, 4, 10, 65) == 1
    assert call(2, 4, 10, 10, None) == 1
    neg = np.array([0, -5], dtype=np.int32)
    assert call(2, 4, 10, 10, neg.ctypes.data) == 1
    assert call(2, 0, 10, 10) == 0                           # empty batch: nothing to do


def test_load_aware_argument_errors(lib):
    th = np.array([0.5, 0.7], np.float32)
    Kh = np.array([5, 10], np.int32)
    il = np.array([0, 1], np.int32)
    ic = np.array([1, 1], np.int32)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    routing = ctypes.c_int32(-1)
    # uniform routing (load below the threshold) without random keys
    assert lib.apc_assign_load_aware(FAKE, 1, 4, 2, p(th), p(Kh), 2, p(il), p(ic), None, None, 0, 1,
                                     ctypes.byref(routing), FAKE, FAKE, FAKE, FAKE, FAKE, None) == E_ARG
    # no place for the routing decision
    rnd = np.array([3, 1], np.uint32)
    assert lib.apc_assign_load_aware(FAKE, 1, 4, 2, p(th), p(Kh), 2, p(il), p(ic), None, p(rnd), 0, 1,
                                     None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == E_ARG
    # table errors are those of apc_assign
    bad = np.array([0, 3], np.int32)
    assert lib.apc_assign_load_aware(FAKE, 1, 4, 2, p(th), p(Kh), 2, p(bad), p(ic), None, p(rnd), 5, 1,
                                     ctypes.byref(routing), FAKE, FAKE, FAKE, FAKE, FAKE, None) == E_TABLE


def test_quantize_and_validate_argument_checks(lib):
    q = lambda dt, n=4, d=16, x=FAKE, out=FAKE, sc=None: lib.apc_quantize_rows(dt, n, d, x, out, sc, None)
    assert q(0) == E_DTYPE                                  # float32 is not a storage target
    assert q(7) == E_DTYPE
    assert q(3) == E_ARG                                    # e4m3 without scales
    assert q(1, sc=FAKE) == E_ARG                           # scales for f16
    assert q(1, x=None) == E_ARG
    assert q(1, x=ctypes.c_void_p(0x100004)) == E_ARG       # x misaligned
    assert q(1, d=12) == E_ARG                              # 24-byte rows
    assert q(1, n=0) == 0                                   # nothing to do
    nb, fb = ctypes.c_int64(7), ctypes.c_int64(7)
    v = lambda dt, n=4, d=16, rows=FAKE, sc=None, nbp=ctypes.byref(nb): lib.apc_validate_rows(
        dt, n, d, rows, sc, None, nbp, ctypes.byref(fb), None)
    assert v(1, nbp=None) == E_ARG
    assert v(9) == E_DTYPE
    assert v(3) == E_ARG                                    # e4m3 without scales
    assert v(0, sc=FAKE) == E_ARG
    assert v(1, rows=ctypes.c_void_p(0x100002)) == E_ARG
    assert v(1, n=0) == 0 and nb.value == 0 and fb.value == -1
