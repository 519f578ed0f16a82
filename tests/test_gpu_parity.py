"""GPU parity of each call of the C ABI against the float64 reference, on small
seeded inputs that span several tiles and ragged tails, plus edge cases."""
import numpy as np
import pytest
import torch

from paper_2502_06798_amd import synth
from tests._util import np_or_none, stored_np
from tests.gpu_check import TOL, check_levels, check_topk, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def apc():
    import paper_2502_06798_amd as apc
    apc.load()
    assert torch.cuda.is_available()
    return apc


def make_rows(n, d, dtype, seed, dev="cuda", clusters=None):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(n, d, generator=g, dtype=torch.float64)
    if clusters is not None:
        c = torch.randn(clusters, d, generator=g, dtype=torch.float64)
        cid = torch.randint(0, clusters, (n,), generator=g)
        x = c[cid] + 0.3 * x
    x = x / x.norm(dim=1, keepdim=True)
    s, sc = synth.to_storage(x.float(), dtype)
    return s.to(dev), (None if sc is None else sc.to(dev))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "e4m3"])
def test_row_factors(apc, orc, dtype):
    say(f"row_factors {dtype}")
    d = 96 if dtype != "e4m3" else 112
    rows, sc = make_rows(300, d, dtype, 1)
    out = torch.empty(300, dtype=torch.float32, device="cuda")
    apc.apc_row_factors(rows, out)
    torch.cuda.synchronize()
    h = stored_np(rows)
    sq, rc, _ = orc.row_sqnorms(dtype, h, None if sc is None else np.ones(300, np.float32))
    want = 1.0 / np.sqrt(sq)
    assert np.max(np.abs(out.cpu().numpy() / want - 1)) <= 1e-6
    # the cache computes the same factors; bad rows are rejected at build
    c = apc.apc_build_cache(rows, sc)
    f2 = torch.empty(300, dtype=torch.float32, device="cuda")
    apc.apc_cache_row_factors(c, f2)
    torch.cuda.synchronize()
    assert torch.equal(f2, out)
    c.close()


def test_build_rejects_bad_rows(apc):
    say("build rejects bad rows")
    x = torch.randn(64, 32, device="cuda")
    x[5] = 0
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_build_cache(x)
    assert ei.value.name == "APC_E_ZERO_NORM" and "row 5" in str(ei.value)
    x[5] = 1
    x[9, 3] = float("nan")
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_build_cache(x)
    assert ei.value.name == "APC_E_NONFINITE"
    c8, sc = make_rows(64, 32, "e4m3", 3)
    sc[7] = -1.0
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_build_cache(c8, sc)
    assert ei.value.name == "APC_E_NONFINITE"
    x[9, 3] = 1
    lat = torch.zeros(8, 32, dtype=torch.uint8, device="cuda")
    soe = torch.full((64,), -1, dtype=torch.int32, device="cuda")
    soe[3] = 8
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_build_cache(x, None, lat, soe)
    assert ei.value.name == "APC_E_ARG"


CASES = [
    # (dtype, b, n, d, k)
    ("f32", 16, 1000, 64, 5),
    ("f32", 7, 4099, 200, 10),
    ("f16", 37, 4099, 200, 10),
    ("f16", 130, 2000, 768, 16),
    ("f16", 1, 300, 8, 1),
    ("bf16", 129, 3000, 512, 33),
    ("bf16", 5, 257, 64, 64),
    ("e4m3", 64, 3000, 768, 32),
    ("e4m3", 200, 1500, 112, 7),
    ("f16", 300, 129, 64, 64),
    # float32 caches of at most 512 blocks of 32 rows (d a multiple of 64,
    # k <= 32, b <= 256): a workgroup per block, d over its wavefronts; a
    # partial last block, one query, the largest cache, k = 32, partial and
    # many query tiles
    ("f32", 16, 5000, 768, 5),
    ("f32", 1, 33, 128, 1),
    ("f32", 17, 16384, 256, 32),
    ("f32", 256, 2000, 64, 12),
    ("f32", 40, 70, 1024, 7),
    ("f32", 3, 1, 64, 1),              # a one-row cache
    ("f32", 256, 16384, 64, 32),       # the largest batch, cache and k together
    # streaming kernel: larger float caches, and 16-bit or e4m3 rows of sizes
    # the query-stationary kernel is not built for (whole groups of 4 x 128
    # bytes, 6 x 128 for e4m3), or k > 32
    ("f32", 16, 20000, 768, 5),
    ("f16", 64, 1000, 1536, 12),
    # query-stationary kernel: 16-bit or e4m3 rows of 512, 768, 1024 or 1536
    # bytes, k <= 32; every shape family (rows, query blocks, 32-row blocks per
    # group, lists of 10, 16 or 32 slots in registers or LDS)
    ("e4m3", 100, 2050, 768, 10),      # 768 B, two query blocks, 10-slot lists
    ("f16", 256, 7777, 768, 10),       # 1536 B, one block, four 32-row blocks
    ("bf16", 3, 17, 256, 17),          # one group, one split
    ("f16", 5, 40, 256, 3),
    ("e4m3", 7, 33, 768, 33),          # k > 32: streaming
    ("bf16", 100, 3000, 768, 20),      # 1536 B, 32-slot lists, two 32-row blocks
    ("f16", 256, 50000, 768, 10),
    ("bf16", 129, 3001, 768, 16),
    ("e4m3", 300, 9000, 768, 10),
    ("f16", 1, 31, 768, 5),
    ("f16", 40, 100, 512, 7),          # 1024 B, lists in LDS
    ("e4m3", 5, 70000, 512, 16),       # 512 B, two query blocks, 16-slot lists
    ("bf16", 512, 20000, 256, 8),
    ("f16", 200, 40000, 256, 3),
    ("f16", 150, 6000, 256, 12),       # 512 B, two query blocks
    ("f16", 150, 6000, 256, 24),       # 512 B, one block, 32-slot lists
    ("bf16", 70, 5000, 384, 16),       # 768 B, two query blocks
    ("f16", 90, 5000, 512, 9),         # 1024 B, two query blocks, lists in LDS
    ("e4m3", 90, 5000, 1024, 20),      # 1024 B e4m3, one block, 32-slot lists
    ("e4m3", 33, 4000, 1536, 11),      # 1536 B e4m3, one block, four 32-row blocks
    ("bf16", 64, 3000, 768, 29),       # 1536 B, 32-slot lists
    ("e4m3", 40, 5000, 1536, 6),       # 1536 B e4m3, 10-slot lists
    ("e4m3", 70, 6000, 1024, 10),      # 1024 B e4m3, two query blocks, 10-slot lists in LDS
    ("f16", 80, 5000, 512, 14),        # 1024 B, 16-slot lists in LDS
    ("f16", 130, 9000, 768, 11),       # 1536 B, 16-slot lists just above 10
]


@pytest.mark.parametrize("dtype,b,n,d,k", CASES)
def test_match_small(apc, orc, dtype, b, n, d, k):
    say(f"match {dtype} b={b} n={n} d={d} k={k}")
    e, es = make_rows(n, d, dtype, 10 + n, clusters=max(1, n // 50))
    q, qs = make_rows(b, d, dtype, 20 + b, clusters=None)
    # queries near entries so the top-k has real structure
    if b > 1:
        q[: b // 2] = e[torch.arange(b // 2, device="cuda") * 7 % n]
        if qs is not None:
            qs[: b // 2] = es[torch.arange(b // 2, device="cuda") * 7 % n]
    c = apc.apc_build_cache(e, es)
    ts = torch.empty((b, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    ws = apc.workspace_tensor(c, b, k)
    apc.apc_match_batch(c, q, qs, k, ts, ti, ws)
    torch.cuda.synchronize()
    qh, eh = stored_np(q), stored_np(e)
    qsh, esh = np_or_none(qs), np_or_none(es)
    rs, ri = orc.topk(dtype, qh, qsh, eh, esh, min(k + 1, n))
    st = check_topk(orc, dtype, qh, qsh, eh, esh, ts.cpu().numpy(), ti.cpu().numpy(), rs, ri)
    say("  ", st)
    # deterministic: a second run is bit-identical
    ts2, ti2 = torch.empty_like(ts), torch.empty_like(ti)
    apc.apc_match_batch(c, q, qs, k, ts2, ti2, ws)
    torch.cuda.synchronize()
    assert torch.equal(ti, ti2) and torch.equal(ts, ts2)
    c.close()


@pytest.mark.parametrize("dtype,b,n,d,k", [("f16", 2048, 40000, 768, 10), ("e4m3", 1024, 60000, 512, 12),
                                            ("e4m3", 4096, 30000, 768, 32), ("f16", 4096, 20000, 512, 16)])
def test_match_many_groups_per_split(apc, orc, dtype, b, n, d, k):
    """Enough query tiles that each split holds many groups: lists fill and
    bounds tighten as the pass goes; a subset of rows is checked.  The row
    counts end in a partial group."""
    say(f"match (many groups per split) {dtype} b={b} n={n} d={d} k={k}")
    e, es = make_rows(n, d, dtype, 30 + n, clusters=max(1, n // 50))
    q, qs = make_rows(b, d, dtype, 40 + b, clusters=None)
    q[: b // 2] = e[torch.arange(b // 2, device="cuda") * 13 % n]
    if qs is not None:
        qs[: b // 2] = es[torch.arange(b // 2, device="cuda") * 13 % n]
    c = apc.apc_build_cache(e, es)
    ts = torch.empty((b, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    apc.apc_match_batch(c, q, qs, k, ts, ti, apc.workspace_tensor(c, b, k))
    torch.cuda.synchronize()
    rows = np.arange(0, b, 61)
    qh, eh = stored_np(q), stored_np(e)
    qsh, esh = np_or_none(qs), np_or_none(es)
    rs, ri = orc.topk(dtype, qh[rows], None if qsh is None else qsh[rows], eh, esh, k + 1)
    st = check_topk(orc, dtype, qh, qsh, eh, esh, ts.cpu().numpy(), ti.cpu().numpy(), rs, ri, rows=rows)
    say("  ", st)
    c.close()


# Batches above 256 queries with 512-, 768- or 1024-byte rows go to the kernel with
# two wavefronts per SIMD (256 queries per workgroup, lists in LDS): every row
# type, both list sizes (k <= 16 and k <= 32), k = 1 and k = 32, a last group
# of fewer than 64 rows, a cache smaller than one group, wavefronts without
# queries (b just above a multiple of 32 and of 256) and many splits.
QS8_CASES = [
    ("e4m3", 257, 5000, 768, 10),
    ("e4m3", 300, 63, 512, 32),        # fewer rows than one group
    ("e4m3", 1000, 20011, 512, 1),
    ("f16", 513, 9000, 384, 16),       # 768-byte f16 rows
    ("bf16", 700, 12345, 256, 17),     # 512-byte bf16 rows, 32-slot lists
    ("f16", 2080, 30001, 256, 32),
    ("bf16", 1024, 7000, 384, 5),
    ("e4m3", 4099, 40000, 768, 32),
    ("f16", 1030, 20001, 512, 16),     # 1024-byte rows: fragments read one step ahead
    ("bf16", 600, 9000, 512, 32),
    ("e4m3", 777, 15000, 1024, 20),
]


@pytest.mark.parametrize("dtype,b,n,d,k", QS8_CASES)
def test_match_two_waves_per_simd(apc, orc, dtype, b, n, d, k):
    say(f"match (two wavefronts per SIMD) {dtype} b={b} n={n} d={d} k={k}")
    e, es = make_rows(n, d, dtype, 50 + n, clusters=max(1, n // 60))
    q, qs = make_rows(b, d, dtype, 60 + b, clusters=None)
    q[: b // 2] = e[torch.arange(b // 2, device="cuda") * 11 % n]
    if qs is not None:
        qs[: b // 2] = es[torch.arange(b // 2, device="cuda") * 11 % n]
    c = apc.apc_build_cache(e, es)
    ts = torch.empty((b, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    ws = apc.workspace_tensor(c, b, k)
    apc.apc_match_batch(c, q, qs, k, ts, ti, ws)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, b, max(1, b // 160)), [b - 1], np.arange(min(b, 40))]))
    qh, eh = stored_np(q), stored_np(e)
    qsh, esh = np_or_none(qs), np_or_none(es)
    rs, ri = orc.topk(dtype, qh[rows], None if qsh is None else qsh[rows], eh, esh, min(k + 1, n))
    st = check_topk(orc, dtype, qh, qsh, eh, esh, ts.cpu().numpy(), ti.cpu().numpy(), rs, ri, rows=rows)
    say("  ", st)
    ts2, ti2 = torch.empty_like(ts), torch.empty_like(ti)
    apc.apc_match_batch(c, q, qs, k, ts2, ti2, ws)
    torch.cuda.synchronize()
    assert torch.equal(ti, ti2) and torch.equal(ts, ts2)
    c.close()


@pytest.mark.parametrize("dtype,d,b,n,k", [
    ("f16", 64, 3, 1000, 20),        # tiled / streaming kernels
    ("f32", 64, 3, 1000, 20),        # small float32 caches, four wavefronts over d
    ("f32", 768, 17, 5000, 32),      # the same, eight wavefronts
    ("f16", 768, 5, 3000, 10),       # query-stationary kernel (1536-byte rows)
    ("e4m3", 768, 300, 2000, 32),    # two wavefronts per SIMD (768-byte rows)
])
def test_match_ties_take_lower_index(apc, orc, dtype, d, b, n, k):
    """Every cache row the same: every score ties, and the top-k is entries
    0 .. k-1 in order, whatever the kernel."""
    say(f"match ties {dtype} d={d} b={b} n={n} k={k}")
    row, rsc = make_rows(1, d, dtype, 77)
    e = row.repeat(n, 1).contiguous()
    es = None if rsc is None else rsc.repeat(n).contiguous()
    q, qs = make_rows(b, d, dtype, 78)
    c = apc.apc_build_cache(e, es)
    ts = torch.empty((b, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    apc.apc_match_batch(c, q, qs, k, ts, ti, apc.workspace_tensor(c, b, k))
    torch.cuda.synchronize()
    assert ti.cpu().tolist() == [list(range(k))] * b
    assert torch.all(ts == ts[:, :1])
    c.close()


@pytest.mark.parametrize("dtype,d", [("f16", 32), ("f16", 256), ("f32", 64)])   # tiled, streaming, small float32
def test_match_invalid_query_rows(apc, dtype, d):
    say(f"match invalid query rows {dtype} d={d}")
    e, _ = make_rows(500, d, dtype, 5)
    q, _ = make_rows(6, d, dtype, 6)
    q[1] = 0
    q[4, 3] = float("inf")
    c = apc.apc_build_cache(e)
    ts = torch.empty((6, 4), dtype=torch.float32, device="cuda")
    ti = torch.empty((6, 4), dtype=torch.int32, device="cuda")
    apc.apc_match_batch(c, q, None, 4, ts, ti, apc.workspace_tensor(c, 6, 4))
    torch.cuda.synchronize()
    for r in (1, 4):
        assert torch.all(ti[r] == -1) and torch.all(torch.isnan(ts[r]))
    for r in (0, 2, 3, 5):
        assert torch.all(ti[r] >= 0)
    c.close()


def test_match_argument_errors(apc):
    say("match argument errors")
    e, _ = make_rows(50, 32, "f16", 5)
    c = apc.apc_build_cache(e)
    q, _ = make_rows(4, 32, "f16", 6)
    ts = torch.empty((4, 51), dtype=torch.float32, device="cuda")
    ti = torch.empty((4, 51), dtype=torch.int32, device="cuda")
    ws = torch.empty(1 << 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_match_batch(c, q, None, 51, ts, ti, ws)       # k > n
    assert ei.value.name == "APC_E_ARG"
    need = apc.apc_match_workspace(c, 4, 8)
    with pytest.raises(apc.ApcError) as ei:
        apc.apc_match_batch(c, q, None, 8, ts, ti, ws[: need - 1])
    assert ei.value.name == "APC_E_WORKSPACE"
    apc.apc_match_batch(c, q[:0], None, 8, ts, ti, ws)        # b = 0 is a no-op
    c.close()


def _random_table(rng, L, I, cap_hi=6):
    il = rng.integers(0, L + 1, I)
    ic = rng.integers(0, cap_hi, I)
    iq = rng.integers(0, 5, I)
    return il, ic, iq


@pytest.mark.parametrize("b,L,I", [(1, 0, 1), (16, 5, 2), (64, 3, 3), (65, 5, 4), (200, 5, 4), (256, 5, 4),
                                    (130, 32, 20), (300, 5, 8), (2500, 10, 40), (5000, 32, 256),
                                    # above 16384 queries: the multi-block placement kernel
                                    (20000, 10, 32), (20000, 32, 64), (65536, 10, 16), (65536, 32, 256)])
def test_assign_bit_exact(apc, orc, b, L, I):
    say(f"assign b={b} L={L} I={I}")
    rng = np.random.default_rng(b + L + I)
    theta = np.sort(rng.uniform(-0.5, 0.99, L)).astype(np.float32)
    theta = np.unique(theta)
    L = theta.size
    K = np.arange(1, L + 1, dtype=np.int32) * 5
    ld = 3
    best = rng.uniform(-1, 1, b).astype(np.float32)
    best[: b // 4] = theta[rng.integers(0, L, b // 4)] if L else best[: b // 4]   # exact boundaries
    ts = torch.zeros((b, ld), dtype=torch.float32)
    ts[:, 0] = torch.from_numpy(best)
    ts = ts.cuda()
    il, ic, iq = _random_table(rng, L, I, cap_hi=max(2, 2 * b // max(I, 1)))
    outs = [torch.full((b,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    fill = torch.full((I,), -7, dtype=torch.int32, device="cuda")
    apc.apc_assign(ts, ld, b, theta, K, il, ic, iq, *outs, fill)
    torch.cuda.synchronize()
    opt, ol, oi, os_ = (o.cpu().numpy() for o in outs)
    assert np.array_equal(opt, orc.levels(best.astype(np.float64), theta))
    r = orc.assign(opt, L, il, ic, iq)
    assert np.array_equal(ol, r[0]) and np.array_equal(oi, r[1]) and np.array_equal(os_, r[2])
    assert np.array_equal(fill.cpu().numpy(), r[3])


def test_assign_empty_and_full(apc, orc):
    say("assign edge cases")
    b = 40
    ts = torch.linspace(-1, 1, b).reshape(b, 1).cuda()
    outs = [torch.empty((b,), dtype=torch.int32, device="cuda") for _ in range(4)]
    fill = torch.empty((3,), dtype=torch.int32, device="cuda")
    # total capacity below demand: the last queries stay unassigned
    apc.apc_assign(ts, 1, b, [0.0, 0.5], [5, 10], [0, 1, 2], [5, 5, 0], None, *outs, fill)
    torch.cuda.synchronize()
    ol = outs[1].cpu().numpy()
    assert (ol >= 0).sum() == 10 and np.all(outs[2].cpu().numpy()[ol < 0] == -1)
    r = orc.assign(outs[0].cpu().numpy(), 2, [0, 1, 2], [5, 5, 0], None)
    assert np.array_equal(ol, r[0]) and np.array_equal(fill.cpu().numpy(), r[3])
    # no instances at all
    apc.apc_assign(ts, 1, b, [0.0], [5], [], [], None, *outs, fill)
    torch.cuda.synchronize()
    assert torch.all(outs[1] == -1)


def test_gather_bit_exact(apc, orc):
    say("gather")
    rng = np.random.default_rng(4)
    n, n_slots, lb = 3000, 700, 4096 + 48
    e, _ = make_rows(n, 64, "f16", 9)
    pool = torch.randint(0, 256, (n_slots, lb), dtype=torch.uint8, device="cuda")
    soe_h = np.full(n, -1, np.int32)
    hot = rng.choice(n, n_slots, replace=False)
    soe_h[hot] = np.arange(n_slots)
    soe = torch.from_numpy(soe_h).cuda()
    c = apc.apc_build_cache(e, None, pool, soe)
    b, n_inst, spi = 500, 5, 128
    top = torch.from_numpy(rng.integers(0, n, (b, 2)).astype(np.int32))
    top[: b // 2, 0] = torch.from_numpy(hot[: b // 2].astype(np.int32))
    top = top.cuda()
    perm = rng.permutation(n_inst * spi)[:b]
    ol = torch.from_numpy(rng.integers(-1, 4, b).astype(np.int32))
    oi = torch.from_numpy((perm // spi).astype(np.int32))
    os_ = torch.from_numpy((perm % spi).astype(np.int32))
    oi[ol < 0] = -1
    os_[ol < 0] = -1
    batch = torch.zeros((n_inst * spi, lb), dtype=torch.uint8, device="cuda")
    hit = torch.empty(b, dtype=torch.int32, device="cuda")
    apc.apc_gather_latents(c, top, 2, b, ol.cuda(), oi.cuda(), os_.cuda(), n_inst, spi, batch, hit)
    torch.cuda.synchronize()
    want = np.zeros((n_inst * spi, lb), np.uint8)
    h = orc.gather(top[:, 0].cpu().numpy(), ol.numpy(), oi.numpy(), os_.numpy(), soe_h, n,
                   pool.cpu().numpy(), n_inst, spi, want)
    assert np.array_equal(hit.cpu().numpy(), h) and h.sum() > 0
    assert np.array_equal(batch.cpu().numpy(), want)
    c.close()
