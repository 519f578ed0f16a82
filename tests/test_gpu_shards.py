"""GPU parity of the merge of per-shard top-k lists.

apc_merge_shards is compared bit for bit with the oracle's merge on the same
seeded lists (ties across shards, invalid entries, fewer candidates than k,
1 to 64 shards).  End to end, a cache split into row shards, matched shard by
shard with apc_match_batch and merged, gives bit for bit the top-k of the
whole cache (every score is the same fixed MFMA sequence wherever its row
lives).
"""
import numpy as np
import pytest
import torch

from paper_2502_06798_amd import synth
from tests.gpu_check import say
from tests.test_gpu_parity import make_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def apc():
    import paper_2502_06798_amd as apc
    apc.load()
    assert torch.cuda.is_available()
    return apc


def _shard_lists(rng, g, b, kin, n_local):
    s = np.round(rng.uniform(-1, 1, (g, b, kin)), 2).astype(np.float32)      # ties across shards
    i = np.stack([[rng.choice(n_local, kin, replace=False) for _ in range(b)] for _ in range(g)]).astype(np.int32)
    for a in range(g):
        for q in range(b):
            o = np.lexsort((i[a, q], -s[a, q].astype(np.float64)))
            s[a, q], i[a, q] = s[a, q][o], i[a, q][o]
            cut = rng.integers(0, kin + 1) if rng.random() < 0.1 else kin     # fewer candidates
            i[a, q, cut:] = -1
            s[a, q, cut:] = np.nan
    return s, i


@pytest.mark.parametrize("g,b,kin,k", [(1, 5, 10, 10), (2, 300, 10, 10), (8, 1000, 32, 32), (8, 77, 16, 40),
                                       (64, 130, 4, 64), (3, 4096, 64, 1), (5, 1, 1, 7)])
def test_merge_shards_bit_exact(apc, orc, g, b, kin, k):
    say(f"merge_shards g={g} b={b} kin={kin} k={k}")
    rng = np.random.default_rng(g * 1000 + b + kin)
    s, i = _shard_lists(rng, g, b, kin, 500)
    offsets = (np.arange(g) * 500).tolist()
    os_ = torch.full((b, k), 7.0, device="cuda")
    oi = torch.full((b, k), 7, dtype=torch.int32, device="cuda")
    apc.apc_merge_shards(torch.from_numpy(s).cuda(), torch.from_numpy(i).cuda(), g, b, kin, offsets, k, os_, oi)
    torch.cuda.synchronize()
    ws, wi = orc.merge_shards(s, i, offsets, k)
    gs = os_.cpu().numpy()
    assert np.array_equal(oi.cpu().numpy(), wi)
    assert np.array_equal(np.isnan(gs), np.isnan(ws)) and np.array_equal(gs[~np.isnan(ws)], ws[~np.isnan(ws)])


@pytest.mark.parametrize("dtype,cuts", [("f16", [0, 20000, 40000]), ("f16", [0, 5000, 5100, 23000, 40000]),
                                        ("e4m3", [0, 13000, 26000, 40000])])
def test_sharded_match_equals_whole_cache(apc, dtype, cuts):
    say(f"sharded match {dtype} cuts={cuts}")
    n, d, b, k = cuts[-1], 768, 300, 10
    e, es = make_rows(n, d, dtype, 21, clusters=50)
    q, qs = make_rows(b, d, dtype, 22, clusters=50)
    whole = apc.apc_build_cache(e, es)
    ts = torch.empty((b, k), device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    apc.apc_match_batch(whole, q, qs, k, ts, ti, apc.workspace_tensor(whole, b, k))
    g = len(cuts) - 1
    ls = torch.empty((g, b, k), device="cuda")
    li = torch.empty((g, b, k), dtype=torch.int32, device="cuda")
    caches = []
    for a in range(g):
        c = apc.apc_build_cache(e[cuts[a]:cuts[a + 1]], None if es is None else es[cuts[a]:cuts[a + 1]])
        caches.append(c)
        apc.apc_match_batch(c, q, qs, k, ls[a], li[a], apc.workspace_tensor(c, b, k))
    ms = torch.empty((b, k), device="cuda")
    mi = torch.empty((b, k), dtype=torch.int32, device="cuda")
    apc.apc_merge_shards(ls, li, g, b, k, cuts[:-1], k, ms, mi)
    torch.cuda.synchronize()
    assert torch.equal(mi, ti) and torch.equal(ms, ts)
    for c in caches + [whole]:
        c.close()


def test_merge_shards_offsets_near_int32_limit(apc, orc):
    # global entry numbers are summed in 64 bits; those of 2^31 - 1 or more are
    # not candidates (they would wrap to negative int32 numbers)
    say("merge_shards offsets near 2^31")
    rng = np.random.default_rng(99)
    g, b, kin, k = 4, 200, 16, 20
    s, i = _shard_lists(rng, g, b, kin, 500)
    offsets = [0, 2**31 - 650, 2**31 - 150, 2**31 - 1]   # disjoint ranges; the last two partly or wholly past the limit
    os_ = torch.full((b, k), 7.0, device="cuda")
    oi = torch.full((b, k), 7, dtype=torch.int32, device="cuda")
    apc.apc_merge_shards(torch.from_numpy(s).cuda(), torch.from_numpy(i).cuda(), g, b, kin, offsets, k, os_, oi)
    torch.cuda.synchronize()
    ws, wi = orc.merge_shards(s, i, offsets, k)
    gs = os_.cpu().numpy()
    assert np.array_equal(oi.cpu().numpy(), wi)
    assert np.array_equal(np.isnan(gs), np.isnan(ws)) and np.array_equal(gs[~np.isnan(ws)], ws[~np.isnan(ws)])
    assert (wi >= -1).all() and (wi[:, 0] >= 0).all()
