"""Pins of the reference's merge of per-shard top-k lists (CPU only).

Merging the exact top-k of every row shard of a cache must give the exact
top-k of the whole cache (the oracle's own brute force, which is pinned
elsewhere); the merge is also checked on hand-made lists with ties across
shards, invalid entries and fewer candidates than k.
"""
import numpy as np

from oracle import oracle


def test_merge_of_shard_topk_is_global_topk():
    rng = np.random.default_rng(61)
    n, d, b, k = 900, 24, 40, 7
    e = rng.standard_normal((n, d)).astype(np.float32)
    e[100:110] = e[5]                                          # duplicate rows: ties across shards
    q = rng.standard_normal((b, d)).astype(np.float32)
    q[:5] = e[5]
    gs, gi = oracle.topk("f32", q, None, e, None, k)
    for cuts in ([0, 450, 900], [0, 100, 333, 334, 900], [0, 7, 900]):
        S = len(cuts) - 1
        ls = np.full((S, b, k), np.nan, np.float32)
        li = np.full((S, b, k), -1, np.int64)
        for s in range(S):
            kk = min(k, cuts[s + 1] - cuts[s])
            ss, ii = oracle.topk("f32", q, None, e[cuts[s]:cuts[s + 1]], None, kk)
            ls[s, :, :kk], li[s, :, :kk] = ss, ii
        ms, mi = oracle.merge_shards(ls, li, cuts[:-1], k)
        assert np.array_equal(mi, gi), cuts
        assert np.array_equal(ms, gs.astype(np.float32))


def test_merge_hand_made_lists():
    s = np.array([[[0.9, 0.5, 0.1]], [[0.9, 0.7, np.nan]], [[0.5, 0.2, 0.0]]], np.float32)
    i = np.array([[[3, 1, 0]], [[0, 2, -1]], [[4, 9, -1]]])
    ms, mi = oracle.merge_shards(s, i, [0, 10, 20], 5)
    # 0.9 at global 3 and 10 (tie: lower entry first), 0.7 at 12, 0.5 at 1 and 24
    assert mi.tolist() == [[3, 10, 12, 1, 24]]
    assert np.allclose(ms, [[0.9, 0.9, 0.7, 0.5, 0.5]])
    ms, mi = oracle.merge_shards(s[:, :, :1] * np.nan, i[:, :, :1], [0, 10, 20], 2)
    assert (mi == -1).all() and np.isnan(ms).all()


def test_merge_drops_entries_past_int32():
    # shard 1 starts 5 entries below 2^31 - 1: its local entries 0..3 fit, 5 and
    # above would reach 2^31 - 1 or wrap, and are not candidates
    top = 2**31 - 1
    s = np.array([[[0.3, 0.2]], [[0.9, 0.8]], [[0.95, 0.1]]], np.float32)
    i = np.array([[[7, 8]], [[9, 3]], [[0, 1]]])
    ms, mi = oracle.merge_shards(s, i, [0, top - 5, top - 1], 6)
    # kept: 0.95 at top - 1, 0.8 at top - 2, 0.3 at 7, 0.2 at 8; dropped: 0.9 at
    # top + 4 and 0.1 at top
    assert mi.tolist() == [[top - 1, top - 2, 7, 8, -1, -1]]
    assert np.allclose(ms[0, :4], [0.95, 0.8, 0.3, 0.2]) and np.isnan(ms[0, 4:]).all()
