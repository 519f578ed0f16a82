"""Handle lifetime, device binding and repeatability on the GPU.

* A cache built, destroyed and built again over the same rows gives the
  same factors and bit for bit the same matches.
* Calls that take a handle check that the handle's device is current
  (APC_E_ARG otherwise; the mismatch needs a second device).
* apc_assign at b = 16,384 repeated 100 times gives identical outputs every
  time (the rank of every query comes from ordered ballots, never from an
  atomic's return order); the similarity + top-k kernel, whose filter
  bounds depend on timing, repeated 20 times gives identical lists.
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


def _match(apc, c, q, qs, k):
    b = q.shape[0]
    ts = torch.empty((b, k), device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    apc.apc_match_batch(c, q, qs, k, ts, ti, apc.workspace_tensor(c, b, k))
    torch.cuda.synchronize()
    return ts, ti


@pytest.mark.parametrize("dtype", ["f16", "e4m3"])
def test_build_destroy_rebuild_identity(apc, dtype):
    say(f"build, destroy, rebuild {dtype}")
    e, es = make_rows(30000, 768, dtype, 5, clusters=40)
    q, qs = make_rows(200, 768, dtype, 6, clusters=40)
    outs = []
    for _ in range(3):
        c = apc.apc_build_cache(e, es)
        f = torch.empty(e.shape[0], device="cuda")
        apc.apc_cache_row_factors(c, f)
        ts, ti = _match(apc, c, q, qs, 16)
        outs.append((f.clone(), ts.clone(), ti.clone()))
        c.close()
    for f, ts, ti in outs[1:]:
        assert torch.equal(f, outs[0][0]) and torch.equal(ts, outs[0][1]) and torch.equal(ti, outs[0][2])


def test_calls_check_the_handle_device(apc):
    say("device check")
    e, _ = make_rows(1000, 256, "f16", 7)
    q, _ = make_rows(8, 256, "f16", 8)
    c = apc.apc_build_cache(e)
    _match(apc, c, q, None, 4)                       # the handle's own device: accepted
    if torch.cuda.device_count() < 2:
        c.close()
        pytest.skip("one GPU: a call from another device cannot be made here")
    with torch.cuda.device(1):
        ts = torch.empty((8, 4), device="cuda:1")
        ti = torch.empty((8, 4), dtype=torch.int32, device="cuda:1")
        ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda:1")
        with pytest.raises(apc.ApcError) as ex:
            apc.apc_match_batch(c, q.to("cuda:1"), None, 4, ts, ti, ws)
        assert ex.value.name == "APC_E_ARG"
    c.close()


def test_assign_repeated_100_times(apc, orc):
    say("apc_assign b=16384 x 100")
    w = synth.WORKLOADS[4]
    rng = np.random.default_rng(2024)
    best = rng.uniform(0.6, 1.0, w.B).astype(np.float32)
    lvl, cap, queue = synth.instances(w)
    theta, K = synth.thresholds(w)
    ts = torch.from_numpy(best).cuda()
    outs = [torch.empty(w.B, dtype=torch.int32, device="cuda") for _ in range(4)]
    fill = torch.empty(w.n_inst, dtype=torch.int32, device="cuda")
    ref = None
    for r in range(100):
        for o in outs:
            o.fill_(-7)
        fill.fill_(-7)
        apc.apc_assign(ts, 1, w.B, theta, K, lvl, cap, queue, *outs, fill)
        torch.cuda.synchronize()
        got = [o.cpu().numpy() for o in outs] + [fill.cpu().numpy()]
        if ref is None:
            ref = got
            want = orc.assign(orc.levels(best.astype(np.float64), theta), w.L, lvl, cap, queue)
            assert np.array_equal(got[0], orc.levels(best.astype(np.float64), theta))
            for g_, w_ in zip(got[1:], want):
                assert np.array_equal(g_, w_)
        else:
            for g_, r_ in zip(got, ref):
                assert np.array_equal(g_, r_), f"repeat {r} differs"


@pytest.mark.parametrize("dtype,n,b,k", [("f16", 100000, 256, 10), ("e4m3", 200000, 1024, 32)])
def test_match_repeated(apc, dtype, n, b, k):
    say(f"match {dtype} n={n} b={b} k={k} x 20")
    e, es = make_rows(n, 768, dtype, 11, clusters=300)
    q, qs = make_rows(b, 768, dtype, 12, clusters=300)
    c = apc.apc_build_cache(e, es)
    ts0, ti0 = _match(apc, c, q, qs, k)
    for r in range(20):
        ts, ti = _match(apc, c, q, qs, k)
        assert torch.equal(ti, ti0) and torch.equal(ts, ts0), f"repeat {r} differs"
    c.close()
