"""GPU parity of the load-aware route-and-batch placement: apc_assign_load_aware
is compared bit for bit with the oracle's reading (greedy routing at or above
the load threshold, uniform routing at batch size 1 below it) on seeded
random scores, thresholds, instance tables and random keys, for batches from
1 to 65,536 queries (every placement kernel)."""
import numpy as np
import pytest
import torch

from tests.gpu_check import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def apc():
    import paper_2502_06798_amd as apc
    apc.load()
    assert torch.cuda.is_available()
    return apc


@pytest.mark.parametrize("b,L,I", [(1, 0, 1), (16, 5, 2), (300, 5, 8), (1000, 10, 40), (5000, 32, 256),
                                    (16384, 10, 32), (20000, 10, 64), (65536, 32, 256)])
@pytest.mark.parametrize("load", [0, 100])
def test_load_aware_bit_exact(apc, orc, b, L, I, load):
    say(f"load-aware assign b={b} L={L} I={I} load={load}")
    rng = np.random.default_rng(b * 7 + L + I + load)
    theta = np.unique(np.sort(rng.uniform(-0.5, 0.99, L)).astype(np.float32))
    L = theta.size
    K = np.arange(1, L + 1, dtype=np.int32) * 5
    best = rng.uniform(-1, 1, b).astype(np.float32)
    ts = torch.from_numpy(best).reshape(b, 1).cuda()
    il = rng.integers(0, L + 1, I).astype(np.int32)
    ic = rng.integers(0, max(2, 2 * b // I) + 1, I).astype(np.int32)
    iq = rng.integers(0, 50, I).astype(np.int32)
    rnd = rng.integers(0, 2**32, I, dtype=np.uint64).astype(np.uint32)
    rnd[: I // 3] = rnd[I // 3: 2 * (I // 3)]                   # some equal keys
    outs = [torch.full((b,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    fill = torch.full((I,), -7, dtype=torch.int32, device="cuda")
    routing = apc.apc_assign_load_aware(ts, 1, b, theta, K, il, ic, iq, rnd, load, 50, *outs, fill)
    torch.cuda.synchronize()
    opt = outs[0].cpu().numpy()
    assert np.array_equal(opt, orc.levels(best.astype(np.float64), theta))
    want = orc.assign_load_aware(opt, L, il, ic, iq, rnd, load, 50)
    assert routing == want[0] == (1 if load >= 50 else 0)
    for g, w in zip([o.cpu().numpy() for o in outs[1:]] + [fill.cpu().numpy()], want[1:]):
        assert np.array_equal(g, w)
