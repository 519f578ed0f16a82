"""apc_match_batch_static (the match on the library's static device
workspace, for callers that cannot allocate) against apc_match_batch with a
caller workspace: bit-identical lists on two calls in a row, the second with
a smaller batch, for the kernel families the plan picks; batches whose
workspace exceeds the static array are rejected with APC_E_WORKSPACE."""
import pytest
import torch

from tests.gpu_check import say
from tests.test_gpu_parity import make_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def apc():
    import paper_2502_06798_amd as apc
    apc.load()
    assert torch.cuda.is_available()
    return apc


def _both(apc, c, q, qs, k):
    b = q.shape[0]
    out = []
    for static in (False, True):
        ts = torch.full((b, k), 7.0, device="cuda")
        ti = torch.full((b, k), 7, dtype=torch.int32, device="cuda")
        if static:
            apc.apc_match_batch_static(c, q, qs, k, ts, ti)
        else:
            apc.apc_match_batch(c, q, qs, k, ts, ti, apc.workspace_tensor(c, b, k))
        torch.cuda.synchronize()
        out.append((ts, ti))
    return out


@pytest.mark.parametrize("dtype,d,n,bs,k", [("e4m3", 768, 60000, (2000, 300), 32),     # two waves per SIMD
                                            ("f16", 768, 40000, (700, 100), 10),        # query-stationary kernel
                                            ("f32", 64, 5000, (300, 17), 5)])           # fp32 rows
def test_static_workspace_matches_caller_workspace(apc, dtype, d, n, bs, k):
    e, es = make_rows(n, d, dtype, 71, clusters=max(1, n // 60))
    c = apc.apc_build_cache(e, es)
    for b in bs:                                   # two calls in a row, the second smaller
        say(f"static workspace {dtype} d={d} n={n} b={b} k={k}")
        q, qs = make_rows(b, d, dtype, 72 + b, clusters=None)
        q[: b // 2] = e[torch.arange(b // 2, device="cuda") * 7 % n]
        if qs is not None:
            qs[: b // 2] = es[torch.arange(b // 2, device="cuda") * 7 % n]
        (s0, i0), (s1, i1) = _both(apc, c, q, qs, k)
        assert torch.equal(i0, i1) and torch.equal(s0, s1)
    c.close()


def test_static_workspace_rejects_oversized_batches(apc):
    e, _ = make_rows(1000, 64, "f16", 73)
    c = apc.apc_build_cache(e)
    b, k = 70000, 64
    assert apc.apc_match_workspace(c, b, k) > (32 << 20)
    q = torch.zeros((b, 64), dtype=torch.float16, device="cuda")
    ts = torch.empty((b, k), device="cuda")
    ti = torch.empty((b, k), dtype=torch.int32, device="cuda")
    with pytest.raises(apc.ApcError) as ex:
        apc.apc_match_batch_static(c, q, None, k, ts, ti)
    assert ex.value.name == "APC_E_WORKSPACE"
    c.close()
