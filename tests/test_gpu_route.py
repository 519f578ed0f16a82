"""GPU parity of the placement that follows a Route-Plan (Eq. 1).

apc_assign_routed is compared bit for bit with the oracle's routed placement
given the same plan: the oracle's LP plan for the batch, the flow that the
rounds placement realises (which must reproduce the rounds placement), and
arbitrary seeded quota matrices (over capacity, over demand, negative).
apc_assign_planned builds the plan in the kernel; plans are not unique, so
its plan is checked for feasibility and for the LP's number served and
minimal degradation, and its placement against apc_assign_routed given that
plan and against the host planner's plan for the oracle's histogram.
"""
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


def _case(rng, b, L, I, tight):
    theta = np.unique(np.sort(rng.uniform(-0.5, 0.99, L)).astype(np.float32))
    L = theta.size
    K = (np.cumsum(rng.integers(1, 9, L)) if L else np.zeros(0)).astype(np.int32)
    best = rng.uniform(-1, 1, b).astype(np.float32)
    if L:
        best[: b // 4] = theta[rng.integers(0, L, b // 4)]         # exact boundaries
    il = rng.integers(0, L + 1, I)
    cap_hi = max(2, (b if tight else 3 * b) // max(I, 1))
    ic = rng.integers(0, cap_hi, I)
    iq = rng.integers(0, 5, I)
    return theta, K, best, il, ic, iq


def _run(apc, fn, best, ld, theta, K, il, ic, iq, plan):
    b = best.size
    ts = torch.zeros((b, ld), dtype=torch.float32)
    ts[:, 0] = torch.from_numpy(best)
    ts = ts.cuda()
    outs = [torch.full((b,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    fill = torch.full((len(il),), -7, dtype=torch.int32, device="cuda")
    fn(ts, ld, b, theta, K, il, ic, iq, plan, *outs, fill)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs] + [fill.cpu().numpy()]


def _hist(level, L):
    return np.bincount(level, minlength=L + 1).astype(np.int64)


def _caps(il, ic, L):
    F = np.zeros(L + 1, dtype=np.int64)
    np.add.at(F, il, ic)
    return F


SIZES = [(1, 0, 1, False), (37, 3, 4, True), (256, 5, 6, True), (256, 8, 12, False), (257, 4, 5, True),
         (1000, 32, 40, True), (1024, 6, 16, True), (3000, 10, 30, True), (4096, 12, 64, False),
         (9000, 32, 256, True), (16384, 8, 64, True)]


@pytest.mark.parametrize("b,L,I,tight", SIZES)
def test_assign_routed_lp_plan_bit_exact(apc, orc, b, L, I, tight):
    say(f"assign_routed lp plan b={b} L={L} I={I} tight={tight}")
    rng = np.random.default_rng(1000 + b + L)
    theta, K, best, il, ic, iq = _case(rng, b, L, I, tight)
    L = theta.size
    level = orc.levels(best.astype(np.float64), theta)
    x, d, served = orc.route_plan(_hist(level, L), _caps(il, ic, L), K)
    plan = torch.from_numpy(x.astype(np.int32)).cuda()
    opt, ol, oi, os_, fill = _run(apc, apc.apc_assign_routed, best, 2, theta, K, il, ic, iq, plan)
    assert np.array_equal(opt, level)
    r = orc.assign_routed(level, L, x, il, ic, iq)
    assert np.array_equal(ol, r[0]) and np.array_equal(oi, r[1]) and np.array_equal(os_, r[2])
    assert np.array_equal(fill, r[3])
    assert (ol >= 0).sum() == served


@pytest.mark.parametrize("b,L,I,tight", SIZES[1:8])
def test_assign_routed_reproduces_rounds(apc, orc, b, L, I, tight):
    say(f"assign_routed rounds flow b={b} L={L} I={I}")
    rng = np.random.default_rng(2000 + b + L)
    theta, K, best, il, ic, iq = _case(rng, b, L, I, tight)
    L = theta.size
    level = orc.levels(best.astype(np.float64), theta)
    g = orc.assign(level, L, il, ic, iq)
    x = np.zeros((L + 1, L + 1), dtype=np.int32)
    for q, j in enumerate(g[0]):
        if j >= 0:
            x[level[q], j] += 1
    got = _run(apc, apc.apc_assign_routed, best, 1, theta, K, il, ic, iq, torch.from_numpy(x).cuda())
    for a, e in zip(got[1:], g):
        assert np.array_equal(a, e)


@pytest.mark.parametrize("b,L,I", [(50, 3, 4), (700, 6, 9), (5000, 12, 30)])
def test_assign_routed_arbitrary_quotas(apc, orc, b, L, I):
    say(f"assign_routed arbitrary quotas b={b} L={L}")
    rng = np.random.default_rng(3000 + b)
    theta, K, best, il, ic, iq = _case(rng, b, L, I, True)
    L = theta.size
    level = orc.levels(best.astype(np.float64), theta)
    x = rng.integers(-3, max(4, 2 * b // (L + 1)), (L + 1, L + 1)).astype(np.int32)
    got = _run(apc, apc.apc_assign_routed, best, 1, theta, K, il, ic, iq, torch.from_numpy(x).cuda())
    r = orc.assign_routed(level, L, x, il, ic, iq)
    for a, e in zip(got[1:], r):
        assert np.array_equal(a, e)


@pytest.mark.parametrize("b,L,I,tight", SIZES)
def test_assign_planned_is_optimal(apc, orc, b, L, I, tight):
    say(f"assign_planned b={b} L={L} I={I} tight={tight}")
    rng = np.random.default_rng(4000 + b + L)
    theta, K, best, il, ic, iq = _case(rng, b, L, I, tight)
    L = theta.size
    level = orc.levels(best.astype(np.float64), theta)
    H, F = _hist(level, L), _caps(il, ic, L)
    plan = torch.full(((L + 1) * (L + 1),), -7, dtype=torch.int32, device="cuda")
    opt, ol, oi, os_, fill = _run(apc, apc.apc_assign_planned, best, 1, theta, K, il, ic, iq, plan)
    X = plan.cpu().numpy().reshape(L + 1, L + 1).astype(np.int64)
    assert np.array_equal(opt, level)
    # the plan: feasible, and the LP's number served and minimal degradation
    assert (X >= 0).all() and (X.sum(axis=1) <= H).all() and (X.sum(axis=0) <= F).all()
    _, d, served = orc.route_plan(H, F, K)
    assert orc.plan_cost(X, K) == (d, served)
    # the placement realises it exactly
    flow = np.zeros_like(X)
    for q, j in enumerate(ol):
        if j >= 0:
            flow[level[q], j] += 1
    assert np.array_equal(flow, X)
    # the host planner gives the same plan for the same histogram
    Xh, dh = apc.apc_route_plan(K, H, F)
    assert np.array_equal(Xh, X) and dh == d
    # and the routed entry point, given that plan, the same placement
    again = _run(apc, apc.apc_assign_routed, best, 1, theta, K, il, ic, iq, plan)
    for a, e in zip(again, (opt, ol, oi, os_, fill)):
        assert np.array_equal(a, e)


def test_plan_placement_edge_cases(apc, orc):
    say("plan placement edge cases")
    theta, K = [0.0, 0.5], [4, 9]
    b = 40
    ts = torch.linspace(-1, 1, b).reshape(b, 1).cuda()
    outs = lambda: [torch.full((b,), -7, dtype=torch.int32, device="cuda") for _ in range(4)]
    plan = torch.full((9,), -7, dtype=torch.int32, device="cuda")
    # no capacity anywhere: nothing served, the plan is all zeros
    o = outs()
    fill = torch.full((2,), -7, dtype=torch.int32, device="cuda")
    apc.apc_assign_planned(ts, 1, b, theta, K, [0, 2], [0, 0], None, plan, *o, fill)
    torch.cuda.synchronize()
    assert (plan == 0).all() and (o[1] == -1).all() and (fill == 0).all()
    # no instances at all
    o = outs()
    apc.apc_assign_planned(ts, 1, b, theta, K, [], [], None, plan, *o, fill)
    torch.cuda.synchronize()
    assert (plan == 0).all() and (o[1] == -1).all() and (o[2] == -1).all()
    # empty batch: the plan is written (zeros), the instance fills are zero
    apc.apc_assign_planned(ts, 1, 0, theta, K, [0, 1], [3, 3], None, plan, *outs(), fill)
    torch.cuda.synchronize()
    assert (plan == 0).all() and (fill == 0).all()
    # capacity exactly the demand, one level only: everything goes there
    o = outs()
    fill1 = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    apc.apc_assign_planned(ts, 1, b, theta, K, [2], [b], None, plan, *o, fill1)
    torch.cuda.synchronize()
    lv = orc.levels(ts[:, 0].cpu().numpy().astype(np.float64), np.array(theta, np.float32))
    Xo = np.zeros((3, 3), dtype=np.int64)                     # the only optimal plan here
    Xo[:, 2] = orc.level_histogram(lv, 2)
    assert np.array_equal(plan.cpu().numpy().reshape(3, 3), Xo) and (o[1] == 2).all() and fill1.item() == b
    r = orc.assign_routed(lv, 2, Xo, [2], [b], None)
    assert np.array_equal(o[2].cpu().numpy(), r[1]) and np.array_equal(o[3].cpu().numpy(), r[2])
    # a caller's plan of all zeros routes nothing
    o = outs()
    apc.apc_assign_routed(ts, 1, b, theta, K, [0, 1, 2], [9, 9, 9], None,
                          torch.zeros(9, dtype=torch.int32, device="cuda"), *o,
                          torch.empty(3, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert (o[1] == -1).all()
