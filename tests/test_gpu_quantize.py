"""GPU parity of the storage step (apc_quantize_rows) and of the row checks
(apc_validate_rows) against the oracle: codes and scales bit-exact, flags,
counts and the first bad row exact."""
import numpy as np
import pytest
import torch

from tests.gpu_check import say

pytestmark = pytest.mark.gpu

TORCH_OF = {"f16": torch.float16, "bf16": torch.bfloat16, "e4m3": torch.float8_e4m3fn, "f32": torch.float32}


@pytest.fixture(scope="module")
def apc():
    import paper_2502_06798_amd as apc
    apc.load()
    assert torch.cuda.is_available()
    return apc


def float_rows(n, d, seed):
    """Normal rows with per-row magnitudes from 2^-140 to 2^120, plus rows
    that hit each special case of the roundings."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d)) * 2.0 ** rng.integers(-140, 120, size=(n, 1))
    x = x.astype(np.float32)
    x[0] = 0.0
    x[1, 7] = np.nan
    x[2, 3] = np.inf
    x[3, :] = -x[3, :]
    x[3, 5] = -np.inf
    x[4] = rng.standard_normal(d).astype(np.float32) * np.float32(1e-40)       # subnormal scale
    x[5] = rng.uniform(-448, 448, d).astype(np.float32)
    # exact float32 midpoints of neighbouring bfloat16 and e4m3 values
    b = rng.integers(0x3000, 0x4F00, d).astype(np.uint32) << 16
    x[6] = (b | np.uint32(0x8000)).view(np.float32)
    x[7] = rng.choice([65504.0, 65519.0, 65520.0, 7e4, 2.0 ** -25, 2.0 ** -24 * 1.5], d).astype(np.float32)
    x[8] = np.float32(2.0 ** -140)
    x[9, :] = 0.0
    x[9, d - 1] = 1.0                                                            # one nonzero in the tail
    return x


def _codes(t):
    return t.view(torch.uint8 if t.element_size() == 1 else torch.int16).cpu().numpy()


@pytest.mark.parametrize("dtype,n,d", [("f16", 1000, 520), ("bf16", 777, 264), ("e4m3", 1000, 784),
                                       ("e4m3", 33, 16), ("f16", 10, 8), ("bf16", 3000, 1024),
                                       ("e4m3", 3000, 1024)])
def test_quantize_rows_bit_exact(apc, orc, dtype, n, d):
    say(f"quantize_rows {dtype} n={n} d={d}")
    x = float_rows(n, d, 11 + n)
    xd = torch.from_numpy(x).cuda()
    out = torch.empty(n, d, dtype=TORCH_OF[dtype], device="cuda")
    sc = torch.full((n,), -7.0, device="cuda") if dtype == "e4m3" else None
    apc.apc_quantize_rows(xd, out, sc)
    torch.cuda.synchronize()
    want, ws = orc.quantize_rows(dtype, x)
    got = _codes(out)
    want = want.view(got.dtype)
    if dtype == "e4m3":
        assert (got == want).all()
        assert (sc.cpu().numpy().view(np.uint32) == ws.view(np.uint32)).all()
        return
    nan = np.isnan(x)
    assert (got[~nan] == want[~nan]).all()
    gv = out.float().cpu().numpy()
    assert np.isnan(gv[nan]).all() and not np.isnan(gv[~nan]).any()


def test_quantize_then_validate_and_build(apc, orc):
    """Rows stored by the library pass its own checks and build a cache."""
    say("quantize then validate")
    rng = np.random.default_rng(5)
    x = torch.from_numpy(rng.standard_normal((500, 256)).astype(np.float32)).cuda()
    for dtype in ("f16", "bf16", "e4m3"):
        out = torch.empty(500, 256, dtype=TORCH_OF[dtype], device="cuda")
        sc = torch.empty(500, device="cuda") if dtype == "e4m3" else None
        apc.apc_quantize_rows(x, out, sc)
        assert apc.apc_validate_rows(out, sc) == (0, -1)
        c = apc.apc_build_cache(out, sc)
        c.close()


def _bad_rows(dtype, n, d, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d)).astype(np.float32)
    picks = rng.choice(n, size=9, replace=False)
    sc = None
    if dtype == "e4m3":
        codes, sc = orc_quant(x)
        codes[picks[0], 3] = 0x7F                                 # NaN codes
        codes[picks[1], d - 1] = 0xFF
        codes[picks[2]] = 0x80                                    # negative zeros only
        codes[picks[3]] = 0
        sc[picks[4]] = 0.0
        sc[picks[5]] = -1.0
        sc[picks[6]] = np.inf
        sc[picks[7]] = np.nan
        codes[picks[8]] = 0
        sc[picks[8]] = np.nan                                     # two flags at once
        return codes, sc
    x[picks[0], 3] = np.nan
    x[picks[1], d - 1] = np.inf
    x[picks[2]] = 0.0
    x[picks[3]] = 2.0 ** -80                                      # squares below float32's range
    x[picks[4]] = 2.0 ** -70
    x[picks[5], 0] = 2e19                                         # the sum of squares overflows
    x[picks[6]] = -0.0
    if dtype == "f32":
        return x, None
    if dtype == "f16":
        with np.errstate(over="ignore"):
            h = x.astype(np.float16)
        h[picks[7], 1] = np.float16(np.inf)
        return h, None
    from oracle import oracle
    return oracle.round_bf16(x), None


def orc_quant(x):
    from oracle import oracle
    return oracle.quantize_rows("e4m3", x)


@pytest.mark.parametrize("dtype,n,d", [("f32", 1000, 100), ("f16", 2001, 264), ("bf16", 999, 512),
                                       ("e4m3", 3000, 784), ("e4m3", 9, 16)])
def test_validate_rows_flags(apc, orc, dtype, n, d):
    say(f"validate_rows {dtype} n={n} d={d}")
    rows, sc = _bad_rows(dtype, n, d, 3 + n)
    want = orc.validate_rows(dtype, rows, sc)
    t = torch.from_numpy(rows.view(np.uint8) if dtype == "e4m3" else rows.view(np.int16) if dtype == "bf16" else rows)
    if dtype == "e4m3":
        t = t.view(torch.float8_e4m3fn)
    elif dtype == "bf16":
        t = t.view(torch.bfloat16)
    t = t.cuda()
    s = None if sc is None else torch.from_numpy(sc).cuda()
    bad = torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda")
    nb, fb = apc.apc_validate_rows(t, s, bad)
    got = bad.cpu().numpy()
    assert (got == want).all(), np.nonzero(got != want)
    assert nb == int((want != 0).sum())
    assert fb == (int(np.nonzero(want)[0][0]) if nb else -1)
    # without the flag array the count and the first bad row are the same
    assert apc.apc_validate_rows(t, s) == (nb, fb)
