"""Pins of the reference's storage of float32 rows (quantisation) and of its
row checks (CPU only).

The roundings are pinned to torch's casts (library routines written from the
same format definitions), to closed forms (every code value maps to itself,
midpoints go to the even code, the clamp at 448) and to the input
generator's recipe; a planted mistake (ties away from zero) is caught.
"""
import numpy as np
import pytest
import torch

from paper_2502_06798_amd import synth

RNG = np.random.default_rng(2502)


def _spread(n, lo=-40, hi=40):
    """float32 values of random sign over a range of binary exponents."""
    m = RNG.uniform(1.0, 2.0, size=n)
    e = RNG.integers(lo, hi, size=n)
    s = RNG.choice([-1.0, 1.0], size=n)
    return (s * m * 2.0 ** e).astype(np.float32)


def test_e4m3_values_match_torch(orc):
    want = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    got = orc.e4m3_values()
    assert ((got == want) | (np.isnan(got) & np.isnan(want))).all()
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9 and got[0x08] == 2.0 ** -6


def _torch_e4m3(y):
    return torch.from_numpy(np.asarray(y, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_round_e4m3_codes_and_midpoints(orc):
    vals = orc.e4m3_values()
    codes = np.array([c for c in range(256) if not np.isnan(vals[c])], dtype=np.uint8)
    # every code value maps to its own code (both zeros keep their sign)
    assert (orc.round_e4m3(vals[codes].astype(np.float32)) == codes).all()
    # midpoints between neighbours go to the even code
    pos = vals[:127]
    mid = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)
    assert (mid.astype(np.float64) == (pos[:-1] + pos[1:]) / 2).all()      # exact in float32
    got = orc.round_e4m3(mid)
    lo = np.arange(126)
    assert (got == np.where(lo % 2 == 0, lo, lo + 1)).all()
    assert (orc.round_e4m3(-mid) == (got | 0x80)).all()
    assert (got == _torch_e4m3(mid)).all()


def test_round_e4m3_matches_torch(orc):
    y = np.concatenate([RNG.uniform(-448, 448, 20000), _spread(20000, -14, 8), _spread(5000, -30, -6)])
    y = np.clip(y, -448, 448).astype(np.float32)
    y = np.concatenate([y, np.array([0.0, -0.0, 448.0, -448.0, 2.0 ** -10, 3 * 2.0 ** -10], np.float32)])
    assert (orc.round_e4m3(y) == _torch_e4m3(y)).all()
    nan = orc.round_e4m3(np.array([np.nan, -np.nan], np.float32))
    assert nan.tolist() == [0x7F, 0xFF]
    with pytest.raises(ValueError):
        orc.round_e4m3(np.array([449.0], np.float32))


def test_planted_rounding_mistake_is_caught(orc, monkeypatch):
    """A rounding that sends ties away from zero (a plausible slip) fails the
    midpoint pin against torch's cast."""
    good = orc.round_e4m3

    def ties_away(y):
        a = np.abs(np.asarray(y, dtype=np.float64))
        codes = good(y)
        mag = (codes & 0x7F).astype(np.int64)
        vals = orc.e4m3_values()
        up = np.minimum(mag + 1, 0x7E)
        went_down = (vals[mag] < a) & ((vals[mag] + vals[up]) / 2 == a)
        return np.where(went_down, codes + 1, codes).astype(np.uint8)

    pos = orc.e4m3_values()[:127]
    mid = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)
    monkeypatch.setattr(orc, "round_e4m3", ties_away)
    assert (orc.round_e4m3(mid) != _torch_e4m3(mid)).any()
    monkeypatch.setattr(orc, "round_e4m3", good)
    assert (orc.round_e4m3(mid) == _torch_e4m3(mid)).all()


def test_round_bf16_matches_torch(orc):
    x = np.concatenate([_spread(40000, -140, 128), RNG.normal(size=5000).astype(np.float32)])
    # exact midpoints between neighbouring bfloat16 values (ties)
    b = (RNG.integers(0, 0x7F7F, 5000).astype(np.uint32) << 16)
    ties = (b | np.uint32(0x8000)).view(np.float32)
    big = np.array([3.3895314e38, 3.3961776e38, 3.4028235e38, np.inf, -np.inf, 0.0, -0.0], np.float32)
    x = np.concatenate([x, ties, -ties, big]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (orc.round_bf16(x) == want).all()
    n = orc.round_bf16(np.array([np.nan], np.float32))
    assert (n & 0x7F80) == 0x7F80 and (n & 0x7F) != 0               # a NaN


def test_f16_matches_torch(orc):
    x = np.concatenate([_spread(40000, -30, 17), np.array([65504.0, 65519.0, 65520.0, 1e-8, 2.0 ** -25], np.float32)])
    got, _ = orc.quantize_rows("f16", x.reshape(1, -1))
    want = torch.from_numpy(x).to(torch.float16).numpy()
    assert (got.view(np.uint16) == want.view(np.uint16)).all()


def test_e4m3_rows_match_the_generator_recipe(orc):
    x = np.concatenate([RNG.normal(size=(6, 64)) * np.array([[1], [1e-3], [300], [1e4], [0], [1e-30]]),
                        np.array([[np.nan] + [1.0] * 63])], axis=0).astype(np.float32)
    codes, s = orc.quantize_rows("e4m3", x)
    t, ts = synth.to_storage(torch.from_numpy(x), "e4m3")
    assert (codes == t.view(torch.uint8).numpy()).all()
    assert (s.view(np.uint32) == ts.numpy().view(np.uint32)).all()
    assert s[4] == 1.0 and s[6] == 1.0                              # zero row, row with NaN
    assert codes[6, 0] == 0x7F and (codes[6, 1:] == 0x38).all()       # NaN, then 1.0
    back = orc.decode("e4m3", codes[:4], s[:4])
    assert (np.abs(back) <= np.abs(x[:4]).max(axis=1)[:, None] * (1 + 2.0 ** -20)).all()
    assert (np.abs(back - x[:4]) <= np.maximum(np.abs(x[:4]) * 2.0 ** -4, s[:4, None] * 2.0 ** -10)).all()


def test_validate_rows(orc):
    f32 = np.zeros((6, 8), np.float32)
    f32[0] = 1.0
    f32[1, 3] = np.nan
    f32[2, 5] = -np.inf
    f32[3] = 2.0 ** -76                                             # squares round to zero in float32
    f32[4] = 2.0 ** -74
    f32[5, 0] = 3e19                                                # its square overflows float32
    assert orc.validate_rows("f32", f32).tolist() == [0, 1, 1, 2, 0, 1]
    zero = np.zeros((1, 8), np.float32)
    assert orc.validate_rows("f32", zero).tolist() == [2]
    bf = orc.round_bf16(np.array([[1.0] * 8, [2.0 ** -80] * 8, [0.0] * 8], np.float32))
    assert orc.validate_rows("bf16", bf).tolist() == [0, 2, 2]
    e = np.full((4, 16), 0x38, np.uint8)
    e[1, 2] = 0xFF                                                  # a NaN code
    e[2] = 0x80                                                     # all negative zeros
    s = np.array([1.0, 1.0, 1.0, 0.0], np.float32)
    assert orc.validate_rows("e4m3", e, s).tolist() == [0, 1, 2, 4]
    s2 = np.array([np.inf, -1.0, np.nan, 2.0], np.float32)
    assert orc.validate_rows("e4m3", e, s2).tolist() == [4, 5, 6, 0]
