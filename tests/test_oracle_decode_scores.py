"""Pins of the reference's decoding and similarity (CPU only).

Decoding is checked against library casts over every code; the cosine
against hand-worked closed forms, invariants and numpy's float64 matmul.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import pyref
from tests._util import np_or_none, stored_np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_decode_f16_all_codes(orc):
    codes = np.arange(65536, dtype=np.uint16).reshape(256, 256)
    got = orc.decode("f16", codes)
    want = codes.view(np.float16).astype(np.float64)
    same = (got == want) | (np.isnan(got) & np.isnan(want))
    assert same.all()


def test_decode_bf16_all_codes(orc):
    codes = np.arange(65536, dtype=np.uint16).reshape(256, 256)
    got = orc.decode("bf16", codes)
    want = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).double().numpy()
    same = (got == want) | (np.isnan(got) & np.isnan(want))
    assert same.all()


def test_decode_e4m3_all_codes(orc):
    codes = np.arange(256, dtype=np.uint8).reshape(16, 16)
    got = orc.decode("e4m3", codes, np.ones(16, dtype=np.float32))
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    same = (got == want) | (np.isnan(got) & np.isnan(want))
    assert same.all()
    # OCP e4m3fn: 448 is the largest finite value; 0x7F/0xFF are the only NaNs
    flat = got.ravel()
    assert np.nanmax(flat) == 448.0 and np.nanmin(flat) == -448.0
    assert set(np.flatnonzero(np.isnan(flat))) == {0x7F, 0xFF}


def test_decode_e4m3_row_scale_exact(orc):
    codes = np.array([[0x38, 0x7E, 0x01]], dtype=np.uint8)   # 1.0, 448, 2^-9
    sc = np.array([0.1], dtype=np.float32)
    got = orc.decode("e4m3", codes, sc)[0]
    s = float(sc[0])
    assert got[0] == s and got[1] == 448.0 * s and got[2] == s * 2.0 ** -9


def _golden_scores():
    rows = []
    for line in open(os.path.join(GOLDEN, "scores_worked.txt")):
        if line.startswith("#") or not line.strip():
            continue
        a, b, c = line.split("|")
        rows.append(([int(x) for x in a.split()], [int(x) for x in b.split()], Fraction(c.strip())))
    return rows


def test_scores_hand_worked(orc):
    for q, e, want in _golden_scores():
        got = orc.pair_scores("f32", np.array([q], np.float32), None, np.array([e], np.float32),
                              None, [0], [0])[0]
        assert abs(got - float(want)) <= 1e-15, (q, e, got, want)


def test_scores_closed_forms(orc):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((8, 37)).astype(np.float32)
    # 2x, -x and x/4 are exact in float32; 3x is rounded per element
    e = np.concatenate([x, np.float32(2.0) * x, -x, np.float32(0.25) * x, np.float32(3.0) * x])
    qi = np.repeat(np.arange(8), 5)
    ei = np.stack([np.arange(8) + 8 * j for j in range(5)], axis=1).ravel()
    s = orc.pair_scores("f32", x, None, e, None, qi, ei).reshape(8, 5)
    assert np.all(np.abs(s[:, 0] - 1) <= 5e-16)          # self-match
    assert np.all(s[:, 1] == s[:, 0])                    # power-of-two multiple: same rounding
    assert np.all(s[:, 2] == -s[:, 0])                   # negation
    assert np.all(s[:, 3] == s[:, 0])
    assert np.all(np.abs(s[:, 4] - 1) <= 1e-14)          # 3x rounded in float32
    # orthogonal integer vectors give exactly 0
    a = np.array([[1, 2, 0, -1]], np.float32)
    b = np.array([[2, -1, 7, 0], [0, 0, 5, 0]], np.float32)
    z = orc.pair_scores("f32", a, None, b, None, [0, 0], [0, 1])
    assert np.all(z == 0.0)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "e4m3"])
def test_scores_match_numpy_normalised_matmul(orc, dtype):
    from paper_2502_06798_amd import synth
    g = torch.Generator().manual_seed(5)
    x = torch.randn(40, 96, generator=g)
    y = torch.randn(300, 96, generator=g)
    xs, xsc = synth.to_storage(x, dtype)
    ys, ysc = synth.to_storage(y, dtype)
    xn, yn = stored_np(xs), stored_np(ys)
    xsc, ysc = np_or_none(xsc), np_or_none(ysc)
    X = orc.decode(dtype, xn, xsc)
    Y = orc.decode(dtype, yn, ysc)
    ref = (X / np.linalg.norm(X, axis=1, keepdims=True)) @ (Y / np.linalg.norm(Y, axis=1, keepdims=True)).T
    qi, ei = np.meshgrid(np.arange(40), np.arange(300), indexing="ij")
    got = orc.pair_scores(dtype, xn, xsc, yn, ysc, qi.ravel(), ei.ravel()).reshape(40, 300)
    assert np.max(np.abs(got - np.clip(ref, -1, 1))) <= 1e-12
    assert np.all(np.abs(got) <= 1.0)
    # symmetry
    back = orc.pair_scores(dtype, yn, ysc, xn, xsc, ei.ravel(), qi.ravel()).reshape(40, 300)
    assert np.max(np.abs(back - got)) <= 1e-15


def test_scores_scale_invariant_e4m3(orc):
    """The cosine does not depend on the positive per-row scales."""
    rng = np.random.default_rng(7)
    codes = rng.integers(0, 256, size=(20, 64), dtype=np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x30                   # no NaN codes
    s1 = rng.uniform(0.01, 3.0, 20).astype(np.float32)
    s2 = rng.uniform(0.01, 3.0, 20).astype(np.float32)
    qi, ei = np.meshgrid(np.arange(20), np.arange(20), indexing="ij")
    a = orc.pair_scores("e4m3", codes, s1, codes, s1, qi.ravel(), ei.ravel())
    b = orc.pair_scores("e4m3", codes, s2, codes, np.ones(20, np.float32), qi.ravel(), ei.ravel())
    assert np.max(np.abs(a - b)) <= 1e-15


def test_row_norm_errors(orc):
    x = np.ones((4, 8), np.float32)
    x[2] = 0.0
    _, rc, bad = orc.row_sqnorms("f32", x)
    assert rc == orc.E_ZERO_NORM and bad == 2
    x[1, 3] = np.inf
    _, rc, bad = orc.row_sqnorms("f32", x)
    assert rc == orc.E_NONFINITE and bad == 1
    codes = np.full((3, 16), 0x38, np.uint8)
    codes[1, 5] = 0xFF
    _, rc, bad = orc.row_sqnorms("e4m3", codes, np.ones(3, np.float32))
    assert rc == orc.E_NONFINITE and bad == 1


def test_cos_key_monotone_matches_float(orc):
    rng = np.random.default_rng(3)
    for _ in range(200):
        q = rng.integers(-3, 4, 4)
        e = rng.integers(-3, 4, 4)
        if not q.any() or not e.any():
            continue
        key = pyref.cos_key(q.tolist(), e.tolist())
        got = orc.pair_scores("f32", q[None].astype(np.float32), None, e[None].astype(np.float32),
                              None, [0], [0])[0]
        assert abs(pyref.cos_float(key) - got) <= 1e-15
