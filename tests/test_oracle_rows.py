"""Pins for the oracle's data-movement definitions: exact rational
arithmetic for fmaf, torch's bfloat16 conversion for the rounding."""
from fractions import Fraction

import numpy as np
import torch

from oracle import rows


def _round32(fr):
    """Correctly rounded binary32 of a Fraction (brute force: candidates)."""
    f = np.float32(float(fr))          # within one ulp of the answer
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - fr),
                                     int(np.float32(c).view(np.uint32)) & 1))
    return best


def test_fmaf_matches_exact_rationals():
    rng = np.random.default_rng(0)
    n = 3000
    r = rng.standard_normal(n).astype(np.float32)
    y = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    x = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    # plant exact binary32 ties: x = -r*y + half an ulp pattern
    got = rows.fmaf(r, y, x)
    for i in range(n):
        want = _round32(Fraction(float(r[i])) * Fraction(float(y[i])) + Fraction(float(x[i])))
        assert got[i] == want, i


def test_fmaf_tie_cases():
    # x + r*y lands exactly between two binary32 values in binary64 but the
    # exact value is not a tie: 1 + 2^-24 + tiny
    r = np.float32(2.0 ** -24)
    y = np.float32(1.0 + 2.0 ** -23)
    x = np.float32(1.0)
    exact = Fraction(1) + Fraction(2) ** -24 * (Fraction(1) + Fraction(2) ** -23)
    assert rows.fmaf(r, y, x) == _round32(exact) == np.nextafter(np.float32(1), np.float32(2))
    # a real binary64 tie: r*y = 2^-24 (1 - 2^-36), x = 1 + 2^-23, so the
    # binary64 sum is the binary32 midpoint 1 + 3*2^-24 while the exact value
    # lies just below it (ties-to-even on the binary64 sum would round up)
    r3 = np.float32(2.0 ** -24 * (1 + 2.0 ** -18))
    y3 = np.float32(1 - 2.0 ** -18)
    x3 = np.float32(1 + 2.0 ** -23)
    exact3 = Fraction(float(r3)) * Fraction(float(y3)) + Fraction(float(x3))
    assert float(r3) * float(y3) + float(x3) == 1 + 3 * 2.0 ** -24
    assert rows.fmaf(r3, y3, x3) == _round32(exact3) == x3
    assert rows.fmaf(r3, -y3, -x3) == -x3


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(200_000) * np.exp2(rng.integers(-60, 60, 200_000))).astype(np.float32)
    x[:6] = [0.0, -0.0, np.inf, -np.inf, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = rows.bf16_round(x)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert np.isnan(rows.bf16_round(np.array([np.nan], np.float32)))[0]
