"""Pins for the oracle's data-movement definitions: exact rational
arithmetic for fmaf, torch's bfloat16 conversion for the rounding."""
from fractions import Fraction

import numpy as np
import pytest
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


# ---- row mapping of the compacted form (gather / scatter-add) -------------
# The efficient form runs f on the kept sequences only and puts the result
# back (Preliminary section); the plain definition is the mask multiply
# X + r M Y over the whole batch.  These tests build that plain form with
# the mask alone (no kept list): Y over the whole batch is the compacted
# rows placed, in ascending sample order, at the samples whose mask is 1.

def _fma32_longdouble(r, y, x):
    """binary32 round of r*y + x evaluated exactly in x87 extended precision
    (r*y has 48 significant bits; the test data keeps the sum inside the
    64-bit significand, which is asserted)."""
    ld = np.longdouble
    p = ld(r) * y.astype(ld)
    s = p + x.astype(ld)
    assert np.all((s - x.astype(ld)) == p), "sum not exact in extended precision"
    return s.astype(np.float32)


def _masked_plain(X, keep, Yk, r, dtype):
    B, S, d = X.shape
    M = np.asarray(keep, bool)
    Y = np.zeros((B, S, d), np.float32)
    Y[M] = np.asarray(Yk, np.float32).reshape(-1, S, d)
    v = _fma32_longdouble(np.float32(r), Y, X.astype(np.float32))
    if dtype == "bf16":
        v = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    return np.where(M[:, None, None], v, X.astype(np.float32))


def _rows_case(keep, dtype, seed):
    B, S, d = len(keep), 5, 24
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((B, S, d)).astype(np.float32)
    n = int(np.sum(keep))
    Yk = rng.standard_normal((n * S, d)).astype(np.float32)
    if dtype == "bf16":   # storage values of the dtype
        X = torch.from_numpy(X).to(torch.bfloat16).to(torch.float32).numpy()
        Yk = torch.from_numpy(Yk).to(torch.bfloat16).to(torch.float32).numpy()
    idx = np.nonzero(np.asarray(keep))[0]
    return X, Yk, idx, n


KEEP_CASES = {
    "ragged": [1, 0, 0, 1, 1, 0, 1, 0],
    "single_last": [0, 0, 0, 0, 0, 0, 0, 1],
    "single_first": [1, 0, 0, 0, 0, 0, 0, 0],
    "empty": [0] * 8,
    "all": [1] * 8,
}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", list(KEEP_CASES))
def test_scatter_add_equals_mask_multiply(case, dtype):
    keep = KEEP_CASES[case]
    X, Yk, idx, n = _rows_case(keep, dtype, 11)
    r = np.float32(1.0 / (1.0 - 0.37))
    got = rows.scatter_add(X, idx, n, r, Yk, dtype)
    want = _masked_plain(X, keep, Yk, r, dtype)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    for b in range(len(keep)):       # dropped samples: bit copies
        if not keep[b]:
            assert np.array_equal(got[b].view(np.uint32), X[b].view(np.uint32))


@pytest.mark.parametrize("case", list(KEEP_CASES))
def test_gather_equals_masked_rows(case):
    keep = KEEP_CASES[case]
    X, _, idx, n = _rows_case(keep, "f32", 12)
    got = rows.gather(X, idx, n, X.shape[1])
    want = X[np.asarray(keep, bool)].reshape(-1, X.shape[2])
    assert got.shape == want.shape and np.array_equal(got, want)
