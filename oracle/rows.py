"""Definitions of the isolated data-movement operations of the compacted form.

Test infrastructure (see the package docstring).

The efficient form of the method runs f only on the kept sequences
(Preliminary section); moving their rows in and out is a bit copy (gather)
and a residual update (scatter-add).  For bit-exact checks of the scatter-add
its rounding is fixed as: out = round_dtype(fmaf(r, y, x)) -- one fused
multiply-add in binary32 (one rounding), then one round-to-nearest-even to the
storage type.  Nothing here depends on the HIP code.
"""

import numpy as np

_MID29 = np.uint64(1 << 28)
_LOW29 = np.uint64((1 << 29) - 1)


def fmaf(r, y, x):
    """Correctly rounded binary32 r*y + x for binary32 inputs (float64 arrays
    holding binary32 values).  r*y is exact in binary64 (24+24 bits); the sum
    and its rounding error come from TwoSum, and a binary32 tie left by the
    binary64 sum is broken by the sign of that error."""
    r, y, x = np.broadcast_arrays(*(np.asarray(v, dtype=np.float64) for v in (r, y, x)))
    shape = r.shape
    r, y, x = (np.atleast_1d(v).ravel() for v in (r, y, x))
    p = r * y
    s = p + x
    bp = s - x
    e = (x - (s - bp)) + (p - bp)
    out = s.astype(np.float32)
    bits = s.view(np.uint64)
    tie = ((bits & _LOW29) == _MID29) & (e != 0) & np.isfinite(s)
    if np.any(tie):
        st = s[tie]
        toward_zero = (bits[tie] & ~_LOW29).view(np.float64).astype(np.float32)
        away = np.nextafter(toward_zero, np.float32(np.inf) * np.sign(st).astype(np.float32))
        same_sign = np.sign(e[tie]) == np.sign(st)
        out[tie] = np.where(same_sign, away, toward_zero)
    return out.reshape(shape)


def bf16_round(x32):
    """Round binary32 values to bfloat16 (nearest, ties to even), returned as
    binary32 values; NaNs stay NaN (quiet)."""
    x32 = np.asarray(x32, dtype=np.float32)
    u = x32.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    out = (rounded & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)
    nan = np.isnan(x32)
    if np.any(nan):
        out = out.copy()
        out[nan] = np.float32(np.nan)
    return out


def gather(X, idx, count, S):
    """Kept rows of X [B, S, d] stacked: row j*S + s comes from idx[j]*S + s."""
    return np.concatenate([X[idx[j]] for j in range(count)], axis=0) if count else X[:0].reshape(0, X.shape[-1])


def scatter_add(X, idx, count, r, Yk, dtype):
    """X with rows of kept sequences replaced by round_dtype(fmaf(r, Yk, X));
    X, Yk hold values of `dtype` ("bf16" or "f32") as float64/float32."""
    out = np.array(X, dtype=np.float32)
    S = out.shape[1]
    r32 = np.float64(np.float32(r))
    for j in range(count):
        b = idx[j]
        v = fmaf(r32, np.asarray(Yk[j * S:(j + 1) * S], dtype=np.float64), out[b].astype(np.float64))
        out[b] = bf16_round(v) if dtype == "bf16" else v
    return out
