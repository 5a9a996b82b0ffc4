"""Pins for the oracle's Philox4x64-10 (not GPU): numpy's independent
implementation and the published known-answer vector."""
import os

import numpy as np
import pytest

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")


def _numpy_philox(c, k):
    cint = sum(int(c[j]) << (64 * j) for j in range(4))
    g = np.random.Philox(counter=(cint - 1) % (1 << 256), key=np.array([int(k[0]), int(k[1])], dtype=np.uint64))
    return [int(v) for v in g.random_raw(4)]


def test_mulhilo_matches_python_ints():
    rng = np.random.default_rng(3)
    a = rng.integers(0, 2**64 - 1, size=2000, dtype=np.uint64, endpoint=True)
    b = rng.integers(0, 2**64 - 1, size=2000, dtype=np.uint64, endpoint=True)
    a[:4] = [0, 1, 2**64 - 1, 2**63]
    b[:4] = [2**64 - 1, 2**64 - 1, 2**64 - 1, 2]
    hi, lo = philox.mulhilo64(a, b)
    for i in range(len(a)):
        p = int(a[i]) * int(b[i])
        assert int(hi[i]) == p >> 64 and int(lo[i]) == p & (2**64 - 1)


def test_known_answer_vector():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    assert rows
    for r in rows:
        c = [int(x, 16) for x in r[:4]]
        k = [int(x, 16) for x in r[4:6]]
        want = [int(x, 16) for x in r[6:10]]
        got = philox.philox4x64_10(*c, *k)
        assert [int(g) for g in got] == want


def test_matches_numpy_on_random_counters():
    rng = np.random.default_rng(11)
    n = 4000
    c = rng.integers(0, 2**64 - 1, size=(n, 4), dtype=np.uint64, endpoint=True)
    k = rng.integers(0, 2**64 - 1, size=(n, 2), dtype=np.uint64, endpoint=True)
    w = philox.philox4x64_10(c[:, 0], c[:, 1], c[:, 2], c[:, 3], k[:, 0], k[:, 1])
    for i in range(n):
        assert [int(w[j][i]) for j in range(4)] == _numpy_philox(c[i], k[i])


def test_matches_numpy_on_mask_counters():
    """The counters the masks use: (sample, layer, step, 0), key (seed, 0),
    including the borrow cases where sample = 0 and layer/step > 0."""
    cases = []
    for seed in (0, 1, 2**63 + 5):
        for step in (0, 1, 500, 1000, 2**40):
            for layer in (0, 1, 15, 31):
                for b in (0, 1, 7, 31):
                    cases.append((b, layer, step, seed))
    for b, layer, step, seed in cases:
        w0 = philox.mask_word(b, layer, step, seed)
        assert int(w0) == _numpy_philox([b, layer, step, 0], [seed, 0])[0]
