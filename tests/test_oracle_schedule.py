"""Pins for the oracle's schedules and masks against what the paper fixes:
closed forms, printed table values, and the Bernoulli law of the mask."""
import math
import os

import numpy as np
import pytest

from oracle import masks, schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "flops_savings.txt")
DIST = dict(uniform=schedule.UNIFORM, ILD=schedule.ILD, ALD=schedule.ALD)
SCHED = dict(const=schedule.CONSTANT, ITS=schedule.ITS, DTS=schedule.DTS)


@pytest.mark.parametrize("L", [2, 3, 12, 13, 16, 17, 32, 40])
@pytest.mark.parametrize("p_max", [0.1, 0.2, 0.5, 0.99])
def test_depth_mean_closed_forms(L, p_max):
    # ILD mean = p_max / 2; ALD mean = floor(L/2)/L * p_max (Dropout Distribution).
    ild = [schedule.depth_rate(schedule.ILD, p_max, l, L) for l in range(L)]
    ald = [schedule.depth_rate(schedule.ALD, p_max, l, L) for l in range(L)]
    assert schedule.p_mean(ild) == pytest.approx(p_max / 2, rel=1e-12)
    assert schedule.p_mean(ald) == pytest.approx((L // 2) / L * p_max, rel=1e-12)
    assert ild[0] == 0.0 and ild[-1] == pytest.approx(p_max)
    # effective depth (1 - p_max/2) L for ILD (larger-scale runs footnote)
    assert schedule.effective_depth(ild) == pytest.approx((1 - 0.5 * p_max) * L, rel=1e-12)


@pytest.mark.parametrize("T", [2, 5, 101, 1001])
def test_time_mean_closed_forms(T):
    # P-bar(ILD, ITS) = P-bar(ILD, DTS) = p_max/4, P-bar(uniform, ITS) = p_max/2.
    for p_max in (0.2, 0.8):
        assert schedule.p_bar(schedule.ILD, schedule.ITS, p_max, 9, T) == pytest.approx(p_max / 4)
        assert schedule.p_bar(schedule.ILD, schedule.DTS, p_max, 9, T) == pytest.approx(p_max / 4)
        assert schedule.p_bar(schedule.UNIFORM, schedule.ITS, p_max, 9, T) == pytest.approx(p_max / 2)
        assert schedule.p_bar(schedule.UNIFORM, schedule.CONSTANT, p_max, 9, T) == pytest.approx(p_max)


def test_time_schedule_endpoints():
    T = 1001
    assert schedule.time_factor(schedule.ITS, 0, T) == 0.0
    assert schedule.time_factor(schedule.ITS, T - 1, T) == 1.0
    assert schedule.time_factor(schedule.ITS, 500, T) == 0.5
    assert schedule.time_factor(schedule.DTS, 0, T) == 1.0
    assert schedule.time_factor(schedule.DTS, T - 1, T) == 0.0
    assert schedule.time_factor(schedule.ITS, 5000, T) == 1.0  # clamped
    assert schedule.time_factor(schedule.DTS, 3, 1) == 1.0     # T = 1


def test_printed_flops_savings():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    assert len(rows) >= 10
    for p_max, dist, sched, pct, printed in rows:
        got = 100 * schedule.p_bar(DIST[dist], SCHED[sched], float(p_max), 13, 1001)
        assert got == pytest.approx(float(pct), abs=1e-9)
        assert round(got) == int(printed)


def test_threshold_special_values():
    assert masks.threshold(0.0) == 0
    assert masks.threshold(-0.0) == 0
    assert masks.threshold(1.0) is None
    assert masks.threshold(0.5) == 2**63
    assert masks.threshold(0.25) == 2**62
    with pytest.raises(ValueError):
        masks.threshold(float("nan"))
    for p in (1e-7, 0.05, 0.2, 0.95, 0.9999999):
        thr = masks.threshold(p)
        assert 0 < thr < 2**64
        assert abs(thr / 2**64 - float(np.float32(p))) <= 2.0**-64


def test_p0_keeps_all_p1_drops_all():
    for step in range(5):
        assert masks.keep_bits(0.0, 0, step, 3, 64).all()
        assert not masks.keep_bits(1.0, 0, step, 3, 64).any()


@pytest.mark.parametrize("p", [0.05, 0.1, 0.2, 0.5, 0.95])
def test_empirical_keep_rate(p):
    n = 1_000_000
    keep = masks.keep_bits(p, 7, 123, 5, n)
    rate = keep.mean()
    sigma = math.sqrt(p * (1 - p) / n)
    assert abs(rate - (1 - p)) < 5 * sigma


def test_masks_independent_across_layers_and_steps():
    n, p = 200_000, 0.5
    a = masks.keep_bits(p, 0, 10, 0, n)
    for other in (masks.keep_bits(p, 0, 10, 1, n), masks.keep_bits(p, 0, 11, 0, n),
                  masks.keep_bits(p, 1, 10, 0, n)):
        agree = (a == other).mean()
        expect = p * p + (1 - p) * (1 - p)
        assert abs(agree - expect) < 5 * math.sqrt(expect * (1 - expect) / n)


def test_masks_are_pure_function_of_counter():
    ps = np.array([0.0, 0.3, 0.6, 1.0], dtype=np.float32)
    k1, i1, c1 = masks.masks(ps, 9, 17, 32)
    masks.masks(ps, 9, 18, 32)          # other steps in between change nothing
    k2, i2, c2 = masks.masks(ps, 9, 17, 32)
    assert (k1 == k2).all() and (i1 == i2).all() and (c1 == c2).all()
    # layer-wise calls with the global layer index give the stack's masks
    for l in range(4):
        kl, il, cl = masks.masks(ps[l:l + 1], 9, 17, 32, first_layer=l)
        assert (kl[0] == k1[l]).all() and (il[0] == i1[l]).all() and cl[0] == c1[l]


def test_compaction_ascending_and_padded():
    ps = np.full(6, 0.5, dtype=np.float32)
    keep, idx, count = masks.masks(ps, 0, 0, 32)
    for l in range(6):
        kept = idx[l, :count[l]]
        assert list(kept) == sorted(kept)
        assert (keep[l, kept] == 1).all() and keep[l].sum() == count[l]
        assert (idx[l, count[l]:] == -1).all()
