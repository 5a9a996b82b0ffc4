"""Per-layer, per-step layer-dropout rates.

Test infrastructure (see the package docstring).

Depth distributions (Dropout Configurations, "Dropout Distribution"):
  uniform  p^l = p_max
  ILD      p^l = l/(L-1) * p_max           (increasing layer distribution)
  ALD      p^l = p_max * [l odd]           (alternating layer distribution)
Time schedules (Dropout Configurations, "Dropout Schedule"):
  constant p^{l,t} = p^l
  ITS      p^{l,t} = p^l * t/(T-1)
  DTS      p^{l,t} = p^l * (1 - t/(T-1))
Readings where the paper is silent or inconsistent:
  * the glossary writes t/T for ITS/DTS while the main text writes t/(T-1);
    t/(T-1) is taken because it is the form whose closed-form mean the paper
    prints (P-bar = p_max/4 for ILD with ITS or DTS);
  * t is clamped to [0, T-1]; with T = 1 the ratio t/(T-1) is taken as 0;
  * ILD with L = 1 gives p = 0 (the distribution "starts at 0 at the first
    layer").
"""

import numpy as np

UNIFORM, ILD, ALD = 0, 1, 2
CONSTANT, ITS, DTS = 0, 1, 2


def depth_rate(dist, p_max, layer, n_layers):
    if dist == UNIFORM:
        return float(p_max)
    if dist == ILD:
        if n_layers <= 1:
            return 0.0
        return layer / (n_layers - 1) * float(p_max)
    if dist == ALD:
        return float(p_max) if layer % 2 == 1 else 0.0
    raise ValueError(f"unknown depth distribution {dist}")


def time_factor(sched, t, n_steps):
    if sched == CONSTANT:
        return 1.0
    t = min(max(int(t), 0), max(int(n_steps) - 1, 0))
    frac = 0.0 if n_steps <= 1 else t / (n_steps - 1)
    if sched == ITS:
        return frac
    if sched == DTS:
        return 1.0 - frac
    raise ValueError(f"unknown time schedule {sched}")


def rate(dist, sched, p_max, layer, n_layers, t, n_steps):
    """p^{l,t} in double precision, returned as the float32 the library takes."""
    return np.float32(depth_rate(dist, p_max, layer, n_layers) * time_factor(sched, t, n_steps))


def rates(dist, sched, p_max, n_layers, t, n_steps):
    return np.array([rate(dist, sched, p_max, l, n_layers, t, n_steps)
                     for l in range(n_layers)], dtype=np.float32)


def p_mean(ps):
    """Average dropout rate over depth at one step = FLOPs savings at that step
    (the p_mean equation of the Dropout Distribution paragraph)."""
    return float(np.mean(np.asarray(ps, dtype=np.float64)))


def p_bar(dist, sched, p_max, n_layers, n_steps):
    """Mean training dropout over depth and time = total FLOPs savings
    (the P-bar equation of the Dropout Schedule paragraph), in double."""
    tot = 0.0
    for t in range(n_steps):
        for l in range(n_layers):
            tot += depth_rate(dist, p_max, l, n_layers) * time_factor(sched, t, n_steps)
    return tot / (n_layers * n_steps)


def effective_depth(ps):
    """Expected number of executed layers, sum_l (1 - p^l) (footnote on the
    effective depth of ILD in the larger-scale runs)."""
    return float(np.sum(1.0 - np.asarray(ps, dtype=np.float64)))
