"""Pins for the oracle's block kind 1, the block of the paper's experiments
(Experimental Setup: ALiBi position embeddings, squared ReLU), not GPU.

What pins it, besides itself:
  * the ALiBi slopes the ALiBi paper states for 8 and 16 heads
    (tests/golden/alibi_slopes.txt), and the stated rule for other head
    counts (power-of-two prefix, then every other slope of the doubled
    sequence);
  * torch float64 autograd of the mask-multiply form with the bias passed as
    an explicit float attention mask to scaled_dot_product_attention and
    torch's relu;
  * central finite differences of the oracle's own forward;
  * zero slopes give the bias-free attention; squared ReLU of a negative
    input and its gradient are zero.
"""
import dataclasses
import os

import numpy as np
import pytest

import ld_inputs as inp
from oracle import block, schedule, stack
from tests import torch_dense_ref as tref

SH = dataclasses.replace(inp.SHAPES["tiny"], kind=1)
CFG = stack.Config(n_heads=SH.n_heads, block_kind=1)
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "alibi_slopes.txt")


def _golden():
    out = {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        h, rest = line.split(":")
        out[int(h)] = [2.0 ** -float(e) for e in rest.split()]
    return out


def test_alibi_slopes_match_the_alibi_paper():
    for h, want in _golden().items():
        assert np.allclose(block.alibi_slopes(h), want, rtol=0, atol=1e-15), h


@pytest.mark.parametrize("h", [1, 3, 5, 6, 9, 10, 12, 14, 21])
def test_alibi_slopes_other_head_counts(h):
    n = 1 << (h.bit_length() - 1)
    got = block.alibi_slopes(h)
    assert len(got) == h
    assert np.array_equal(got[:n], block.alibi_slopes(n))
    assert np.array_equal(got[n:], block.alibi_slopes(2 * n)[0::2][:h - n])
    assert len(set(got.tolist())) == h and (got > 0).all() and (got < 1).all()


def _problem(layers=None):
    sh = dataclasses.replace(SH, n_layers=layers or SH.n_layers)
    X = inp.f64(inp.hidden(sh))
    G = inp.f64(inp.upstream_grad(sh))
    W = [{k: inp.f64(v) for k, v in inp.layer_weights(sh, l, gain_jitter=True).items()}
         for l in range(sh.n_layers)]
    assert W[0]["w_gate_up"].shape == (sh.d_ff, sh.d_model)
    return sh, X, G, W


def _rs(ps, keep):
    return [stack.residual_scale(p, CFG) if keep[l].any() else 1.0 for l, p in enumerate(ps)]


def _close(a, b, tol):
    a, b = np.asarray(a), np.asarray(b)
    return np.max(np.abs(a - b)) <= tol * max(1.0, np.max(np.abs(b)))


@pytest.mark.parametrize("p_max", [0.0, 0.2, 0.6])
def test_matches_torch_mask_multiply(p_max):
    sh, X, G, W = _problem()
    ps = np.full(sh.n_layers, p_max, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 3, G, CFG)
    XL, G0, grads = tref.stack_step(X, W, out["keep"], _rs(ps, out["keep"]), G, sh.n_heads,
                                    CFG.rms_eps, kind=1)
    assert _close(out["X_L"], XL, 1e-12)
    assert _close(out["G_0"], G0, 1e-11)
    for l in range(sh.n_layers):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11), (l, k)


def test_forced_masks_against_torch():
    sh, X, G, W = _problem(layers=3)
    keep = np.zeros((3, sh.batch), dtype=np.uint8)
    keep[0, 5] = 1
    keep[1, [0, 2, 3, 7]] = 1
    keep[2, :] = 1
    ps = np.full(3, 0.5, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 0, G, CFG, keep=keep)
    XL, G0, grads = tref.stack_step(X, W, keep, _rs(ps, keep), G, sh.n_heads, CFG.rms_eps, kind=1)
    assert _close(out["X_L"], XL, 1e-12) and _close(out["G_0"], G0, 1e-11)
    for l in range(3):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11)


def test_finite_differences():
    sh, X, G, W = _problem()
    ps = schedule.rates(schedule.ILD, schedule.CONSTANT, 0.5, sh.n_layers, 0, 1)
    out = stack.stack_step(X, W, ps, 0, 1, G, CFG)
    keep = out["keep"]
    assert out["count"].min() > 0

    def loss(Xp, Wp):
        return float(np.sum(G * stack.stack_forward(Xp, Wp, ps, 0, 1, CFG, keep=keep)[0]))

    rng = np.random.default_rng(11)
    h = 1e-5
    for l in range(sh.n_layers):
        for k in stack.WEIGHT_KEYS:
            for _ in range(3):
                i = tuple(rng.integers(0, n) for n in W[l][k].shape)
                Wp = [{kk: v.copy() for kk, v in w.items()} for w in W]
                Wp[l][k][i] += h
                lp = loss(X, Wp)
                Wp[l][k][i] -= 2 * h
                lm = loss(X, Wp)
                fd = (lp - lm) / (2 * h)
                an = out["grads"][l][k][i]
                assert abs(fd - an) / max(1.0, abs(an)) < 1e-6, (l, k, i, fd, an)
    for _ in range(6):
        i = tuple(rng.integers(0, n) for n in X.shape)
        Xp = X.copy(); Xp[i] += h
        lp = loss(Xp, W)
        Xp[i] -= 2 * h
        lm = loss(Xp, W)
        assert abs((lp - lm) / (2 * h) - out["G_0"][i]) / max(1.0, abs(out["G_0"][i])) < 1e-6


def test_special_cases():
    rng = np.random.default_rng(2)
    S, d, H = 12, 16, 4
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    a0, p0 = block.causal_attention(q, k, v, H)
    a1, p1 = block.causal_attention(q, k, v, H, np.zeros(H))
    assert np.allclose(a0, a1, atol=1e-14) and np.allclose(p0, p1, atol=1e-14)
    # with a bias the first row still attends only to itself
    a2, p2 = block.causal_attention(q, k, v, H, block.alibi_slopes(H))
    assert np.allclose(p2[:, 0, 0], 1.0) and np.allclose(a2[0], v[0])
    u = np.array([-2.0, -0.0, 0.0, 0.5, 3.0])
    assert np.array_equal(block.relu2(u), [0.0, 0.0, 0.0, 0.25, 9.0])
    assert np.array_equal(block.relu2_grad(u), [0.0, 0.0, 0.0, 1.0, 6.0])
