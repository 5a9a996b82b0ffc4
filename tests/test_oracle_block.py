"""Pins for the oracle's block, layer and stack (not GPU).

What pins it, besides itself:
  * torch float64 autograd of the mask-multiply form H + r M f(H) built from
    library routines (rms_norm, scaled_dot_product_attention, silu) -- the
    paper's plain definition, against which the oracle's per-sequence skip
    form must agree (Preliminary section: executing f only on kept sequences
    gives the same result);
  * central finite differences of the oracle's own forward (gradients);
  * the special cases p = 0 (dense stack) and p = 1 (identity, zero grads);
  * per-sequence independence and the Monte-Carlo mean under r = 1/(1-p).
"""
import numpy as np
import pytest

import ld_inputs as inp
from oracle import masks, schedule, stack
from tests import torch_dense_ref as tref

SH = inp.SHAPES["tiny"]
CFG = stack.Config(n_heads=SH.n_heads)


def _problem(gain_jitter=True, batch=None, seq=None, layers=None):
    sh = inp.Shape(layers or SH.n_layers, SH.d_model, SH.n_heads, SH.d_ff,
                   seq or SH.seq, batch or SH.batch, "f32")
    X = inp.f64(inp.hidden(sh))
    G = inp.f64(inp.upstream_grad(sh))
    W = [{k: inp.f64(v) for k, v in inp.layer_weights(sh, l, gain_jitter=gain_jitter).items()}
         for l in range(sh.n_layers)]
    return sh, X, G, W


def _ild(sh, p_max=0.2):
    return schedule.rates(schedule.ILD, schedule.CONSTANT, p_max, sh.n_layers, 0, 1)


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
    XL, G0, grads = tref.stack_step(X, W, out["keep"], _rs(ps, out["keep"]), G,
                                    sh.n_heads, CFG.rms_eps)
    assert _close(out["X_L"], XL, 1e-12)
    assert _close(out["G_0"], G0, 1e-11)
    for l in range(sh.n_layers):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11), (l, k)


def test_forced_masks_count_0_1_ragged_all():
    sh, X, G, W = _problem(layers=4)
    keep = np.zeros((4, sh.batch), dtype=np.uint8)
    keep[1, 5] = 1                      # count 1
    keep[2, [0, 2, 3, 7]] = 1           # ragged
    keep[3, :] = 1                      # all
    ps = np.full(4, 0.5, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 0, G, CFG, keep=keep)
    assert list(out["count"]) == [0, 1, 4, 8]
    XL, G0, grads = tref.stack_step(X, W, keep, _rs(ps, keep), G, sh.n_heads, CFG.rms_eps)
    assert _close(out["X_L"], XL, 1e-12) and _close(out["G_0"], G0, 1e-11)
    for l in range(4):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11)
    for k in stack.WEIGHT_KEYS:
        assert not out["grads"][0][k].any()


def test_p1_is_identity_and_zero_grads():
    sh, X, G, W = _problem()
    ps = np.ones(sh.n_layers, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 0, G, CFG)
    assert np.array_equal(out["X_L"], X) and np.array_equal(out["G_0"], G)
    assert all(not g[k].any() for g in out["grads"] for k in stack.WEIGHT_KEYS)
    assert (out["count"] == 0).all()


def test_p0_is_dense_and_equals_forced_all_keep():
    sh, X, G, W = _problem()
    ps = np.zeros(sh.n_layers, dtype=np.float32)
    a = stack.stack_step(X, W, ps, 0, 0, G, CFG)
    b = stack.stack_step(X, W, ps, 0, 0, G, CFG, keep=np.ones((sh.n_layers, sh.batch), np.uint8))
    assert (a["count"] == sh.batch).all()
    assert np.array_equal(a["X_L"], b["X_L"]) and np.array_equal(a["G_0"], b["G_0"])


def test_finite_differences():
    """Central differences of L = sum(G * X_L) at the tiny shape, float64."""
    sh, X, G, W = _problem()
    ps = _ild(sh, 0.5)
    out = stack.stack_step(X, W, ps, 0, 1, G, CFG)
    assert out["count"].min() > 0, "want every layer exercised"
    keep = out["keep"]

    def loss(Xp, Wp):
        XL = stack.stack_forward(Xp, Wp, ps, 0, 1, CFG, keep=keep)[0]
        return float(np.sum(G * XL))

    rng = np.random.default_rng(5)
    h = 1e-5
    worst = 0.0
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
                err = abs(fd - an) / max(1.0, abs(an))
                worst = max(worst, err)
                assert err < 1e-6, (l, k, i, fd, an)
    for _ in range(6):
        i = tuple(rng.integers(0, n) for n in X.shape)
        Xp = X.copy(); Xp[i] += h
        lp = loss(Xp, W)
        Xp[i] -= 2 * h
        lm = loss(Xp, W)
        fd = (lp - lm) / (2 * h)
        assert abs(fd - out["G_0"][i]) / max(1.0, abs(out["G_0"][i])) < 1e-6


def test_dropped_rows_bitwise_and_samples_independent():
    sh, X, G, W = _problem()
    ps = np.full(sh.n_layers, 0.5, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 2, G, CFG)
    # a sample dropped by every layer passes through bit for bit
    for b in range(sh.batch):
        if not out["keep"][:, b].any():
            assert np.array_equal(out["X_L"][b], X[b]) and np.array_equal(out["G_0"][b], G[b])
    # changing another sample's input leaves sample b's outputs unchanged
    X2 = X.copy(); X2[3] += 1.0
    G2 = G.copy(); G2[3] -= 0.5
    out2 = stack.stack_step(X2, W, ps, 0, 2, G2, CFG)
    for b in range(sh.batch):
        if b != 3:
            assert np.array_equal(out["X_L"][b], out2["X_L"][b])
            assert np.array_equal(out["G_0"][b], out2["G_0"][b])


@pytest.mark.parametrize("zeroed", ["w_down", "w_o"])
def test_rescaled_mean_matches_dense_one_block(zeroed):
    """r = 1/(1-p): averaging one residual block's output over steps gives
    x + f(x) (Hyperparameters section: r_eval = 1 makes the eval output the
    expected training output).  This is exact in expectation for a single
    residual block only -- with both sub-blocks live the FFN sees the rescaled
    attention output -- so the other sub-block is switched off by zeroing its
    output projection."""
    sh, X, G, W = _problem(layers=1, batch=4)
    W[0][zeroed][:] = 0.0
    p = np.float32(0.5)
    dense, _ = stack.layer_forward(X, W[0], np.ones(sh.batch, np.uint8), 0.0, CFG)
    n = 400
    acc = np.zeros_like(X)
    for t in range(n):
        keep = masks.keep_bits(p, 0, t, 0, sh.batch)
        acc += stack.layer_forward(X, W[0], keep, p, CFG)[0]
    mean = acc / n
    fx = dense - X
    assert np.max(np.abs(fx)) > 1e-3
    bound = 5 * np.sqrt(p * (1 - p) / n) / (1 - p)   # CLT bound on |r*mean(M) - 1|
    assert np.all(np.abs(mean - dense) <= bound * np.abs(fx) + 1e-12)
    # and not r = 1 (which would give x + (1-p) f(x))
    assert np.max(np.abs(mean - (X + (1 - p) * fx))) > 0.1 * np.max(np.abs(fx))
