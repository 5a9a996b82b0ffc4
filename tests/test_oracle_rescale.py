"""Pins for the oracle's residual scale r (not GPU).

The layer-dropout training equation multiplies the kept branch by r_train;
the paper's choice is r_train = 1/rho with rho = 1 - p (Hyperparameters
section, "Dropout Scale"), and the parameterisation table carries a constant
residual-branch multiplier.  The oracle's r is res_scale / (1 - p) with
rescaling on and res_scale with it off.  What pins it, besides itself:

  * torch float64 autograd of the mask-multiply form H + r M f(H) over the
    whole batch, for rescale on and off and res_scale in {0.5, 1, 1.7};
  * expectations over the Philox masks: for one residual block, the mean
    output over steps is x + res_scale f(x) with rescaling (the rescale
    makes the expected training output the evaluation output) and
    x + (1 - p) res_scale f(x) without it;
  * exact identities: without rescaling the branch is homogeneous of degree
    one in res_scale for an attention-only block, and at p = 0 rescaling on
    and off coincide.
A mistake such as dropping res_scale when rescaling is off, applying 1/(1-p)
twice, or rescaling by (1 - p) instead of 1/(1 - p), fails one of these.
"""
import numpy as np
import pytest

import ld_inputs as inp
from oracle import masks, schedule, stack
from tests import torch_dense_ref as tref

SH = inp.SHAPES["tiny"]


def _problem(layers=None, batch=None):
    sh = inp.Shape(layers or SH.n_layers, SH.d_model, SH.n_heads, SH.d_ff, SH.seq,
                   batch or SH.batch, "f32")
    X = inp.f64(inp.hidden(sh))
    G = inp.f64(inp.upstream_grad(sh))
    W = [{k: inp.f64(v) for k, v in inp.layer_weights(sh, l, gain_jitter=True).items()}
         for l in range(sh.n_layers)]
    return sh, X, G, W


def _close(a, b, tol):
    a, b = np.asarray(a), np.asarray(b)
    return np.max(np.abs(a - b)) <= tol * max(1.0, np.max(np.abs(b)))


@pytest.mark.parametrize("rescale", [True, False])
@pytest.mark.parametrize("res_scale", [0.5, 1.0, 1.7])
def test_matches_torch_mask_multiply(rescale, res_scale):
    sh, X, G, W = _problem()
    cfg = stack.Config(n_heads=sh.n_heads, rescale=rescale, res_scale=res_scale)
    ps = schedule.rates(schedule.UNIFORM, schedule.CONSTANT, 0.4, sh.n_layers, 0, 1)
    out = stack.stack_step(X, W, ps, 0, 7, G, cfg)
    assert out["count"].min() > 0 and out["count"].max() < sh.batch, "want ragged layers"
    # the branch multiplier of each layer, from the paper's r_train = 1/rho
    # (rho = 1 - p, the float32 p the masks use) and the constant multiplier
    rs = [res_scale * (1.0 / (1.0 - float(np.float32(p))) if rescale else 1.0) for p in ps]
    XL, G0, grads = tref.stack_step(X, W, out["keep"], rs, G, sh.n_heads, cfg.rms_eps)
    assert _close(out["X_L"], XL, 1e-12)
    assert _close(out["G_0"], G0, 1e-11)
    for l in range(sh.n_layers):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11), (l, k)


@pytest.mark.parametrize("rescale", [True, False])
@pytest.mark.parametrize("res_scale", [0.5, 1.7])
def test_mean_over_masks_one_block(rescale, res_scale):
    """Mean over steps of one residual block (FFN switched off by zeroing its
    output projection): x + res_scale f(x) with rescaling, x + (1 - p)
    res_scale f(x) without; within a CLT bound of the mask mean."""
    sh, X, G, W = _problem(layers=1, batch=4)
    W[0]["w_down"][:] = 0.0
    p = np.float32(0.5)
    cfg = stack.Config(n_heads=sh.n_heads, rescale=rescale, res_scale=res_scale)
    plain = stack.Config(n_heads=sh.n_heads)
    fx = stack.layer_forward(X, W[0], np.ones(sh.batch, np.uint8), 0.0, plain)[0] - X
    assert np.max(np.abs(fx)) > 1e-3
    n = 400
    acc = np.zeros_like(X)
    for t in range(n):
        keep = masks.keep_bits(p, 1, t, 0, sh.batch)
        acc += stack.layer_forward(X, W[0], keep, p, cfg)[0]
    mean = acc / n
    want = X + (res_scale if rescale else (1 - p) * res_scale) * fx
    # |mean(M) - (1-p)| <= 5 sigma; the branch carries r * mean(M)
    r = res_scale / (1 - p) if rescale else res_scale
    bound = 5 * np.sqrt(p * (1 - p) / n) * r
    assert np.all(np.abs(mean - want) <= bound * np.abs(fx) + 1e-12)
    # and not the other rule
    other = X + ((1 - p) * res_scale if rescale else res_scale) * fx
    assert np.max(np.abs(mean - other)) > 0.1 * res_scale * np.max(np.abs(fx))


def test_no_rescale_is_homogeneous_in_res_scale():
    """Without rescaling an attention-only block adds res_scale f(x): the
    branch at res_scale c is exactly c times the branch at res_scale 1 (up to
    one rounding of the sum), for every p and every kept sample."""
    sh, X, G, W = _problem(layers=1)
    W[0]["w_down"][:] = 0.0
    p = np.float32(0.3)
    keep = masks.keep_bits(p, 0, 3, 0, sh.batch)
    assert 0 < keep.sum() < sh.batch
    one = stack.layer_forward(X, W[0], keep, p, stack.Config(n_heads=sh.n_heads, rescale=False))[0]
    for c in (0.5, 1.7, -2.0):
        got = stack.layer_forward(X, W[0], keep, p,
                                  stack.Config(n_heads=sh.n_heads, rescale=False, res_scale=c))[0]
        assert _close(got - X, c * (one - X), 1e-13)
        for b in range(sh.batch):
            if not keep[b]:
                assert np.array_equal(got[b], X[b])


def test_p0_rescale_on_equals_off():
    sh, X, G, W = _problem()
    ps = np.zeros(sh.n_layers, np.float32)
    for c in (0.5, 1.7):
        on = stack.stack_step(X, W, ps, 0, 0, G, stack.Config(n_heads=sh.n_heads, res_scale=c))
        off = stack.stack_step(X, W, ps, 0, 0, G,
                               stack.Config(n_heads=sh.n_heads, rescale=False, res_scale=c))
        assert np.array_equal(on["X_L"], off["X_L"]) and np.array_equal(on["G_0"], off["G_0"])


def test_rescale_off_gradient_scales_with_res_scale():
    """The weight gradients of an FFN-only block (attention switched off)
    without rescaling are res_scale times those at res_scale 1 for the
    down projection, whose gradient is linear in the branch scale."""
    sh, X, G, W = _problem(layers=1)
    W[0]["w_o"][:] = 0.0
    keep = np.ones(sh.batch, np.uint8)
    base = stack.Config(n_heads=sh.n_heads, rescale=False)
    _, ctx1 = stack.layer_forward(X, W[0], keep, 0.25, base)
    _, g1 = stack.layer_backward(ctx1, G, base)
    cfg = stack.Config(n_heads=sh.n_heads, rescale=False, res_scale=1.7)
    _, ctx2 = stack.layer_forward(X, W[0], keep, 0.25, cfg)
    _, g2 = stack.layer_backward(ctx2, G, cfg)
    assert _close(g2["w_down"], 1.7 * g1["w_down"], 1e-13)
