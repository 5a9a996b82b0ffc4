"""Pins for the oracle's depth-elastic inference (not GPU): the evaluation
form over an active-layer set and KV-cached incremental decoding.

What pins them, besides the oracle itself:
  * torch float64 built from library routines (rms_norm,
    scaled_dot_product_attention with is_causal or an explicit float mask
    carrying the causal cut and the ALiBi bias, silu / relu) for the
    evaluation form, the cached keys/values and one decoded layer;
  * the training forward at p = 0 (r_train = 1), which the evaluation form
    with r_eval = 1 must equal exactly;
  * causality: decoding rows pos..pos+n-1 from the cache of positions
    0..pos-1 gives the evaluation forward's rows at those positions;
  * attention over explicit query positions reduces to causal attention when
    the queries are all positions.
"""
import dataclasses

import numpy as np
import pytest

import ld_inputs as inp
from oracle import block, infer, stack
from tests import torch_dense_ref as tref

KINDS = [0, 1]


def _problem(kind, layers=3, seq=None, batch=3):
    base = inp.SHAPES["tiny"]
    sh = dataclasses.replace(base, n_layers=layers, seq=seq or base.seq, batch=batch, kind=kind)
    X = inp.f64(inp.hidden(sh))
    W = [{k: inp.f64(v) for k, v in inp.layer_weights(sh, l, gain_jitter=True).items()}
         for l in range(layers)]
    return sh, X, W


def _close(a, b, tol):
    a, b = np.asarray(a), np.asarray(b)
    return np.max(np.abs(a - b)) <= tol * max(1.0, np.max(np.abs(b)))


ACTIVE_SETS = {"all": [1, 1, 1, 1], "exit2": [1, 1, 0, 0], "exit1": [1, 0, 0, 0],
               "skip_odd": [1, 0, 1, 0], "skip_first": [0, 1, 1, 1], "none": [0, 0, 0, 0]}


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("name", list(ACTIVE_SETS))
def test_eval_matches_torch(kind, name):
    sh, X, W = _problem(kind, layers=4)
    act = ACTIVE_SETS[name]
    r = [1.0, 0.8, 1.25, 1.0]
    XL, kv = infer.eval_forward(X, W, act, sh.n_heads, kind=kind, r_eval=r)
    XT, kvT = tref.eval_stack(X, W, act, r, sh.n_heads, 1e-5, kind)
    assert _close(XL, XT, 1e-12)
    for l in range(4):
        if act[l]:
            assert _close(kv[l][0], kvT[l][0], 1e-12) and _close(kv[l][1], kvT[l][1], 1e-12)
        else:
            assert kv[l] is None
    if name == "none":
        assert np.array_equal(XL, X)


@pytest.mark.parametrize("kind", KINDS)
def test_eval_r1_all_active_is_training_forward_at_p0(kind):
    sh, X, W = _problem(kind)
    XL, _ = infer.eval_forward(X, W, [1] * sh.n_layers, sh.n_heads, kind=kind)
    cfg = stack.Config(n_heads=sh.n_heads, block_kind=kind)
    XT = stack.stack_forward(X, W, np.zeros(sh.n_layers, np.float32), 0, 0, cfg)[0]
    assert np.array_equal(XL, XT)


@pytest.mark.parametrize("kind", KINDS)
def test_early_exit_is_the_truncated_stack(kind):
    sh, X, W = _problem(kind, layers=4)
    for exit_at in range(5):
        act = [1 if l < exit_at else 0 for l in range(4)]
        a, _ = infer.eval_forward(X, W, act, sh.n_heads, kind=kind)
        b, _ = infer.eval_forward(X, W[:exit_at], [1] * exit_at, sh.n_heads, kind=kind)
        assert np.array_equal(a, b)


@pytest.mark.parametrize("kind", KINDS)
def test_attention_rows_reduce_to_causal_attention(kind):
    rng = np.random.default_rng(4)
    S, d, H = 19, 24, 3
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    slopes = block.alibi_slopes(H) if kind == 1 else None
    want, _ = block.causal_attention(q, k, v, H, slopes)
    got = infer.attention_rows(q, k, v, np.arange(S), H, slopes)
    assert _close(got, want, 1e-13)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("name", ["all", "skip_odd", "exit2"])
@pytest.mark.parametrize("pos,n", [(0, 1), (0, 4), (7, 1), (9, 3), (31, 1)])
def test_decode_equals_eval_rows(kind, name, pos, n):
    sh, X, W = _problem(kind, layers=4, seq=32)
    act = ACTIVE_SETS[name]
    if pos + n > 32:
        pytest.skip("past the sequence")
    full, _ = infer.eval_forward(X[:, :pos + n], W, act, sh.n_heads, kind=kind)
    if pos == 0:
        kv = [None if not a else (np.zeros((sh.batch, 0, sh.d_model)),) * 2 for a in act]
    else:
        _, kv = infer.eval_forward(X[:, :pos], W, act, sh.n_heads, kind=kind)
    got, new_kv = infer.decode(X[:, pos:pos + n], W, act, kv, pos, sh.n_heads, kind=kind)
    assert _close(got, full[:, pos:pos + n], 1e-12)
    # the new keys/values are the evaluation forward's at those positions
    _, kv_full = infer.eval_forward(X[:, :pos + n], W, act, sh.n_heads, kind=kind)
    for l in range(4):
        if act[l]:
            assert _close(new_kv[l][0], kv_full[l][0][:, pos:], 1e-12)
            assert _close(new_kv[l][1], kv_full[l][1][:, pos:], 1e-12)


@pytest.mark.parametrize("kind", KINDS)
def test_draft_decode_over_full_model_cache_matches_torch(kind):
    """Drafting: a subset of layers decodes over the keys/values the full
    model wrote for earlier positions (so the layer inputs of cached rows come
    from the full model, not from the subset)."""
    sh, X, W = _problem(kind, layers=4, seq=24)
    pos, n = 17, 3
    _, kv = infer.eval_forward(X[:, :pos], W, [1, 1, 1, 1], sh.n_heads, kind=kind)
    draft = [1, 0, 1, 0]
    got, _ = infer.decode(X[:, pos:pos + n], W, draft, kv, pos, sh.n_heads, kind=kind)
    x = X[:, pos:pos + n]
    for l in range(4):
        if draft[l]:
            x = tref.decode_layer(x, W[l], kv[l][0], kv[l][1], pos, 1.0, sh.n_heads, 1e-5, kind)
    assert _close(got, x, 1e-12)
    # and it is not what the subset's own prefill would give
    own, _ = infer.eval_forward(X[:, :pos + n], W, draft, sh.n_heads, kind=kind)
    assert not _close(got, own[:, pos:], 1e-6)


def test_decode_r_eval_scales_branches():
    sh, X, W = _problem(0, layers=2, seq=16)
    pos, n = 10, 2
    r = [0.5, 2.0]
    _, kv = infer.eval_forward(X[:, :pos], W, [1, 1], sh.n_heads, r_eval=r)
    got, _ = infer.decode(X[:, pos:pos + n], W, [1, 1], kv, pos, sh.n_heads, r_eval=r)
    full, _ = infer.eval_forward(X[:, :pos + n], W, [1, 1], sh.n_heads, r_eval=r)
    assert _close(got, full[:, pos:], 1e-12)
    XT, _ = tref.eval_stack(X[:, :pos + n], W, [1, 1], r, sh.n_heads, 1e-5)
    assert _close(got, XT[:, pos:], 1e-12)
