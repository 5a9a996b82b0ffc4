"""Pins for the oracle's mask granularities (not GPU): sub-layer dropout
(independent attention and FFN masks) and per-batch dropout (one draw per
layer and step), Dropout Granularity section.

What pins them, besides the oracle itself:
  * numpy's independent Philox4x64-10 for every word the masks use;
  * keep rates, the joint keep rate (1-p)^2 of independent sub-block masks,
    and per-batch masks constant over the batch;
  * torch float64 autograd of the mask-multiply form with separate
    attention and FFN masks (Z = X + r M_attn f_attn(X), X' = Z + r M_ffn
    f_ffn(Z)), built from library routines;
  * central finite differences under sub-layer masks;
  * the reductions the definitions give: equal sub-layer masks are layer
    dropout, per-batch dropout is layer dropout under an all-or-none mask.
"""
import numpy as np
import pytest

import ld_inputs as inp
from oracle import masks, stack
from tests import torch_dense_ref as tref
from tests.test_oracle_philox import _numpy_philox

SH = inp.SHAPES["tiny"]
GRANS = (masks.LAYER_SEQ, masks.SUBLAYER_SEQ, masks.LAYER_BATCH, masks.SUBLAYER_BATCH)


def _cfg(gran):
    return stack.Config(n_heads=SH.n_heads, granularity=gran)


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


def _rs(ps, keep, cfg):
    return [stack.residual_scale(p, cfg) if np.asarray(keep[l]).any() else 1.0
            for l, p in enumerate(ps)]


# ------------------------------------------------------------------ masks

@pytest.mark.parametrize("gran", GRANS)
def test_mask_words_match_numpy_philox(gran):
    p = 0.37
    thr = masks.threshold(p)
    for seed in (0, 9, 2**63 + 1):
        for step in (0, 1, 999, 2**41):
            for layer in (0, 3, 31):
                B = 13
                got = masks.keep_bits_granular(p, seed, step, layer, B, gran)
                assert got.shape == (masks.n_masks(gran), B)
                for m in range(got.shape[0]):
                    for b in range(B):
                        if gran & 2:
                            w = _numpy_philox([0, layer, step, 1], [seed, 0])[m]
                        else:
                            w = _numpy_philox([b, layer, step, 0], [seed, 0])[m]
                        assert got[m, b] == (0 if w < thr else 1)


def test_attention_mask_is_the_layer_mask():
    for layer in range(4):
        a = masks.keep_bits_granular(0.3, 5, 17, layer, 200, masks.SUBLAYER_SEQ)[0]
        assert np.array_equal(a, masks.keep_bits(0.3, 5, 17, layer, 200))


@pytest.mark.parametrize("gran", GRANS)
def test_p0_keeps_all_p1_drops_all(gran):
    nm = masks.n_masks(gran)
    assert (masks.keep_bits_granular(0.0, 1, 2, 3, 50, gran) == 1).all()
    assert (masks.keep_bits_granular(1.0, 1, 2, 3, 50, gran) == 0).all()
    assert masks.keep_bits_granular(1.0, 1, 2, 3, 50, gran).shape == (nm, 50)


@pytest.mark.parametrize("p", [0.1, 0.5, 0.9])
def test_sublayer_rates_and_independence(p):
    """10^6 (sample, layer) pairs: each sub-block keeps with 1 - p and both
    together with (1 - p)^2, each within 5 sigma."""
    n, L = 100_000, 10
    ka = np.zeros(0, dtype=np.uint8)
    kf = np.zeros(0, dtype=np.uint8)
    for l in range(L):
        k = masks.keep_bits_granular(p, 123, 7, l, n, masks.SUBLAYER_SEQ)
        ka = np.concatenate([ka, k[0]])
        kf = np.concatenate([kf, k[1]])
    N = n * L
    for rate, want in ((ka.mean(), 1 - p), (kf.mean(), 1 - p),
                       ((ka & kf).mean(), (1 - p) ** 2)):
        sigma = np.sqrt(want * (1 - want) / N)
        assert abs(rate - want) < 5 * sigma, (rate, want)


@pytest.mark.parametrize("gran", [masks.LAYER_BATCH, masks.SUBLAYER_BATCH])
def test_per_batch_constant_over_batch_and_rate(gran):
    p = 0.3
    vals = []
    for step in range(200):
        for layer in range(100):
            k = masks.keep_bits_granular(p, 77, step, layer, 9, gran)
            assert (k == k[:, :1]).all()
            vals.append(k[:, 0])
    v = np.array(vals)
    N = len(v)
    sigma = np.sqrt(p * (1 - p) / N)
    for m in range(v.shape[1]):
        assert abs(v[:, m].mean() - (1 - p)) < 5 * sigma
    if v.shape[1] == 2:
        want = (1 - p) ** 2
        assert abs((v[:, 0] & v[:, 1]).mean() - want) < 5 * np.sqrt(want * (1 - want) / N)
    # the per-batch stream is not sample 0's per-sequence stream
    seq0 = np.array([masks.keep_bits(p, 77, s, l, 1)[0] for s in range(200) for l in range(100)])
    assert not np.array_equal(seq0, v[:, 0])


def test_masks_granular_lists():
    ps = np.array([0.0, 0.5, 1.0, 0.2], dtype=np.float32)
    for gran in GRANS:
        keep, idx, count = masks.masks_granular(ps, 3, 4, 37, gran)
        nm = masks.n_masks(gran)
        assert keep.shape == (4, nm, 37) and idx.shape == (4, nm, 37) and count.shape == (4, nm)
        for l in range(4):
            for m in range(nm):
                kept = np.nonzero(keep[l, m])[0]
                assert count[l, m] == len(kept)
                assert list(idx[l, m, :len(kept)]) == list(kept)
                assert (idx[l, m, len(kept):] == -1).all()


# ------------------------------------------------------------ layer / stack

@pytest.mark.parametrize("gran", [masks.SUBLAYER_SEQ, masks.SUBLAYER_BATCH, masks.LAYER_BATCH])
@pytest.mark.parametrize("p_max", [0.2, 0.6])
@pytest.mark.parametrize("kind", [0, 1])
def test_matches_torch_mask_multiply(gran, p_max, kind):
    sh, X, G, W = _problem(layers=3)
    if kind == 1:
        sh1 = inp.Shape(3, SH.d_model, SH.n_heads, SH.d_ff, SH.seq, SH.batch, "f32", 1)
        W = [{k: inp.f64(v) for k, v in inp.layer_weights(sh1, l, gain_jitter=True).items()}
             for l in range(3)]
    cfg = stack.Config(n_heads=SH.n_heads, granularity=gran, block_kind=kind)
    ps = np.full(3, p_max, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 4, 11, G, cfg)
    XL, G0, grads = tref.stack_step(X, W, out["keep"], _rs(ps, out["keep"], cfg), G,
                                    sh.n_heads, cfg.rms_eps, kind)
    assert _close(out["X_L"], XL, 1e-12)
    assert _close(out["G_0"], G0, 1e-11)
    for l in range(3):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11), (l, k)


def _forced_sublayer(L, B):
    keep = np.zeros((L, 2, B), dtype=np.uint8)
    keep[0, 0, [1, 4]] = 1                  # attention only on two samples
    keep[1, 1, [0, 2, 3, 7]] = 1            # FFN only, ragged
    keep[2, 0, :] = 1                       # attention on all, FFN on one
    keep[2, 1, 5] = 1
    keep[3, 0, [0, 3, 6]] = 1               # overlapping, both partial
    keep[3, 1, [3, 4, 6, 7]] = 1
    return keep


def test_forced_sublayer_masks_match_torch():
    sh, X, G, W = _problem(layers=5)
    cfg = _cfg(masks.SUBLAYER_SEQ)
    keep = _forced_sublayer(5, sh.batch)      # layer 4: nothing kept anywhere
    ps = np.full(5, 0.5, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 0, G, cfg, keep=keep)
    assert out["count"].tolist() == [[2, 0], [0, 4], [8, 1], [3, 4], [0, 0]]
    XL, G0, grads = tref.stack_step(X, W, keep, _rs(ps, keep, cfg), G, sh.n_heads, cfg.rms_eps)
    assert _close(out["X_L"], XL, 1e-12) and _close(out["G_0"], G0, 1e-11)
    for l in range(5):
        for k in stack.WEIGHT_KEYS:
            assert _close(out["grads"][l][k], grads[l][k], 1e-11), (l, k)
    # a sub-block kept on no sample has zero weight gradients
    for k in ("g_mlp", "w_gate_up", "w_down"):
        assert not out["grads"][0][k].any()
    for k in ("g_attn", "w_qkv", "w_o"):
        assert not out["grads"][1][k].any()
    for k in stack.WEIGHT_KEYS:
        assert not out["grads"][4][k].any()


def test_sublayer_finite_differences():
    sh, X, G, W = _problem(layers=4)
    cfg = _cfg(masks.SUBLAYER_SEQ)
    keep = _forced_sublayer(4, sh.batch)
    ps = np.full(4, 0.25, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 0, 0, G, cfg, keep=keep)

    def loss(Xp, Wp):
        return float(np.sum(G * stack.stack_forward(Xp, Wp, ps, 0, 0, cfg, keep=keep)[0]))

    rng = np.random.default_rng(8)
    h = 1e-5
    for l in range(4):
        for k in stack.WEIGHT_KEYS:
            for _ in range(2):
                i = tuple(rng.integers(0, n) for n in W[l][k].shape)
                Wp = [{kk: v.copy() for kk, v in w.items()} for w in W]
                Wp[l][k][i] += h
                lp = loss(X, Wp)
                Wp[l][k][i] -= 2 * h
                fd = (lp - loss(X, Wp)) / (2 * h)
                an = out["grads"][l][k][i]
                assert abs(fd - an) / max(1.0, abs(an)) < 1e-6, (l, k, i, fd, an)
    for _ in range(6):
        i = tuple(rng.integers(0, n) for n in X.shape)
        Xp = X.copy(); Xp[i] += h
        lp = loss(Xp, W)
        Xp[i] -= 2 * h
        fd = (lp - loss(Xp, W)) / (2 * h)
        assert abs(fd - out["G_0"][i]) / max(1.0, abs(out["G_0"][i])) < 1e-6


def test_equal_sublayer_masks_are_layer_dropout():
    sh, X, G, W = _problem()
    ps = np.full(sh.n_layers, 0.5, dtype=np.float32)
    lay = stack.stack_step(X, W, ps, 2, 9, G, _cfg(masks.LAYER_SEQ))
    pair = np.stack([lay["keep"], lay["keep"]], axis=1)
    sub = stack.stack_step(X, W, ps, 2, 9, G, _cfg(masks.SUBLAYER_SEQ), keep=pair)
    assert np.array_equal(sub["X_L"], lay["X_L"]) and np.array_equal(sub["G_0"], lay["G_0"])
    for l in range(sh.n_layers):
        for k in stack.WEIGHT_KEYS:
            assert np.array_equal(sub["grads"][l][k], lay["grads"][l][k])


def test_per_batch_is_layer_dropout_under_all_or_none_masks():
    sh, X, G, W = _problem(layers=6)
    ps = np.full(6, 0.5, dtype=np.float32)
    pb = stack.stack_step(X, W, ps, 1, 3, G, _cfg(masks.LAYER_BATCH))
    assert set(pb["count"].tolist()) <= {0, sh.batch}
    assert 0 < (pb["count"] == 0).sum() < 6, "want kept and dropped layers at this seed"
    lay = stack.stack_step(X, W, ps, 1, 3, G, _cfg(masks.LAYER_SEQ), keep=pb["keep"])
    assert np.array_equal(pb["X_L"], lay["X_L"]) and np.array_equal(pb["G_0"], lay["G_0"])
    for l in range(6):
        if pb["count"][l] == 0:
            assert all(not pb["grads"][l][k].any() for k in stack.WEIGHT_KEYS)


def test_sublayer_dropped_everywhere_passes_through_bitwise():
    sh, X, G, W = _problem()
    ps = np.full(sh.n_layers, 0.6, dtype=np.float32)
    out = stack.stack_step(X, W, ps, 6, 1, G, _cfg(masks.SUBLAYER_SEQ))
    any_kept = out["keep"].any(axis=(0, 1))
    assert not any_kept.all(), "want a sample dropped by every sub-block at this seed"
    for b in range(sh.batch):
        if not any_kept[b]:
            assert np.array_equal(out["X_L"][b], X[b]) and np.array_equal(out["G_0"][b], G[b])
