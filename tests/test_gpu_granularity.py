"""Mask granularities on the HIP path against the oracle (needs a GPU):
sub-layer dropout (independent attention / FFN masks) and per-batch dropout
(one draw per layer and step), Dropout Granularity section.  Masks and kept
lists bit-exact; outputs and gradients within the dtype's tolerance; rows
that no sub-block keeps bitwise untouched; weight gradients of skipped
sub-blocks exactly zero (their buffers start filled with garbage); the
per-batch path whose draws the host takes itself bitwise equal to the device
path under the same masks."""
import numpy as np
import pytest
import torch

import ld_inputs as inp
import paper_2609_05275_amd as ld
from oracle import masks, schedule, stack
from tests.gpu_util import DEV, f64, layer_weights_dev, rel, tol, zero_grads
from tests.test_gpu_layer import SMALL_BF16, SMALL_P, _buf, _cfg, _check_grads, _ocfg

pytestmark = pytest.mark.gpu

GRANS = [ld.LD_GRAN_LAYER_SEQ, ld.LD_GRAN_SUBLAYER_SEQ, ld.LD_GRAN_LAYER_BATCH,
         ld.LD_GRAN_SUBLAYER_BATCH]
GRAN_IDS = ["layer_seq", "sublayer_seq", "layer_batch", "sublayer_batch"]
SHAPES = [inp.SHAPES["tiny"], SMALL_BF16, SMALL_P]
SHAPE_IDS = ["tiny_f32", "small_bf16", "paper_small_bf16"]


def _garbage_grads(sh):
    dw = zero_grads(sh)
    for v in dw.values():
        v.fill_(7.0)
    return dw


@pytest.mark.parametrize("gran", GRANS, ids=GRAN_IDS)
@pytest.mark.parametrize("batch", [1, 8, 1000, 3001])
def test_masks_bit_exact(gran, batch):
    ps = np.float32([0.0, 0.05, 0.5, 0.95, 1.0, 0.3])
    L, nm = len(ps), masks.n_masks(gran)
    keep = torch.full((L, nm, batch), 9, dtype=torch.uint8, device=DEV)
    idx = torch.full((L, nm, batch), -7, dtype=torch.int32, device=DEV)
    cnt = torch.full((L, nm), -7, dtype=torch.int32, device=DEV)
    for seed, step in ((0, 0), (5, 1000), (2**63 + 3, 2**40 + 1)):
        ld.ld_masks_granular(gran, list(ps), seed, step, keep, idx, cnt, first_layer=3)
        torch.cuda.synchronize()
        k, i, c = masks.masks_granular(ps, seed, step, batch, gran, first_layer=3)
        assert np.array_equal(keep.cpu().numpy(), k)
        assert np.array_equal(idx.cpu().numpy(), i)
        assert np.array_equal(cnt.cpu().numpy(), c)


def _pair(B, kind):
    k = np.zeros((2, B), np.uint8)
    if kind == "split":          # attention on some samples, FFN on others, overlap
        k[0, [b for b in (0, 2, 3) if b < B]] = 1
        k[1, [b for b in (1, 2, B - 1)]] = 1
    elif kind == "attn_only":
        k[0, :] = 1
    elif kind == "ffn_only":
        k[1, [b for b in range(B) if b % 2 == 0]] = 1
    elif kind == "none":
        pass
    return k


@pytest.mark.parametrize("sh", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("forced", [None, "split", "attn_only", "ffn_only", "none"])
def test_sublayer_layer_fwd_bwd(sh, forced):
    cfg = _cfg(sh, granularity=ld.LD_GRAN_SUBLAYER_SEQ)
    layer, p, seed, step = 2, np.float32(0.45), 8, 31
    wd, w64 = layer_weights_dev(sh, layer, gain_jitter=True)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    keep = None if forced is None else _pair(sh.batch, forced)
    xd, gd = x.to(DEV), gy.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    kov = None if keep is None else torch.from_numpy(keep).to(DEV)
    ld.ld_layer_fwd(cfg, wd, layer, float(p), seed, step, xd, ctx, ws, keep_override=kov)
    dw = _garbage_grads(sh)
    ld.ld_layer_bwd(cfg, wd, ctx, gd, dw, ws)
    torch.cuda.synchronize()
    if keep is None:
        keep = masks.keep_bits_granular(p, seed, step, layer, sh.batch, masks.SUBLAYER_SEQ)
    assert np.array_equal(ctx[:2 * sh.batch].cpu().numpy().reshape(2, -1), keep)
    oc = _ocfg(sh, granularity=masks.SUBLAYER_SEQ)
    X1, octx = stack.layer_forward(inp.f64(x), w64, keep, p, oc)
    G0, grads = stack.layer_backward(octx, inp.f64(gy), oc)
    t = tol(sh.dtype)
    xo, go = f64(xd), f64(gd)
    for b in range(sh.batch):
        if keep[:, b].any():
            assert rel(xo[b], X1[b]) < t, b
            assert rel(go[b], G0[b]) < t, b
        else:
            assert np.array_equal(xo[b], inp.f64(x)[b]) and np.array_equal(go[b], inp.f64(gy)[b])
    _check_grads(dw, grads, t, forced)


def _stack_case(sh, gran, ps, seed, step, keep_override=None):
    cfg = _cfg(sh, granularity=gran)
    L, B, nm = sh.n_layers, sh.batch, masks.n_masks(gran)
    W = [layer_weights_dev(sh, l, gain_jitter=True) for l in range(L)]
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dws = [_garbage_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    keep = torch.zeros(L, nm, B, dtype=torch.uint8, device=DEV)
    idx = torch.zeros(L, nm, B, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(L, nm, dtype=torch.int32, device=DEV)
    kov = None if keep_override is None else torch.from_numpy(keep_override).to(DEV)
    ld.ld_stack_step(cfg, [w[0] for w in W], list(ps), seed, step, xd, gd, dws, ws,
                     keep_override=kov, keep_out=keep, idx_out=idx, count_out=cnt)
    torch.cuda.synchronize()
    return dict(x=x, gy=gy, W=W, xd=xd, gd=gd, dws=dws, keep=keep.cpu().numpy(),
                idx=idx.cpu().numpy(), cnt=cnt.cpu().numpy())


@pytest.mark.parametrize("sh", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("gran", GRANS[1:], ids=GRAN_IDS[1:])
@pytest.mark.parametrize("p_max", [0.2, 0.6])
def test_stack_step(sh, gran, p_max):
    ps = schedule.rates(schedule.UNIFORM, schedule.CONSTANT, p_max, sh.n_layers, 0, 1)
    seed, step = 3, 12
    g = _stack_case(sh, gran, ps, seed, step)
    ref = stack.stack_step(inp.f64(g["x"]), [w[1] for w in g["W"]], ps, seed, step,
                           inp.f64(g["gy"]), _ocfg(sh, granularity=gran))
    nm = masks.n_masks(gran)
    L, B = sh.n_layers, sh.batch
    assert np.array_equal(g["keep"], np.asarray(ref["keep"]).reshape(L, nm, B))
    assert np.array_equal(g["idx"], np.asarray(ref["idx"]).reshape(L, nm, B))
    assert np.array_equal(g["cnt"], np.asarray(ref["count"]).reshape(L, nm))
    t = tol(sh.dtype)
    assert rel(f64(g["xd"]), ref["X_L"]) < t
    assert rel(f64(g["gd"]), ref["G_0"]) < t
    for l in range(L):
        _check_grads(g["dws"][l], ref["grads"][l], t, l)
    untouched = ~g["keep"].reshape(L * nm, B).any(axis=0)
    for b in np.nonzero(untouched)[0]:
        assert torch.equal(g["xd"][b].cpu(), g["x"][b]) and torch.equal(g["gd"][b].cpu(), g["gy"][b])


def _per_batch_seed(sh, gran, p):
    """A (seed, step) whose per-batch draws keep some sub-blocks and drop others."""
    ps = np.full(sh.n_layers, p, np.float32)
    for seed in range(100):
        k, _, _ = masks.masks_granular(ps, seed, 4, sh.batch, gran)
        rows = k[:, :, 0].ravel()
        if rows.any() and not rows.all():
            return ps, seed, 4
    raise AssertionError("no mixed seed")


@pytest.mark.parametrize("sh", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("gran", [ld.LD_GRAN_LAYER_BATCH, ld.LD_GRAN_SUBLAYER_BATCH],
                         ids=["layer_batch", "sublayer_batch"])
def test_per_batch_host_skip_equals_device_path(sh, gran):
    """Without an override the host takes the per-batch draws and launches
    nothing for a dropped sub-block; with the same masks as an override every
    launch is made and the device decides.  Both must agree bit for bit, and
    with the oracle."""
    ps, seed, step = _per_batch_seed(sh, gran, 0.5)
    a = _stack_case(sh, gran, ps, seed, step)
    b = _stack_case(sh, gran, ps, seed, step, keep_override=a["keep"])
    assert np.array_equal(a["keep"], b["keep"]) and np.array_equal(a["cnt"], b["cnt"])
    assert torch.equal(a["xd"], b["xd"]) and torch.equal(a["gd"], b["gd"])
    for l in range(sh.n_layers):
        for k in ld.WEIGHT_KEYS:
            assert torch.equal(a["dws"][l][k], b["dws"][l][k]), (l, k)
    ref = stack.stack_step(inp.f64(a["x"]), [w[1] for w in a["W"]], ps, seed, step,
                           inp.f64(a["gy"]), _ocfg(sh, granularity=gran))
    t = tol(sh.dtype)
    assert rel(f64(a["xd"]), ref["X_L"]) < t and rel(f64(a["gd"]), ref["G_0"]) < t
    for l in range(sh.n_layers):
        _check_grads(a["dws"][l], ref["grads"][l], t, l)


def test_per_batch_layer_fwd_skips_and_bwd_zero_grads():
    """ld_layer_fwd under per-batch granularity with a dropping draw leaves x
    untouched; ld_layer_bwd on that ctx leaves dx untouched and writes zero
    gradients."""
    sh = SMALL_BF16
    cfg = _cfg(sh, granularity=ld.LD_GRAN_LAYER_BATCH)
    p = np.float32(0.5)
    layer, step = 1, 4
    seed = next(s for s in range(100)
                if not masks.keep_bits_granular(p, s, step, layer, sh.batch, masks.LAYER_BATCH).any())
    wd, _ = layer_weights_dev(sh, layer)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    ld.ld_layer_fwd(cfg, wd, layer, float(p), seed, step, xd, ctx, ws)
    dw = _garbage_grads(sh)
    ld.ld_layer_bwd(cfg, wd, ctx, gd, dw, ws)
    torch.cuda.synchronize()
    assert torch.equal(xd.cpu(), x) and torch.equal(gd.cpu(), gy)
    assert not ctx[:sh.batch].cpu().numpy().any()
    for k in ld.WEIGHT_KEYS:
        assert not dw[k].any(), k


@pytest.mark.parametrize("gran", GRANS, ids=GRAN_IDS)
@pytest.mark.parametrize("p", [0.0, 0.7, 0.95])
def test_host_counts_plan_only(gran, p):
    """The host takes the mask draws again to know each layer's kept counts
    (they plan split counts and skip sub-blocks no sample keeps).  Under
    profiling the device counts are read back and must agree (the step fails
    otherwise), the counts are the oracle's, and the results are bitwise
    those of the unprofiled step."""
    sh = SMALL_BF16
    ps = [p] * sh.n_layers
    a = _stack_case(sh, gran, ps, 11, 40)
    ld.ld_prof_start("ld_mask_compact")
    try:
        b = _stack_case(sh, gran, ps, 11, 40)
    finally:
        ld.ld_prof_stop()
    _, _, c = masks.masks_granular(ps, 11, 40, sh.batch, gran)
    assert np.array_equal(a["cnt"], c) and np.array_equal(b["cnt"], c)
    assert torch.equal(a["xd"], b["xd"]) and torch.equal(a["gd"], b["gd"])
    for da, db in zip(a["dws"], b["dws"]):
        for k in da:
            assert torch.equal(da[k], db[k]), k
