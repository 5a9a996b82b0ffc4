"""Layer and stack parity of the HIP path against the oracle (needs a GPU):
ld_layer_fwd / ld_layer_bwd / ld_stack_step through the C ABI, masks and
kept lists bit-exact, dropped rows bitwise untouched, activations and
gradients within the dtype's tolerance of the float64 oracle."""
import dataclasses

import numpy as np
import pytest
import torch

import ld_inputs as inp
import paper_2609_05275_amd as ld
from oracle import masks, schedule, stack
from tests.gpu_util import DEV, f64, layer_weights_dev, rel, tol, zero_grads

pytestmark = pytest.mark.gpu

SMALL_BF16 = inp.Shape(3, 256, 4, 704, 192, 5, "bf16")      # d_head 64, ragged q tile
SMALL_BF16_128 = inp.Shape(2, 256, 2, 512, 128, 3, "bf16")  # d_head 128
# large enough that every projection GEMM takes the 256x256 kernel path
MID_BF16 = inp.Shape(2, 1024, 8, 2816, 512, 4, "bf16")
# the block of the paper's experiments (ALiBi + squared ReLU, W_up only);
# 6 heads: not a power of two, so both ALiBi slope rules are exercised
TINY_P = dataclasses.replace(inp.SHAPES["tiny"], kind=1)
SMALL_P = inp.Shape(3, 256, 4, 1024, 192, 5, "bf16", 1)
SMALL_P_128 = inp.Shape(2, 768, 6, 2048, 256, 2, "bf16", 1)
MID_P = inp.Shape(2, 1024, 8, 4096, 512, 4, "bf16", 1)


def _cfg(sh, **kw):
    return ld.config(sh.batch, sh.seq, sh.d_model, sh.n_heads, sh.d_ff,
                     ld.LD_BF16 if sh.dtype == "bf16" else ld.LD_F32, block_kind=sh.kind, **kw)


def _ocfg(sh, **kw):
    return stack.Config(n_heads=sh.n_heads, block_kind=sh.kind, **kw)


def _buf(nbytes):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=DEV)


def _check_grads(got, want, t, where=""):
    for k in ld.WEIGHT_KEYS:
        g, w = f64(got[k]), want[k]
        if not np.any(w):
            assert not np.any(g), (where, k)
        else:
            assert rel(g, w) < t, (where, k, rel(g, w))


@pytest.mark.parametrize("sh", [inp.SHAPES["tiny"], SMALL_BF16, SMALL_BF16_128, MID_BF16,
                                TINY_P, SMALL_P, SMALL_P_128, MID_P],
                         ids=["tiny_f32", "small_bf16", "small_bf16_dh128", "mid_bf16",
                              "paper_tiny_f32", "paper_small_bf16", "paper_small_bf16_dh128_h6",
                              "paper_mid_bf16"])
@pytest.mark.parametrize("forced", [None, "none", "one", "ragged", "all"])
def test_layer_fwd_bwd(sh, forced):
    cfg = _cfg(sh)
    layer, p, seed, step = 1, np.float32(0.4), 3, 17
    wd, w64 = layer_weights_dev(sh, layer, gain_jitter=True)
    x = inp.hidden(sh)
    gy = inp.upstream_grad(sh)
    keep = None
    if forced is not None:
        k = np.zeros(sh.batch, np.uint8)
        k[{"none": [], "one": [sh.batch - 1], "ragged": [b for b in (0, 2, 3) if b < sh.batch - 1],
           "all": list(range(sh.batch))}[forced]] = 1
        keep = k
    xd, gd = x.to(DEV), gy.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    kov = None if keep is None else torch.from_numpy(keep).to(DEV)
    ld.ld_layer_fwd(cfg, wd, layer, float(p), seed, step, xd, ctx, ws, keep_override=kov)
    dw = zero_grads(sh)
    for v in dw.values():
        v.fill_(7.0)            # must be overwritten
    ld.ld_layer_bwd(cfg, wd, ctx, gd, dw, ws)
    torch.cuda.synchronize()
    if keep is None:
        keep = masks.keep_bits(p, seed, step, layer, sh.batch)
    oc = _ocfg(sh)
    X1, octx = stack.layer_forward(inp.f64(x), w64, keep, p, oc)
    G0, grads = stack.layer_backward(octx, inp.f64(gy), oc)
    t = tol(sh.dtype)
    xo, go = f64(xd), f64(gd)
    for b in range(sh.batch):
        if keep[b]:
            assert rel(xo[b], X1[b]) < t, b
            assert rel(go[b], G0[b]) < t, b
        else:   # dropped: bitwise untouched
            assert np.array_equal(xo[b], inp.f64(x)[b]) and np.array_equal(go[b], inp.f64(gy)[b])
    _check_grads(dw, grads, t, forced)


@pytest.mark.parametrize("sh", [inp.SHAPES["tiny"], SMALL_BF16, TINY_P, SMALL_P],
                         ids=["tiny_f32", "small_bf16", "paper_tiny_f32", "paper_small_bf16"])
@pytest.mark.parametrize("p_max", [0.0, 0.2, 0.6, 1.0])
def test_stack_step(sh, p_max):
    cfg = _cfg(sh)
    L = sh.n_layers
    ps = schedule.rates(schedule.ILD if p_max < 1 else schedule.UNIFORM, schedule.CONSTANT,
                        p_max, L, 0, 1)
    seed, step = 0, 5
    W = [layer_weights_dev(sh, l, gain_jitter=True) for l in range(L)]
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dws = [zero_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    keep = torch.zeros(L, sh.batch, dtype=torch.uint8, device=DEV)
    idx = torch.zeros(L, sh.batch, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, [w[0] for w in W], list(ps), seed, step, xd, gd, dws, ws,
                     keep_out=keep, idx_out=idx, count_out=cnt)
    torch.cuda.synchronize()
    ref = stack.stack_step(inp.f64(x), [w[1] for w in W], ps, seed, step, inp.f64(gy), _ocfg(sh))
    assert np.array_equal(keep.cpu().numpy(), ref["keep"])
    assert np.array_equal(idx.cpu().numpy(), ref["idx"])
    assert np.array_equal(cnt.cpu().numpy(), ref["count"])
    t = tol(sh.dtype)
    if p_max == 1.0:
        assert torch.equal(xd.cpu(), x) and torch.equal(gd.cpu(), gy)
    assert rel(f64(xd), ref["X_L"]) < t
    assert rel(f64(gd), ref["G_0"]) < t
    for l in range(L):
        _check_grads(dws[l], ref["grads"][l], t, l)


def test_stack_mask_edges_forced():
    """Kept counts 0, 1, ragged and all through the stack (keep override)."""
    sh = inp.Shape(4, 256, 4, 704, 128, 6, "bf16")
    cfg = _cfg(sh)
    L, B = sh.n_layers, sh.batch
    k = np.zeros((L, B), np.uint8)
    k[1, 4] = 1
    k[2, [0, 3, 5]] = 1
    k[3, :] = 1
    ps = [0.0, 0.95, 0.5, 0.05]
    W = [layer_weights_dev(sh, l) for l in range(L)]
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dws = [zero_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    cnt = torch.zeros(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, [w[0] for w in W], ps, 0, 0, xd, gd, dws, ws,
                     keep_override=torch.from_numpy(k).to(DEV), count_out=cnt)
    torch.cuda.synchronize()
    ref = stack.stack_step(inp.f64(x), [w[1] for w in W], np.float32(ps), 0, 0, inp.f64(gy),
                           _ocfg(sh), keep=k)
    assert list(cnt.cpu().numpy()) == [0, 1, 3, 6]
    assert rel(f64(xd), ref["X_L"]) < 2e-2
    assert rel(f64(gd), ref["G_0"]) < 2e-2
    for l in range(L):
        _check_grads(dws[l], ref["grads"][l], 2e-2, l)
    # sample 1 and 2 are kept only by layer 3; their rows before it are copies
    assert np.array_equal(k[:3, 1], [0, 0, 0])


def test_stack_deterministic():
    sh = SMALL_BF16
    cfg = _cfg(sh)
    L = sh.n_layers
    ps = [0.0, 0.3, 0.6]
    W = [layer_weights_dev(sh, l)[0] for l in range(L)]
    outs = []
    for _ in range(2):
        xd, gd = inp.hidden(sh).to(DEV), inp.upstream_grad(sh).to(DEV)
        dws = [zero_grads(sh) for _ in range(L)]
        ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
        ld.ld_stack_step(cfg, W, ps, 1, 2, xd, gd, dws, ws)
        torch.cuda.synchronize()
        outs.append((xd.cpu(), gd.cpu(), [{k: v.cpu() for k, v in d.items()} for d in dws]))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    for a, b in zip(outs[0][2], outs[1][2]):
        for k in a:
            assert torch.equal(a[k], b[k]), k


def test_layer_masks_match_stack_masks():
    """ld_layer_fwd with the global layer index draws the stack's masks."""
    sh = SMALL_BF16
    cfg = _cfg(sh)
    ps = np.float32([0.1, 0.5, 0.7])
    keep = torch.zeros(3, sh.batch, dtype=torch.uint8, device=DEV)
    idx = torch.zeros(3, sh.batch, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(3, dtype=torch.int32, device=DEV)
    ld.ld_masks(list(ps), 4, 9, keep, idx, cnt)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    for l in range(3):
        xd = inp.hidden(sh).to(DEV)
        ld.ld_layer_fwd(cfg, layer_weights_dev(sh, l)[0], l, float(ps[l]), 4, 9, xd, ctx)
        torch.cuda.synchronize()
        assert torch.equal(ctx[:sh.batch], keep[l])


RESCALE_CASES = [(False, 1.0), (False, 1.7), (True, 0.5), (True, 1.7)]


@pytest.mark.parametrize("sh", [inp.SHAPES["tiny"], SMALL_BF16], ids=["tiny_f32", "small_bf16"])
@pytest.mark.parametrize("rescale,res_scale", RESCALE_CASES,
                         ids=[f"rescale{int(a)}-c{b}" for a, b in RESCALE_CASES])
def test_residual_scale_options_layer(sh, rescale, res_scale):
    """r = res_scale / (1 - p) with rescaling, res_scale without (Dropout
    Scale; the parameterisation table's branch multiplier): one layer
    forward and backward against the oracle."""
    cfg = _cfg(sh, rescale=rescale, res_scale=res_scale)
    layer, p, seed, step = 1, np.float32(0.4), 3, 17
    wd, w64 = layer_weights_dev(sh, layer, gain_jitter=True)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    keep = masks.keep_bits(p, seed, step, layer, sh.batch)
    assert 0 < keep.sum() < sh.batch
    xd, gd = x.to(DEV), gy.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    ld.ld_layer_fwd(cfg, wd, layer, float(p), seed, step, xd, ctx, ws)
    dw = zero_grads(sh)
    ld.ld_layer_bwd(cfg, wd, ctx, gd, dw, ws)
    torch.cuda.synchronize()
    oc = _ocfg(sh, rescale=rescale, res_scale=res_scale)
    X1, octx = stack.layer_forward(inp.f64(x), w64, keep, p, oc)
    G0, grads = stack.layer_backward(octx, inp.f64(gy), oc)
    t = tol(sh.dtype)
    xo, go = f64(xd), f64(gd)
    for b in range(sh.batch):
        if keep[b]:
            assert rel(xo[b], X1[b]) < t, b
            assert rel(go[b], G0[b]) < t, b
        else:
            assert np.array_equal(xo[b], inp.f64(x)[b]) and np.array_equal(go[b], inp.f64(gy)[b])
    _check_grads(dw, grads, t, (rescale, res_scale))


@pytest.mark.parametrize("sh", [inp.SHAPES["tiny"], SMALL_BF16], ids=["tiny_f32", "small_bf16"])
@pytest.mark.parametrize("rescale,res_scale", RESCALE_CASES,
                         ids=[f"rescale{int(a)}-c{b}" for a, b in RESCALE_CASES])
def test_residual_scale_options_stack(sh, rescale, res_scale):
    cfg = _cfg(sh, rescale=rescale, res_scale=res_scale)
    L = sh.n_layers
    ps = schedule.rates(schedule.ILD, schedule.CONSTANT, 0.6, L, 0, 1)
    seed, step = 2, 9
    W = [layer_weights_dev(sh, l, gain_jitter=True) for l in range(L)]
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dws = [zero_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    cnt = torch.zeros(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, [w[0] for w in W], list(ps), seed, step, xd, gd, dws, ws, count_out=cnt)
    torch.cuda.synchronize()
    ref = stack.stack_step(inp.f64(x), [w[1] for w in W], ps, seed, step, inp.f64(gy),
                           _ocfg(sh, rescale=rescale, res_scale=res_scale))
    assert np.array_equal(cnt.cpu().numpy(), ref["count"])
    t = tol(sh.dtype)
    assert rel(f64(xd), ref["X_L"]) < t
    assert rel(f64(gd), ref["G_0"]) < t
    for l in range(L):
        _check_grads(dws[l], ref["grads"][l], t, l)
