"""Parity at the full workload sizes (needs a GPU).

The oracle cannot run whole steps of these shapes in seconds, so each test
checks outputs it can compute one at a time, or properties that hold at any
size, through the same entry points and kernel plans the benchmark drives:

- 1B layer, and a layer of the paper's 3.9B architecture with its block
  (ALiBi, squared ReLU; batch 8, the real ILD mask): the first kept sequence's output,
  input gradient and weight gradients against the float64 oracle; dropped
  sequences bitwise untouched; the weight gradients of the whole launch equal
  the sum of single-sequence launches (gradients are sums over kept
  sequences), so every kept sequence's contribution is covered.
- 1B, three layers through ld_stack_step: one sampled sequence's X_L and
  dL/dX^0 against the oracle run on that sequence alone with the same
  (global-index) masks; masks and counts bit-exact.
- 125M full stack step: every output against the oracle.
- 7B layer forward: the first 64 rows of every kept sequence; causal
  attention makes a prefix depend on itself only, so the oracle on the
  prefix is exact.
- Batch 32 at the 1B width (stress configuration), two layers, uniform p in
  {0, 0.05, 0.5, 0.95, 1} and forced kept counts 1 / 32 and 0 / ragged.
"""
import numpy as np
import pytest
import torch

import ld_inputs as inp
import paper_2609_05275_amd as ld
from oracle import masks, schedule, stack
from tests.gpu_util import DEV, TOL_BF16, f64, layer_weights_dev, rel, zero_grads

pytestmark = pytest.mark.gpu

# float32 sums of the same products in another order (split-K partials vs
# per-sequence sums)
TOL_REORDER = 1e-4


def _cfg(sh):
    return ld.config(sh.batch, sh.seq, sh.d_model, sh.n_heads, sh.d_ff, ld.LD_BF16,
                     block_kind=sh.kind)


def _buf(nbytes):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=DEV)


def _ild(p_max, layer, n_layers):
    # the benchmark's rates: ILD at the end of the increasing ramp
    return np.float32(schedule.rate(schedule.ILD, schedule.ITS, p_max, layer, n_layers, 1000, 1001))


def _step_with(p, layer, batch, want):
    """First step >= 1000 whose mask for `layer` satisfies want(keep)."""
    for step in range(1000, 1200):
        k = masks.keep_bits(p, 0, step, layer, batch)
        if want(k):
            return step, k
    raise AssertionError("no such step")


def _layer_run(cfg, sh, wd, layer, p, step, x, gy, keep=None):
    xd, gd = x.to(DEV), gy.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    kov = None if keep is None else torch.from_numpy(np.asarray(keep, np.uint8)).to(DEV)
    ld.ld_layer_fwd(cfg, wd, layer, float(p), 0, step, xd, ctx, ws, keep_override=kov)
    x1 = xd.clone()
    dw = zero_grads(sh)
    ld.ld_layer_bwd(cfg, wd, ctx, gd, dw, ws)
    torch.cuda.synchronize()
    del ctx, ws
    return x1, gd, dw


@pytest.mark.parametrize("name", ["1b", "paper_3p9b"])
def test_layer_sampled_and_additive(name):
    sh = inp.SHAPES[name]
    cfg = _cfg(sh)
    layer = sh.n_layers - 1
    p = _ild(0.2, layer, sh.n_layers)
    step, keep = _step_with(p, layer, sh.batch, lambda k: 2 <= k.sum() < sh.batch)
    wd, w64 = layer_weights_dev(sh, layer)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    x1, g0, dw = _layer_run(cfg, sh, wd, layer, p, step, x, gy)
    kept = [b for b in range(sh.batch) if keep[b]]
    for b in range(sh.batch):
        if not keep[b]:
            assert torch.equal(x1[b].cpu(), x[b]), b
            assert torch.equal(g0[b].cpu(), gy[b]), b
    # the first kept sequence against the oracle
    b0 = kept[0]
    oc = stack.Config(n_heads=sh.n_heads, block_kind=sh.kind)
    X1, octx = stack.layer_forward(inp.f64(x[b0:b0 + 1]), w64, np.ones(1, np.uint8), p, oc)
    G0, grads = stack.layer_backward(octx, inp.f64(gy[b0:b0 + 1]), oc)
    assert rel(f64(x1[b0]), X1[0]) < TOL_BF16
    assert rel(f64(g0[b0]), G0[0]) < TOL_BF16
    # that sequence's weight gradients, from a launch that keeps only it
    single = {}
    for b in kept:
        only = np.zeros(sh.batch, np.uint8)
        only[b] = 1
        _, _, single[b] = _layer_run(cfg, sh, wd, layer, p, step, x, gy, keep=only)
    for k in ld.WEIGHT_KEYS:
        assert rel(f64(single[b0][k]), grads[k]) < TOL_BF16, k
    # additivity over the kept sequences
    for k in ld.WEIGHT_KEYS:
        total = sum(f64(single[b][k]) for b in kept)
        assert rel(f64(dw[k]), total) < TOL_REORDER, k


def test_1b_three_layer_stack_sampled_sequence():
    sh = inp.SHAPES["1b"]
    L = 3
    cfg = _cfg(sh)
    ps = [np.float32(v) for v in (0.25, 0.5, 0.25)]
    # a step where the sampled sequence is kept in some layers, dropped in one
    b_s = 5
    for step in range(1000, 1200):
        kp, _, _ = masks.masks(ps, 0, step, sh.batch)
        if 0 < kp[:, b_s].sum() < L and kp.sum(axis=1).min() >= 1:
            break
    else:
        raise AssertionError("no such step")
    W, W64 = [], []
    for l in range(L):
        wd, w64 = layer_weights_dev(sh, l)
        W.append(wd)
        W64.append(w64)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dW = [zero_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    keep_d = torch.empty(L, sh.batch, dtype=torch.uint8, device=DEV)
    idx_d = torch.empty(L, sh.batch, dtype=torch.int32, device=DEV)
    cnt_d = torch.empty(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, W, ps, 0, step, xd, gd, dW, ws, keep_out=keep_d, idx_out=idx_d,
                     count_out=cnt_d)
    torch.cuda.synchronize()
    kp, idx, cnt = masks.masks(ps, 0, step, sh.batch)
    assert np.array_equal(keep_d.cpu().numpy(), kp)
    assert np.array_equal(idx_d.cpu().numpy(), idx)
    assert np.array_equal(cnt_d.cpu().numpy(), cnt)
    oc = stack.Config(n_heads=sh.n_heads)
    res = stack.stack_step(inp.f64(x[b_s:b_s + 1]), W64, ps, 0, step, inp.f64(gy[b_s:b_s + 1]), oc,
                           keep=kp[:, b_s:b_s + 1])
    assert rel(f64(xd[b_s]), res["X_L"][0]) < TOL_BF16
    assert rel(f64(gd[b_s]), res["G_0"][0]) < TOL_BF16
    for b in range(sh.batch):
        if not kp[:, b].any():   # dropped everywhere: bitwise untouched
            assert torch.equal(xd[b].cpu(), x[b]) and torch.equal(gd[b].cpu(), gy[b]), b


def test_125m_full_stack_step():
    sh = inp.SHAPES["125m"]
    L = sh.n_layers
    cfg = _cfg(sh)
    ps = [_ild(0.2, l, L) for l in range(L)]
    step = 1000
    W, W64 = [], []
    for l in range(L):
        wd, w64 = layer_weights_dev(sh, l, gain_jitter=True)
        W.append(wd)
        W64.append(w64)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dW = [zero_grads(sh) for _ in range(L)]
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    cnt_d = torch.empty(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, W, ps, 0, step, xd, gd, dW, ws, count_out=cnt_d)
    torch.cuda.synchronize()
    oc = stack.Config(n_heads=sh.n_heads)
    res = stack.stack_step(inp.f64(x), W64, ps, 0, step, inp.f64(gy), oc)
    assert np.array_equal(cnt_d.cpu().numpy(), res["count"])
    assert rel(f64(xd), res["X_L"]) < TOL_BF16
    assert rel(f64(gd), res["G_0"]) < TOL_BF16
    for l in range(L):
        for k in ld.WEIGHT_KEYS:
            want = res["grads"][l][k]
            got = f64(dW[l][k])
            if not np.any(want):
                assert not np.any(got), (l, k)
            else:
                assert rel(got, want) < TOL_BF16, (l, k)


def test_7b_layer_forward_prefix():
    sh = inp.SHAPES["7b"]
    cfg = _cfg(sh)
    layer = sh.n_layers - 1
    p = _ild(0.2, layer, sh.n_layers)
    step, keep = _step_with(p, layer, sh.batch, lambda k: 1 <= k.sum() < sh.batch)
    wd, w64 = layer_weights_dev(sh, layer)
    x = inp.hidden(sh)
    xd = x.to(DEV)
    ctx = _buf(ld.ld_layer_ctx_bytes(cfg))
    ws = _buf(ld.ld_layer_ws_bytes(cfg))
    ld.ld_layer_fwd(cfg, wd, layer, float(p), 0, step, xd, ctx, ws)
    torch.cuda.synchronize()
    oc = stack.Config(n_heads=sh.n_heads)
    rows = 64
    for b in range(sh.batch):
        if keep[b]:
            X1, _ = stack.layer_forward(inp.f64(x[b:b + 1, :rows]), w64, np.ones(1, np.uint8), p, oc)
            assert rel(f64(xd[b, :rows]), X1[0]) < TOL_BF16, b
        else:
            assert torch.equal(xd[b].cpu(), x[b]), b


def _forced(kind, L, B):
    k = np.zeros((L, B), np.uint8)
    if kind == "one_then_all":
        k[0, 17] = 1
        k[1, :] = 1
    elif kind == "none_then_ragged":
        k[1, [0, 3, 4, 9, 10, 11, 20, 31]] = 1
    return k


@pytest.mark.parametrize("case", [("p", 0.0), ("p", 0.05), ("p", 0.5), ("p", 0.95), ("p", 1.0),
                                  ("forced", "one_then_all"), ("forced", "none_then_ragged")],
                         ids=lambda c: f"{c[0]}-{c[1]}")
def test_stress_b32_two_layers(case):
    """Batch 32 at the 1B width (stress configuration), two layers: masks
    and counts bit-exact, a sampled sequence kept somewhere against the
    oracle, sequences dropped everywhere bitwise untouched, weight gradients
    zero where nothing is kept."""
    sh = inp.SHAPES["1b_b32"]
    L = 2
    cfg = _cfg(sh)
    kind, val = case
    ps = [np.float32(val if kind == "p" else 0.3)] * L
    kov = _forced(val, L, sh.batch) if kind == "forced" else None
    step = 1000
    W, W64 = [], []
    for l in range(L):
        wd, w64 = layer_weights_dev(sh, l)
        W.append(wd)
        W64.append(w64)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    xd, gd = x.to(DEV), gy.to(DEV)
    dW = [zero_grads(sh) for _ in range(L)]
    for g in dW:
        for v in g.values():
            v.fill_(7.0)   # must be overwritten
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    keep_d = torch.empty(L, sh.batch, dtype=torch.uint8, device=DEV)
    cnt_d = torch.empty(L, dtype=torch.int32, device=DEV)
    ld.ld_stack_step(cfg, W, ps, 0, step, xd, gd, dW, ws,
                     keep_override=None if kov is None else torch.from_numpy(kov).to(DEV),
                     keep_out=keep_d, count_out=cnt_d)
    torch.cuda.synchronize()
    kp = kov if kov is not None else masks.masks(ps, 0, step, sh.batch)[0]
    assert np.array_equal(keep_d.cpu().numpy(), kp)
    assert np.array_equal(cnt_d.cpu().numpy(), kp.sum(axis=1).astype(np.int32))
    for l in range(L):
        if kp[l].sum() == 0:
            for k in ld.WEIGHT_KEYS:
                assert not torch.any(dW[l][k]), (l, k)
    for b in range(sh.batch):
        if not kp[:, b].any():
            assert torch.equal(xd[b].cpu(), x[b]) and torch.equal(gd[b].cpu(), gy[b]), b
    somewhere = [b for b in range(sh.batch) if kp[:, b].any()]
    if somewhere:
        b_s = somewhere[len(somewhere) // 2]
        oc = stack.Config(n_heads=sh.n_heads)
        res = stack.stack_step(inp.f64(x[b_s:b_s + 1]), W64, ps, 0, step, inp.f64(gy[b_s:b_s + 1]), oc,
                               keep=kp[:, b_s:b_s + 1])
        assert rel(f64(xd[b_s]), res["X_L"][0]) < TOL_BF16
        assert rel(f64(gd[b_s]), res["G_0"][0]) < TOL_BF16
