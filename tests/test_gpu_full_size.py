"""Parity at the full workload sizes (needs a GPU).

The oracle cannot run whole steps of these shapes in seconds, so each test
checks outputs it can compute one sequence at a time, or properties that
hold at any size, through the same entry points and kernel plans the
benchmark drives.  Two facts of the method make one-sequence checks exact:

  * sequences are independent (per-sequence masks; attention within a
    sequence), so the oracle run on one sequence alone, with that sequence's
    column of the global-index masks, gives its rows of X_L and dL/dX^0;
  * weight gradients are sums over kept sequences, so a launch whose keep
    override keeps only one sequence's mask column gives that sequence's
    weight gradients, and the whole launch's gradients equal the sum of such
    launches up to float32 reordering.

Workloads:
- 1B shape, all 16 layers at the benchmark's rates (ILD p_max 0.2 at the end
  of the 0..1000 ramp, step 1000): masks, kept lists and counts bit-exact;
  X_L and dL/dX^0 of a sequence kept by every layer and of one dropped by
  some layers against the oracle; those sequences' weight gradients of every
  layer against the oracle; additivity over all kept sequences.
- 1B layer and a layer of the paper's 3.9B architecture with its block.
- 125M-shape full stack step: every output against the oracle.
- 7B shape, layers 0 and 31 forward and backward: the first kept sequence's
  output, dL/dX and six weight gradients against the oracle; additivity.
- Stress configuration (1B width, batch 32), all 16 layers: uniform p in
  {0, 0.05, 0.5, 0.95, 1}, the same p on the last 4 layers only, and mixed
  p_l = set[l mod 5], Philox seeds 0, 1, 2; plus forced kept counts 0, 1,
  32 and ragged.  Masks, kept lists and counts bit-exact; sequences dropped
  everywhere bitwise untouched; zero weight gradients for empty layers; two
  sampled sequences against the oracle.  For those the upstream gradient is
  zero past row R: causal attention then makes every output row < R and
  every gradient depend on rows < R only (dL/dX^0 rows >= R are exactly 0,
  checked), so the oracle on the first R rows is exact while the GPU runs
  the full 2048-row shape.  One case also runs the full upstream gradient
  against the oracle on a whole sequence.
"""
import time

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

_WCACHE = {}


def _weights(sh, layer):
    """(device, float64) weights of one layer; the 1B and stress shapes share
    them (same widths), so they are drawn once."""
    key = (sh.d_model, sh.n_heads, sh.d_ff, sh.kind, layer)
    if key not in _WCACHE:
        _WCACHE[key] = layer_weights_dev(sh, layer)
    return _WCACHE[key]


def _say(msg):
    print(f"[full-size] {msg}", flush=True)


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


def _check_grads(got, want, t, where):
    for k in ld.WEIGHT_KEYS:
        g = f64(got[k])
        if not np.any(want[k]):
            assert not np.any(g), (where, k)
        else:
            assert rel(g, want[k]) < t, (where, k, rel(g, want[k]))


def _only(keep, b):
    """Keep override with only sequence b's mask column."""
    k = np.zeros_like(keep)
    k[..., b] = keep[..., b]
    return k


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


def _layer_parity(sh, layer, p, step, keep):
    """One layer forward + backward at full size: dropped sequences bitwise
    untouched, the first kept sequence against the oracle (output, dL/dX,
    weight gradients from a launch keeping only it), additivity of the
    single-sequence weight gradients."""
    cfg = _cfg(sh)
    wd, w64 = _weights(sh, layer)
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    x1, g0, dw = _layer_run(cfg, sh, wd, layer, p, step, x, gy)
    kept = [b for b in range(sh.batch) if keep[b]]
    for b in range(sh.batch):
        if not keep[b]:
            assert torch.equal(x1[b].cpu(), x[b]), b
            assert torch.equal(g0[b].cpu(), gy[b]), b
    b0 = kept[0]
    oc = stack.Config(n_heads=sh.n_heads, block_kind=sh.kind)
    t0 = time.time()
    X1, octx = stack.layer_forward(inp.f64(x[b0:b0 + 1]), w64, np.ones(1, np.uint8), p, oc)
    G0, grads = stack.layer_backward(octx, inp.f64(gy[b0:b0 + 1]), oc)
    del octx
    _say(f"layer {layer} oracle {time.time() - t0:.1f} s")
    assert rel(f64(x1[b0]), X1[0]) < TOL_BF16
    assert rel(f64(g0[b0]), G0[0]) < TOL_BF16
    total = {k: torch.zeros(v.shape, dtype=torch.float64, device=DEV) for k, v in dw.items()}
    for b in kept:
        _, _, single = _layer_run(cfg, sh, wd, layer, p, step, x, gy, keep=_only(np.asarray(keep, np.uint8), b))
        if b == b0:
            _check_grads(single, grads, TOL_BF16, (layer, b0))
        for k in ld.WEIGHT_KEYS:
            total[k] += single[k].double()
    for k in ld.WEIGHT_KEYS:
        assert rel(f64(dw[k]), f64(total[k])) < TOL_REORDER, k


@pytest.mark.parametrize("name", ["1b", "paper_3p9b"])
def test_layer_sampled_and_additive(name):
    sh = inp.SHAPES[name]
    layer = sh.n_layers - 1
    p = _ild(0.2, layer, sh.n_layers)
    step, keep = _step_with(p, layer, sh.batch, lambda k: 2 <= k.sum() < sh.batch)
    _layer_parity(sh, layer, p, step, keep)
    if name != "1b":
        for key in [k for k in _WCACHE if k[3] == 1]:
            del _WCACHE[key]


def _stack_run(cfg, W, ps, seed, step, x, gy, ws, L, B, keep_override=None, nm=1):
    xd, gd = x.to(DEV), gy.to(DEV)
    dW = [{k: torch.full(v.shape, 7.0, dtype=torch.float32, device=DEV) for k, v in W[0].items()}
          for _ in range(L)]   # must be overwritten
    keep_d = torch.empty(L, B, dtype=torch.uint8, device=DEV)
    idx_d = torch.empty(L, B, dtype=torch.int32, device=DEV)
    cnt_d = torch.empty(L, dtype=torch.int32, device=DEV)
    kov = None if keep_override is None else torch.from_numpy(np.ascontiguousarray(keep_override)).to(DEV)
    ld.ld_stack_step(cfg, W, ps, seed, step, xd, gd, dW, ws, keep_override=kov, keep_out=keep_d,
                     idx_out=idx_d, count_out=cnt_d)
    torch.cuda.synchronize()
    return xd, gd, dW, keep_d.cpu().numpy(), idx_d.cpu().numpy(), cnt_d.cpu().numpy()


def test_1b_full_depth_stack():
    """All 16 layers of the 1B shape at the benchmark's rates and step."""
    sh = inp.SHAPES["1b"]
    L, B = sh.n_layers, sh.batch
    cfg = _cfg(sh)
    ps = [_ild(0.2, l, L) for l in range(L)]
    step = 1000
    kp, idx, cnt = masks.masks(ps, 0, step, B)
    per = kp.sum(axis=0)
    b_all = int(np.argmax(per == L))
    assert per[b_all] == L, "a sequence kept by every layer"
    b_drop = int(np.argmin(np.where(per > 0, per, L + 1)))
    assert 0 < per[b_drop] < L
    t0 = time.time()
    W = [_weights(sh, l) for l in range(L)]
    _say(f"1B weights {time.time() - t0:.1f} s")
    x, gy = inp.hidden(sh), inp.upstream_grad(sh)
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    Wd = [w[0] for w in W]
    xd, gd, dW, keep_g, idx_g, cnt_g = _stack_run(cfg, Wd, ps, 0, step, x, gy, ws, L, B)
    assert np.array_equal(keep_g, kp)
    assert np.array_equal(idx_g, idx)
    assert np.array_equal(cnt_g, cnt)
    for b in range(B):
        if not kp[:, b].any():
            assert torch.equal(xd[b].cpu(), x[b]) and torch.equal(gd[b].cpu(), gy[b]), b
    oc = stack.Config(n_heads=sh.n_heads)
    W64 = [w[1] for w in W]
    total = [{k: torch.zeros(v.shape, dtype=torch.float64, device=DEV) for k, v in d.items()} for d in dW]
    for b in range(B):
        if not kp[:, b].any():
            continue
        _, _, single, *_ = _stack_run(cfg, Wd, ps, 0, step, x, gy, ws, L, B, keep_override=_only(kp, b))
        for l in range(L):
            for k in ld.WEIGHT_KEYS:
                total[l][k] += single[l][k].double()
        if b in (b_all, b_drop):
            t0 = time.time()
            res = stack.stack_step(inp.f64(x[b:b + 1]), W64, ps, 0, step, inp.f64(gy[b:b + 1]), oc,
                                   keep=kp[:, b:b + 1])
            _say(f"1B oracle, sequence {b} kept by {per[b]} layers: {time.time() - t0:.1f} s")
            assert rel(f64(xd[b]), res["X_L"][0]) < TOL_BF16, b
            assert rel(f64(gd[b]), res["G_0"][0]) < TOL_BF16, b
            for l in range(L):
                _check_grads(single[l], res["grads"][l], TOL_BF16, (b, l))
            del res
        del single
    for l in range(L):
        for k in ld.WEIGHT_KEYS:
            assert rel(f64(dW[l][k]), f64(total[l][k])) < TOL_REORDER, (l, k)


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
        _check_grads(dW[l], res["grads"][l], TOL_BF16, l)


@pytest.mark.parametrize("layer", [0, 31])
def test_7b_layer_fwd_bwd(layer):
    """7B shape (batch 4, S 4096, d 4096, d_ff 11008): the first and last
    layers forward and backward at the benchmark's rates."""
    sh = inp.SHAPES["7b"]
    p = _ild(0.2, layer, sh.n_layers)
    if layer == 0:
        step, keep = 1000, masks.keep_bits(p, 0, 1000, layer, sh.batch)   # p = 0: all kept
        assert keep.all()
    else:
        step, keep = _step_with(p, layer, sh.batch, lambda k: 1 <= k.sum() < sh.batch)
    t0 = time.time()
    _layer_parity(sh, layer, p, step, keep)
    _say(f"7B layer {layer}: {time.time() - t0:.1f} s")
    for key in [k for k in _WCACHE if k[0] == sh.d_model]:
        del _WCACHE[key]


# ------------------------------------------------------------------ stress

STRESS_P = [0.0, 0.05, 0.5, 0.95, 1.0]
STRESS_CASES = ([("uniform", v) for v in STRESS_P] + [("last4", v) for v in STRESS_P] + [("mixed", None)])
PREFIX = 256     # rows of the truncated upstream gradient
_ORACLE_CACHE = {}


def _stress_rates(kind, val, L):
    if kind == "uniform":
        return [np.float32(val)] * L
    if kind == "last4":   # the last L/4 layers only
        return [np.float32(0.0)] * (L - L // 4) + [np.float32(val)] * (L // 4)
    return [np.float32(STRESS_P[l % len(STRESS_P)]) for l in range(L)]


@pytest.fixture(scope="module")
def stress_setup():
    sh = inp.SHAPES["1b_b32"]
    L = sh.n_layers
    cfg = _cfg(sh)
    t0 = time.time()
    W = [_weights(sh, l) for l in range(L)]
    _say(f"stress weights {time.time() - t0:.1f} s")
    x = inp.hidden(sh)
    gy_full = inp.upstream_grad(sh)
    gy = gy_full.clone()
    gy[:, PREFIX:] = 0
    ws = _buf(ld.ld_stack_ws_bytes(cfg, L))
    return dict(sh=sh, cfg=cfg, W=W, x=x, gy=gy, gy_full=gy_full, ws=ws)


def _stress_oracle(st, b, keep_col, ps, rows, gy):
    """Oracle for sequence b alone over its first `rows` rows.  Returns
    (X_L, G_0, grads or None): results are cached on (b, its mask column, the
    rates of the layers that keep it, rows) without the weight gradients, as
    a repeat of the same single-sequence launch is bitwise the same launch
    and its gradients were compared the first time."""
    L = len(ps)
    key = (b, tuple(int(v) for v in keep_col), tuple(float(ps[l]) for l in range(L) if keep_col[l]), rows)
    if key in _ORACLE_CACHE:
        return _ORACLE_CACHE[key] + (None,)
    oc = stack.Config(n_heads=st["sh"].n_heads)
    t0 = time.time()
    res = stack.stack_step(inp.f64(st["x"][b:b + 1, :rows]), [w[1] for w in st["W"]], ps, 0, 0,
                           inp.f64(gy[b:b + 1, :rows]), oc, keep=np.asarray(keep_col, np.uint8).reshape(L, 1))
    _say(f"stress oracle, sequence {b}, {int(np.sum(keep_col))} kept layers, {rows} rows: "
         f"{time.time() - t0:.1f} s")
    _ORACLE_CACHE[key] = (res["X_L"][0], res["G_0"][0])
    return res["X_L"][0], res["G_0"][0], res["grads"]


def _stress_check(st, ps, seed, kp, forced):
    """One stack step of the stress shape with the truncated upstream
    gradient; kp is the expected mask (Philox or forced)."""
    sh, cfg, ws = st["sh"], st["cfg"], st["ws"]
    L, B = sh.n_layers, sh.batch
    Wd = [w[0] for w in st["W"]]
    x, gy = st["x"], st["gy"]
    step = 1000
    xd, gd, dW, keep_g, idx_g, cnt_g = _stack_run(cfg, Wd, ps, seed, step, x, gy, ws, L, B,
                                                  keep_override=kp if forced else None)
    assert np.array_equal(keep_g, kp)
    want_idx = np.full((L, B), -1, np.int32)
    for l in range(L):
        kept = np.nonzero(kp[l])[0]
        want_idx[l, :len(kept)] = kept
    assert np.array_equal(idx_g, want_idx)
    assert np.array_equal(cnt_g, kp.sum(axis=1).astype(np.int32))
    x_d, gy_d = x.to(DEV), gy.to(DEV)
    per = kp.sum(axis=0)
    for b in range(B):
        if per[b] == 0:   # dropped everywhere: bitwise untouched
            assert torch.equal(xd[b], x_d[b]) and torch.equal(gd[b], gy_d[b]), b
        else:             # rows past the truncation carry no gradient
            assert not torch.any(gd[b, PREFIX:]), b
    for l in range(L):
        if kp[l].sum() == 0:
            for k in ld.WEIGHT_KEYS:
                assert not torch.any(dW[l][k]), (l, k)
    del x_d, gy_d
    some = [b for b in range(B) if per[b] > 0]
    if not some:
        return
    if all(np.array_equal(kp[:, b], kp[:, some[0]]) for b in some):
        sel = [0, B - 1] if (0 in some and B - 1 in some) else some[:2]
    else:   # the sequences kept by the fewest layers (cheapest oracle runs)
        order = sorted(some, key=lambda b: (per[b], -b))
        sel = order[:2]
    for b in sel:
        XL, G0, grads = _stress_oracle(st, b, kp[:, b], ps, PREFIX, gy)
        assert rel(f64(xd[b, :PREFIX]), XL) < TOL_BF16, b
        assert rel(f64(gd[b, :PREFIX]), G0) < TOL_BF16, b
        if grads is None:
            continue
        _, _, single, *_ = _stack_run(cfg, Wd, ps, seed, step, x, gy, ws, L, B, keep_override=_only(kp, b))
        for l in range(L):
            _check_grads(single[l], grads[l], TOL_BF16, (b, l))
        del single, grads


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("case", STRESS_CASES, ids=lambda c: f"{c[0]}-{c[1]}")
def test_stress_b32_full_depth(stress_setup, case, seed):
    st = stress_setup
    L, B = st["sh"].n_layers, st["sh"].batch
    ps = _stress_rates(*case, L)
    kp = masks.masks(ps, seed, 1000, B)[0]
    _stress_check(st, ps, seed, kp, forced=False)


def test_stress_b32_forced_counts(stress_setup):
    """Kept counts forced to 0, 1, 32 and ragged, cycling over the 16 layers."""
    st = stress_setup
    L, B = st["sh"].n_layers, st["sh"].batch
    kp = np.zeros((L, B), np.uint8)
    ragged = [0, 3, 4, 9, 10, 11, 20, 31]
    for l in range(L):
        m = l % 4
        if m == 1:
            kp[l, 17] = 1
        elif m == 2:
            kp[l, :] = 1
        elif m == 3:
            kp[l, ragged] = 1
    ps = [np.float32(0.3)] * L
    _stress_check(st, ps, 0, kp, forced=True)


def test_stress_b32_full_gradient_one_sequence(stress_setup):
    """Mixed rates at seed 0 with the full N(0, 1) upstream gradient: the
    sequence kept by the fewest layers against the oracle over all rows."""
    st = stress_setup
    sh, cfg, ws = st["sh"], st["cfg"], st["ws"]
    L, B = sh.n_layers, sh.batch
    ps = _stress_rates("mixed", None, L)
    kp = masks.masks(ps, 0, 1000, B)[0]
    per = kp.sum(axis=0)
    b = min((b for b in range(B) if per[b] > 0), key=lambda b: (per[b], b))
    Wd = [w[0] for w in st["W"]]
    xd, gd, dW, *_ = _stack_run(cfg, Wd, ps, 0, 1000, st["x"], st["gy_full"], ws, L, B)
    XL, G0, grads = _stress_oracle(st, b, kp[:, b], ps, sh.seq, st["gy_full"])
    assert grads is not None
    assert rel(f64(xd[b]), XL) < TOL_BF16
    assert rel(f64(gd[b]), G0) < TOL_BF16
    _, _, single, *_ = _stack_run(cfg, Wd, ps, 0, 1000, st["x"], st["gy_full"], ws, L, B,
                                  keep_override=_only(kp, b))
    for l in range(L):
        _check_grads(single[l], grads[l], TOL_BF16, (b, l))
