"""Kernel-level parity of the HIP path against the oracle (needs a GPU).

Masks, kept lists, gather and scatter-add are bit-exact; the floating-point
kernels are within the tolerance of their dtype (normwise max relative error
against the float64 oracle, see gpu_util)."""
import numpy as np
import pytest
import torch

import paper_2609_05275_amd as ld
from oracle import block, masks, rows
from tests.gpu_util import DEV, TOL_BF16, TOL_F32, f64, rel

pytestmark = pytest.mark.gpu

TD = {"bf16": torch.bfloat16, "f32": torch.float32}


def _run_masks(ps, B, seed, step, first_layer=0):
    L = len(ps)
    keep = torch.full((L, B), 7, dtype=torch.uint8, device=DEV)
    idx = torch.full((L, B), 12345, dtype=torch.int32, device=DEV)
    cnt = torch.full((L,), -5, dtype=torch.int32, device=DEV)
    ld.ld_masks(ps, seed, step, keep, idx, cnt, first_layer=first_layer)
    torch.cuda.synchronize()
    return keep.cpu().numpy(), idx.cpu().numpy(), cnt.cpu().numpy()


@pytest.mark.parametrize("case", [
    ("tiny_ild", [0.0, 0.2], 8, 0, 0, 0),
    ("1b_ild", list(np.linspace(0, 0.2, 16)), 8, 0, 1000, 0),
    ("stress", [0.0, 0.05, 0.5, 0.95, 1.0] * 3 + [0.5], 32, 2, 7, 0),
    ("layer_offset", [0.3, 0.6], 4, 9, 123456789, 5),
    ("one_sample", [0.5] * 4, 1, 1, 3, 0),
    ("big_batch", [0.0, 0.1, 0.5, 0.9, 1.0], 100_003, 3, 2**40 + 5, 0),
    ("many_layers", [0.37] * 128, 64, 11, 1, 0),
])
def test_masks_bit_exact(case):
    name, ps, B, seed, step, first = case
    ps = np.asarray(ps, dtype=np.float32)
    k, i, c = _run_masks(list(ps), B, seed, step, first)
    ek, ei, ec = masks.masks(ps, seed, step, B, first_layer=first)
    assert np.array_equal(k, ek), name
    assert np.array_equal(c, ec), name
    assert np.array_equal(i, ei), name


def test_masks_empirical_rate_on_device():
    B, p = 1 << 20, np.float32(0.2)
    k, _, c = _run_masks([float(p)], B, 5, 77)
    rate = c[0] / B
    assert abs(rate - (1 - p)) < 5 * np.sqrt(p * (1 - p) / B)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_gather_scatter_bit_exact(dt):
    B, S, d = 6, 128, 256
    cfg = ld.config(B, S, d, 4 if dt == "bf16" else 8, 512, ld.LD_BF16 if dt == "bf16" else ld.LD_F32)
    g = torch.Generator().manual_seed(0)
    x = torch.randn(B, S, d, generator=g).to(TD[dt]).to(DEV)
    yk = torch.randn(B * S, d, generator=g).to(TD[dt]).to(DEV)
    kept = [0, 2, 3, 5]
    idx = torch.tensor(kept + [-1, -1], dtype=torch.int32, device=DEV)
    cnt = torch.tensor([len(kept)], dtype=torch.int32, device=DEV)
    xk = torch.zeros(B * S, d, dtype=TD[dt], device=DEV)
    ld.ld_gather_rows(cfg, idx, cnt, x, xk)
    torch.cuda.synchronize()
    want = x.reshape(B, S, d)[kept].reshape(-1, d)
    assert torch.equal(xk[:len(kept) * S], want)
    assert not xk[len(kept) * S:].any()
    r = 1.0 / (1.0 - 0.3)
    x0 = x.clone()
    ld.ld_scatter_add_rows(cfg, idx, cnt, r, yk, x)
    torch.cuda.synchronize()
    want = rows.scatter_add(f64(x0), kept, len(kept), r, f64(yk), dt)
    assert np.array_equal(f64(x).astype(np.float32).view(np.uint32), want.view(np.uint32))
    assert torch.equal(x[1], x0[1]) and torch.equal(x[4], x0[4])


@pytest.mark.parametrize("dt,d", [("bf16", 2048), ("bf16", 768), ("bf16", 4096), ("f32", 64),
                                  ("f32", 1000)])
def test_rmsnorm_fwd_bwd(dt, d):
    rows, eps = 333, 1e-5
    g = torch.Generator().manual_seed(1)
    x = torch.randn(rows, d, generator=g).to(TD[dt])
    gam = (1 + 0.1 * torch.randn(d, generator=g)).to(TD[dt])
    gy = torch.randn(rows, d, generator=g).to(TD[dt])
    gres = torch.randn(rows, d, generator=g).to(TD[dt])
    xd, gd, gyd, grd = (t.to(DEV) for t in (x, gam, gy, gres))
    y = torch.empty_like(xd)
    rstd = torch.empty(rows, dtype=torch.float32, device=DEV)
    ld.ld_rmsnorm_fwd(xd, gd, y, rstd, eps)
    gx = torch.empty_like(xd)
    dg = torch.empty(d, dtype=torch.float32, device=DEV)
    ws = torch.empty(ld.ld_rmsnorm_bwd_ws_bytes(rows, d), dtype=torch.uint8, device=DEV)
    ld.ld_rmsnorm_bwd(xd, gd, rstd, gyd, grd, gx, dg, ws)
    torch.cuda.synchronize()
    ey, er = block.rmsnorm(f64(x), f64(gam), eps)
    egx, edg = block.rmsnorm_bwd(f64(x), f64(gam), er, f64(gy))
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    assert rel(f64(y), ey) < tol
    assert rel(f64(rstd), er) < 1e-5
    assert rel(f64(gx), egx + f64(gres)) < tol
    assert rel(f64(dg), edg) < tol


@pytest.mark.parametrize("dt,f", [("bf16", 16384), ("bf16", 2048), ("f32", 172)])
def test_relu2_fwd_bwd(dt, f):
    rows = 257
    g = torch.Generator().manual_seed(6)
    u = (2 * torch.randn(rows, f, generator=g)).to(TD[dt])
    gs = torch.randn(rows, f, generator=g).to(TD[dt])
    ud, gsd = u.to(DEV), gs.to(DEV)
    s = torch.empty(rows, f, dtype=TD[dt], device=DEV)
    gu = torch.empty(rows, f, dtype=TD[dt], device=DEV)
    ld.ld_relu2_fwd(ud, s)
    ld.ld_relu2_bwd(ud, gsd, gu)
    torch.cuda.synchronize()
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    assert rel(f64(s), block.relu2(f64(u))) < tol
    assert rel(f64(gu), f64(gs) * block.relu2_grad(f64(u))) < tol
    # negative inputs give exactly zero
    neg = f64(u) <= 0
    assert not f64(s)[neg].any() and not f64(gu)[neg].any()


@pytest.mark.parametrize("dt,f", [("bf16", 5504), ("bf16", 2048), ("f32", 172)])
def test_swiglu_fwd_bwd(dt, f):
    rows = 257
    g = torch.Generator().manual_seed(2)
    uv = (2 * torch.randn(rows, 2 * f, generator=g)).to(TD[dt])
    gs = torch.randn(rows, f, generator=g).to(TD[dt])
    uvd, gsd = uv.to(DEV), gs.to(DEV)
    s = torch.empty(rows, f, dtype=TD[dt], device=DEV)
    guv = torch.empty(rows, 2 * f, dtype=TD[dt], device=DEV)
    ld.ld_swiglu_fwd(uvd, s)
    ld.ld_swiglu_bwd(uvd, gsd, guv)
    torch.cuda.synchronize()
    u, v, go = f64(uv)[:, :f], f64(uv)[:, f:], f64(gs)
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    assert rel(f64(s), block.silu(u) * v) < tol
    assert rel(f64(guv)[:, :f], go * v * block.silu_grad(u)) < tol
    assert rel(f64(guv)[:, f:], go * block.silu(u)) < tol


@pytest.mark.parametrize("layout", [(1, 1), (1, 0), (0, 0), (0, 1)])
@pytest.mark.parametrize("shape", [(256, 384, 512), (200, 136, 72), (128, 128, 0), (1000, 264, 1256)])
def test_gemm_bf16(layout, shape):
    ak, bk = layout
    M, N, K = shape
    g = torch.Generator().manual_seed(3)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    B = torch.randn(N, K, generator=g).to(torch.bfloat16)
    R = torch.randn(M, N, generator=g).to(torch.bfloat16)
    Ad = (A if ak else A.t().contiguous()).to(DEV)
    Bd = (B if bk else B.t().contiguous()).to(DEV)
    Cd = torch.empty(M, N, dtype=torch.bfloat16, device=DEV)
    ld.ld_gemm(ak, bk, M, N, K, Ad, K if ak else M, Bd, K if bk else N, Cd, N, alpha=0.5,
               R=R.to(DEV), ldr=N)
    Cf = torch.empty(M, N, dtype=torch.float32, device=DEV)
    ld.ld_gemm(ak, bk, M, N, K, Ad, K if ak else M, Bd, K if bk else N, Cf, N, alpha=1.0, c_f32=True)
    torch.cuda.synchronize()
    ref = f64(A) @ f64(B).T
    assert rel(f64(Cd), f64(R) + 0.5 * ref) < TOL_BF16
    if K > 0:
        assert rel(f64(Cf), ref) < 1e-5
    else:
        assert not Cf.any()


@pytest.mark.parametrize("layout", [(1, 1), (1, 0), (0, 0), (0, 1)])
@pytest.mark.parametrize("shape", [(2048, 2048, 2048), (2048, 2048, 2000), (4096, 1000, 512),
                                   (1536, 2304, 1024)])
def test_gemm_bf16_big_tiles(layout, shape):
    """Shapes routed to the 256x256 kernel: K tail, ragged N, M not a tile multiple."""
    ak, bk = layout
    M, N, K = shape
    g = torch.Generator().manual_seed(6)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    B = torch.randn(N, K, generator=g).to(torch.bfloat16)
    R = torch.randn(M, N, generator=g).to(torch.bfloat16)
    Ad = (A if ak else A.t().contiguous()).to(DEV)
    Bd = (B if bk else B.t().contiguous()).to(DEV)
    Cd = torch.empty(M, N, dtype=torch.bfloat16, device=DEV)
    ld.ld_gemm(ak, bk, M, N, K, Ad, K if ak else M, Bd, K if bk else N, Cd, N, alpha=-1.5,
               R=R.to(DEV), ldr=N)
    torch.cuda.synchronize()
    ref = f64(A) @ f64(B).T
    assert rel(f64(Cd), f64(R) - 1.5 * ref) < TOL_BF16


@pytest.mark.parametrize("layout", [(0, 0), (1, 0)])
def test_gemm_bf16_split_k(layout):
    """float32 output with split-K partials summed in a fixed order."""
    ak, bk = layout
    M, N, K = 2048, 2048, 8192
    g = torch.Generator().manual_seed(7)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    B = torch.randn(N, K, generator=g).to(torch.bfloat16)
    Ad = (A if ak else A.t().contiguous()).to(DEV)
    Bd = (B if bk else B.t().contiguous()).to(DEV)
    wsb = ld.ld_gemm_ws_bytes(ld.LD_BF16, ak, bk, M, N, K, N, 1)
    assert wsb > 0
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        Cd = torch.full((M, N), 3.0, dtype=torch.float32, device=DEV)
        ld.ld_gemm(ak, bk, M, N, K, Ad, K if ak else M, Bd, K if bk else N, Cd, N, alpha=0.25,
                   c_f32=True, ws=ws)
        torch.cuda.synchronize()
        outs.append(Cd.cpu())
    assert torch.equal(outs[0], outs[1])
    assert rel(outs[0].double().numpy(), 0.25 * (f64(A) @ f64(B).T)) < 1e-5


@pytest.mark.parametrize("layout", [(1, 1), (1, 0), (0, 0)])
def test_gemm_f32(layout):
    ak, bk = layout
    M, N, K = 100, 172, 64
    g = torch.Generator().manual_seed(4)
    A = torch.randn(M, K, generator=g)
    B = torch.randn(N, K, generator=g)
    Ad = (A if ak else A.t().contiguous()).to(DEV)
    Bd = (B if bk else B.t().contiguous()).to(DEV)
    Cd = torch.empty(M, N, device=DEV)
    ld.ld_gemm(ak, bk, M, N, K, Ad, K if ak else M, Bd, K if bk else N, Cd, N, alpha=2.0)
    torch.cuda.synchronize()
    assert rel(f64(Cd), 2.0 * (f64(A) @ f64(B).T)) < TOL_F32


def _attn_ref(qkv, n, S, H, dh, alibi=0):
    d = H * dh
    q64 = f64(qkv).reshape(n, S, 3 * d)
    outs, probs = [], []
    slopes = block.alibi_slopes(H) if alibi else None
    for b in range(n):
        o, p = block.causal_attention(q64[b, :, :d], q64[b, :, d:2 * d], q64[b, :, 2 * d:], H, slopes)
        outs.append(o)
        probs.append(p)
    return q64, outs, probs


@pytest.mark.parametrize("alibi", [0, 1])
@pytest.mark.parametrize("dt,n,S,H,dh", [("bf16", 2, 64, 2, 128), ("bf16", 2, 192, 2, 64), ("bf16", 2, 256, 2, 128),
                                         ("bf16", 1, 1024, 1, 128), ("bf16", 1, 512, 6, 128),
                                         ("f32", 3, 32, 4, 16), ("f32", 2, 100, 2, 64)])
def test_attention_fwd_bwd(dt, n, S, H, dh, alibi):
    d = H * dh
    g = torch.Generator().manual_seed(5)
    qkv = torch.randn(n * S, 3 * d, generator=g).to(TD[dt])
    go = torch.randn(n * S, d, generator=g).to(TD[dt])
    qd, god = qkv.to(DEV), go.to(DEV)
    o = torch.empty(n * S, d, dtype=TD[dt], device=DEV)
    lse = torch.empty(n, H, S, dtype=torch.float32, device=DEV)
    ld.ld_attn_fwd(n, S, H, dh, qd, o, lse, alibi=alibi)
    gq = torch.empty(n * S, 3 * d, dtype=TD[dt], device=DEV)
    ws = torch.empty(ld.ld_attn_bwd_ws_bytes(n, S, H), dtype=torch.uint8, device=DEV)
    ld.ld_attn_bwd(n, S, H, dh, qd, o, lse, god, gq, ws, alibi=alibi)
    torch.cuda.synchronize()
    q64, outs, probs = _attn_ref(qkv, n, S, H, dh, alibi)
    go64 = f64(go).reshape(n, S, d)
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    of, gf = f64(o).reshape(n, S, d), f64(gq).reshape(n, S, 3 * d)
    lsef = f64(lse)
    for b in range(n):
        assert rel(of[b], outs[b]) < tol
        gq_, gk_, gv_ = block.causal_attention_bwd(q64[b, :, :d], q64[b, :, d:2 * d],
                                                   q64[b, :, 2 * d:], probs[b], go64[b], H)
        assert rel(gf[b, :, :d], gq_) < tol, "dq"
        assert rel(gf[b, :, d:2 * d], gk_) < tol, "dk"
        assert rel(gf[b, :, 2 * d:], gv_) < tol, "dv"
        # log-sum-exp of the scaled causal scores (with the ALiBi bias)
        slopes = block.alibi_slopes(H) if alibi else np.zeros(H)
        dist = np.arange(S)[:, None] - np.arange(S)[None, :]
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            s = q64[b, :, cols] @ q64[b, :, d:2 * d][:, cols].T / np.sqrt(dh) - slopes[h] * dist
            s[np.triu(np.ones((S, S), bool), 1)] = -np.inf
            m = s.max(axis=1)
            want = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
            assert np.max(np.abs(lsef[b, h] - want)) < (2e-2 if dt == "bf16" else 1e-4)


@pytest.mark.parametrize("dh", [64, 128])
def test_attention_bwd_bf16_repeatable(dh):
    """The bf16 backward passes P between waves through LDS under barriers;
    repeated runs on the same inputs must give the same bits (a missing
    wait would show up as run-to-run differences)."""
    n, S, H = 3, 1024, 2
    d = H * dh
    g = torch.Generator().manual_seed(11)
    qd = torch.randn(n * S, 3 * d, generator=g).to(torch.bfloat16).to(DEV)
    god = torch.randn(n * S, d, generator=g).to(torch.bfloat16).to(DEV)
    o = torch.empty(n * S, d, dtype=torch.bfloat16, device=DEV)
    lse = torch.empty(n, H, S, dtype=torch.float32, device=DEV)
    ld.ld_attn_fwd(n, S, H, dh, qd, o, lse)
    ws = torch.empty(ld.ld_attn_bwd_ws_bytes(n, S, H), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(4):
        gq = torch.full((n * S, 3 * d), float("nan"), dtype=torch.bfloat16, device=DEV)
        ld.ld_attn_bwd(n, S, H, dh, qd, o, lse, god, gq, ws)
        torch.cuda.synchronize()
        outs.append(gq.view(torch.int16).cpu())
    assert not torch.isnan(gq.float()).any()
    for x in outs[1:]:
        assert torch.equal(x, outs[0])
