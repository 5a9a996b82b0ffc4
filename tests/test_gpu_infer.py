"""Depth-elastic inference on the HIP path against the oracle (needs a GPU):
the evaluation form over active-layer sets (ld_stack_eval), KV-cached
decoding (ld_stack_decode) including a draft/verify sequence, and the
decoding kernels in isolation (skinny GEMM, KV store, decode attention).
Inputs given to the oracle are built on the host (the caches it reads are
host copies of host data), never read back from the GPU."""
import dataclasses

import numpy as np
import pytest
import torch

import ld_inputs as inp
import paper_2609_05275_amd as ld
from oracle import block, infer
from tests.gpu_util import DEV, f64, layer_weights_dev, rel, tol
from tests.test_gpu_layer import SMALL_BF16, SMALL_BF16_128, SMALL_P, SMALL_P_128, _buf, _cfg

pytestmark = pytest.mark.gpu

BF16_SHAPES = [SMALL_BF16, SMALL_P, SMALL_BF16_128, SMALL_P_128]
BF16_IDS = ["small_bf16", "paper_small_bf16", "small_bf16_dh128", "paper_small_dh128_h6"]


def _bf16(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)


def _rng_bf16(rng, shape, scale=1.0):
    return _bf16(rng.standard_normal(shape) * scale)


# ------------------------------------------------------------- kernels

@pytest.mark.parametrize("M", [1, 8, 31, 33, 48, 64])
@pytest.mark.parametrize("N,K", [(96, 64), (130, 200), (2048, 2048), (704, 5504)])
@pytest.mark.parametrize("resid", [False, True])
def test_gemm_skinny(M, N, K, resid):
    rng = np.random.default_rng(M * 7 + N + K)
    A = _rng_bf16(rng, (M, K))
    W = _rng_bf16(rng, (N, K), 0.05)
    R = _rng_bf16(rng, (M, N)) if resid else None
    alpha = 0.75
    Ad, Wd = A.to(DEV), W.to(DEV)
    Rd = None if R is None else R.to(DEV)
    ws_n = ld.ld_gemm_skinny_ws_bytes(M, N, K)
    ws = _buf(ws_n) if ws_n else None
    outs = []
    for _ in range(2):
        C = torch.full((M, N), 3.0, dtype=torch.bfloat16, device=DEV)
        ld.ld_gemm_skinny(Ad, Wd, C, alpha=alpha, R=Rd, ws=ws)
        torch.cuda.synchronize()
        outs.append(C.cpu())
    assert torch.equal(outs[0], outs[1])
    want = alpha * (f64(A) @ f64(W).T) + (f64(R) if resid else 0.0)
    assert rel(f64(outs[0]), want) < 1e-2


def test_gemm_skinny_rejects():
    A = torch.zeros(65, 64, dtype=torch.bfloat16, device=DEV)
    W = torch.zeros(32, 64, dtype=torch.bfloat16, device=DEV)
    C = torch.zeros(65, 32, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ld.LdError):
        ld.ld_gemm_skinny(A, W, C)


DEC_MODES = ["plain", "resid", "norm", "norm_resid", "swiglu", "norm_swiglu", "norm_relu2"]


@pytest.mark.parametrize("M", [1, 3, 8])
@pytest.mark.parametrize("N,K", [(96, 64), (130, 200), (2048, 2048), (704, 5504), (11008, 2048)])
@pytest.mark.parametrize("mode", DEC_MODES)
def test_gemm_dec(M, N, K, mode):
    """Fused decoding projection: RMSNorm of the input rows, projection,
    residual or activation in one launch, against the oracle's RMSNorm and
    activations in float64 on the same bf16 inputs (16 waves per workgroup
    for N = 2048, 8 for the 11008-column SwiGLU, ragged column tiles for
    N = 130 and 704, a ragged k chunk for K = 200)."""
    norm = mode.startswith("norm")
    act = ld.DEC_ACT_SWIGLU if "swiglu" in mode else ld.DEC_ACT_RELU2 if "relu2" in mode else ld.DEC_ACT_NONE
    rng = np.random.default_rng(M * 131 + N * 7 + K + len(mode))
    wrows = 2 * N if act == ld.DEC_ACT_SWIGLU else N
    A = _rng_bf16(rng, (M, K))
    W = _rng_bf16(rng, (wrows, K), 0.05)
    G = _bf16(1.0 + 0.2 * rng.standard_normal(K)) if norm else None
    R = _rng_bf16(rng, (M, N)) if "resid" in mode else None
    alpha = 0.75
    eps = 1e-5
    Ad, Wd = A.to(DEV), W.to(DEV)
    Gd = None if G is None else G.to(DEV)
    Rd = None if R is None else R.to(DEV)
    if norm and K > 4096:
        # the fused RMSNorm stages at most 4096 columns: refused, nothing launched
        C = torch.full((M, N), 3.0, dtype=torch.bfloat16, device=DEV)
        with pytest.raises(ld.LdError) as e:
            ld.ld_gemm_dec(Ad, Wd, C, g=Gd, eps=eps, alpha=alpha, R=Rd, act=act)
        assert e.value.status == 3   # LD_E_UNSUPPORTED
        torch.cuda.synchronize()
        assert bool((C == 3.0).all())
        return
    outs = []
    for _ in range(2):
        C = torch.full((M, N), 3.0, dtype=torch.bfloat16, device=DEV)
        ld.ld_gemm_dec(Ad, Wd, C, g=Gd, eps=eps, alpha=alpha, R=Rd, act=act)
        torch.cuda.synchronize()
        outs.append(C.cpu())
    assert torch.equal(outs[0], outs[1])
    a = f64(A)
    if norm:
        a, _ = block.rmsnorm(a, f64(G), eps)
    y = alpha * (a @ f64(W).T)
    if act == ld.DEC_ACT_SWIGLU:
        want = block.silu(y[:, :N]) * y[:, N:]
    elif act == ld.DEC_ACT_RELU2:
        want = block.relu2(y)
    else:
        want = y + (f64(R) if R is not None else 0.0)
    assert rel(f64(outs[0]), want) < 1e-2


def test_gemm_dec_rejects():
    A = torch.zeros(9, 64, dtype=torch.bfloat16, device=DEV)
    W = torch.zeros(32, 64, dtype=torch.bfloat16, device=DEV)
    C = torch.zeros(9, 32, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ld.LdError):
        ld.ld_gemm_dec(A, W, C)                                       # 9 rows
    A8, C8 = A[:8], C[:8]
    with pytest.raises(ld.LdError):
        ld.ld_gemm_dec(A8, W, C8, R=C8, act=ld.DEC_ACT_RELU2)       # residual with an activation
    Ak = torch.zeros(8, 4104, dtype=torch.bfloat16, device=DEV)
    Wk = torch.zeros(32, 4104, dtype=torch.bfloat16, device=DEV)
    g = torch.ones(4104, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ld.LdError):
        ld.ld_gemm_dec(Ak, Wk, C8, g=g)                               # norm over more than 4096 columns


@pytest.mark.parametrize("pos,n", [(0, 1), (5, 3), (248, 8)])
def test_kv_store_bit_exact(pos, n):
    rng = np.random.default_rng(pos + n)
    B, d, s_max = 3, 256, 256
    qkv = _rng_bf16(rng, (B * n, 3 * d))
    kv = _rng_bf16(rng, (B, s_max, 2 * d))
    want = kv.clone()
    for b in range(B):
        for j in range(n):
            want[b, pos + j] = qkv[b * n + j, d:]
    kd = kv.to(DEV)
    ld.ld_kv_store(B, n, d, pos, qkv.to(DEV), kd, s_max)
    torch.cuda.synchronize()
    assert torch.equal(kd.cpu(), want)


@pytest.mark.parametrize("dh,H", [(64, 4), (128, 3)])
@pytest.mark.parametrize("alibi", [0, 1])
@pytest.mark.parametrize("pos,n", [(0, 1), (0, 8), (5, 3), (255, 1), (250, 8), (256, 2), (700, 8)])
def test_attn_decode(dh, H, alibi, pos, n):
    rng = np.random.default_rng(pos * 31 + n + dh + alibi)
    B, d = 2, H * dh
    s_max = max(pos + n, 64) + 16
    qkv = _rng_bf16(rng, (B * n, 3 * d))
    kv = _rng_bf16(rng, (B, s_max, 2 * d))
    for b in range(B):                       # the cache holds the new rows' keys/values
        for j in range(n):
            kv[b, pos + j] = qkv[b * n + j, d:]
    o = torch.zeros(B * n, d, dtype=torch.bfloat16, device=DEV)
    ws = _buf(ld.ld_attn_decode_ws_bytes(B, H, dh, s_max))
    ld.ld_attn_decode(B, H, dh, pos, n, qkv.to(DEV), kv.to(DEV), s_max, o, ws, alibi=alibi)
    torch.cuda.synchronize()
    slopes = block.alibi_slopes(H) if alibi else None
    q64, kv64 = f64(qkv), f64(kv)
    got = f64(o)
    for b in range(B):
        want = infer.attention_rows(q64[b * n:(b + 1) * n, :d], kv64[b, :pos + n, :d],
                                    kv64[b, :pos + n, d:], pos + np.arange(n), H, slopes)
        assert rel(got[b * n:(b + 1) * n], want) < 1e-2, b


# ------------------------------------------------------ evaluation form

ACTIVE = {"all": None, "exit": "exit", "skip": "skip"}


def _active(name, L):
    if name == "all":
        return [1] * L
    if name == "exit":
        return [1] * (L - 1) + [0]
    return [0 if l % 2 else 1 for l in range(L)]


def _weights(sh):
    return [layer_weights_dev(sh, l, gain_jitter=True) for l in range(sh.n_layers)]


@pytest.mark.parametrize("sh", [inp.SHAPES["tiny"]] + BF16_SHAPES, ids=["tiny_f32"] + BF16_IDS)
@pytest.mark.parametrize("name", list(ACTIVE))
def test_stack_eval(sh, name):
    cfg = _cfg(sh)
    L, B, S, d = sh.n_layers, sh.batch, sh.seq, sh.d_model
    act = _active(name, L)
    r = [1.0] * L if name != "skip" else [0.9 + 0.1 * l for l in range(L)]
    W = _weights(sh)
    x = inp.hidden(sh)
    xd = x.to(DEV)
    bf = sh.dtype == "bf16"
    s_max = S + 64
    kv = None
    if bf:
        kv = [torch.full((B, s_max, 2 * d), 5.0, dtype=torch.bfloat16, device=DEV) for _ in range(L)]
    ld.ld_stack_eval(cfg, [w[0] for w in W], xd, _buf(ld.ld_eval_ws_bytes(cfg)), active=act,
                     r_eval=r, kv=kv, s_max=s_max)
    torch.cuda.synchronize()
    XL, okv = infer.eval_forward(inp.f64(x), [w[1] for w in W], act, sh.n_heads, kind=sh.kind,
                                 r_eval=r)
    t = tol(sh.dtype)
    assert rel(f64(xd), XL) < t
    if bf:
        for l in range(L):
            c = f64(kv[l])
            if act[l]:
                assert rel(c[:, :S, :d], okv[l][0]) < t and rel(c[:, :S, d:], okv[l][1]) < t
                assert (c[:, S:] == 5.0).all()
            else:
                assert (c == 5.0).all()


# ------------------------------------------------------------- decoding

def _decode_case(sh, steps, s_max, batch=None):
    """Prefill 64 positions with the full model, then run (n_new, active)
    decoding steps in order; compare every step with the oracle: full-model
    steps against the evaluation forward's rows, draft steps against oracle
    decoding over the full model's keys/values."""
    if batch:
        sh = dataclasses.replace(sh, batch=batch)
    L, B, d = sh.n_layers, sh.batch, sh.d_model
    total = 64 + sum(n for n, _ in steps)
    shf = dataclasses.replace(sh, seq=((total + 63) // 64) * 64)
    X = inp.hidden(shf)                       # [B, >= total, d]: the row inputs of every position
    W = _weights(sh)
    wd, w64 = [w[0] for w in W], [w[1] for w in W]
    cfg = _cfg(dataclasses.replace(sh, seq=64))
    kv = [torch.zeros(B, s_max, 2 * d, dtype=torch.bfloat16, device=DEV) for _ in range(L)]
    x0 = X[:, :64].contiguous().to(DEV)
    ld.ld_stack_eval(cfg, wd, x0, _buf(ld.ld_eval_ws_bytes(cfg)), kv=kv, s_max=s_max)
    X64 = inp.f64(X)
    full_out, full_kv = infer.eval_forward(X64[:, :total], w64, [1] * L, sh.n_heads, kind=sh.kind)
    t = tol(sh.dtype)
    pos = 64
    ws = _buf(max(ld.ld_decode_ws_bytes(cfg, n, s_max) for n, _ in steps))
    for n, act in steps:
        xd = X[:, pos:pos + n].contiguous().to(DEV)
        ld.ld_stack_decode(cfg, wd, xd, kv, s_max, pos, n, ws, active=act)
        torch.cuda.synchronize()
        if act is None:
            want = full_out[:, pos:pos + n]
        else:
            okv = [(full_kv[l][0], full_kv[l][1]) for l in range(L)]
            want, _ = infer.decode(X64[:, pos:pos + n], w64, act, okv, pos, sh.n_heads, kind=sh.kind)
        assert rel(f64(xd), want) < t, (pos, n, act)
        if act is None:
            pos += n                           # a draft step is verified (overwritten) next
    return sh


@pytest.mark.parametrize("sh", BF16_SHAPES, ids=BF16_IDS)
def test_decode_draft_and_verify(sh):
    L = sh.n_layers
    draft = [1 if l % 2 == 0 else 0 for l in range(L)]
    steps = [(3, None), (1, draft), (1, draft), (2, None), (8, None), (1, None)]
    _decode_case(sh, steps, s_max=192)


@pytest.mark.parametrize("sh", BF16_SHAPES, ids=BF16_IDS)
def test_decode_draft_several_rows(sh):
    """Draft steps of 2 and 3 rows per sequence (9 to 64 rows in all: the
    reductions that carry the next active layer's RMSNorm skip the inactive
    layers, and the last active layer's carries none)."""
    L = sh.n_layers
    draft = [1 if l % 2 == 0 else 0 for l in range(L)]
    late = [0] * (L - 1) + [1]
    steps = [(2, None), (2, draft), (3, draft), (3, late), (2, None)]
    _decode_case(sh, steps, s_max=192)


@pytest.mark.parametrize("sh", [SMALL_BF16, SMALL_P_128], ids=["small_bf16", "paper_small_dh128_h6"])
def test_decode_across_key_chunks(sh):
    """Decoding steps of 8 from position 64 to past 256 (the attention's key
    chunk boundary) with a cache that ends exactly at the last position."""
    steps = [(8, None)] * 26
    _decode_case(sh, steps, s_max=64 + 8 * 26)


def test_decode_more_rows_than_the_skinny_kernel():
    """batch 9 x 8 rows = 72 > 64: the projections take the general GEMM."""
    _decode_case(SMALL_BF16, [(8, None), (1, None)], s_max=128, batch=9)


def test_decode_rejects_bad_positions():
    sh = SMALL_BF16
    cfg = _cfg(sh)
    W = [w[0] for w in _weights(sh)]
    kv = [torch.zeros(sh.batch, 64, 2 * sh.d_model, dtype=torch.bfloat16, device=DEV)] * sh.n_layers
    x = torch.zeros(sh.batch, 1, sh.d_model, dtype=torch.bfloat16, device=DEV)
    ws = _buf(ld.ld_decode_ws_bytes(cfg, 8, 64))
    with pytest.raises(ld.LdError):
        ld.ld_stack_decode(cfg, W, x, kv, 64, 64, 1, ws)       # past the cache
    with pytest.raises(ld.LdError):
        ld.ld_stack_decode(cfg, W, x, kv, 64, 0, 9, ws)        # n_new > 8
