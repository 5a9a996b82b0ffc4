"""One pre-norm decoder block on one sequence, float64, forward and backward.

Test infrastructure (see the package docstring).

The block is f^l of the transformer form of the layer-dropout training
equation (Preliminary section, "Layer Dropout for a Transformer"):
    Z  = X + r * f_attn(X)        f_attn(X) = MHA(RMSNorm(X; g_attn)) W_o^T
    X' = Z + r * f_ffn(Z)         f_ffn(Z)  = SwiGLU(RMSNorm(Z; g_mlp)) W_down^T
with the sub-block choices of this hot path (kind 0): RMSNorm, causal
multi-head attention without positional bias, SwiGLU.  The paper's footnote
on that equation states the formulation holds for any pre-norm attention/FFN
variant with a residual connection.  Kind 1 is the block of the paper's
experiments (Experimental Setup: ALiBi position embeddings, squared ReLU):
the attention scores get the ALiBi bias, and f_ffn(Z) = relu(RMSNorm(Z) W_up^T)^2
W_down^T with two matrices.

Readings (the paper is silent on these):
  * RMSNorm(x; g) = x / sqrt(mean_d(x^2) + eps) * g, eps from the config;
  * attention scale 1/sqrt(d_head), causal with the diagonal kept (j <= i);
  * no biases anywhere;
  * w_qkv rows are [q | k | v], each d rows, head h owning rows h*dh..h*dh+dh
    of each part; w_gate_up rows [0, f) are the gate, [f, 2f) the up
    projection; SwiGLU(u, v) = silu(u) * v, silu(u) = u * sigmoid(u);
  * weights are stored [out, in] and applied as x @ W^T;
  * kind 1: the normalisation stays RMSNorm with a gain and there are no
    biases (the paper names a pre-norm parameter and a hidden-bias learning
    rate in its parameterisation table but not which layers carry biases);
    ALiBi is added to the scaled scores, s_ij = q_i.k_j / sqrt(dh) - m_h (i - j),
    with the slopes of alibi_slopes; w_gate_up holds W_up [f, d].

The backward is the chain rule of the forward written out by hand; it is
pinned against finite differences and against torch float64 autograd.
"""

import numpy as np


def rmsnorm(x, g, eps):
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)
    return x * rstd[:, None] * g[None, :], rstd


def rmsnorm_bwd(x, g, rstd, gy):
    """Gradient of y = x * rstd * g: returns (dx, dg)."""
    dg = np.sum(gy * x * rstd[:, None], axis=0)
    mean_term = np.mean(x * g[None, :] * gy, axis=-1)
    dx = rstd[:, None] * (g[None, :] * gy) - x * (rstd ** 3 * mean_term)[:, None]
    return dx, dg


def alibi_slopes(n_heads):
    """Head slopes of ALiBi (Press et al., ICLR 2022, section 3): for n heads
    with n a power of two, the geometric sequence starting at 2^(-8/n) with
    that ratio; for other head counts, the n' = largest power of two below
    gets its own sequence and the remaining heads take every other slope of
    the 2n'-head sequence, starting with its first."""
    if n_heads < 1:
        return np.zeros(0)
    n = 1 << (int(n_heads).bit_length() - 1)
    own = [2.0 ** (-8.0 * (i + 1) / n) for i in range(n)]
    twice = [2.0 ** (-8.0 * (i + 1) / (2 * n)) for i in range(2 * n)]
    return np.array(own + twice[0::2][:n_heads - n], dtype=np.float64)


def causal_attention(q, k, v, n_heads, slopes=None):
    """softmax(q k^T / sqrt(dh) + bias, causal j <= i) v per head, with the
    ALiBi bias -m_h (i - j) when `slopes` is given (else no bias).
    q, k, v: [S, d].  Returns (out [S, d], probs [H, S, S])."""
    S, d = q.shape
    dh = d // n_heads
    out = np.zeros((S, d))
    probs = np.zeros((n_heads, S, S))
    future = np.triu(np.ones((S, S), dtype=bool), k=1)
    dist = np.arange(S)[:, None] - np.arange(S)[None, :]   # i - j
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        s = q[:, cols] @ k[:, cols].T / np.sqrt(dh)
        if slopes is not None:
            s = s - slopes[h] * dist
        s[future] = -np.inf
        s = s - np.max(s, axis=-1, keepdims=True)
        e = np.exp(s)
        pr = e / np.sum(e, axis=-1, keepdims=True)
        probs[h] = pr
        out[:, cols] = pr @ v[:, cols]
    return out, probs


def causal_attention_bwd(q, k, v, probs, gout, n_heads):
    """Gradients of causal_attention with respect to q, k, v."""
    S, d = q.shape
    dh = d // n_heads
    gq, gk, gv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        pr = probs[h]
        go = gout[:, cols]
        gv[:, cols] = pr.T @ go
        dp = go @ v[:, cols].T
        ds = pr * (dp - np.sum(dp * pr, axis=-1, keepdims=True))
        gq[:, cols] = ds @ k[:, cols] / np.sqrt(dh)
        gk[:, cols] = ds.T @ q[:, cols] / np.sqrt(dh)
    return gq, gk, gv


def relu2(u):
    return np.maximum(u, 0.0) ** 2


def relu2_grad(u):
    return 2.0 * np.maximum(u, 0.0)


def silu(u):
    return u / (1.0 + np.exp(-u))


def silu_grad(u):
    sg = 1.0 / (1.0 + np.exp(-u))
    return sg * (1.0 + u * (1.0 - sg))


def attn_forward(x, w, r, n_heads, eps, kind=0):
    """Attention residual sub-block on one sequence: z = x + r f_attn(x)."""
    d = x.shape[1]
    h1, rstd1 = rmsnorm(x, w["g_attn"], eps)
    qkv = h1 @ w["w_qkv"].T
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    a, probs = causal_attention(q, k, v, n_heads, alibi_slopes(n_heads) if kind == 1 else None)
    z = x + r * (a @ w["w_o"].T)
    return z, dict(x=x, h1=h1, rstd1=rstd1, q=q, k=k, v=v, a=a, probs=probs)


def ffn_forward(z, w, r, eps, kind=0):
    """FFN residual sub-block on one sequence: x' = z + r f_ffn(z)."""
    f = w["w_down"].shape[1]
    h2, rstd2 = rmsnorm(z, w["g_mlp"], eps)
    uv = h2 @ w["w_gate_up"].T
    if kind == 1:
        u, vv = uv, None
        s = relu2(u)
    else:
        u, vv = uv[:, :f], uv[:, f:]
        s = silu(u) * vv
    x_next = z + r * (s @ w["w_down"].T)
    return x_next, dict(z=z, h2=h2, rstd2=rstd2, u=u, vv=vv, s=s, kind=kind)


def forward(x, w, r, n_heads, eps, kind=0):
    """Apply the block to one kept sequence x [S, d]: the attention sub-block,
    then the FFN sub-block on its output.

    w: dict with g_attn [d], w_qkv [3d, d], w_o [d, d], g_mlp [d],
    w_gate_up [2f, d] (kind 0) or [f, d] (kind 1), w_down [d, f].  r is the
    residual-branch scale.  Returns (x_next, cache)."""
    z, ca = attn_forward(x, w, r, n_heads, eps, kind)
    x_next, cf = ffn_forward(z, w, r, eps, kind)
    return x_next, dict(ca, **cf)


def ffn_backward(cache, g, w, r):
    """Backward of ffn_forward given g = dL/dx'.  Returns (dL/dz, grads of
    g_mlp, w_gate_up, w_down)."""
    c = cache
    gy = r * g
    d_down = gy.T @ c["s"]
    gs = gy @ w["w_down"]
    if c["kind"] == 1:
        guv = gs * relu2_grad(c["u"])
    else:
        gu = gs * c["vv"] * silu_grad(c["u"])
        gvv = gs * silu(c["u"])
        guv = np.concatenate([gu, gvv], axis=1)
    d_gate_up = guv.T @ c["h2"]
    gh2 = guv @ w["w_gate_up"]
    gz_norm, d_g_mlp = rmsnorm_bwd(c["z"], w["g_mlp"], c["rstd2"], gh2)
    return g + gz_norm, dict(g_mlp=d_g_mlp, w_gate_up=d_gate_up, w_down=d_down)


def attn_backward(cache, gz, w, r, n_heads):
    """Backward of attn_forward given gz = dL/dz.  Returns (dL/dx, grads of
    g_attn, w_qkv, w_o)."""
    c = cache
    go = r * gz
    d_o = go.T @ c["a"]
    ga = go @ w["w_o"]
    gq, gk, gv = causal_attention_bwd(c["q"], c["k"], c["v"], c["probs"], ga, n_heads)
    gqkv = np.concatenate([gq, gk, gv], axis=1)
    d_qkv = gqkv.T @ c["h1"]
    gh1 = gqkv @ w["w_qkv"]
    gx_norm, d_g_attn = rmsnorm_bwd(c["x"], w["g_attn"], c["rstd1"], gh1)
    return gz + gx_norm, dict(g_attn=d_g_attn, w_qkv=d_qkv, w_o=d_o)


def backward(cache, g, w, r, n_heads):
    """Backward of `forward` for one kept sequence given g = dL/dx_next.
    Returns (dL/dx, grads dict with the same keys as w)."""
    gz, gf = ffn_backward(cache, g, w, r)
    gx, ga = attn_backward(cache, gz, w, r, n_heads)
    return gx, dict(ga, **gf)
