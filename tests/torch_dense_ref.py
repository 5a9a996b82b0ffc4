"""A second, independent statement of the block for the oracle's pins:
torch float64 autograd built from library routines (rms_norm,
scaled_dot_product_attention with is_causal or with an explicit float mask,
silu, relu), applied to the whole batch and gated by the mask multiply of the
layer-dropout training equation (H + r M f(H)), with one mask per layer or
separate attention and FFN masks (sub-layer dropout).  Kind 1 adds the ALiBi bias
through the attention mask and uses the squared-ReLU feed-forward.  Used only
by the CPU pin tests of the oracle."""
import numpy as np
import torch
import torch.nn.functional as F

KEYS = ("g_attn", "w_qkv", "w_o", "g_mlp", "w_gate_up", "w_down")


def alibi_mask(n_heads, S):
    """Float attention mask [H, S, S]: -m_h (i - j) on and below the diagonal,
    -inf above.  Slopes: powers of two of the head count get 2^(-8/n) raised
    to 1..n; otherwise the largest power of two n below takes those and the
    rest are the odd-numbered terms 1, 3, 5, ... of the 2n-head sequence."""
    n = 2 ** int(np.floor(np.log2(n_heads)))
    base = torch.tensor(2.0, dtype=torch.float64) ** (-8.0 / n)
    sl = [base ** (i + 1) for i in range(n)]
    base2 = torch.tensor(2.0, dtype=torch.float64) ** (-8.0 / (2 * n))
    sl += [base2 ** (2 * i + 1) for i in range(n_heads - n)]
    slopes = torch.stack(sl)
    i = torch.arange(S, dtype=torch.float64)
    dist = i[:, None] - i[None, :]
    mask = -slopes[:, None, None] * dist
    return mask.masked_fill(dist < 0, float("-inf"))


def block_full_batch(X, w, n_heads, eps, kind=0):
    B, S, d = X.shape
    dh = d // n_heads
    h1 = F.rms_norm(X, (d,), w["g_attn"], eps)
    qkv = h1 @ w["w_qkv"].T
    q, k, v = (qkv[..., i * d:(i + 1) * d].reshape(B, S, n_heads, dh).transpose(1, 2)
               for i in range(3))
    if kind == 1:
        a = F.scaled_dot_product_attention(q, k, v, attn_mask=alibi_mask(n_heads, S))
    else:
        a = F.scaled_dot_product_attention(q, k, v, is_causal=True)
    a = a.transpose(1, 2).reshape(B, S, d)
    return h1, a


def layer_masked(X, w, keep, r, n_heads, eps, kind=0):
    """X + r M_attn f_attn, then + r M_ffn f_ffn, over the full batch (mask
    multiply).  keep: [B] (one mask for both sub-blocks) or [2, B]."""
    B, S, d = X.shape
    f = w["w_down"].shape[1]
    k = np.asarray(keep).reshape(-1, B)
    m_a = torch.as_tensor(k[0], dtype=X.dtype).reshape(B, 1, 1)
    m = torch.as_tensor(k[-1], dtype=X.dtype).reshape(B, 1, 1)
    _, a = block_full_batch(X, w, n_heads, eps, kind)
    Z = X + r * m_a * (a @ w["w_o"].T)
    h2 = F.rms_norm(Z, (d,), w["g_mlp"], eps)
    uv = h2 @ w["w_gate_up"].T
    if kind == 1:
        s = F.relu(uv) ** 2
    else:
        s = F.silu(uv[..., :f]) * uv[..., f:]
    return Z + r * m * (s @ w["w_down"].T)


def stack_step(X0, weights, keep, rs, G, n_heads, eps, kind=0):
    """Returns X_L, dL/dX0, grads (numpy float64) with L = sum(G * X_L)."""
    X = torch.tensor(X0, dtype=torch.float64, requires_grad=True)
    ws = [{k: torch.tensor(np.asarray(w[k], dtype=np.float64), requires_grad=True) for k in KEYS}
          for w in weights]
    H = X
    for l, w in enumerate(ws):
        H = layer_masked(H, w, keep[l], rs[l], n_heads, eps, kind)
    loss = (H * torch.as_tensor(G, dtype=torch.float64)).sum()
    loss.backward()
    grads = [{k: w[k].grad.numpy().copy() for k in KEYS} for w in ws]
    return H.detach().numpy(), X.grad.numpy().copy(), grads
