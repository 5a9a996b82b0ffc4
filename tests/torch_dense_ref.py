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


def eval_stack(X0, weights, active, r_eval, n_heads, eps, kind=0):
    """Evaluation form over an active set with torch library routines: an
    active layer is layer_masked with every sequence kept and r = r_eval[l];
    a skipped layer is the identity.  Returns X_L (numpy float64) and the
    per-layer keys/values (k, v) [B, S, d] of active layers (None otherwise)."""
    H = torch.tensor(np.asarray(X0, dtype=np.float64))
    B, S, d = H.shape
    kv = []
    for l, w in enumerate(weights):
        if not active[l]:
            kv.append(None)
            continue
        wt = {k: torch.tensor(np.asarray(w[k], dtype=np.float64)) for k in KEYS}
        h1 = F.rms_norm(H, (d,), wt["g_attn"], eps)
        qkv = h1 @ wt["w_qkv"].T
        kv.append((qkv[..., d:2 * d].numpy().copy(), qkv[..., 2 * d:].numpy().copy()))
        H = layer_masked(H, wt, np.ones(B), float(r_eval[l]), n_heads, eps, kind)
    return H.numpy(), kv


def decode_layer(x_new, w, K, V, pos, r, n_heads, eps, kind=0):
    """One active layer on rows x_new [B, n, d] at positions pos..pos+n-1,
    attending to cached K, V [B, >= pos, d] plus their own keys/values:
    scaled_dot_product_attention with an explicit [n, pos+n] mask (-inf past
    each row's position, plus the ALiBi bias for kind 1)."""
    X = torch.tensor(np.asarray(x_new, dtype=np.float64))
    B, n, d = X.shape
    dh = d // n_heads
    wt = {k: torch.tensor(np.asarray(w[k], dtype=np.float64)) for k in KEYS}
    f = wt["w_down"].shape[1]
    h1 = F.rms_norm(X, (d,), wt["g_attn"], eps)
    qkv = h1 @ wt["w_qkv"].T
    Kc = torch.cat([torch.tensor(np.asarray(K, dtype=np.float64)[:, :pos]), qkv[..., d:2 * d]], 1)
    Vc = torch.cat([torch.tensor(np.asarray(V, dtype=np.float64)[:, :pos]), qkv[..., 2 * d:]], 1)
    P = pos + n
    qpos = torch.arange(pos, P, dtype=torch.float64)[:, None]
    kpos = torch.arange(P, dtype=torch.float64)[None, :]
    mask = torch.zeros(n_heads, n, P, dtype=torch.float64)
    if kind == 1:
        full = alibi_mask(n_heads, P)            # [H, P, P], rows are query positions
        mask = full[:, pos:P, :]
    mask = mask.masked_fill((kpos > qpos)[None], float("-inf"))
    q = qkv[..., :d].reshape(B, n, n_heads, dh).transpose(1, 2)
    k = Kc.reshape(B, P, n_heads, dh).transpose(1, 2)
    v = Vc.reshape(B, P, n_heads, dh).transpose(1, 2)
    a = F.scaled_dot_product_attention(q, k, v, attn_mask=mask)
    a = a.transpose(1, 2).reshape(B, n, d)
    Z = X + r * (a @ wt["w_o"].T)
    h2 = F.rms_norm(Z, (d,), wt["g_mlp"], eps)
    uv = h2 @ wt["w_gate_up"].T
    s = F.relu(uv) ** 2 if kind == 1 else F.silu(uv[..., :f]) * uv[..., f:]
    return (Z + r * (s @ wt["w_down"].T)).numpy()
