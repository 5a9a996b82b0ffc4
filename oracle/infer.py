"""Depth-elastic inference: the evaluation form of the layer and KV-cached
incremental decoding over a static set of active layers.

Test infrastructure (see the package docstring).

Definitions followed:
  * Evaluation equation (Preliminary section, transformer form at inference):
        Z^l     = X^l + r_eval^l f_attn^l(X^l)
        X^{l+1} = Z^l + r_eval^l f_ffn^l(Z^l)
    with no masks; the paper sets r_eval = 1 (Hyperparameters section,
    "Dropout Scale": it makes the evaluation output the expected training
    output under r_train = 1/rho).
  * Static early exit at l' runs layers 0..l'-1 only, i.e. skips l'..L-1, and
    intermediate layer skipping skips a chosen set (Inference Optimizations
    section, Early Exit and Intermediate Layer Skipping): both are an active
    set, active[l] in {0, 1}, applied to every sequence; a skipped layer is
    the identity.
  * Incremental (KV-cached) decoding: the rows at positions pos..pos+n-1 of
    the evaluation forward, computed from those rows alone plus the keys and
    values of positions 0..pos-1 held for each active layer (causal
    attention lets a row see only itself and earlier positions).  Drafting in
    self-speculative decoding (Inference Optimizations section,
    Self-Speculative Decoding: a subset of the model's own layers drafts,
    the full model verifies) is decoding with a smaller active set over the
    cache the full model wrote.

All float64.  Weights as in block.py.
"""

import numpy as np

from . import block


def _r(r_eval, L):
    if r_eval is None:
        return [1.0] * L
    r = np.broadcast_to(np.asarray(r_eval, dtype=np.float64), (L,))
    return [float(v) for v in r]


def eval_forward(X, weights, active, n_heads, eps=1e-5, kind=0, r_eval=None):
    """X [B, S, d] -> (X_L, kv) where kv[l] is None for a skipped layer and
    (K, V), each [B, S, d], the keys and values layer l formed, otherwise."""
    X = np.asarray(X, dtype=np.float64).copy()
    L = len(weights)
    r = _r(r_eval, L)
    kv = [None] * L
    for l in range(L):
        if not active[l]:
            continue
        w = {k: np.asarray(v, dtype=np.float64) for k, v in weights[l].items()}
        K = np.zeros_like(X)
        V = np.zeros_like(X)
        for b in range(X.shape[0]):
            X[b], c = block.forward(X[b], w, r[l], n_heads, eps, kind)
            K[b], V[b] = c["k"], c["v"]
        kv[l] = (K, V)
    return X, kv


def attention_rows(q, K, V, q_pos, n_heads, slopes=None):
    """Attention of queries q [n, d] at positions q_pos [n] over keys and
    values K, V [P, d] at positions 0..P-1: per head softmax over keys j <= its
    position of q.k_j / sqrt(dh) (minus m_h (pos - j) with ALiBi slopes)."""
    n, d = q.shape
    dh = d // n_heads
    P = K.shape[0]
    out = np.zeros((n, d))
    kpos = np.arange(P)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        for i in range(n):
            s = K[:, cols] @ q[i, cols] / np.sqrt(dh)
            if slopes is not None:
                s = s - slopes[h] * (q_pos[i] - kpos)
            s = np.where(kpos <= q_pos[i], s, -np.inf)
            e = np.exp(s - np.max(s))
            out[i, cols] = (e / np.sum(e)) @ V[:, cols]
    return out


def decode(x_new, weights, active, kv, pos, n_heads, eps=1e-5, kind=0, r_eval=None):
    """Rows x_new [B, n, d] at positions pos..pos+n-1 through the active
    layers.  kv[l] = (K, V) with at least pos positions [B, >= pos, d] for
    every active layer (entries past pos are ignored).  Returns (x_out, new_kv)
    where new_kv[l] = (k, v) [B, n, d] of the new rows (None if skipped)."""
    X = np.asarray(x_new, dtype=np.float64).copy()
    B, n, d = X.shape
    L = len(weights)
    r = _r(r_eval, L)
    slopes = block.alibi_slopes(n_heads) if kind == 1 else None
    q_pos = pos + np.arange(n)
    new_kv = [None] * L
    for l in range(L):
        if not active[l]:
            continue
        w = {k: np.asarray(v, dtype=np.float64) for k, v in weights[l].items()}
        kn = np.zeros((B, n, d))
        vn = np.zeros((B, n, d))
        for b in range(B):
            x = X[b]
            h1, _ = block.rmsnorm(x, w["g_attn"], eps)
            qkv = h1 @ w["w_qkv"].T
            q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
            Kc = np.concatenate([kv[l][0][b, :pos], k], axis=0)
            Vc = np.concatenate([kv[l][1][b, :pos], v], axis=0)
            a = attention_rows(q, Kc, Vc, q_pos, n_heads, slopes)
            z = x + r[l] * (a @ w["w_o"].T)
            X[b], _ = block.ffn_forward(z, w, r[l], eps, kind)
            kn[b], vn[b] = k, v
        new_kv[l] = (kn, vn)
    return X, new_kv
