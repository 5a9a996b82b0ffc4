"""Layer and stack forward+backward under per-sequence layer dropout.

Test infrastructure (see the package docstring).

Definition followed (Preliminary section): for layer l at step t,
    H^{l+1}[b] = H^l[b]                                  if M^{l,t}[b] = 0
    H^{l+1}[b] = H^l[b] + r f^l(H^l[b])  (both sub-blocks) if M^{l,t}[b] = 1
with r = res_scale / (1 - p^{l,t}) when rescaling is on (the paper's choice
r_train = 1/rho, rho = 1 - p, Hyperparameters section "Dropout Scale"), and
r = res_scale otherwise.  res_scale is a constant residual multiplier (the
depth multiplier of the parameterisation table; 1 by default).  The same r
multiplies both sub-blocks (transformer form of the training equation).

Sub-layer dropout (Dropout Granularity section, model granularity) draws the
attention and FFN masks independently:
    Z[b]       = H^l[b] + r M_attn[b] f_attn(H^l[b])
    H^{l+1}[b] = Z[b]   + r M_ffn[b]  f_ffn(Z[b])
with the layer's p and r for both; layer dropout is the case M_attn = M_ffn.
Per-batch dropout (tensor granularity) changes only how the masks are drawn
(masks.py); the arithmetic is the same.

Samples are visited in ascending order and each kept sample is processed on
its own; dropped samples are copied bit for bit and their gradient passes
through unchanged.  Weight gradients are sums over kept samples (no 1/B);
they start at zero on every call, so a layer with no kept sample has zero
gradients.
"""

from dataclasses import dataclass

import numpy as np

from . import block
from .masks import masks_granular, n_masks

WEIGHT_KEYS = ("g_attn", "w_qkv", "w_o", "g_mlp", "w_gate_up", "w_down")


@dataclass
class Config:
    n_heads: int
    rms_eps: float = 1e-5
    rescale: bool = True
    res_scale: float = 1.0
    block_kind: int = 0     # 0: RMSNorm/MHA/SwiGLU; 1: ALiBi + squared ReLU (block.py)
    granularity: int = 0    # masks.LAYER_SEQ, SUBLAYER_SEQ, LAYER_BATCH, SUBLAYER_BATCH


def residual_scale(p, cfg):
    """r^{l,t}; only evaluated for layers with at least one kept sample."""
    p = float(np.float32(p))
    return cfg.res_scale / (1.0 - p) if cfg.rescale else cfg.res_scale


def _as64(w):
    return {k: np.asarray(w[k], dtype=np.float64) for k in WEIGHT_KEYS}


def _sub_masks(keep_row):
    """(attention mask, FFN mask) from a layer mask [B] or a pair [2, B]."""
    k = np.asarray(keep_row)
    if k.ndim == 1:
        return k, k
    return k[0], k[1]


def layer_forward(X, w, keep_row, p, cfg):
    """X [B, S, d] float64 -> (X_next, ctx).  keep_row: uint8[B] (one mask for
    both sub-blocks) or uint8[2, B] (attention mask, FFN mask)."""
    w = _as64(w)
    X = np.asarray(X, dtype=np.float64)
    keep_a, keep_f = _sub_masks(keep_row)
    X_next = X.copy()
    cache_a, cache_f = {}, {}
    r = None
    for b in range(X.shape[0]):
        if not (keep_a[b] or keep_f[b]):
            continue                      # dropped: H^{l+1}[b] = H^l[b]
        if r is None:
            r = residual_scale(p, cfg)
        z = X[b]
        if keep_a[b]:
            z, cache_a[b] = block.attn_forward(z, w, r, cfg.n_heads, cfg.rms_eps, cfg.block_kind)
        if keep_f[b]:
            z, cache_f[b] = block.ffn_forward(z, w, r, cfg.rms_eps, cfg.block_kind)
        X_next[b] = z
    return X_next, dict(cache_a=cache_a, cache_f=cache_f, r=r, w=w)


def layer_backward(ctx, G, cfg):
    """G = dL/dH^{l+1} [B, S, d] -> (dL/dH^l, grads summed over kept samples)."""
    G = np.asarray(G, dtype=np.float64)
    G_prev = G.copy()
    grads = {k: np.zeros(v.shape) for k, v in ctx["w"].items()}
    for b in sorted(set(ctx["cache_a"]) | set(ctx["cache_f"])):
        g = G[b]
        if b in ctx["cache_f"]:
            g, gb = block.ffn_backward(ctx["cache_f"][b], g, ctx["w"], ctx["r"])
            for k in gb:
                grads[k] += gb[k]
        if b in ctx["cache_a"]:
            g, gb = block.attn_backward(ctx["cache_a"][b], g, ctx["w"], ctx["r"], cfg.n_heads)
            for k in gb:
                grads[k] += gb[k]
        G_prev[b] = g
    return G_prev, grads


def stack_forward(X0, weights, ps, seed, step, cfg, keep=None):
    """Forward through all layers; returns (X_L, ctxs, keep, idx, count).
    keep, idx are [L, B] and count [L] for layer granularity, [L, 2, B] and
    [L, 2] for sub-layer granularity (attention row, then FFN row).  keep of
    that shape overrides the Philox masks when given."""
    B = X0.shape[0]
    L = len(weights)
    nm = n_masks(cfg.granularity)
    if keep is None:
        keep, idx, count = masks_granular(ps, seed, step, B, cfg.granularity)
    else:
        keep = np.asarray(keep, dtype=np.uint8).reshape(L, nm, B)
        idx = np.full((L, nm, B), -1, dtype=np.int32)
        count = np.zeros((L, nm), dtype=np.int32)
        for l in range(L):
            for m in range(nm):
                kept = np.nonzero(keep[l, m])[0]
                idx[l, m, :len(kept)] = kept
                count[l, m] = len(kept)
    if nm == 1:
        keep, idx, count = keep[:, 0], idx[:, 0], count[:, 0]
    X = np.asarray(X0, dtype=np.float64)
    ctxs = []
    for l in range(L):
        X, ctx = layer_forward(X, weights[l], keep[l], ps[l], cfg)
        ctxs.append(ctx)
    return X, ctxs, keep, idx, count


def stack_step(X0, weights, ps, seed, step, G_L, cfg, keep=None):
    """One forward+backward step.  Returns dict with X_L, G_0 (dL/dX^0),
    grads (list per layer), keep, idx, count."""
    X_L, ctxs, keep, idx, count = stack_forward(X0, weights, ps, seed, step, cfg, keep)
    G = np.asarray(G_L, dtype=np.float64)
    grads = [None] * len(weights)
    for l in reversed(range(len(weights))):
        G, grads[l] = layer_backward(ctxs[l], G, cfg)
    return dict(X_L=X_L, G_0=G, grads=grads, keep=keep, idx=idx, count=count)
