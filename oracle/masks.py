"""Per-sequence layer-dropout masks and the kept-sample lists.

Test infrastructure (see the package docstring).

The mask M^{l,t} in {0,1}^B is Bernoulli(1 - p^{l,t}), one draw per sequence
b, shared by the attention and FFN sub-blocks of the layer (Preliminary
section, layer-dropout training equation and its per-sequence case form;
Dropout Granularity: layer granularity, per-sequence tensor granularity).
M = 1 keeps the sequence.

Reading of the Bernoulli draw (the paper fixes no generator):
  w    = word 0 of Philox4x64-10, counter (b, l, t, 0), key (seed, 0)
  thr  = floor(p * 2^64) for 0 < p < 1      (exact in binary64)
  drop = p >= 1  or  (p > 0 and w < thr)
so P(drop) = thr / 2^64, within 2^-64 of p, and p = 0 / p = 1 are exact.

The kept list is the ascending set { b : M[b] = 1 } -- the sequences on which
f is executed in the efficient form of the method (Preliminary section, the
paragraph after the per-sequence case form).
"""

import math

import numpy as np

from .philox import block_words, mask_word


def threshold(p):
    """Integer drop threshold for a float32 rate; None means drop all."""
    p = float(np.float32(p))
    if math.isnan(p):
        raise ValueError("p is NaN")
    if p >= 1.0:
        return None
    if p <= 0.0:
        return 0
    return int(math.floor(math.ldexp(p, 64)))


def keep_bits(p, seed, step, layer, batch):
    """uint8[batch]: 1 where sample b keeps layer `layer` at step `step`."""
    thr = threshold(p)
    if thr is None:
        return np.zeros(batch, dtype=np.uint8)
    w = mask_word(np.arange(batch, dtype=np.uint64), layer, step, seed)
    # uint64 against uint64: exact on the full 64-bit range.
    return np.where(w < np.uint64(thr), 0, 1).astype(np.uint8)


def compact(keep_row):
    """Ascending kept indices, padded with -1 to the batch size, and the count."""
    kept = [b for b in range(len(keep_row)) if keep_row[b]]
    idx = np.full(len(keep_row), -1, dtype=np.int32)
    idx[:len(kept)] = kept
    return idx, len(kept)


def masks(ps, seed, step, batch, first_layer=0):
    """keep uint8[L,B], idx int32[L,B] (ascending, -1 padded), count int32[L]
    for layers first_layer .. first_layer+L-1."""
    ps = np.asarray(ps, dtype=np.float32)
    L = len(ps)
    keep = np.zeros((L, batch), dtype=np.uint8)
    idx = np.full((L, batch), -1, dtype=np.int32)
    count = np.zeros(L, dtype=np.int32)
    for i in range(L):
        keep[i] = keep_bits(ps[i], seed, step, first_layer + i, batch)
        idx[i], count[i] = compact(keep[i])
    return keep, idx, count


# ------------------------------------------------------------ granularity
# Dropout Granularity section: model granularity (one mask per layer shared by
# both sub-blocks, or independent attention and FFN masks: sub-layer dropout)
# and tensor granularity (one draw per sequence, or one draw per layer and step
# shared by the whole batch: per-batch dropout).  Encoded as two bits:
LAYER_SEQ = 0        # layer granularity, per sequence (the paper's choice)
SUBLAYER_SEQ = 1     # M_attn, M_ffn drawn independently, per sequence
LAYER_BATCH = 2      # one draw per (layer, step) for all sequences
SUBLAYER_BATCH = 3   # independent attention / FFN draws, per (layer, step)

# Reading of the draws (the paper fixes no generator):
#   per sequence: block (b, l, t, 0); per batch: block (0, l, t, 1); key (seed, 0)
#   the attention mask (and the layer mask) takes word 0 of the block, the
#   FFN mask of sub-layer dropout takes word 1.  So the attention mask of
#   sub-layer dropout is the layer-dropout mask, and both sub-block masks are
#   Bernoulli(1 - p^{l,t}) with the layer's rate.


def n_masks(granularity):
    """Masks per layer: 2 (attention, FFN) for sub-layer dropout, else 1."""
    if granularity not in (LAYER_SEQ, SUBLAYER_SEQ, LAYER_BATCH, SUBLAYER_BATCH):
        raise ValueError(f"unknown granularity {granularity}")
    return 2 if granularity & 1 else 1


def keep_bits_granular(p, seed, step, layer, batch, granularity):
    """uint8[n_masks, batch]: row 0 the attention (or whole-layer) mask, row 1
    the FFN mask of sub-layer dropout."""
    nm = n_masks(granularity)
    thr = threshold(p)
    if thr is None:
        return np.zeros((nm, batch), dtype=np.uint8)
    if granularity & 2:
        words = block_words(0, layer, step, seed, 1)
        rows = [np.full(batch, words[m], dtype=np.uint64) for m in range(nm)]
    else:
        words = block_words(np.arange(batch, dtype=np.uint64), layer, step, seed, 0)
        rows = [words[m] for m in range(nm)]
    return np.stack([np.where(w < np.uint64(thr), 0, 1) for w in rows]).astype(np.uint8)


def masks_granular(ps, seed, step, batch, granularity, first_layer=0):
    """keep uint8[L, n_masks, B], idx int32[L, n_masks, B], count int32[L, n_masks]."""
    ps = np.asarray(ps, dtype=np.float32)
    L, nm = len(ps), n_masks(granularity)
    keep = np.zeros((L, nm, batch), dtype=np.uint8)
    idx = np.full((L, nm, batch), -1, dtype=np.int32)
    count = np.zeros((L, nm), dtype=np.int32)
    for i in range(L):
        keep[i] = keep_bits_granular(ps[i], seed, step, first_layer + i, batch, granularity)
        for m in range(nm):
            idx[i, m], count[i, m] = compact(keep[i, m])
    return keep, idx, count
