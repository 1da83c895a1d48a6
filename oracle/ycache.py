"""Y-caching variant of the masked step (test infrastructure only).

Sec. 3.1, "How does it work" and Fig. 5 (bottom): the paper's primary way of
reusing a template's inference. Per block, the cache holds the block's input
activations of the unmasked tokens, from a prior inference of the same
template (cache shape (B, (1 - m) L, H) in Table 1). The masked rows are
extracted, projected into Q and carried through the block; the unmasked rows
are replenished from the cache, which is all a block needs of them: their K
and V, the only place unmasked tokens enter the masked rows' computation.
Those are recomputed here from the cached activations with the block's own
LayerNorm and K/V projection. The final hidden state is replenished from the
cached output as in the K/V variant.

Fig. 7 caches the K and V that this variant recomputes, so for a K/V cache
derived from the same activations the two variants give the same result
(tested).

Arrays: ``yin_cache`` is ``[L][B][N][d]`` over the image grid (rows of
recomputed tokens are never read; text tokens are always recomputed), the
rest as in ``oracle.stack``.
"""
from __future__ import annotations

import numpy as np

from .stack import block_rows, layer_norm, linear, masked_tokens, rounder


def _image_weights(layer_w):
    return layer_w[0] if isinstance(layer_w, (tuple, list)) else layer_w


def kv_of_inputs(x_rows, layer_w, shape, rnd) -> np.ndarray:
    """K and V of image-token rows from their block input: LN1, then the K/V part
    of the QKV projection, with the bf16 rounding points of the block. Returns
    ``[m][2][d]``."""
    w = _image_weights(layer_w)
    d = shape.d_model
    a = rnd(layer_norm(np.asarray(x_rows, np.float64), w["ln1_g"], w["ln1_b"], shape.ln_eps))
    qkv = rnd(linear(a, w["w_qkv"], w["b_qkv"]))
    return np.stack([qkv[:, d:2 * d], qkv[:, 2 * d:]], axis=1)


def kv_cache_of_inputs(yin_cache, mask, weights, shape) -> np.ndarray:
    """The Fig. 7 cache that holds what Y-caching recomputes: K/V of the unmasked
    image tokens from ``yin_cache``; every other row zero. ``[L][B][T][2][d]``."""
    rnd = rounder(shape.dtype)
    yin = np.asarray(yin_cache, np.float64)
    L, B, N, d = yin.shape
    T = shape.n_text + N
    kv = np.zeros((L, B, T, 2, d), np.float64)
    for l in range(L):
        for b in range(B):
            un = np.flatnonzero(np.asarray(mask[b]) == 0)
            if un.size:
                kv[l, b, shape.n_text + un] = kv_of_inputs(yin[l, b, un], weights[l], shape, rnd)
    return kv


def masked_stack_y(x, mask, yin_cache, y_cache, weights, shape, dense_prefix: int = 0,
                   round_p: bool = False):
    """Mask-aware step with Y caching.

    Blocks ``0..k-1`` (``k = dense_prefix``) run over every token without the
    cache (Sec. 4.2, Alg. 1: with per-block input caches a block can skip its
    cache only while every earlier block did, so the choice is again a
    prefix); blocks ``k..L-1`` recompute the K/V of the unmasked image tokens
    from ``yin_cache[l]`` and everything else for the recomputed rows only.
    ``round_p``: the bf16 softmax-weight switch of ``oracle.stack.attention_head``.
    """
    rnd = rounder(shape.dtype)
    x = np.asarray(x, np.float64)
    B, T, d = x.shape
    L = len(weights)
    k = int(dense_prefix)
    if not 0 <= k <= L:
        raise ValueError("dense_prefix out of range")
    y = np.array(y_cache, dtype=np.float64, copy=True)
    all_toks = np.arange(T)
    for b in range(B):
        toks = masked_tokens(mask[b], shape.n_text)
        if toks.size == 0:
            continue
        un = np.flatnonzero(np.asarray(mask[b]) == 0)
        xb = x[b]
        for l in range(k):
            xb, _ = block_rows(xb, all_toks, weights[l], np.zeros((T, 2, d)), shape, rnd, round_p)
        xm = xb[toks]
        for l in range(k, L):
            kv_b = np.zeros((T, 2, d), np.float64)
            if un.size:
                kv_b[shape.n_text + un] = kv_of_inputs(np.asarray(yin_cache[l][b], np.float64)[un],
                                                       weights[l], shape, rnd)
            xm, _ = block_rows(xm, toks, weights[l], kv_b, shape, rnd, round_p)
        y[b, toks] = xm
    return y


def dense_inputs(x, weights, shape, round_p: bool = False) -> np.ndarray:
    """Input hidden state of every block of the dense flow (Fig. 5 top), image
    tokens only: what a Y cache of this inference holds. ``[L][B][N][d]``."""
    rnd = rounder(shape.dtype)
    x = np.asarray(x, np.float64)
    B, T, d = x.shape
    L = len(weights)
    nt = shape.n_text
    out = np.empty((L, B, T - nt, d), np.float64)
    toks = np.arange(T)
    for b in range(B):
        xb = x[b]
        for l, w in enumerate(weights):
            out[l, b] = xb[nt:]
            xb, _ = block_rows(xb, toks, w, np.zeros((T, 2, d)), shape, rnd, round_p)
    return out
