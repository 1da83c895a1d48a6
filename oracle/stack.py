"""CPU oracle for one denoising step of a mask-aware, K/V-cached block stack.

TEST INFRASTRUCTURE. Only the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this module. It shares no code with the
GPU path and imports nothing from it.

What is computed (InstGenIE, arXiv 2505.20600):

* Sec. 3.1 ("How does it work"): every operator of a transformer block except
  the attention score/softmax is token-wise, so per-token work can be limited
  to the masked tokens.
* Sec. 3.1 ("Mask-aware attention", Fig. 5): only the masked tokens are
  queried; they attend over the keys/values of all tokens (the LLM-decoding
  analogy at the end of that subsection).
* Sec. 3.1 ("Alternative approaches", Fig. 7): the K/V-caching variant. Each
  block's K and V of the unmasked tokens come from a cache of an earlier
  inference of the same template; the masked rows of K and V are recomputed.
  The unmasked rows of the stack's output are replenished from the cached
  final hidden state.
* Table 1: the per-layer work of projections, feed-forward and
  ``QK^T / sqrt(.)`` is proportional to the masked-row count.

The block is pre-LayerNorm: LN -> QKV projection -> multi-head attention ->
out projection + residual -> LN -> Linear/GELU/Linear + residual. The paper
omits LayerNorm, GELU and dropout from its figure (Fig. 5 caption); the
readings taken for them (pre-LN, eps in the model description, exact erf-GELU,
no dropout at inference, attention scale 1/sqrt(head_dim)) are the block of
standard DiT stacks.

Precision: everything is evaluated in float64. For the bf16 workloads,
``bf16_round`` (round to nearest even) is applied at each point where the GPU
holds a value in bf16 storage: LN outputs; Q, K, V; the attention output O;
the out-projection result H (residual included); the GELU output U; the block
output. Between those points there is no rounding. The fp32 workload uses no
rounding at all. The switch ``round_p`` (bf16 workloads only, off by default)
also rounds the softmax weights to bf16 before the PV product, the operand
type of a bf16 matrix unit; the normaliser is then the sum of the same
rounded weights, so the weights applied still sum to one.

Arrays: hidden ``[B][T][d]``, K/V ``[B][T][2][d]`` (K then V per token), mask
``uint8 [B][N]`` over the image grid (nonzero = masked). Token ``t`` of a
request is ``n_text + row * grid_w + col`` for image cells (raster order,
Sec. 2.1) and ``0..n_text-1`` for text tokens, which are always recomputed.
Linear weights are ``[out][in]``.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

BF16_MAX = float.fromhex("0x1.fep127")


def bf16_round(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits. For |x| in [2^(e-1), 2^e) one unit in
    the last place is 2^(e-8); below the normal range the spacing stays at
    2^-133. Rounding is done in float64, where scaling by a power of two and
    ``np.rint`` (ties to even) are exact. Overflow gives +-inf, NaN stays NaN.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x) & (x != 0)
    xf = x[fin]
    _, e = np.frexp(xf)
    q = np.maximum(e - 8, -133)
    r = np.ldexp(np.rint(np.ldexp(xf, -q)), q)
    r = np.where(np.abs(r) > BF16_MAX, np.copysign(np.inf, r), r)
    out[fin] = r
    return out


def _identity(x):
    return np.asarray(x, dtype=np.float64)


def rounder(dtype: str):
    return bf16_round if dtype == "bf16" else _identity


def layer_norm(x, gamma, beta, eps: float) -> np.ndarray:
    """(x - mean) / sqrt(var + eps) * gamma + beta over the last axis; population variance."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)


def gelu(x) -> np.ndarray:
    """Exact GELU: x * Phi(x) with the standard normal CDF Phi(x) = (1 + erf(x / sqrt 2)) / 2."""
    x = np.asarray(x, dtype=np.float64)
    return x * 0.5 * (1.0 + erf(x / np.sqrt(2.0)))


def attention_head(q, k, v, scale: float, round_p: bool = False) -> np.ndarray:
    """softmax(q k^T * scale) v for one head; full softmax over every key (Sec. 3.1).

    With ``round_p`` the unnormalised weights ``exp(s - max s)`` (the largest is
    exactly 1) are rounded to bf16 before they multiply V, and each row is
    divided by the sum of its rounded weights.
    """
    s = (np.asarray(q, np.float64) @ np.asarray(k, np.float64).T) * scale
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    if round_p:
        p = bf16_round(p)
        return (p @ np.asarray(v, np.float64)) / p.sum(axis=1, keepdims=True)
    p /= p.sum(axis=1, keepdims=True)
    return p @ np.asarray(v, np.float64)


def linear(x, w, b) -> np.ndarray:
    """x W^T + b with W stored [out][in]."""
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T + np.asarray(b, np.float64)


# ---------------------------------------------------------------------------
# Mask -> masked-row index (token selection of Sec. 3.1, "extract the matrix of
# masked tokens")
# ---------------------------------------------------------------------------


def masked_tokens(mask_b, n_text: int) -> np.ndarray:
    """Ascending token ids that are recomputed for one request: all text tokens, then masked cells."""
    cells = [n for n in range(len(mask_b)) if mask_b[n] != 0]
    return np.array(list(range(n_text)) + [n_text + n for n in cells], dtype=np.int64)


def compact(mask, n_text: int = 0, dual_stream: bool = False) -> dict:
    """Packed masked-row layout shared by every kernel of the step.

    Returns ``tokens`` (per request, ascending), ``rows`` (flat ``b*T + t`` of
    each packed row), ``seg_start`` / ``seg_req`` (packed segments) and
    ``inv`` (``[B*T]``: packed row of a token, -1 if not recomputed).

    Packing: request-major for a single weight set. With a separate text
    weight set the text rows of all requests come first (request-major),
    followed by the image rows of all requests (request-major), so each weight
    set owns one contiguous packed range.
    """
    mask = np.asarray(mask)
    B, N = mask.shape
    T = n_text + N
    tokens = [masked_tokens(mask[b], n_text) for b in range(B)]
    segs = []  # (request, token list)
    if dual_stream and n_text > 0:
        for b in range(B):
            segs.append((b, tokens[b][tokens[b] < n_text]))
        for b in range(B):
            segs.append((b, tokens[b][tokens[b] >= n_text]))
    else:
        for b in range(B):
            segs.append((b, tokens[b]))
    rows, seg_start, seg_req = [], [0], []
    for b, toks in segs:
        rows.extend(int(b * T + t) for t in toks)
        seg_start.append(len(rows))
        seg_req.append(b)
    inv = np.full(B * T, -1, np.int64)
    for m, r in enumerate(rows):
        inv[r] = m
    return {
        "tokens": tokens,
        "rows": np.array(rows, np.int64),
        "seg_start": np.array(seg_start, np.int64),
        "seg_req": np.array(seg_req, np.int64),
        "inv": inv,
        "M": len(rows),
    }


# ---------------------------------------------------------------------------
# One block over a subset of one request's tokens
# ---------------------------------------------------------------------------


def _weights_for(layer_w, is_text: bool):
    if isinstance(layer_w, (tuple, list)):
        return layer_w[1] if is_text else layer_w[0]
    return layer_w


def _token_wise(fn, x_rows, toks, layer_w, n_text):
    """Apply a token-wise function with the weight set of each row's stream."""
    x_rows = np.asarray(x_rows, np.float64)
    is_text = np.asarray(toks) < n_text
    out = None
    for flag in (False, True):
        sel = is_text == flag
        if not sel.any():
            continue
        y = fn(x_rows[sel], _weights_for(layer_w, bool(flag)))
        if out is None:
            out = np.empty((x_rows.shape[0],) + y.shape[1:], np.float64)
        out[sel] = y
    return out


def block_rows(x_rows, toks, layer_w, kv_b, shape, rnd, round_p: bool = False, return_h: bool = False):
    """One pre-LN block for the rows ``toks`` of one request.

    ``x_rows [m][d]`` are the hidden rows of tokens ``toks``; ``kv_b [T][2][d]``
    holds K/V for every token of the request (cache contents). The K/V of
    ``toks`` are recomputed from ``x_rows`` and replace the cached rows
    (Fig. 7); every row in ``toks`` then queries all ``T`` keys (Fig. 5).
    ``round_p`` rounds the softmax weights to bf16 (bf16 workloads only; see
    ``attention_head``).

    Returns ``(x_out [m][d], kv_work [T][2][d])``, and with ``return_h`` also the
    rows' value between the two residual additions, ``H = x + O W_o^T + b_o``.
    """
    d, h = shape.d_model, shape.n_heads
    hd = d // h
    eps = shape.ln_eps
    nt = shape.n_text

    def pre_attn(x, w):
        a = rnd(layer_norm(x, w["ln1_g"], w["ln1_b"], eps))
        return rnd(linear(a, w["w_qkv"], w["b_qkv"]))

    qkv = _token_wise(pre_attn, x_rows, toks, layer_w, nt)
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]

    kv_work = np.array(kv_b, dtype=np.float64, copy=True)
    kv_work[toks, 0, :] = k
    kv_work[toks, 1, :] = v

    o = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    rp = bool(round_p) and shape.dtype == "bf16"
    for j in range(h):
        cs = slice(j * hd, (j + 1) * hd)
        o[:, cs] = attention_head(q[:, cs], kv_work[:, 0, cs], kv_work[:, 1, cs], scale, rp)
    o = rnd(o)

    def post_attn(pair, w):
        x, oo = pair[:, :d], pair[:, d:]
        hh = rnd(x + linear(oo, w["w_o"], w["b_o"]))
        a2 = rnd(layer_norm(hh, w["ln2_g"], w["ln2_b"], eps))
        u = rnd(gelu(linear(a2, w["w_1"], w["b_1"])))
        return np.concatenate([rnd(hh + linear(u, w["w_2"], w["b_2"])), hh], axis=1)

    out = _token_wise(post_attn, np.concatenate([x_rows, o], axis=1), toks, layer_w, nt)
    if return_h:
        return out[:, :d], kv_work, out[:, d:]
    return out[:, :d], kv_work


# ---------------------------------------------------------------------------
# Stacks
# ---------------------------------------------------------------------------


def dense_stack(x, weights, shape, round_p: bool = False):
    """Full computation over every token (the Fig. 5 top flow), layer by layer.

    Returns ``(y [B][T][d], kv [L][B][T][2][d])``; ``kv`` is what a cache of
    this inference holds (Fig. 7), ``y`` its final hidden state.
    """
    rnd = rounder(shape.dtype)
    x = np.asarray(x, np.float64)
    B, T, d = x.shape
    toks = np.arange(T)
    y = np.empty_like(x)
    kv = np.empty((len(weights), B, T, 2, d), np.float64)
    for b in range(B):
        xb = x[b]
        for l, w in enumerate(weights):
            xb, kvw = block_rows(xb, toks, w, np.zeros((T, 2, d)), shape, rnd, round_p)
            kv[l, b] = kvw
        y[b] = xb
    return y, kv


def masked_stack(x, mask, kv_cache, y_cache, weights, shape, return_kv: bool = False,
                 dense_prefix: int = 0, round_p: bool = False):
    """Mask-aware step with K/V caching (Sec. 3.1, Fig. 5 bottom and Fig. 7).

    ``kv_cache[l]`` is ``[B][T][2][d]`` (rows of recomputed tokens are ignored),
    ``y_cache [B][T][d]`` the cached final hidden state. Only recomputed rows
    are touched; the output's other rows are copied from ``y_cache``.
    With ``return_kv`` the per-layer working K/V (cache with fresh rows) is
    returned too.

    ``dense_prefix = k`` computes blocks ``0..k-1`` over every token without
    the cache (the "compute all tokens" choice of the bubble-free pipeline,
    Sec. 4.2 and Alg. 1) and blocks ``k..L-1`` with the cache. With K/V
    caching a block can only skip the cache if all earlier blocks did (only
    then do the unmasked tokens' hidden states exist), so the choice is a
    prefix. ``round_p``: see ``attention_head``.
    """
    rnd = rounder(shape.dtype)
    x = np.asarray(x, np.float64)
    B, T, d = x.shape
    L = len(weights)
    k = int(dense_prefix)
    if not 0 <= k <= L:
        raise ValueError("dense_prefix out of range")
    y = np.array(y_cache, dtype=np.float64, copy=True)
    kv_out = [] if return_kv else None
    if return_kv:
        kv_out = np.empty((L, B, T, 2, d), np.float64)
    all_toks = np.arange(T)
    for b in range(B):
        toks = masked_tokens(mask[b], shape.n_text)
        if toks.size == 0:
            if return_kv:
                for l in range(L):
                    kv_out[l, b] = kv_cache[l][b]
            continue
        xb = x[b]
        for l in range(k):
            xb, kvw = block_rows(xb, all_toks, weights[l], np.zeros((T, 2, d)), shape, rnd, round_p)
            if return_kv:
                kv_out[l, b] = kvw
        xm = xb[toks]
        for l in range(k, L):
            xm, kvw = block_rows(xm, toks, weights[l], kv_cache[l][b], shape, rnd, round_p)
            if return_kv:
                kv_out[l, b] = kvw
        y[b, toks] = xm
    if return_kv:
        return y, kv_out
    return y


def masked_rows_of_stack(x, mask, kv_cache, weights, shape, b: int, dense_prefix: int = 0,
                         round_p: bool = False):
    """Final hidden rows of request ``b`` for its recomputed tokens only: ``(toks, rows)``.

    The same steps as ``masked_stack`` for that one request (requests never
    attend across each other): blocks ``0..k-1`` over every token of the
    request (``k = dense_prefix``), then the cached blocks over its recomputed
    rows. ``kv_cache[l]`` only needs ``[b]`` indexing, so a caller may pass
    per-layer arrays of any batch size that hold request ``b``.
    """
    rnd = rounder(shape.dtype)
    k = int(dense_prefix)
    L = len(weights)
    if not 0 <= k <= L:
        raise ValueError("dense_prefix out of range")
    toks = masked_tokens(mask[b], shape.n_text)
    if toks.size == 0:
        return toks, np.zeros((0, shape.d_model))
    xb = np.asarray(x[b], np.float64)
    T, d = xb.shape
    all_toks = np.arange(T)
    for l in range(k):
        xb, _ = block_rows(xb, all_toks, weights[l], np.zeros((T, 2, d)), shape, rnd, round_p)
    xm = xb[toks]
    for l in range(k, L):
        xm, _ = block_rows(xm, toks, weights[l], kv_cache[l][b], shape, rnd, round_p)
    return toks, xm


# ---------------------------------------------------------------------------
# Work accounting (Table 1)
# ---------------------------------------------------------------------------


def layer_flops(m_rows: int, n_tokens: int, d: int, mlp_mult: int = 4) -> int:
    """Algorithmic FLOPs of one block for ``m_rows`` recomputed rows of one request.

    Projections (QKV 3d^2, out d^2) and feed-forward (2 * mlp_mult * d^2)
    scale with the row count, and so do ``QK^T`` and ``PV`` over all
    ``n_tokens`` keys (Table 1); one multiply-add = 2 FLOPs.
    """
    gemm = 2 * m_rows * d * d * (3 + 1 + 2 * mlp_mult)
    attn = 2 * 2 * m_rows * n_tokens * d
    return gemm + attn
