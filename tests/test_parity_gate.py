"""The per-block bf16 gate (tests/parity_gate) admits a correct implementation in
another precision and rejects plausible mistakes.

* A correct block evaluated the way the matrix units do it (float32
  accumulation, bf16 rounding at the same storage points, online softmax over
  64-key tiles with a running maximum that is only raised when it grows by more
  than 2^8, softmax weights rounded to bf16 against that running maximum, the
  normaliser summed from the same rounded weights) stays within 2e-2
  element-wise of the oracle with ``round_p``, for head_dim 64 / 72 / 128.
* The oracle with a planted mistake (on the CPU: a dropped ragged key tail, a
  wrong softmax scale (that of the zero-padded head_dim 80 for head_dim 72; an
  exp2 without the log2(e) prescale otherwise), keys misaligned with their
  values by one token, a dropped out-projection bias) fails the same gate
  against the unaltered oracle.

Inputs as in the GPU per-block tests: weights N(0, 0.05), random LayerNorm
affine parameters, hidden states N(0, 1), a random cache. At this scale a
correct float32 block stays at about 1.45e-2 while every planted mistake
reaches 3e-2 or more; at 0.06-0.08 the mistakes show more but correct blocks
reach 1.6-2.0e-2 (the Q/K roundings move a sharper softmax).
"""
import numpy as np
import pytest
from scipy.special import erf

import oracle
from oracle import stack as OS
from paper_2505_20600_amd import workloads as W
from tests import parity_gate as PG

STD = 0.05
SHAPES = [
    W.ModelShape("hd64_T256", 1, 256, 4, 4, 16, 16, dtype="bf16"),
    W.ModelShape("hd72_T144", 1, 576, 8, 4, 12, 12, dtype="bf16"),
    W.ModelShape("hd128_T192", 1, 256, 2, 4, 12, 16, dtype="bf16"),
]
RATIOS = (0.05, 0.45, 1.0)


def _b16(a):
    return OS.bf16_round(np.asarray(a, np.float64)).astype(np.float32)


def _ln32(x, g, b, eps):
    mu = x.mean(-1, keepdims=True, dtype=np.float32)
    var = ((x - mu) ** 2).mean(-1, keepdims=True, dtype=np.float32)
    return (x - mu) / np.sqrt(var + np.float32(eps)) * g + b


def _attention32(q, k, v, scale, tile=64, lazy_log2=8.0):
    c = np.float32(scale * np.log2(np.e))
    m = np.full(q.shape[0], -np.inf, np.float32)
    l = np.zeros(q.shape[0], np.float32)
    o = np.zeros((q.shape[0], v.shape[1]), np.float32)
    for t0 in range(0, k.shape[0], tile):
        s = q @ k[t0:t0 + tile].T
        m_new = np.maximum(m, s.max(1))
        if np.any((m_new - m) * c > lazy_log2):
            corr = np.where(np.isinf(m), 0.0, np.exp2((m - m_new) * c)).astype(np.float32)
            o *= corr[:, None]
            l *= corr
            m = m_new
        p = _b16(np.exp2(s * c - (m * c)[:, None]))
        l += p.sum(1)
        o += p @ v[t0:t0 + tile]
    return o / l[:, None]


def _block32(x, toks, w, kv_b, shape):
    """One block in float32 with bf16 storage points (an implementation other than the oracle)."""
    f = {k: np.asarray(v, np.float32) for k, v in w.items()}
    d, h = shape.d_model, shape.n_heads
    hd = d // h
    a = _b16(_ln32(np.asarray(x, np.float32), f["ln1_g"], f["ln1_b"], shape.ln_eps))
    qkv = _b16(a @ f["w_qkv"].T + f["b_qkv"])
    kv = np.array(kv_b, np.float32)
    kv[toks, 0], kv[toks, 1] = qkv[:, d:2 * d], qkv[:, 2 * d:]
    o = np.empty((len(toks), d), np.float32)
    for j in range(h):
        c = slice(j * hd, (j + 1) * hd)
        o[:, c] = _attention32(qkv[:, c], kv[:, 0, c], kv[:, 1, c], 1.0 / np.sqrt(hd))
    hh = _b16(np.asarray(x, np.float32) + _b16(o) @ f["w_o"].T + f["b_o"])
    pre = _b16(_ln32(hh, f["ln2_g"], f["ln2_b"], shape.ln_eps)) @ f["w_1"].T + f["b_1"]
    u = _b16(pre * np.float32(0.5) * (1 + erf(pre / np.sqrt(2)).astype(np.float32)))
    return _b16(hh + u @ f["w_2"].T + f["b_2"])


def _case(shape, ratio):
    ws = W.stack_weights(shape, 33, random_ln=True, std=STD)
    x = W.template_hidden(shape, 33)[0]
    kv = W.synthetic_kv_cache(shape, 33, 0)[0]
    n = shape.n_image
    toks = np.sort(np.random.default_rng(5).choice(n, max(1, int(round(ratio * n))), replace=False))
    return ws[0], x[toks], toks, kv


def _ref(w, x, toks, kv, shape):
    """The oracle's block output and its value between the two residual additions."""
    out, _, h = oracle.block_rows(x, toks, w, kv, shape, oracle.bf16_round, round_p=True, return_h=True)
    return out, h


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
@pytest.mark.parametrize("ratio", RATIOS)
def test_float32_block_passes_the_block_gate(shape, ratio):
    w, x, toks, kv = _case(shape, ratio)
    ref, h = _ref(w, x, toks, kv, shape)
    ok, e1, e2, lim = PG.check(_block32(x, toks, w, kv, shape), ref, "bf16", 1, inp=h)
    assert ok, (e1, e2, lim)


def _planted(name, shape):
    """attention_head replacements (and weight edits) that each plant one mistake."""
    orig = OS.attention_head
    hd = shape.head_dim
    T = shape.n_tokens
    tail = T % 64 or 16
    if name == "dropped key tail":
        return lambda q, k, v, s, rp=False: orig(q, k[:T - tail], v[:T - tail], s, rp), None
    if name == "wrong softmax scale":
        if hd % 16:      # the scale of the head_dim padded to the matrix-unit step
            return lambda q, k, v, s, rp=False: orig(q, k, v, 1.0 / np.sqrt((hd + 15) // 16 * 16), rp), None
        # exp2 of scores that miss the log2(e) prescale: exp(s ln 2)
        return lambda q, k, v, s, rp=False: orig(q, k, v, s * np.log(2.0), rp), None
    if name == "keys one token off":
        return lambda q, k, v, s, rp=False: orig(q, np.roll(k, 1, axis=0), v, s, rp), None
    if name == "out-projection bias dropped":
        return orig, "b_o"
    raise KeyError(name)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
@pytest.mark.parametrize("mistake", ["dropped key tail", "wrong softmax scale", "keys one token off",
                                     "out-projection bias dropped"])
def test_planted_mistake_fails_the_block_gate(shape, mistake, monkeypatch):
    for ratio in RATIOS:
        w, x, toks, kv = _case(shape, ratio)
        good, h = _ref(w, x, toks, kv, shape)
        fn, zero = _planted(mistake, shape)
        monkeypatch.setattr(OS, "attention_head", fn)
        wb = dict(w)
        if zero:
            wb[zero] = np.zeros_like(w[zero])
        bad = _ref(wb, x, toks, kv, shape)[0]
        monkeypatch.setattr(OS, "attention_head", oracle.attention_head)
        ok, e1, e2, lim = PG.check(bad, good, "bf16", 1, inp=h)
        assert not ok, f"{mistake} at ratio {ratio} passed: {e1:.3e} / {e2:.3e}"


def test_stack_bound_grows_with_the_square_root_of_depth():
    assert PG.tol("bf16", 1) == 2e-2
    assert PG.tol("bf16", 4) == pytest.approx(4e-2)
    assert PG.tol("fp32", 1) == 1e-4
    with pytest.raises(ValueError):
        PG.tol("bf16", 0)


@pytest.mark.parametrize("d,heads,grid,seed", [(768, 12, 32, 4), (1152, 16, 24, 3)])
def test_two_correct_implementations_drift_within_the_stack_bound(d, heads, grid, seed):
    """The float64 oracle and the float32 block above through 28 blocks of a workload-like
    stack (weights N(0, 0.02), LayerNorm 1/0, 10% of the tokens recomputed, a random
    cache): at every depth both measures stay within 2e-2 sqrt(L), and after 28 blocks
    the element-wise divergence is beyond a fixed 2e-2 (a depth allowance is needed)."""
    L = 28
    shape = W.ModelShape("deep", L, d, heads, 4, grid, grid, dtype="bf16")
    ws = W.stack_weights(shape, seed)
    x0 = W.template_hidden(shape, seed)[0]
    n = shape.n_image
    toks = np.sort(np.random.default_rng(seed).choice(n, n // 10, replace=False))
    xr = x0[toks].astype(np.float64)
    xe = xr.astype(np.float32)
    for l in range(L):
        kv = W.synthetic_kv_cache(shape, seed, l)[0]
        xr = oracle.block_rows(xr, toks, ws[l], kv, shape, oracle.bf16_round, round_p=True)[0]
        xe = _block32(xe, toks, ws[l], kv, shape)
        ok, e1, e2, lim = PG.check(xe, xr, "bf16", l + 1, inp=x0[toks])
        assert ok, (l + 1, e1, e2, lim)
    assert PG.elem_rel_err(xe, xr, x0[toks]) > PG.TOL["bf16"]
