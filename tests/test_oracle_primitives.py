"""Pins of the oracle's primitives against library routines, closed forms and special cases."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


# ---------------------------------------------------------------- bf16 rounding

def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_round_matches_torch_conversion_on_fp32_values():
    g = np.random.default_rng(1)
    x = np.concatenate([
        g.standard_normal(20000),
        g.standard_normal(2000) * 1e-30,
        g.standard_normal(2000) * 1e30,
        g.standard_normal(2000) * 1e-39,   # fp32 subnormals / bf16 subnormals
        np.clip(g.standard_normal(2000), -1.1, 1.1) * 3e38,
    ]).astype(np.float32)
    got = oracle.bf16_round(x.astype(np.float64))
    want = _torch_bf16(x)
    np.testing.assert_array_equal(got, want)


def test_bf16_round_ties_to_even_and_specials():
    one_ulp = 2.0 ** -7  # spacing of bf16 in [1, 2)
    # exactly halfway between 1 and 1+ulp -> even (1); between 1+ulp and 1+2ulp -> 1+2ulp
    assert oracle.bf16_round(1.0 + one_ulp / 2) == 1.0
    assert oracle.bf16_round(1.0 + 1.5 * one_ulp) == 1.0 + 2 * one_ulp
    assert oracle.bf16_round(-(1.0 + 1.5 * one_ulp)) == -(1.0 + 2 * one_ulp)
    # just above a tie rounds up
    assert oracle.bf16_round(1.0 + one_ulp / 2 + 2.0 ** -30) == 1.0 + one_ulp
    # largest finite bf16 and overflow
    mx = float.fromhex("0x1.fep127")
    assert oracle.bf16_round(mx) == mx
    assert np.isinf(oracle.bf16_round(float.fromhex("0x1.ffp127")))
    assert np.isnan(oracle.bf16_round(np.nan))
    assert oracle.bf16_round(np.inf) == np.inf
    assert oracle.bf16_round(0.0) == 0.0
    # smallest bf16 subnormal is 2^-133; half of it ties to 0 (even)
    assert oracle.bf16_round(2.0 ** -133) == 2.0 ** -133
    assert oracle.bf16_round(2.0 ** -134) == 0.0
    assert oracle.bf16_round(1.5 * 2.0 ** -133) == 2.0 ** -132


def test_bf16_round_is_idempotent_and_monotone():
    g = np.random.default_rng(2)
    x = np.sort(g.standard_normal(5000) * 10)
    r = oracle.bf16_round(x)
    np.testing.assert_array_equal(oracle.bf16_round(r), r)
    assert np.all(np.diff(r) >= 0)
    assert np.max(np.abs(r - x) / np.abs(x)) <= 2.0 ** -8 + 1e-15


# ---------------------------------------------------------------- LayerNorm, GELU

def test_layer_norm_matches_torch():
    g = np.random.default_rng(3)
    x = g.standard_normal((7, 48)) * 3 + 1.5
    gam, bet = g.standard_normal(48), g.standard_normal(48)
    want = F.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(gam), torch.from_numpy(bet), 1e-5).numpy()
    np.testing.assert_allclose(oracle.layer_norm(x, gam, bet, 1e-5), want, rtol=1e-12, atol=1e-12)


def test_layer_norm_closed_form_properties():
    g = np.random.default_rng(4)
    x = g.standard_normal((5, 32)) * 4 - 2
    y = oracle.layer_norm(x, np.ones(32), np.zeros(32), 0.0)
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1, atol=1e-12)
    # shift/scale invariance, and gamma/beta are an affine map afterwards
    np.testing.assert_allclose(oracle.layer_norm(3 * x + 7, np.ones(32), np.zeros(32), 0.0), y, atol=1e-12)
    np.testing.assert_allclose(oracle.layer_norm(x, 2 * np.ones(32), np.ones(32), 0.0), 2 * y + 1, atol=1e-12)


def test_gelu_matches_torch_and_limits():
    x = np.linspace(-9, 9, 1001)
    want = F.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(oracle.gelu(x), want, rtol=1e-13, atol=1e-15)
    assert oracle.gelu(0.0) == 0.0
    assert abs(oracle.gelu(1.0) - 0.5 * (1 + math.erf(1 / math.sqrt(2)))) < 1e-15
    assert abs(oracle.gelu(12.0) - 12.0) < 1e-12
    assert abs(oracle.gelu(-12.0)) < 1e-12


# ---------------------------------------------------------------- attention

def test_attention_head_matches_torch_sdpa():
    g = np.random.default_rng(5)
    q, k, v = g.standard_normal((9, 16)), g.standard_normal((33, 16)), g.standard_normal((33, 16))
    want = F.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None]).numpy()[0]
    np.testing.assert_allclose(oracle.attention_head(q, k, v, 1 / 4.0), want, rtol=1e-12, atol=1e-12)


def test_attention_head_special_cases():
    g = np.random.default_rng(6)
    q, v = g.standard_normal((4, 8)), g.standard_normal((1, 8))
    # one key: the output is that key's value
    np.testing.assert_allclose(oracle.attention_head(q, g.standard_normal((1, 8)), v, 0.3), np.repeat(v, 4, 0))
    # identical keys: uniform weights, the output is the mean of the values
    k = np.repeat(g.standard_normal((1, 8)), 5, 0)
    v5 = g.standard_normal((5, 8))
    np.testing.assert_allclose(oracle.attention_head(q, k, v5, 0.3), np.repeat(v5.mean(0, keepdims=True), 4, 0),
                               atol=1e-14)
    # a dominant key wins
    k2 = np.zeros((3, 8)); k2[1] = 100 * q[0]
    out = oracle.attention_head(q[:1], k2, v5[:3], 1.0)
    np.testing.assert_allclose(out[0], v5[1], atol=1e-12)


def test_linear_matches_torch():
    g = np.random.default_rng(7)
    x, w, b = g.standard_normal((6, 10)), g.standard_normal((4, 10)), g.standard_normal(4)
    want = F.linear(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(oracle.linear(x, w, b), want, rtol=1e-13, atol=1e-13)


def test_layer_flops_linear_in_rows():
    f1 = oracle.layer_flops(1, 4096, 768)
    for m in (2, 205, 4096):
        assert oracle.layer_flops(m, 4096, 768) == m * f1
    # Table 1: full recomputation of every token equals the dense block's count
    d, T = 64, 100
    dense = 2 * T * d * 3 * d + 2 * T * T * d * 2 + 2 * T * d * d + 2 * T * d * 4 * d * 2
    assert oracle.layer_flops(T, T, d) == dense
