"""Pins of the pipeline-loading planner (Sec. 4.2, Alg. 1) and of the dense-prefix
variant of the masked stack in the oracle."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2505_20600_amd import workloads as W

TINY = W.ModelShape("tiny", 4, 32, 4, 4, 3, 4, dtype="fp32")


# ---------------------------------------------------------------- latency recurrence

def test_latency_closed_forms():
    # all blocks computed in full: N * C_wo
    assert oracle.pipeline_latency([False] * 7, 3.0, 1.0, 5.0) == 35.0
    # all cached, loads slower than compute: loads back to back, last block's compute after its load
    assert oracle.pipeline_latency([True] * 7, 3.0, 1.0, 5.0) == 7 * 3.0 + 1.0
    # all cached, compute slower than loads: first load, then computes back to back
    assert oracle.pipeline_latency([True] * 7, 1.0, 3.0, 5.0) == 1.0 + 7 * 3.0


def test_latency_hand_example():
    # F, F, T, T with L=4, C_w=1, C_wo=3:
    # comp: 3, 6; load chain 4 -> comp max(4,6)+1 = 7; load 8 -> comp max(8,7)+1 = 9
    assert oracle.pipeline_latency([False, False, True, True], 4.0, 1.0, 3.0) == 9.0


def test_greedy_is_the_papers_rule_on_a_hand_example():
    # L=4, C_w=1, C_wo=3, N=4:
    # block 1: max(0+4, 0)+1 = 5 > 0+3 -> full (comp 3)
    # block 2: max(4, 3)+1 = 5 <= 3+3 -> cache (load 4, comp 5)
    # block 3: max(8, 5)+1 = 9 > 5+3 = 8 -> full (comp 8)
    # block 4: max(8, 8)+1 = 9 <= 8+3 -> cache (load 8, comp 9)
    choice, lat = oracle.greedy_choice(4, 4.0, 1.0, 3.0)
    assert choice == [False, True, False, True]
    assert lat == 9.0
    assert lat == oracle.pipeline_latency(choice, 4.0, 1.0, 3.0)


def test_best_prefix_is_the_brute_force_minimum_over_prefixes():
    g = np.random.default_rng(0)
    for _ in range(200):
        n = int(g.integers(1, 12))
        L, cw, cwo = g.uniform(0.1, 5), g.uniform(0.01, 2), g.uniform(0.5, 6)
        k, lat = oracle.best_dense_prefix(n, L, cw, cwo)
        lats = [oracle.pipeline_latency([False] * j + [True] * (n - j), L, cw, cwo) for j in range(n + 1)]
        assert lat == min(lats)
        assert k == lats.index(min(lats))


def test_prefix_optimum_never_beats_the_unconstrained_optimum_and_matches_it_when_loads_are_cheap():
    g = np.random.default_rng(1)
    for _ in range(100):
        n = int(g.integers(1, 9))
        L, cw = g.uniform(0.1, 3), g.uniform(0.01, 1)
        cwo = cw + g.uniform(0.0, 4)          # a full block never costs less than a cached one
        best_any = min(oracle.pipeline_latency(c, L, cw, cwo) for c in itertools.product([False, True], repeat=n))
        _, best_prefix = oracle.best_dense_prefix(n, L, cw, cwo)
        assert best_any <= best_prefix + 1e-12
        if L <= cw and cwo >= cw + L:   # loads hide under compute: caching every block is optimal
            assert abs(best_prefix - (L + n * cw)) < 1e-9


# ---------------------------------------------------------------- dense prefix in the oracle

def _setup(shape, cfg=21):
    ws = W.stack_weights(shape, cfg, random_ln=True, std=0.2)
    x = W.template_hidden(shape, cfg)
    yc = W.synthetic_y_cache(shape, cfg)
    kv = np.stack([W.synthetic_kv_cache(shape, cfg, l) for l in range(shape.n_layers)])
    mask = np.zeros((1, shape.n_image), np.uint8)
    mask[0, [0, 4, 5, 11]] = 1
    return ws, x, yc, kv, mask


def test_dense_prefix_zero_is_the_masked_stack():
    ws, x, yc, kv, mask = _setup(TINY)
    np.testing.assert_array_equal(oracle.masked_stack(x, mask, kv, yc, ws, TINY, dense_prefix=0),
                                  oracle.masked_stack(x, mask, kv, yc, ws, TINY))


def test_full_dense_prefix_gives_the_dense_rows_and_the_cached_rest():
    ws, x, yc, kv, mask = _setup(TINY)
    y = oracle.masked_stack(x, mask, kv, yc, ws, TINY, dense_prefix=TINY.n_layers)
    y_dense, _ = oracle.dense_stack(x, ws, TINY)
    sel = mask[0] != 0
    np.testing.assert_array_equal(y[0, sel], y_dense[0, sel])
    np.testing.assert_array_equal(y[0, ~sel], yc[0, ~sel])


@pytest.mark.parametrize("k", [1, 2, 3])
def test_dense_prefix_reads_no_cache_of_its_blocks_and_keeps_own_cache_exactness(k):
    ws, x, yc, kv, mask = _setup(TINY)
    poisoned = kv.copy()
    poisoned[:k] = np.nan
    y = oracle.masked_stack(x, mask, poisoned, yc, ws, TINY, dense_prefix=k)
    np.testing.assert_array_equal(y, oracle.masked_stack(x, mask, kv, yc, ws, TINY, dense_prefix=k))
    # own cache: any prefix reproduces the dense result
    y_dense, kv_dense = oracle.dense_stack(x, ws, TINY)
    y_own = oracle.masked_stack(x, mask, kv_dense, y_dense, ws, TINY, dense_prefix=k)
    np.testing.assert_allclose(y_own, y_dense, rtol=1e-12, atol=1e-12)
    # and a prefix changes the result with a foreign cache (the dense blocks see fresh unmasked K/V)
    y0 = oracle.masked_stack(x, mask, kv, yc, ws, TINY)
    assert np.max(np.abs(y - y0)) > 1e-6
