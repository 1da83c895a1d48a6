"""Pins of the worker-load estimate and the mask-aware routing (Sec. 4.3, Alg. 2) in the oracle."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2505_20600_amd import workloads as W

SHAPE = W.ModelShape("route", 6, 64, 2, 4, 4, 4, n_text=3, dtype="bf16")   # N = 16 image tokens, T = 19


def _model(comp0=0.5, comp_b=2.0, load0=0.25, load_b=3.0):
    return oracle.CostModel(comp0, comp_b, load0, load_b, 2 * SHAPE.d_model * 2)


# ---------------------------------------------------------------- regression models

def test_fit_textbook_example():
    # x = 1..5, y = 2 4 5 4 5: slope 6/10, intercept 4 - 0.6 * 3, SS_res 2.4 of SS_tot 6
    a, b, r2 = oracle.fit_linear([1, 2, 3, 4, 5], [2, 4, 5, 4, 5])
    assert a == pytest.approx(2.2, abs=1e-12)
    assert b == pytest.approx(0.6, abs=1e-12)
    assert r2 == pytest.approx(0.6, abs=1e-12)


def test_fit_recovers_an_exact_line_with_unit_r2():
    x = [0.5, 1.0, 7.0, 3.25, 11.0]
    a, b, r2 = oracle.fit_linear(x, [1.75 + 0.125 * xi for xi in x])
    assert (a, b) == (pytest.approx(1.75, abs=1e-12), pytest.approx(0.125, abs=1e-12))
    assert r2 == pytest.approx(1.0, abs=1e-12)


def test_fit_matches_the_library_least_squares():
    g = np.random.default_rng(5)
    for _ in range(50):
        n = int(g.integers(2, 40))
        x, y = g.uniform(-3, 9, n), g.normal(0, 4, n)
        a, b, r2 = oracle.fit_linear(list(x), list(y))
        b_ref, a_ref = np.polyfit(x, y, 1)
        assert a == pytest.approx(a_ref, rel=1e-9, abs=1e-9)
        assert b == pytest.approx(b_ref, rel=1e-9, abs=1e-9)
        assert r2 == pytest.approx(np.corrcoef(x, y)[0, 1] ** 2, rel=1e-9, abs=1e-12)


def test_fit_rejects_degenerate_inputs():
    for x, y in (([1.0], [2.0]), ([2.0, 2.0, 2.0], [1.0, 2.0, 3.0]), ([1.0, 2.0], [1.0])):
        with pytest.raises(ValueError):
            oracle.fit_linear(x, y)


# ---------------------------------------------------------------- per-block costs of a batch

def test_block_costs_follow_table1():
    m = _model(0.0, 1.0, 0.0, 1.0)
    L, cw, cwo = oracle.block_costs([5], SHAPE, m)
    d, T = SHAPE.d_model, SHAPE.n_tokens
    rows = 5 + SHAPE.n_text
    assert cw == pytest.approx((24 * rows * d * d + 4 * rows * T * d) / 1e9, rel=1e-12)
    assert cwo == pytest.approx((24 * T * d * d + 4 * T * T * d) / 1e9, rel=1e-12)
    assert L == pytest.approx((SHAPE.n_image - 5) * 4 * d / 1e6, rel=1e-12)


def test_all_masked_request_loads_nothing_and_costs_a_full_block():
    m = _model()
    L, cw, cwo = oracle.block_costs([SHAPE.n_image], SHAPE, m)
    assert L == 0.0 and cw == cwo
    k, lat = oracle.batch_latency([SHAPE.n_image] * 3, SHAPE, m)
    assert (k, lat) == (0, pytest.approx(SHAPE.n_layers * oracle.block_costs([SHAPE.n_image] * 3, SHAPE, m)[1]))


def test_batch_costs_add_over_requests_through_the_models():
    m0 = _model(0.0, 2.0, 0.0, 3.0)     # no intercepts: costs are additive over requests
    parts = [oracle.block_costs([k], SHAPE, m0) for k in (0, 4, 16)]
    whole = oracle.block_costs([0, 4, 16], SHAPE, m0)
    for j in range(3):
        assert whole[j] == pytest.approx(sum(p[j] for p in parts), rel=1e-12)


def test_empty_batch_costs_nothing():
    assert oracle.batch_latency([], SHAPE, _model()) == (0, 0.0)


# ---------------------------------------------------------------- CalcCost and routing (Alg. 2)

def test_adding_a_request_never_lowers_the_latency():
    g = np.random.default_rng(8)
    m = _model()
    for _ in range(200):
        batch = list(g.integers(0, SHAPE.n_image + 1, int(g.integers(0, 6))))
        r = int(g.integers(0, SHAPE.n_image + 1))
        assert oracle.calc_cost(r, batch, SHAPE, m) >= oracle.batch_latency(batch, SHAPE, m)[1] - 1e-12


def test_route_is_the_brute_force_argmin_with_first_index_ties_and_full_workers_skipped():
    g = np.random.default_rng(9)
    m = _model()
    for _ in range(300):
        nw = int(g.integers(1, 6))
        cap = int(g.integers(1, 4))
        workers = [list(g.integers(0, SHAPE.n_image + 1, int(g.integers(0, cap + 1)))) for _ in range(nw)]
        r = int(g.integers(0, SHAPE.n_image + 1))
        w, c = oracle.route(r, workers, cap, SHAPE, m)
        costs = [oracle.calc_cost(r, wk, SHAPE, m) if len(wk) < cap else None for wk in workers]
        free = [i for i, ci in enumerate(costs) if ci is not None]
        if not free:
            assert (w, c) == (-1, 0.0)
            continue
        best = min(costs[i] for i in free)
        assert w == min(i for i in free if costs[i] == best)
        assert c == best


def test_route_hand_example():
    # Comp = GFLOP, Load = MB (no intercepts), one layer: latency = max(L, 0) + C_w, or C_wo when
    # the block is computed in full. Worker 0 runs one all-masked request, worker 1 one request
    # with 4 masked tokens; a new request with 8 masked tokens:
    m = oracle.CostModel(0.0, 1.0, 0.0, 1.0, 4 * SHAPE.d_model)
    one = SHAPE.replace(n_layers=1)
    L0, cw0, cwo0 = oracle.block_costs([16, 8], one, m)
    L1, cw1, cwo1 = oracle.block_costs([4, 8], one, m)
    expect = [min(L0 + cw0, cwo0), min(L1 + cw1, cwo1)]
    w, c = oracle.route(8, [[16], [4]], 4, one, m)
    assert c == min(expect) and w == expect.index(min(expect))


def test_prefix_latency_is_alg1_over_the_batch_costs():
    m = _model()
    for batch in itertools.product([0, 3, 9, 16], repeat=2):
        k, lat = oracle.batch_latency(list(batch), SHAPE, m)
        L, cw, cwo = oracle.block_costs(list(batch), SHAPE, m)
        lats = [oracle.pipeline_latency([False] * j + [True] * (SHAPE.n_layers - j), L, cw, cwo)
                for j in range(SHAPE.n_layers + 1)]
        assert lat == min(lats) and k == lats.index(min(lats))
