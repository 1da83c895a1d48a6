"""The native worker-load estimate and router (Sec. 4.3, Alg. 2) against the oracle (host-only)."""
import numpy as np
import pytest

import oracle
from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W

SHAPES = [W.ModelShape("route", 6, 64, 2, 4, 4, 4, n_text=3, dtype="bf16"),
          W.CONFIGS["c4"], W.CONFIGS["c5"]]


def _models(g, shape):
    bpt = 2 * shape.d_model * (2 if shape.dtype == "bf16" else 4)
    vals = [g.uniform(0, 2), g.uniform(0, 0.2), g.uniform(0, 1), g.uniform(0, 0.05)]
    return oracle.CostModel(*vals, bpt), MS.CostModel(*vals, bpt)


def test_fit_matches_the_oracle():
    g = np.random.default_rng(3)
    for _ in range(100):
        n = int(g.integers(2, 30))
        x, y = list(g.uniform(0, 50, n)), list(g.normal(3, 2, n))
        got = MS.mask_fit_linear(x, y)
        ref = oracle.fit_linear(x, y)
        assert got == pytest.approx(ref, rel=1e-10, abs=1e-12)


def test_fit_rejects_degenerate_inputs():
    for x, y in (([1.0], [2.0]), ([2.0, 2.0], [1.0, 3.0]), ([1.0, float("nan")], [1.0, 2.0])):
        with pytest.raises(MS.MaskStepError):
            MS.mask_fit_linear(x, y)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
def test_batch_cost_matches_the_oracle(shape):
    g = np.random.default_rng(4)
    desc = MS.model_desc(shape)
    for _ in range(60):
        om, nm = _models(g, shape)
        masked = [int(v) for v in g.integers(0, shape.n_image + 1, int(g.integers(0, 9)))]
        costs, k, lat = MS.mask_batch_cost(desc, nm, masked)
        ref = oracle.block_costs(masked, shape, om) if masked else (0.0, 0.0, 0.0)
        assert costs == pytest.approx(ref, rel=1e-12, abs=0)
        assert (k, lat) == (oracle.batch_latency(masked, shape, om)[0],
                            pytest.approx(oracle.batch_latency(masked, shape, om)[1], rel=1e-12, abs=0))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
def test_route_matches_the_oracle(shape):
    g = np.random.default_rng(6)
    desc = MS.model_desc(shape)
    for _ in range(60):
        om, nm = _models(g, shape)
        cap = int(g.integers(1, 5))
        workers = [[int(v) for v in g.integers(0, shape.n_image + 1, int(g.integers(0, cap + 1)))]
                   for _ in range(int(g.integers(0, 6)))]
        r = int(g.integers(0, shape.n_image + 1))
        w, c = MS.mask_route_request(desc, nm, workers, cap, r)
        w_ref, c_ref = oracle.route(r, workers, cap, shape, om)
        assert w == w_ref
        assert c == pytest.approx(c_ref, rel=1e-12, abs=0)


def test_cost_calls_reject_bad_arguments():
    shape = SHAPES[0]
    desc = MS.model_desc(shape)
    good = MS.CostModel(1.0, 0.1, 0.5, 0.01, 256.0)
    with pytest.raises(MS.MaskStepError):
        MS.mask_batch_cost(desc, good, [shape.n_image + 1])
    with pytest.raises(MS.MaskStepError):
        MS.mask_batch_cost(desc, MS.CostModel(-1.0, 0.1, 0.5, 0.01, 256.0), [1])
    with pytest.raises(MS.MaskStepError):
        MS.mask_route_request(desc, good, [[1]], 0, 1)
    with pytest.raises(MS.MaskStepError):
        MS.mask_route_request(desc, good, [[-1]], 2, 1)
    assert MS.mask_route_request(desc, good, [[1, 2], [3, 4]], 2, 5) == (-1, 0.0)
    assert MS.mask_route_request(desc, good, [], 2, 5) == (-1, 0.0)
