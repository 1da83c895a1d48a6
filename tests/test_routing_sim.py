"""The host-only routing simulation (Sec. 4.3, Alg. 2): invariants and the mask-aware
policy's decisions against the oracle's router."""
import numpy as np
import pytest

import oracle
from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import routing as R
from paper_2505_20600_amd import workloads as W

SHAPE = W.ModelShape("route", 6, 64, 2, 4, 8, 8, n_text=0, dtype="bf16")   # 64 image tokens
BPT = 2.0 * SHAPE.d_model * 2
VALS = (0.4, 2.0, 0.3, 5.0)


def _run(n_workers=3, max_batch=3, steps=4, n=60, rate=40.0, decisions=None):
    desc = MS.model_desc(SHAPE, max_batch=max_batch)
    model = MS.CostModel(*VALS, BPT)
    reqs = R.draw_requests(n, rate, SHAPE.n_image, seed=3)
    return reqs, R.simulate(desc, model, reqs, n_workers, max_batch, steps, decisions)


def test_every_request_is_served_no_faster_than_alone():
    desc = MS.model_desc(SHAPE, max_batch=3)
    model = MS.CostModel(*VALS, BPT)
    reqs, lat = _run()
    assert all(v is not None for v in lat)
    for (t, m), v in zip(reqs, lat):
        alone = MS.mask_batch_cost(desc, model, [m])[2] / 1e3
        assert v >= 4 * alone * (1 - 1e-12)


def test_one_worker_serves_in_arrival_order_batches():
    """With one worker every request that finds room joins it; more workers never make the
    mean latency worse on the same arrivals."""
    one = _run(n_workers=1)[1]
    three = _run(n_workers=3)[1]
    assert all(v is not None for v in one)
    assert np.mean(three) <= np.mean(one) + 1e-12


def test_mask_aware_decisions_are_the_oracle_router():
    dec = []
    _run(n_workers=4, max_batch=2, n=80, rate=2000.0, decisions=dec)
    model = oracle.CostModel(*VALS, BPT)
    assert any(w >= 0 for _, _, w in dec) and any(w < 0 for _, _, w in dec)   # full cluster reached
    for masked, workers, chosen in dec:
        assert chosen == oracle.route(masked, workers, 2, SHAPE, model)[0]

