"""Worker-load estimate and mask-aware request routing (Sec. 4.3, Alg. 2) — test
infrastructure only.

Sec. 4.3 estimates a worker's load with two linear regression models fitted
offline. One maps the computation of a batch, as FLOPs from Table 1 at the
requests' mask ratios, to a block's latency. The other maps the bytes of
cached activations a block loads to the loading latency. ``fit_linear`` is
ordinary least squares with an intercept, written out (slope = covariance /
variance), with the coefficient of determination R^2 = 1 - SS_res / SS_tot.

``block_costs`` turns a batch (masked image tokens per request) into Alg. 1's
per-block inputs:

* C_w, a cached block: the masked and text rows of every request;
* C_wo, a block over every token;
* L, the cache of the unmasked image rows.

A zero amount of work or bytes costs nothing, so the intercepts apply only
to work that is issued. ``batch_latency`` runs Alg. 1 over these in its
dense-prefix form (the K/V variant, see ``planner``). ``calc_cost`` is
Alg. 2's CalcCost: the pipeline latency of the worker's running batch with
the new request added. ``route`` picks the candidate of least cost, the
first on ties; candidates are the workers whose running batch has room.
"""
from __future__ import annotations

from .planner import best_dense_prefix
from .stack import layer_flops


def fit_linear(x, y):
    """(intercept, slope, r2) of the least-squares line y ~ intercept + slope * x."""
    n = len(x)
    if n != len(y) or n < 2:
        raise ValueError("need two or more (x, y) pairs")
    xm = sum(x) / n
    ym = sum(y) / n
    sxx = sum((xi - xm) ** 2 for xi in x)
    if not sxx > 0:
        raise ValueError("x has no spread")
    sxy = sum((xi - xm) * (yi - ym) for xi, yi in zip(x, y))
    slope = sxy / sxx
    intercept = ym - slope * xm
    ss_res = sum((yi - (intercept + slope * xi)) ** 2 for xi, yi in zip(x, y))
    ss_tot = sum((yi - ym) ** 2 for yi in y)
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else (1.0 if ss_res == 0 else 0.0)
    return intercept, slope, r2


class CostModel:
    """Comp(F) = comp_ms0 + comp_ms_per_gflop * F / 1e9 and Load(B) = load_ms0 + load_ms_per_mb * B / 1e6,
    per block; ``cache_bytes_per_token`` is what one unmasked image token's cache holds per block."""

    def __init__(self, comp_ms0, comp_ms_per_gflop, load_ms0, load_ms_per_mb, cache_bytes_per_token):
        self.comp_ms0 = comp_ms0
        self.comp_ms_per_gflop = comp_ms_per_gflop
        self.load_ms0 = load_ms0
        self.load_ms_per_mb = load_ms_per_mb
        self.cache_bytes_per_token = cache_bytes_per_token

    def comp(self, flops):
        return 0.0 if flops == 0 else self.comp_ms0 + self.comp_ms_per_gflop * flops / 1e9

    def load(self, nbytes):
        return 0.0 if nbytes == 0 else self.load_ms0 + self.load_ms_per_mb * nbytes / 1e6


def block_costs(masked, shape, model: CostModel):
    """(L, C_w, C_wo) of one block for a batch with ``masked[b]`` masked image tokens per request."""
    T, d, mlp = shape.n_tokens, shape.d_model, shape.mlp_mult
    f_cached = sum(layer_flops(m + shape.n_text, T, d, mlp) for m in masked)
    f_full = len(masked) * layer_flops(T, T, d, mlp)
    nbytes = sum((shape.n_image - m) * model.cache_bytes_per_token for m in masked)
    return model.load(nbytes), model.comp(f_cached), model.comp(f_full)


def batch_latency(masked, shape, model: CostModel):
    """(dense prefix k, pipeline latency) of Alg. 1 for the batch."""
    if not masked:
        return 0, 0.0
    L, cw, cwo = block_costs(masked, shape, model)
    return best_dense_prefix(shape.n_layers, L, cw, cwo)


def calc_cost(request_masked, running, shape, model: CostModel):
    return batch_latency(list(running) + [request_masked], shape, model)[1]


def route(request_masked, workers, max_batch, shape, model: CostModel):
    """(worker index or -1 when no worker has room, its cost)."""
    best, best_cost = -1, None
    for i, running in enumerate(workers):
        if len(running) >= max_batch:
            continue
        c = calc_cost(request_masked, running, shape, model)
        if best_cost is None or c < best_cost:
            best, best_cost = i, c
    return best, (best_cost if best_cost is not None else 0.0)
