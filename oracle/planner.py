"""Pipeline-loading planner (Sec. 4.2, Alg. 1) — test infrastructure only.

Alg. 1 walks the blocks in order and keeps two clocks: when the load stream
has finished the cached activations of block i (``load``) and when the
compute stream has finished block i (``comp``). A block that uses its cache
must wait for its load (``max(load + L, comp)``) and then takes ``C_w``; a
block computed over all tokens needs no load and takes ``C_wo``. The
pipeline latency is ``comp`` after the last block.

``pipeline_latency`` evaluates those two recurrences for a given per-block
choice. ``greedy_choice`` is the algorithm's own rule: a block uses the cache
when doing so finishes no later than computing it in full. With K/V caching
only prefix choices are feasible (a full block needs every token's hidden
state, which exists only while every earlier block was full), so
``best_dense_prefix`` evaluates the same latency for every prefix length and
keeps the smallest (earliest minimum).
"""
from __future__ import annotations


def pipeline_latency(use_cache, load_ms: float, cached_ms: float, full_ms: float) -> float:
    comp, load = 0.0, 0.0
    for uc in use_cache:
        if uc:
            load = load + load_ms
            comp = max(load, comp) + cached_ms
        else:
            comp = comp + full_ms
    return comp


def greedy_choice(n_blocks: int, load_ms: float, cached_ms: float, full_ms: float):
    comp, load, out = 0.0, 0.0, []
    for _ in range(n_blocks):
        if max(load + load_ms, comp) + cached_ms <= comp + full_ms:
            load = load + load_ms
            comp = max(load, comp) + cached_ms
            out.append(True)
        else:
            comp = comp + full_ms
            out.append(False)
    return out, comp


def best_dense_prefix(n_blocks: int, load_ms: float, cached_ms: float, full_ms: float):
    best_k, best = 0, None
    for k in range(n_blocks + 1):
        lat = pipeline_latency([False] * k + [True] * (n_blocks - k), load_ms, cached_ms, full_ms)
        if best is None or lat < best - 1e-12:
            best_k, best = k, lat
    return best_k, best
