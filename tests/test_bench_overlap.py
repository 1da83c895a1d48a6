"""Host logic of the benchmark's cache-load overlap figures (interval unions and
their intersection), checked on hand-made timelines."""
import importlib.util
import os

import numpy as np
import pytest

_spec = importlib.util.spec_from_file_location(
    "bench", os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "bench.py"))
bench = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(bench)


def test_union_merges_touching_and_nested_intervals():
    assert bench._union([(3, 4), (0, 1), (0.5, 2), (2, 2.5), (5, 9), (6, 7)]) == [[0, 2.5], [3, 4], [5, 9]]
    assert bench._length(bench._union([(0, 1), (0.5, 2)])) == 2


def test_intersection_of_unions():
    u = [[0, 2], [4, 6]]
    v = [[1, 5]]
    assert bench._intersection(u, v) == pytest.approx(2.0)   # [1,2] + [4,5]
    assert bench._intersection(u, [[10, 11]]) == 0.0


def test_stream_overlap_figures():
    # two steps; per step: copies 0-4 and 10-14, kernels 1-3, 3-6, 11-12 (+ a kernel-only span)
    iv = [("copy", 0.0, 4.0), ("attention", 1.0, 3.0), ("gemm_qkv", 3.0, 6.0),
          ("copy", 10.0, 14.0), ("gemm_up", 11.0, 12.0), ("gemm_down", 20.0, 22.0)]
    r = bench.stream_overlap(iv, steps=2)
    # copy union [0,4] + [10,14] = 8; kernel union [1,6] + [11,12] + [20,22] = 8
    assert r["sum_copy_ms"] == pytest.approx(4.0)
    assert r["sum_kernel_ms"] == pytest.approx(4.0)
    # overlap: [1,4] (3) + [11,12] (1) = 4 of min(8, 8)
    assert r["overlap"] == pytest.approx(0.5)
    assert r["first_layer_copy_ms"] == pytest.approx(4.0)
    assert r["bound_ms"] == pytest.approx(8.0)


def test_stream_overlap_without_copies():
    r = bench.stream_overlap([("attention", 0.0, 1.0)], steps=1)
    assert r["overlap"] is None and r["sum_copy_ms"] == 0


def test_step_fit_is_the_least_squares_line_over_the_common_prefix():
    rows = [[0.1, 400, 0.8 + 0.0003 * 400, 0], [0.3, 1200, 0.8 + 0.0003 * 1200, 0],
            [0.5, 2000, 0.8 + 0.0003 * 2000, 0], [0.9, 3600, 5.0, 2]]
    f = bench.step_fit(rows)
    assert f["points"] == 3 and f["dense_prefix"] == 0
    assert abs(f["ms0"] - 0.8) < 1e-4 and abs(f["ms_per_1k_rows"] - 0.3) < 1e-4 and f["r2"] == 1.0
    noisy = [[0, m, t, 0] for m, t in ((100, 1.0), (200, 1.3), (300, 1.1), (400, 1.6))]
    x = np.array([100, 200, 300, 400.0]); y = np.array([1.0, 1.3, 1.1, 1.6])
    r = np.corrcoef(x, y)[0, 1]
    assert abs(bench.step_fit(noisy)["r2"] - r * r) < 1e-3
    assert bench.step_fit(rows[:2]) is None and bench.step_fit([]) is None
