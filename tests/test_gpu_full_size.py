"""The workloads at full size, in the launch configurations the benchmark times.

Inputs follow each workload's recipe (weights N(0, 0.02), LayerNorm 1/0,
hidden states N(0, 1), the workload's own mask generator); the cache is a
seeded random stand-in (the masked computation is defined for any cache
contents), so the oracle runs only what one request needs.

* c2 (12 x d768, HBM-resident cache) at mask ratios 5 / 25 / 60 / 100%: the
  step through mask_stack_forward equals the step through the per-block calls
  bit for bit; every block matches the oracle's block on the GPU's own block
  input at the one-block bound; request 0's output rows match the oracle's
  whole stack in the max norm; untouched rows are the cached state, bit for bit.
* c3 (28 x d1152, head_dim 72, cache streamed from pinned host memory): all 28
  layers block by block through cache_prefetch_layer with a two-slot ring,
  equal bit for bit to mask_stack_forward with one slot per layer (as the
  benchmark runs it); and the bubble-free pipeline's dense prefix (Alg. 1)
  over 5 layers with one slot per layer, against the oracle's dense-prefix path.
* c5 (19 x d3072 dual stream, 512 text rows, batch 4, pinned cache): 3 layers
  with a dense prefix of 1 against the oracle, and block by block without a
  prefix; the request with the fewest recomputed rows is checked.
* c4 (28 x d1152, batch 8, HBM-resident, varlen): all layers, the smallest request.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")
    yield


def _inputs(key, shape):
    cfg = W.CONFIG_IDS[key]
    ws = W.stack_weights(shape, cfg)
    xt = W.template_hidden(shape, cfg)
    kv = [W.synthetic_kv_cache(shape, cfg, l) for l in range(shape.n_layers)]
    yc = W.synthetic_y_cache(shape, cfg)
    return ws, xt, kv, yc


def _kv_rows(kv, shape):
    def of(l, b):
        k = np.array(kv[l][b], np.float64)
        k[:shape.n_text] = 0.0
        return k
    return of


def _untouched_rows_exact(y, yc, mask, shape, b):
    keep = np.concatenate([np.zeros(shape.n_text, bool), mask[b] == 0])
    np.testing.assert_array_equal(y[b, keep], yc[b, keep])


@pytest.mark.parametrize("ratio", [0.05, 0.25, 0.60, 1.00])
def test_c2_full_size_block_by_block(ratio):
    shape = W.CONFIGS["c2"]
    ws, xt, kv, yc = _inputs("c2", shape)
    mask = W.workload_mask("c2", shape, ratio=ratio)
    x = W.edited_hidden(shape, W.CONFIG_IDS["c2"], xt, mask)
    y, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, return_kv=False)
    y_blocks, snaps, rows = G.run_block_by_block(shape, mask, x, kv, yc, ws, form="resident")
    np.testing.assert_array_equal(y_blocks, y)
    G.check_blocks(shape, snaps, rows, _kv_rows(kv, shape), ws, f"c2 {ratio:.0%}")
    toks, ref = oracle.masked_rows_of_stack(x, mask, kv, ws, shape, 0, round_p=True)
    G.assert_close(y[0, toks], ref, "bf16", f"c2 {ratio:.0%} stack", blocks=shape.n_layers, inp=x[0, toks])
    _untouched_rows_exact(y, yc, mask, shape, 0)


def test_c3_full_size_streamed_block_by_block():
    shape = W.CONFIGS["c3"]
    ws, xt, kv, yc = _inputs("c3", shape)
    mask = W.workload_mask("c3", shape, ratio=0.10)
    x = W.edited_hidden(shape, W.CONFIG_IDS["c3"], xt, mask)
    y_blocks, snaps, rows = G.run_block_by_block(shape, mask, x, kv, yc, ws, form="kv", n_slots=2)
    y, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=shape.n_layers)
    np.testing.assert_array_equal(y_blocks, y)
    G.check_blocks(shape, snaps, rows, _kv_rows(kv, shape), ws, "c3 10%")
    toks, ref = oracle.masked_rows_of_stack(x, mask, kv, ws, shape, 0, round_p=True)
    G.assert_close(y[0, toks], ref, "bf16", "c3 10% stack", blocks=shape.n_layers, inp=x[0, toks])
    _untouched_rows_exact(y, yc, mask, shape, 0)


@pytest.mark.parametrize("ratio,k", [(0.05, 2), (0.50, 3)])
def test_c3_full_size_dense_prefix(ratio, k):
    """Blocks [0, k) over every token, the rest with the streamed cache (every load
    issued at the start, under the prefix): 5 of the 28 layers."""
    shape = W.CONFIGS["c3"].replace(n_layers=5)
    ws, xt, kv, yc = _inputs("c3", shape)
    mask = W.workload_mask("c3", shape, ratio=ratio)
    x = W.edited_hidden(shape, W.CONFIG_IDS["c3"], xt, mask)
    y, _, step = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=shape.n_layers, dense_prefix=k)
    assert step.info().dense_prefix == k
    y2, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=2, dense_prefix=k)
    np.testing.assert_array_equal(y2, y)
    toks, ref = oracle.masked_rows_of_stack(x, mask, kv, ws, shape, 0, dense_prefix=k, round_p=True)
    G.assert_close(y[0, toks], ref, "bf16", f"c3 {ratio:.0%} dense prefix {k}", blocks=shape.n_layers,
                   inp=x[0, toks])
    _untouched_rows_exact(y, yc, mask, shape, 0)


def test_c5_full_size_dense_prefix_and_block_by_block():
    shape = W.CONFIGS["c5"].replace(n_layers=3)
    ws, xt, kv, yc = _inputs("c5", shape)
    mask = W.workload_mask("c5", shape)
    x = W.edited_hidden(shape, W.CONFIG_IDS["c5"], xt, mask)
    b = int(np.argmin(mask.sum(1)))
    y, _, step = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=shape.n_layers, dense_prefix=1)
    assert step.info().dense_prefix == 1
    toks, ref = oracle.masked_rows_of_stack(x, mask, kv, ws, shape, b, dense_prefix=1, round_p=True)
    G.assert_close(y[b, toks], ref, "bf16", f"c5 dense prefix 1, request {b}", blocks=shape.n_layers,
                   inp=x[b, toks])
    _untouched_rows_exact(y, yc, mask, shape, b)
    y0, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=shape.n_layers)
    y_blocks, snaps, rows = G.run_block_by_block(shape, mask, x, kv, yc, ws, form="kv", n_slots=2)
    np.testing.assert_array_equal(y_blocks, y0)
    G.check_blocks(shape, snaps, rows, _kv_rows(kv, shape), ws, f"c5 request {b}", requests=[b])


def test_c4_full_size_batched_stack():
    shape = W.CONFIGS["c4"]
    ws, xt, kv, yc = _inputs("c4", shape)
    mask = W.workload_mask("c4", shape)
    x = W.edited_hidden(shape, W.CONFIG_IDS["c4"], xt, mask)
    y, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, return_kv=False)
    b = int(np.argmin(mask.sum(1)))
    toks, ref = oracle.masked_rows_of_stack(x, mask, kv, ws, shape, b, round_p=True)
    G.assert_close(y[b, toks], ref, "bf16", f"c4 request {b}", blocks=shape.n_layers, inp=x[b, toks])
    _untouched_rows_exact(y, yc, mask, shape, b)
