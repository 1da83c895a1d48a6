"""The per-block boundary calls, block by block against the oracle.

A step driven through the calls the paper's pipeline is made of (Sec. 3.1 with
Fig. 7 for the block, Sec. 4.2 with Fig. 8 for the block-wise cache loading):
mask_gather_rows, then per layer cache_prefetch_layer on a copy stream (a ring
of two device slots ordered by events, the paper's double buffer) and
mask_block_forward on the compute stream, then mask_scatter_rows. For Y
caching the layer's block inputs stream in with cache_prefetch_inputs and
mask_recompute_kv rebuilds the unmasked tokens' K/V before the block.

Checked per block: the block output against the oracle's block applied to the
GPU's own block input (element-wise at the one-block bound, 2e-2 for bf16),
the fresh K/V rows likewise, the cached K/V rows the block leaves alone bit for
bit (K/V caching) or at the one-block bound (Y caching, where they are
recomputed); and the final output bit for bit against mask_stack_forward and
the HBM-resident cache. Weights N(0, 0.05): the scale at which the gate
rejects attention mistakes with room for correct rounding (tests/test_parity_gate).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

STD = 0.05

SHAPES = [
    W.ModelShape("hd64_T256_L3_b2", 3, 256, 4, 4, 16, 16, dtype="bf16", batch=2),
    W.ModelShape("hd72_T144", 2, 576, 8, 4, 12, 12, dtype="bf16"),
    W.ModelShape("hd128_b3", 2, 256, 2, 4, 12, 16, dtype="bf16", batch=3),
    W.ModelShape("dual_txt40_b2", 2, 256, 2, 4, 10, 10, n_text=40, dual_stream=True, dtype="bf16", batch=2),
]


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")
    yield


def _mask(shape, ratio, seed):
    g = np.random.default_rng(seed)
    m = np.zeros((shape.batch, shape.n_image), np.uint8)
    for b in range(shape.batch):
        r = ratio * (1 - 0.3 * b) if ratio < 1 else 1.0
        m[b, g.choice(shape.n_image, max(1, int(round(r * shape.n_image))), replace=False)] = 1
    return m


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
@pytest.mark.parametrize("ratio", [0.05, 0.45, 1.0])
def test_kv_cache_block_by_block(shape, ratio):
    ws = W.stack_weights(shape, 120, random_ln=True, std=STD)
    xt = W.template_hidden(shape, 120)
    kv = np.stack([W.synthetic_kv_cache(shape, 120, l) for l in range(shape.n_layers)])
    yc = W.synthetic_y_cache(shape, 120)
    mask = _mask(shape, ratio, 31)
    x = W.edited_hidden(shape, 120, xt, mask)
    y, snaps, rows = G.run_block_by_block(shape, mask, x, kv, yc, ws, form="kv", n_slots=2)

    def kv_of_layer(l, b):
        k = np.array(kv[l][b], np.float64)
        k[:shape.n_text] = 0.0            # text rows are never cached: every block recomputes them
        return k

    G.check_blocks(shape, snaps, rows, kv_of_layer, ws, f"{shape.name} K/V")
    y_stack, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=2)
    np.testing.assert_array_equal(y, y_stack)
    y_res, _, _ = G.run_stack(shape, mask, x, kv, yc, ws)
    np.testing.assert_array_equal(y, y_res)
    for b in range(shape.batch):
        keep = np.concatenate([np.zeros(shape.n_text, bool), mask[b] == 0])
        np.testing.assert_array_equal(y[b, keep], yc[b, keep])


@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[3]], ids=lambda s: s.name)
@pytest.mark.parametrize("ratio", [0.05, 0.45])
def test_y_cache_block_by_block(shape, ratio):
    ws = W.stack_weights(shape, 121, random_ln=True, std=STD)
    xt = W.template_hidden(shape, 121)
    yin = np.stack([W.to_bf16_values(W.rng(121, 6, l).standard_normal((shape.batch, shape.n_image,
                                                                        shape.d_model)))
                    for l in range(shape.n_layers)])
    yc = W.synthetic_y_cache(shape, 121)
    mask = _mask(shape, ratio, 32)
    x = W.edited_hidden(shape, 121, xt, mask)
    y, snaps, rows = G.run_block_by_block(shape, mask, x, yin, yc, ws, form="y", n_slots=2)
    kv_y = oracle.kv_cache_of_inputs(yin, mask, ws, shape)     # what the recomputation must produce
    G.check_blocks(shape, snaps, rows, lambda l, b: kv_y[l, b], ws, f"{shape.name} Y", loaded_exact=False)
    y_stack, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True, pinned=True, n_slots=2)
    np.testing.assert_array_equal(y, y_stack)
