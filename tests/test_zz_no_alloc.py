"""mask_step_init_static (the entry point that allocates nothing) against mask_step_init.

Two calls in a row on the library's static scratch, the second with a smaller
input (fewer requests, a smaller mask): each step's output equals, bit for bit,
the same step on a caller workspace (same kernels, same launch configuration)
and matches the oracle; the scratch is refused while a context holds it and
for a step larger than it, and is usable again after destroy.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

SHAPE = W.ModelShape("noalloc", 2, 256, 4, 4, 16, 16, n_text=8, dual_stream=True, dtype="bf16", batch=3)


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")
    yield


def _step_on(step, shape, x, kv, yc, ws, pinned):
    """mask_stack_forward on an existing context; returns the output as float64."""
    wc = MS.weights_array(G.dev_weights(ws, shape))
    d_x, d_yc = G.to_dev(x, shape), G.to_dev(yc, shape)
    if pinned:
        layers = []
        for l in range(shape.n_layers):
            t = torch.empty((shape.batch, shape.n_image, 2, shape.d_model), dtype=torch.bfloat16, pin_memory=True)
            t.copy_(torch.as_tensor(np.ascontiguousarray(kv[l][:, shape.n_text:], np.float32)).to(torch.bfloat16))
            layers.append(t)
        slots = [torch.full((shape.batch, shape.n_tokens, 2, shape.d_model), float("nan"), dtype=torch.bfloat16,
                            device=G.DEV) for _ in range(2)]
    else:
        layers, slots = [G.to_dev(kv[l], shape) for l in range(shape.n_layers)], ()
    y = torch.empty_like(d_yc)
    step.stack_forward(wc, d_x, d_yc, layers, y, pinned=pinned, slots=slots, copy_stream=torch.cuda.Stream())
    torch.cuda.synchronize()
    return G.to_np(y)


@pytest.mark.parametrize("pinned", [False, True], ids=["resident", "streamed"])
def test_static_scratch_step_equals_the_workspace_step(pinned):
    cases = [(SHAPE, (0.45, 0.2, 0.7)), (SHAPE.replace(batch=1), (0.1,))]   # the second smaller
    for i, (shape, ratios) in enumerate(cases):
        print(f"[no-alloc] call {i}: batch {shape.batch}, ratios {ratios}, pinned {pinned}", flush=True)
        ws = W.stack_weights(shape, 140, random_ln=True, std=0.03)
        xt = W.template_hidden(shape, 140)
        kv = np.stack([W.synthetic_kv_cache(shape, 140, l) for l in range(shape.n_layers)])
        yc = W.synthetic_y_cache(shape, 140)
        g = np.random.default_rng(40 + i)
        mask = np.zeros((shape.batch, shape.n_image), np.uint8)
        for b, r in enumerate(ratios):
            mask[b, g.choice(shape.n_image, int(round(r * shape.n_image)), replace=False)] = 1
        x = W.edited_hidden(shape, 140, xt, mask)
        desc = MS.model_desc(shape)
        assert MS.mask_workspace_bytes(desc, shape.batch) <= MS.STATIC_SCRATCH_BYTES
        d_mask = torch.as_tensor(mask).to(G.DEV)
        st = MS.MaskStep(desc, shape.batch, d_mask, None)
        try:
            with pytest.raises(MS.MaskStepError) as busy:
                MS.MaskStep(desc, shape.batch, d_mask, None)
            assert busy.value.status == MS.MS_ESTATE
            y_static = _step_on(st, shape, x, kv, yc, ws, pinned)
            info = st.info()
        finally:
            st.close()
        ref_step = G.new_step(shape, mask)
        y_ws = _step_on(ref_step, shape, x, kv, yc, ws, pinned)
        assert info.rows == ref_step.info().rows
        ref_step.close()
        np.testing.assert_array_equal(y_static, y_ws)
        y_ref = oracle.masked_stack(x, mask, kv, yc, ws, shape, round_p=True)
        G.assert_close(y_static, y_ref, "bf16", f"static scratch call {i}", blocks=shape.n_layers, inp=x)


def test_static_scratch_refuses_a_step_larger_than_it():
    big = W.CONFIGS["c3"]
    desc = MS.model_desc(big)
    assert MS.mask_workspace_bytes(desc, big.batch) > MS.STATIC_SCRATCH_BYTES
    d_mask = torch.ones((1, big.n_image), dtype=torch.uint8, device=G.DEV)
    with pytest.raises(MS.MaskStepError) as err:
        MS.MaskStep(desc, big.batch, d_mask, None)
    assert err.value.status == MS.MS_EWORKSPACE
    small = SHAPE.replace(batch=1)
    st = MS.MaskStep(MS.model_desc(small), 1, torch.ones((1, small.n_image), dtype=torch.uint8, device=G.DEV), None)
    st.close()
