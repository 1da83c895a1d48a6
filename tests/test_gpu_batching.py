"""Step-level continuous batching (Sec. 4.2 "Continuous Batching") on the GPU: per-request
pinned caches, requests that recompute nothing, and requests joining and leaving a running
batch, each against the oracle or the contiguous-batch path."""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_20600_amd import batching as CB
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

PLAIN = W.ModelShape("cb", 2, 256, 4, 4, 8, 8, dtype="bf16", batch=3)
TEXT = W.ModelShape("cbt", 2, 256, 4, 4, 8, 8, n_text=8, dual_stream=True, dtype="bf16", batch=3)


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")
    yield


def _inputs(shape, cfg):
    ws = W.stack_weights(shape, cfg, random_ln=True, std=0.03)
    xt = W.template_hidden(shape, cfg)
    kv = np.stack([W.synthetic_kv_cache(shape, cfg, l) for l in range(shape.n_layers)])
    yc = W.synthetic_y_cache(shape, cfg)
    return ws, xt, kv, yc


def _masks(shape, ratios, seed):
    g = np.random.default_rng(seed)
    m = np.zeros((shape.batch, shape.n_image), np.uint8)
    for b, r in enumerate(ratios):
        m[b, g.choice(shape.n_image, int(round(r * shape.n_image)), replace=False)] = 1
    return m


def _pinned_layers(kv, shape, per_request):
    """[L] contiguous [B][N][2][d] pinned buffers, or [L][B] per-request [N][2][d] ones."""
    out = []
    for l in range(shape.n_layers):
        img = np.ascontiguousarray(np.asarray(kv[l])[:, shape.n_text:], np.float32)
        if per_request:
            row = []
            for b in range(shape.batch):
                t = torch.empty(img.shape[1:], dtype=torch.bfloat16, pin_memory=True)
                t.copy_(torch.as_tensor(img[b]).to(torch.bfloat16))
                row.append(t)
            out.append(row)
        else:
            t = torch.empty(img.shape, dtype=torch.bfloat16, pin_memory=True)
            t.copy_(torch.as_tensor(img).to(torch.bfloat16))
            out.append(t)
    return out


def _run_pinned(shape, mask, x, kv, yc, ws, per_request, drop=()):
    wc = G.MS.weights_array(G.dev_weights(ws, shape))
    step = G.new_step(shape, mask)
    layers = _pinned_layers(kv, shape, per_request)
    if per_request:
        layers = [[None if b in drop else t for b, t in enumerate(row)] for row in layers]
    slots = [torch.full((shape.batch, shape.n_tokens, 2, shape.d_model), float("nan"), dtype=torch.bfloat16,
                        device=G.DEV) for _ in range(2)]
    y = torch.empty((shape.batch, shape.n_tokens, shape.d_model), dtype=torch.bfloat16, device=G.DEV)
    step.stack_forward(wc, G.to_dev(x, shape), G.to_dev(yc, shape), None if per_request else layers, y,
                       pinned=True, slots=slots, copy_stream=torch.cuda.Stream(),
                       per_request=layers if per_request else None)
    torch.cuda.synchronize()
    return G.to_np(y)


@pytest.mark.parametrize("shape", [PLAIN, TEXT], ids=lambda s: s.name)
def test_per_request_host_caches_equal_the_contiguous_layout(shape):
    ws, xt, kv, yc = _inputs(shape, 71)
    mask = _masks(shape, (0.3, 0.1, 0.55), 5)
    x = W.edited_hidden(shape, 71, xt, mask)
    y_c = _run_pinned(shape, mask, x, kv, yc, ws, per_request=False)
    y_r = _run_pinned(shape, mask, x, kv, yc, ws, per_request=True)
    np.testing.assert_array_equal(y_r, y_c)
    G.assert_close(y_r, oracle.masked_stack(x, mask, kv, yc, ws, shape, round_p=True), "bf16",
                   "per-request caches", blocks=shape.n_layers, inp=x)


def test_request_that_recomputes_nothing_reads_no_cache():
    shape = PLAIN
    ws, xt, kv, yc = _inputs(shape, 72)
    mask = _masks(shape, (0.3, 0.0, 0.2), 6)
    x = W.edited_hidden(shape, 72, xt, mask)
    y_c = _run_pinned(shape, mask, x, kv, yc, ws, per_request=False)
    y_r = _run_pinned(shape, mask, x, kv, yc, ws, per_request=True, drop=(1,))   # its caches are NULL
    np.testing.assert_array_equal(y_r, y_c)
    np.testing.assert_array_equal(y_r[1], np.asarray(yc[1], np.float64))


@pytest.mark.parametrize("streamed", [True, False], ids=["streamed", "resident"])
def test_requests_joining_and_leaving_match_the_oracle(streamed):
    """Three requests with their own masks, caches and per-step inputs: r0 runs steps 0-2, r1
    joins at step 1 for two steps, r2 at step 2 for one; every step's output of every request
    equals the oracle's masked stack of that request alone."""
    shape = TEXT if streamed else PLAIN
    one = shape.replace(batch=1)
    ws, xt, kv, yc = _inputs(shape, 73)
    mask = _masks(shape, (0.25, 0.5, 0.05), 7)
    wc = G.MS.weights_array(G.dev_weights(ws, shape))
    eng = CB.ContinuousBatcher(shape, wc, 3, streamed=streamed)
    layers = _pinned_layers(kv, shape, True) if streamed else None
    reqs = []
    for b, (join, steps) in enumerate(((0, 3), (1, 2), (2, 1))):
        cache = [layers[l][b] for l in range(shape.n_layers)] if streamed else \
                [G.to_dev(kv[l][b], shape) for l in range(shape.n_layers)]
        reqs.append((join, CB.Request(mask[b], None, G.to_dev(yc[b], shape), cache, steps)))
    xs = {}   # per (request, step) seeded inputs
    for b in range(3):
        for s in range(3):
            xs[b, s] = W.edited_hidden(one, 100 + 10 * b + s, xt[b:b + 1], mask[b:b + 1])[0]
    active = []
    for s in range(3):
        for b, (join, r) in enumerate(reqs):
            if join == s:
                assert eng.join(r)
                active.append(b)
        for b in active:
            reqs[b][1].x = G.to_dev(xs[b, s], shape)
        running = list(active)
        done = eng.step()
        torch.cuda.synchronize()
        for b in running:
            r = reqs[b][1]
            ref = oracle.masked_stack(xs[b, s][None], mask[b:b + 1], kv[:, b:b + 1], yc[b:b + 1], ws, one,
                                      round_p=True)[0]
            G.assert_close(G.to_np(r.y), ref, "bf16", f"request {b} step {s}", blocks=shape.n_layers,
                           inp=xs[b, s])
        for r in done:
            active.remove(next(b for b in active if reqs[b][1] is r))
        if s == 1:   # three running (r2 joins next step): the batch is full for a fourth
            assert eng.free() == 1 and eng.join(CB.Request(mask[0], None, None, None, 1)) and eng.free() == 0
            assert not eng.join(CB.Request(mask[0], None, None, None, 1))
            eng.joining.clear()
    assert not active   # every request left after its last step
    assert eng.step() == []
