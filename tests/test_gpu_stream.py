"""The copy figures of a step context (the planned host-to-device copies of one
cached block) and the profiler's interval timeline, through the C ABI."""
import numpy as np
import pytest
import torch

from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the gpu-marked tests must run on an MI355X")


@pytest.mark.parametrize("d_model", [256, 3072])
def test_copy_figures_are_the_planned_copies(d_model):
    """copy_spans / copy_rows of a step context are the cache-load plans of its
    recomputing requests (mask_plan_copies, a command priced at 512 KiB)."""
    shape = W.ModelShape("spans", 2, d_model, d_model // 64, 4, 32, 32, dtype="bf16", batch=4)
    g = np.random.default_rng(5)
    mask = np.zeros((4, shape.n_image), np.uint8)
    mask[0, g.choice(shape.n_image, 300, replace=False)] = 1      # scattered: many short gaps
    mask[1, 100:400] = 1                                           # one long gap
    mask[2].reshape(32, 32)[8:24, 4:28] = 1                        # a rectangle: a strided copy at d 3072
    # request 3 recomputes nothing: no copies for it
    step = G.new_step(shape, mask)
    info = step.info()
    C = (512 * 1024) / (2 * d_model * 2)
    plans = [MS.mask_plan_copies(mask[b], 32, 32, C) for b in range(3)]
    assert info.copy_spans == sum(len(p) for p in plans)
    assert info.copy_rows == sum(w * h for p in plans for _, w, h in p)
    assert info.copy_rows >= int((mask[:3] == 0).sum())
    if d_model == 3072:
        assert any(h > 1 for p in plans for _, _, h in p)
    plans_y = [MS.mask_plan_copies(mask[b], 32, 32, 2 * C) for b in range(3)]   # Y rows: half the bytes
    assert info.copy_spans_y == sum(len(p) for p in plans_y)
    assert info.copy_rows_y == sum(w * h for p in plans_y for _, w, h in p)


def test_strided_cache_loads_match_resident(monkeypatch):
    """Blob masks with a command priced at 8 KiB (a few 1 KiB K/V rows), so the
    loads are strided 2-D copies around the blobs: streamed == resident, bit for
    bit, in both cache forms."""
    monkeypatch.setenv("MS_COPY_GAP_BYTES", "8192")
    shape = W.ModelShape("strided", 3, 256, 2, 4, 16, 16, n_text=0, dtype="bf16", batch=2)
    ws = W.stack_weights(shape, 91, random_ln=True, std=0.03)
    xt = W.template_hidden(shape, 91)
    kv = np.stack([W.synthetic_kv_cache(shape, 91, l) for l in range(shape.n_layers)])
    yc = W.synthetic_y_cache(shape, 91)
    mask = np.stack([W.blob_mask(16, 16, r, W.rng(91, 3, b)) for b, r in enumerate((0.3, 0.5))])
    x = W.edited_hidden(shape, 91, xt, mask)
    plans = [MS.mask_plan_copies(m, 16, 16, 8192 / (2 * 256 * 2)) for m in mask]
    assert any(h > 1 for p in plans for _, _, h in p)
    y_res, _, step = G.run_stack(shape, mask, x, kv, yc, ws)
    assert step.info().copy_spans == sum(len(p) for p in plans)
    y_kv, _, _ = G.run_stack(shape, mask, x, kv, yc, ws, pinned=True, n_slots=2)
    np.testing.assert_array_equal(y_kv, y_res)
    yin = np.stack([np.asarray(yc)[:, shape.n_text:]] * shape.n_layers)
    y_y, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True, pinned=True, n_slots=2)
    y_yres, _, _ = G.run_stack(shape, mask, x, yin, yc, ws, inputs=True)
    np.testing.assert_array_equal(y_y, y_yres)


def test_profiler_intervals_match_the_totals():
    shape = W.ModelShape("prof", 3, 256, 2, 4, 16, 16, dtype="bf16", batch=2)
    ws = W.stack_weights(shape, 90, random_ln=True, std=0.03)
    xt = W.template_hidden(shape, 90)
    kv = np.stack([W.synthetic_kv_cache(shape, 90, l) for l in range(shape.n_layers)])
    yc = W.synthetic_y_cache(shape, 90)
    mask = np.zeros((2, shape.n_image), np.uint8)
    mask[:, 40:120] = 1
    MS.profiler_start(MS.KERNEL_CLASSES, capacity=4096)
    G.run_stack(shape, mask, xt, kv, yc, ws, pinned=True, n_slots=2)
    tot = MS.profiler_stop()
    iv = MS.profiler_intervals()
    dropped = tot.pop("_dropped")
    assert dropped == 0
    assert len(iv) == sum(n for _, n in tot.values())
    assert any(c == "copy" for c, _, _ in iv) and any(c == "attention" for c, _, _ in iv)
    assert min(a for _, a, _ in iv) == pytest.approx(0.0, abs=1e-6)
    for c, a, b in iv:
        assert 0.0 <= a <= b
    for c, (ms, n) in tot.items():
        assert sum(b - a for cc, a, b in iv if cc == c) == pytest.approx(ms, rel=1e-3, abs=1e-3)


@pytest.mark.parametrize("n_slots,prefix,form", [(2, 0, "kv"), (5, 0, "kv"), (5, 2, "kv"), (2, 3, "kv"),
                                                 (5, 0, "y"), (2, 2, "y")])
def test_back_to_back_steps_of_two_contexts_share_slots_exactly(n_slots, prefix, form):
    """Steps of two step contexts (different masks, different host caches) issued
    back to back through the same slots, with no synchronisation between the
    calls: a call's loads must not overwrite a slot the previous call's blocks
    still read (with MS_KV_LOADS_AHEAD the next call's first loads start under them). With a dense
    prefix on one context the two stream different numbers of blocks; a third
    context (every token masked) streams nothing, and the same context may run
    twice in a row. Every output equals the same step run alone."""
    shape = W.ModelShape("b2b", 5, 256, 2, 4, 16, 16, n_text=0, dtype="bf16", batch=2)
    ws = W.stack_weights(shape, 93, random_ln=True, std=0.03)
    dw = G.dev_weights(ws, shape)
    wc = MS.weights_array(dw)
    xt = W.template_hidden(shape, 93)
    d_yc = G.to_dev(W.synthetic_y_cache(shape, 93), shape)
    masks = [np.stack([W.blob_mask(16, 16, r, W.rng(93, 3, 10 * c + b)) for b, r in enumerate(rs)])
             for c, rs in enumerate(((0.2, 0.4), (0.35, 0.1)))]
    masks.append(np.ones_like(masks[0]))   # a third context that streams nothing (every token masked)
    steps = [G.new_step(shape, m) for m in masks]
    if prefix:
        steps[1].set_dense_prefix(prefix)   # the two contexts stream different numbers of blocks
    hosts = []
    for c in range(3):
        layers = []
        for l in range(shape.n_layers):
            # K/V form: [B][N][2][d] rows; Y form: the block inputs [B][N][d]
            img = (W.synthetic_kv_cache(shape, 200 + c, l) if form == "kv"
                   else W.synthetic_y_cache(shape, 200 + 10 * c + l))[:, shape.n_text:]
            t = torch.empty(img.shape, dtype=torch.bfloat16, pin_memory=True)
            t.copy_(torch.as_tensor(np.ascontiguousarray(img, np.float32)).to(torch.bfloat16))
            layers.append(t)
        hosts.append(layers)
    xs = [G.to_dev(W.edited_hidden(shape, 93, xt, m), shape) for m in masks]
    slot_shape = ((shape.batch, shape.n_tokens, 2, shape.d_model) if form == "kv"
                  else (shape.batch, shape.n_image, shape.d_model))
    slots = [torch.full(slot_shape, float("nan"), dtype=torch.bfloat16, device=G.DEV) for _ in range(n_slots)]
    copy = torch.cuda.Stream()

    def call(c, y):
        steps[c].stack_forward(wc, xs[c], d_yc, hosts[c], y, pinned=True, slots=slots, copy_stream=copy,
                               inputs=form == "y", loads_ahead=True)

    alone = []
    for c in range(3):
        y = torch.empty_like(d_yc)
        call(c, y)
        torch.cuda.synchronize()
        alone.append(y)
    outs = []
    order = [0, 1] * 3 if n_slots == 5 else [0, 1, 2, 0, 2, 1, 1, 0]
    for c in order:
        y = torch.empty_like(d_yc)
        call(c, y)
        outs.append((c, y))
    torch.cuda.synchronize()
    assert not torch.equal(alone[0], alone[1])
    for c, y in outs:
        assert torch.equal(y, alone[c]), f"context {c}"


def test_many_slot_lists_back_to_back():
    """Steps of one context through 18 different lists of slot buffers in turn,
    then the first list again, back to back with MS_KV_LOADS_AHEAD and no
    synchronisation: more lists than the library keeps release rings for (16
    per device), so entries pass from list to list and the first list's entry
    is gone when it returns. Every output equals the step run alone."""
    shape = W.ModelShape("rings", 4, 256, 2, 4, 16, 16, n_text=0, dtype="bf16", batch=2)
    ws = W.stack_weights(shape, 94, random_ln=True, std=0.03)
    wc = MS.weights_array(G.dev_weights(ws, shape))
    xt = W.template_hidden(shape, 94)
    d_yc = G.to_dev(W.synthetic_y_cache(shape, 94), shape)
    mask = np.stack([W.blob_mask(16, 16, r, W.rng(94, 3, b)) for b, r in enumerate((0.25, 0.45))])
    step = G.new_step(shape, mask)
    host = [G._pinned(W.synthetic_kv_cache(shape, 94, l)[:, shape.n_text:], shape) for l in range(shape.n_layers)]
    x = G.to_dev(W.edited_hidden(shape, 94, xt, mask), shape)
    lists = [[torch.full((shape.batch, shape.n_tokens, 2, shape.d_model), float("nan"), dtype=torch.bfloat16,
                         device=G.DEV) for _ in range(2)] for _ in range(18)]
    copy = torch.cuda.Stream()

    def call(slots, y):
        step.stack_forward(wc, x, d_yc, host, y, pinned=True, slots=slots, copy_stream=copy, loads_ahead=True)

    alone = torch.empty_like(d_yc)
    call(lists[0], alone)
    torch.cuda.synchronize()
    outs = []
    for i in list(range(18)) + [0, 0, 5]:
        y = torch.empty_like(d_yc)
        call(lists[i], y)
        outs.append((i, y))
    torch.cuda.synchronize()
    for i, y in outs:
        assert torch.equal(y, alone), f"slot list {i}"


@pytest.mark.parametrize("pinned", [False, True], ids=["resident", "streamed"])
def test_step_replays_as_a_graph(pinned):
    """One step captured as a HIP graph (torch.cuda.graph) and replayed three times,
    with eager steps of another context through the same slots in between: every
    replay equals the eager step bit for bit. A captured call orders its loads after
    its own start, and so do the eager calls, which run without MS_KV_LOADS_AHEAD (a
    replay touches the slots between them)."""
    shape = W.ModelShape("graph", 3, 256, 2, 4, 16, 16, n_text=0, dtype="bf16", batch=2)
    ws = W.stack_weights(shape, 95, random_ln=True, std=0.03)
    wc = MS.weights_array(G.dev_weights(ws, shape))
    xt = W.template_hidden(shape, 95)
    d_yc = G.to_dev(W.synthetic_y_cache(shape, 95), shape)
    masks = [np.stack([W.blob_mask(16, 16, r, W.rng(95, 3, 10 * c + b)) for b, r in enumerate(rs)])
             for c, rs in enumerate(((0.3, 0.15), (0.2, 0.45)))]
    steps = [G.new_step(shape, m) for m in masks]
    xs = [G.to_dev(W.edited_hidden(shape, 95, xt, m), shape) for m in masks]
    kvs = []
    for c in range(2):
        layers = []
        for l in range(shape.n_layers):
            full = W.synthetic_kv_cache(shape, 300 + c, l)
            if pinned:
                t = torch.empty(full[:, shape.n_text:].shape, dtype=torch.bfloat16, pin_memory=True)
                t.copy_(torch.as_tensor(np.ascontiguousarray(full[:, shape.n_text:], np.float32)).to(torch.bfloat16))
            else:
                t = G.to_dev(full, shape)
            layers.append(t)
        kvs.append(layers)
    slots = [torch.empty((shape.batch, shape.n_tokens, 2, shape.d_model), dtype=torch.bfloat16, device=G.DEV)
             for _ in range(2)] if pinned else []
    copy = torch.cuda.Stream() if pinned else None

    def run(c, y, stream=None):
        if not pinned:   # the resident cache is also the working K/V: start each step from the cache
            kv = [t.clone() for t in kvs[c]]
        else:
            kv = kvs[c]
        steps[c].stack_forward(wc, xs[c], d_yc, kv, y, pinned=pinned, slots=slots, stream=stream,
                               copy_stream=copy)
        return kv

    y_ref = torch.empty_like(d_yc)
    run(0, y_ref)
    torch.cuda.synchronize()
    y_other = torch.empty_like(d_yc)
    run(1, y_other)
    torch.cuda.synchronize()
    # capture step 0 (resident: on a private copy of the cache that each replay restarts from)
    y_g = torch.empty_like(d_yc)
    kv_g = [t.clone() for t in kvs[0]] if not pinned else None
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    with torch.cuda.stream(cap):
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            steps[0].stack_forward(wc, xs[0], d_yc, kv_g if not pinned else kvs[0], y_g, pinned=pinned, slots=slots,
                                   copy_stream=copy)
    torch.cuda.synchronize()
    for i in range(3):
        if not pinned:
            for dst, src in zip(kv_g, kvs[0]):
                dst.copy_(src)
        y_g.fill_(float("nan"))
        graph.replay()
        y_o = torch.empty_like(d_yc)
        run(1, y_o)   # eager work of another context through the same slots
        torch.cuda.synchronize()
        assert torch.equal(y_g, y_ref), f"replay {i}"
        assert torch.equal(y_o, y_other), f"eager step after replay {i}"
