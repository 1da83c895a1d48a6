"""The copy figures of a step context (span-merged host-to-device copies of one
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


def _spans(mask, gap_rows, recomputes):
    """Unmasked runs of each recomputing request, merged across masked gaps of <= gap_rows."""
    out = []
    for b, m in enumerate(mask):
        if not recomputes[b]:
            continue
        runs, n, N = [], 0, len(m)
        while n < N:
            while n < N and m[n]:
                n += 1
            if n >= N:
                break
            n0 = n
            while n < N and not m[n]:
                n += 1
            if runs and n0 - runs[-1][1] <= gap_rows:
                runs[-1][1] = n
            else:
                runs.append([n0, n])
        out += runs
    return out


@pytest.mark.parametrize("d_model", [256, 3072])
def test_copy_rows_are_the_merged_unmasked_runs(d_model):
    shape = W.ModelShape("spans", 2, d_model, d_model // 64, 4, 32, 32, dtype="bf16", batch=3)
    g = np.random.default_rng(5)
    mask = np.zeros((3, shape.n_image), np.uint8)
    mask[0, g.choice(shape.n_image, 300, replace=False)] = 1      # scattered: many short gaps
    mask[1, 100:400] = 1                                           # one long gap
    # request 2 recomputes nothing: no copies for it
    step = G.new_step(shape, mask)
    info = step.info()
    row_bytes = 2 * d_model * 2
    spans = _spans(mask, (512 * 1024) // row_bytes, [True, True, False])   # gaps up to 512 KiB merge
    assert info.copy_spans == len(spans)
    assert info.copy_rows == sum(b - a for a, b in spans)
    unmasked = int((mask[:2] == 0).sum())
    assert info.copy_rows >= unmasked


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
