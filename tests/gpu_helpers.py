"""Shared helpers of the GPU parity tests: device copies of the seeded inputs,
one step through the C ABI, and the error metric."""
from __future__ import annotations

import numpy as np
import torch

from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W

DEV = "cuda:0"
# Max relative error of a tensor in the max norm, max|g - r| / max|r|.
TOL = {"fp32": 1e-4, "bf16": 2e-2}
# Element-wise guard, |g_i - r_i| / max(|r_i|, rms(r)): fp32 keeps the same
# 1e-4; for bf16 it is derived from the arithmetic. Rounding the softmax
# probabilities to bf16 before the PV product (the MFMA operand type) already
# moves the oracle by 0.0144 after one block and 0.021 after three under this
# measure, and two bf16 trajectories (GPU fp32 accumulation vs oracle float64)
# differ by about sqrt(2) times that, growing with depth; 0.1 leaves room for
# 28 layers while an indexing or algebra mistake gives O(1).
ELEM_TOL = {"fp32": 1e-4, "bf16": 1e-1}


def tdtype(shape):
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


def to_dev(a, shape):
    return torch.as_tensor(np.ascontiguousarray(a, np.float32)).to(DEV).to(tdtype(shape)).contiguous()


def to_np(t):
    return t.detach().to(torch.float64).cpu().numpy()


def dev_weights(weights, shape):
    out = []
    for w in weights:
        if isinstance(w, (tuple, list)):
            out.append(tuple({k: to_dev(v, shape) for k, v in ws.items()} for ws in w))
        else:
            out.append({k: to_dev(v, shape) for k, v in w.items()})
    return out


def max_rel_err(got, ref):
    """max_i |g_i - r_i| / max_i |r_i|: relative error in the max norm."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def elem_rel_err(got, ref):
    """max_i |g_i - r_i| / max(|r_i|, rms(r)): element-wise relative error with an RMS floor."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref ** 2))
    den = np.maximum(np.abs(ref), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(got - ref) / den))


def assert_close(got, ref, dtype, what=""):
    e1, e2 = max_rel_err(got, ref), elem_rel_err(got, ref)
    print(f"[parity] {what} max-norm rel err {e1:.3e} (tol {TOL[dtype]}), element-wise {e2:.3e} "
          f"(tol {ELEM_TOL[dtype]})", flush=True)
    assert e1 <= TOL[dtype], f"{what}: max-norm relative error {e1:.3e} > {TOL[dtype]}"
    assert e2 <= ELEM_TOL[dtype], f"{what}: element-wise relative error {e2:.3e} > {ELEM_TOL[dtype]}"


def new_step(shape, mask_np, stream=None):
    desc = MS.model_desc(shape)
    nbytes = MS.mask_workspace_bytes(desc, shape.batch)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    d_mask = torch.as_tensor(np.ascontiguousarray(mask_np, np.uint8)).to(DEV)
    return MS.MaskStep(desc, shape.batch, d_mask, ws, stream)


def run_stack(shape, mask, x, kv_cache, y_cache, weights, *, pinned=False, serialize=False,
              aliased=False, poison_cache=False, n_slots=2, dense_prefix=0, inputs=False):
    """One step through mask_stack_forward; returns (y, working kv per layer or None, step).
    With ``inputs`` the cache is Y caching's per-layer block inputs ``[L][B][N][d]``."""
    if inputs:
        return _run_stack_y(shape, mask, x, kv_cache, y_cache, weights, pinned=pinned, serialize=serialize,
                            n_slots=n_slots, dense_prefix=dense_prefix)
    dw = dev_weights(weights, shape)
    wc = MS.weights_array(dw)
    d_x = to_dev(x, shape)
    d_yc = to_dev(y_cache, shape) if y_cache is not None else None
    step = new_step(shape, mask)
    L = shape.n_layers
    if pinned:
        host = []
        for l in range(L):
            img = np.asarray(kv_cache[l])[:, shape.n_text:]
            t = torch.empty(img.shape, dtype=tdtype(shape), pin_memory=True)
            t.copy_(torch.as_tensor(np.ascontiguousarray(img, np.float32)).to(tdtype(shape)))
            host.append(t)
        slots = [torch.full((shape.batch, shape.n_tokens, 2, shape.d_model), float("nan"),
                            dtype=tdtype(shape), device=DEV) for _ in range(n_slots)]
        kv_layers = host
    else:
        kv_layers = [to_dev(kv_cache[l], shape) for l in range(L)]
        if poison_cache:
            for t in kv_layers:
                t.fill_(float("nan"))
        slots = ()
    if dense_prefix:
        step.set_dense_prefix(dense_prefix)
    y = d_yc if aliased else torch.empty((shape.batch, shape.n_tokens, shape.d_model),
                                         dtype=tdtype(shape), device=DEV)
    cs = torch.cuda.current_stream()
    copy = cs if serialize else torch.cuda.Stream()
    step.stack_forward(wc, d_x, d_yc, kv_layers, y, pinned=pinned, slots=slots, stream=cs,
                       copy_stream=copy)
    torch.cuda.synchronize()
    kv_out = None if pinned else [to_np(t) for t in kv_layers]
    return to_np(y), kv_out, step


def _run_stack_y(shape, mask, x, yin, y_cache, weights, *, pinned, serialize, n_slots, dense_prefix):
    dw = dev_weights(weights, shape)
    wc = MS.weights_array(dw)
    d_x = to_dev(x, shape)
    d_yc = to_dev(y_cache, shape) if y_cache is not None else None
    step = new_step(shape, mask)
    L = shape.n_layers
    layers = []
    for l in range(L):
        t = torch.as_tensor(np.ascontiguousarray(yin[l], np.float32)).to(tdtype(shape))
        layers.append(t.pin_memory() if pinned else t.to(DEV))
    slots = ()
    if pinned:
        slots = [torch.full((shape.batch, shape.n_image, shape.d_model), float("nan"), dtype=tdtype(shape),
                            device=DEV) for _ in range(n_slots)]
    if dense_prefix:
        step.set_dense_prefix(dense_prefix)
    y = torch.empty((shape.batch, shape.n_tokens, shape.d_model), dtype=tdtype(shape), device=DEV)
    cs = torch.cuda.current_stream()
    copy = cs if serialize else torch.cuda.Stream()
    step.stack_forward(wc, d_x, d_yc, layers, y, pinned=pinned, slots=slots, stream=cs, copy_stream=copy,
                       inputs=True)
    torch.cuda.synchronize()
    return to_np(y), None, step
