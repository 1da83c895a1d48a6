"""Shared helpers of the GPU parity tests: device copies of the seeded inputs,
one step through the C ABI (whole-stack call or per-block calls), and the
parity gate."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W
from tests import parity_gate as PG

DEV = "cuda:0"
TOL = PG.TOL


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


max_rel_err = PG.max_rel_err
elem_rel_err = PG.elem_rel_err


def assert_close(got, ref, dtype, what="", *, blocks, inp=None):
    """Both error measures within the bound after ``blocks`` blocks between the shared
    input and the compared tensor; ``inp``: the compared rows' values on entering those
    blocks when they travel the residual path (tests/parity_gate)."""
    ok, e1, e2, lim = PG.check(got, ref, dtype, blocks, inp)
    print(f"[parity] {what}: max-norm rel err {e1:.3e}, element-wise {e2:.3e} (bound {lim:.3g}, "
          f"{blocks} block(s))", flush=True)
    assert e1 <= lim, f"{what}: max-norm relative error {e1:.3e} > {lim:.3g} ({blocks} block(s))"
    assert e2 <= lim, f"{what}: element-wise relative error {e2:.3e} > {lim:.3g} ({blocks} block(s))"


def new_step(shape, mask_np, stream=None):
    desc = MS.model_desc(shape)
    nbytes = MS.mask_workspace_bytes(desc, shape.batch)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    d_mask = torch.as_tensor(np.ascontiguousarray(mask_np, np.uint8)).to(DEV)
    return MS.MaskStep(desc, shape.batch, d_mask, ws, stream)


def run_stack(shape, mask, x, kv_cache, y_cache, weights, *, pinned=False, serialize=False,
              aliased=False, poison_cache=False, n_slots=2, dense_prefix=0, inputs=False, return_kv=True):
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
    kv_out = None if (pinned or not return_kv) else [to_np(t) for t in kv_layers]
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


# ------------------------------------------------------------------ a step through the per-block calls

def _pinned(a, shape):
    t = torch.empty(a.shape, dtype=tdtype(shape), pin_memory=True)
    t.copy_(torch.as_tensor(np.ascontiguousarray(a, np.float32)).to(tdtype(shape)))
    return t


def run_block_by_block(shape, mask, x, cache, yc, weights, *, form="kv", n_slots=2, keep_kv=True):
    """One step through the per-block calls: mask_gather_rows; per layer the cache load
    (form "kv": cache_prefetch_layer of the image rows of ``cache`` [L][B][T][2][d] from
    pinned host memory; "y": cache_prefetch_inputs of the block inputs [L][B][N][d] and
    mask_recompute_kv; "resident": ``cache`` copied to HBM, the layer's buffer passed as
    the working K/V) and mask_block_forward; mask_scatter_rows. Loads run on a copy
    stream through a ring of ``n_slots`` device slots ordered by events.

    Returns ``(y, snaps, rows)``: the output, per layer (block input rows, block output
    rows, working K/V after the block or None) as float64, and the packed row table."""
    L, B, T, N, d = shape.n_layers, shape.batch, shape.n_tokens, shape.n_image, shape.d_model
    dt = tdtype(shape)
    dw = dev_weights(weights, shape)
    step = new_step(shape, mask)
    M = step.info().rows
    xm = torch.empty((max(M, 1), d), dtype=dt, device=DEV)
    d_x, d_yc = to_dev(x, shape), to_dev(yc, shape)
    cs = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    copied = [torch.cuda.Event() for _ in range(n_slots)]
    consumed = [torch.cuda.Event() for _ in range(n_slots)]
    for e in copied + consumed:
        e.record(copy)                      # creates the HIP events before the library records them
    if form == "kv":
        host = [_pinned(np.asarray(cache[l])[:, shape.n_text:], shape) for l in range(L)]
        slots = [torch.full((B, T, 2, d), float("nan"), dtype=dt, device=DEV) for _ in range(n_slots)]
    elif form == "y":
        host = [_pinned(cache[l], shape) for l in range(L)]
        slots = [torch.full((B, N, d), float("nan"), dtype=dt, device=DEV) for _ in range(n_slots)]
        kv_work = torch.full((B, T, 2, d), float("nan"), dtype=dt, device=DEV)
    elif form == "resident":
        resident = [to_dev(cache[l], shape) for l in range(L)]
    else:
        raise ValueError(form)
    step.gather_rows(d_x, xm)
    snaps = []
    for l in range(L):
        j = l % n_slots
        wait = consumed[j] if l >= n_slots else None
        if form == "kv":
            step.prefetch_layer(l, host[l], slots[j], copy, wait_event=wait, signal_event=copied[j])
        elif form == "y":
            step.prefetch_inputs(l, host[l], slots[j], copy, wait_event=wait, signal_event=copied[j])
        if form != "resident":
            cs.wait_event(copied[j])
        x_in = xm[:M].clone()
        if form == "kv":
            kvbuf = slots[j]
        elif form == "y":
            step.recompute_kv(l, dw[l], slots[j], kv_work)
            kvbuf = kv_work
        else:
            kvbuf = resident[l]
        step.block_forward(l, dw[l], xm, kvbuf)
        snaps.append((x_in, xm[:M].clone(), kvbuf.clone() if keep_kv else None))
        if form != "resident":
            consumed[j].record(cs)
    y = torch.empty((B, T, d), dtype=dt, device=DEV)
    step.scatter_rows(xm, d_yc, y)
    torch.cuda.synchronize()
    out = [(to_np(a), to_np(b), None if c is None else to_np(c)) for a, b, c in snaps]
    rows = oracle.compact(mask, shape.n_text, shape.dual_stream)["rows"]
    step.close()
    return to_np(y), out, rows


def request_rows(rows, b, T):
    """Packed positions and token ids of request b's recomputed rows, in token order."""
    pos = np.flatnonzero(rows // T == b)
    toks = rows[pos] % T
    order = np.argsort(toks, kind="stable")
    return pos[order], toks[order]


def check_blocks(shape, snaps, rows, kv_of_layer, weights, what, *, requests=None, loaded_exact=True):
    """Each block's output (and fresh K/V rows) against the oracle's block applied to the
    GPU's own block input, at the one-block bound. ``kv_of_layer(l, b)``: request b's
    [T][2][d] K/V for the unmasked tokens as the block must see them. ``loaded_exact``:
    those rows were loaded (K/V caching), so the GPU's working K/V must hold them bit for
    bit; otherwise they were recomputed (Y caching) and are held to the one-block bound."""
    T = shape.n_tokens
    reqs = range(shape.batch) if requests is None else requests
    for l, (x_in, x_out, kv_gpu) in enumerate(snaps):
        got, ref, ins, kv_got, kv_ref, un_got, un_ref = [], [], [], [], [], [], []
        for b in reqs:
            pos, toks = request_rows(rows, b, T)
            if pos.size == 0:
                continue
            kv_b = kv_of_layer(l, b)
            out_b, kvw, h_b = oracle.block_rows(x_in[pos], toks, weights[l], kv_b, shape, oracle.bf16_round,
                                                round_p=True, return_h=True)
            got.append(x_out[pos])
            ref.append(out_b)
            ins.append(h_b)
            if kv_gpu is None:
                continue
            kv_got.append(kv_gpu[b, toks])
            kv_ref.append(kvw[toks])
            keep = np.setdiff1d(np.arange(shape.n_text, T), toks)
            if loaded_exact:
                np.testing.assert_array_equal(kv_gpu[b, keep], kv_b[keep], err_msg=f"{what} layer {l} request {b}")
            else:
                un_got.append(kv_gpu[b, keep])
                un_ref.append(kv_b[keep])
        if not got:
            continue
        assert_close(np.concatenate(got), np.concatenate(ref), shape.dtype, f"{what} block {l} output", blocks=1,
                     inp=np.concatenate(ins))
        if kv_got:
            assert_close(np.concatenate(kv_got), np.concatenate(kv_ref), shape.dtype, f"{what} block {l} fresh K/V",
                         blocks=1)
        if un_got and sum(a.size for a in un_got):
            assert_close(np.concatenate(un_got), np.concatenate(un_ref), shape.dtype,
                         f"{what} block {l} recomputed unmasked K/V", blocks=1)
