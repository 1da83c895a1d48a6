"""Step-level continuous batching of mask-aware editing requests on one GPU
(Sec. 4.2 "Continuous Batching").

A request joins the running batch at the next denoising-step boundary and
leaves as soon as its last step is done; every step runs the whole stack
(``mask_stack_forward``) once over the batch as it stands. Two cache forms:

* streamed (pinned host caches): the batch is re-formed every step from the
  running requests, whose caches stay in their own pinned buffers (the
  ``per_request`` host pointers of ``ms_kv_source``); device slots of
  ``max_batch`` requests carry the loads;
* resident (caches in HBM): ``max_batch`` fixed slots with one per-layer
  working K/V buffer each; a joining request's cache is copied into its slot
  once, and a free slot runs as a request with an empty mask, which
  recomputes and loads nothing (models without text rows).

The step's output for each request is left in ``Request.y``; what the next
step's input is (the sampler's update) is the caller's business: it sets
``Request.x`` before the next ``step()``.

``python -m paper_2505_20600_amd.batching --workload c4`` measures the
throughput of full batches against ``max_batch`` (one JSON line).
"""
from __future__ import annotations

import argparse
import json
import time

import numpy as np
import torch

from . import maskstep as MS
from . import workloads as W


class Request:
    """mask: uint8 [N] (nonzero = masked); x, ycache: device [T][d]; cache: [L] per-layer cache,
    device [T][2][d] (resident) or pinned host [N][2][d] (streamed); steps: denoising steps left."""

    def __init__(self, mask, x, ycache, cache, steps):
        self.mask = np.ascontiguousarray(mask, np.uint8)
        self.x = x
        self.ycache = ycache
        self.cache = cache
        self.steps = steps
        self.y = None
        self.slot = None


class ContinuousBatcher:
    def __init__(self, shape, weights_c, max_batch, *, streamed, stream=None, copy_stream=None):
        if not streamed and shape.n_text > 0:
            raise ValueError("resident slots need a model without text rows (a free slot must recompute nothing)")
        self.shape = shape
        self.wc = weights_c
        self.max_batch = max_batch
        self.streamed = streamed
        dev, tdt = "cuda", (torch.bfloat16 if shape.dtype == "bf16" else torch.float32)
        T, N, d, L = shape.n_tokens, shape.n_image, shape.d_model, shape.n_layers
        self.desc = MS.model_desc(shape, max_batch=max_batch)
        self.ws = torch.empty(MS.mask_workspace_bytes(self.desc, max_batch), dtype=torch.uint8, device=dev)
        self.x = torch.empty((max_batch, T, d), dtype=tdt, device=dev)
        self.yc = torch.empty_like(self.x)
        self.y = torch.empty_like(self.x)
        self.stream = stream or torch.cuda.current_stream()
        self.copy_stream = copy_stream or (torch.cuda.Stream() if streamed else None)
        if streamed:
            self.slots = [torch.empty((max_batch, T, 2, d), dtype=tdt, device=dev) for _ in range(L)]
            self.running = []
        else:
            self.kv = [torch.empty((max_batch, T, 2, d), dtype=tdt, device=dev) for _ in range(L)]
            self.slot_req = [None] * max_batch
        self.joining = []

    def free(self):
        n = len(self.running) if self.streamed else sum(r is not None for r in self.slot_req)
        return self.max_batch - n - len(self.joining)

    def join(self, req: Request) -> bool:
        """Queue ``req`` for the next step; False when the batch is full."""
        if self.free() <= 0:
            return False
        self.joining.append(req)
        return True

    def _admit(self):
        for req in self.joining:
            if self.streamed:
                self.running.append(req)
                continue
            s = self.slot_req.index(None)
            self.slot_req[s] = req
            req.slot = s
            with torch.cuda.stream(self.stream):
                for l, t in enumerate(req.cache):
                    self.kv[l][s].copy_(t)     # the request's working K/V from now on
        self.joining = []

    def step(self):
        """One denoising step of the running batch; returns the requests that finished."""
        self._admit()
        N = self.shape.n_image
        if self.streamed:
            reqs = list(self.running)
            if not reqs:
                return []
            B = len(reqs)
            order = list(range(B))
        else:
            reqs = self.slot_req
            if all(r is None for r in reqs):
                return []
            B = self.max_batch
            order = [i for i, r in enumerate(reqs) if r is not None]
        mask = np.zeros((B, N), np.uint8)
        with torch.cuda.stream(self.stream):
            for i in order:
                r = reqs[i]
                mask[i] = r.mask
                self.x[i].copy_(r.x)
                self.yc[i].copy_(r.ycache)
            d_mask = torch.as_tensor(mask).to(self.x.device, non_blocking=False)
        st = MS.MaskStep(self.desc, B, d_mask, self.ws, self.stream)
        if self.streamed:
            per_req = [[r.cache[l] for r in reqs] for l in range(self.shape.n_layers)]
            st.stack_forward(self.wc, self.x[:B], self.yc[:B], None, self.y[:B], pinned=True, slots=self.slots,
                             stream=self.stream, copy_stream=self.copy_stream, per_request=per_req)
        else:
            st.stack_forward(self.wc, self.x, self.yc, self.kv, self.y, stream=self.stream)
        st.close()
        done = []
        with torch.cuda.stream(self.stream):
            for i in order:
                r = reqs[i]
                r.y = self.y[i].clone()
                r.steps -= 1
                if r.steps <= 0:
                    done.append(r)
        for r in done:
            if self.streamed:
                self.running.remove(r)
            else:
                self.slot_req[r.slot] = None
        return done


def main(argv=None):
    ap = argparse.ArgumentParser(description="throughput of step-level continuous batching vs max batch size")
    ap.add_argument("--workload", default="c4", choices=("c2", "c3", "c4", "c5"))
    ap.add_argument("--batches", default="1,2,4,8")
    ap.add_argument("--layers", type=int, default=0, help="layers of the stack (0: the workload's)")
    ap.add_argument("--steps", type=int, default=4, help="denoising steps per request")
    ap.add_argument("--requests", type=int, default=24)
    ap.add_argument("--streamed", action="store_true", help="pinned host caches streamed per step")
    args = ap.parse_args(argv)
    shape = W.CONFIGS[args.workload]
    if args.layers:
        shape = shape.replace(n_layers=args.layers)
    cfg = W.CONFIG_IDS[args.workload]
    dev = "cuda"
    tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    g = torch.Generator(device=dev)
    g.manual_seed(4000 + cfg)
    T, N, d, L = shape.n_tokens, shape.n_image, shape.d_model, shape.n_layers
    # weights by the seeded device recipe (N(0, 0.02), LN identity)
    ws = []
    for _ in range(L):
        def one():
            f = shape.mlp_mult * d
            w = {k: (torch.randn(s, generator=g, device=dev) * 0.02).to(tdt) for k, s in
                 {"w_qkv": (3 * d, d), "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,), "w_1": (f, d), "b_1": (f,),
                  "w_2": (d, f), "b_2": (d,)}.items()}
            w.update({"ln1_g": torch.ones(d, device=dev, dtype=tdt), "ln2_g": torch.ones(d, device=dev, dtype=tdt),
                      "ln1_b": torch.zeros(d, device=dev, dtype=tdt), "ln2_b": torch.zeros(d, device=dev, dtype=tdt)})
            return w
        ws.append((one(), one()) if shape.dual_stream else one())
    wc = MS.weights_array(ws)
    # one template cache shared by all requests (each joins with its own working copy)
    if args.streamed:
        cache = []
        for _ in range(L):
            h = torch.empty((N, 2, d), dtype=tdt, pin_memory=True)
            h.copy_((torch.randn((N, 2, d), generator=g, device=dev) * 0.5).to(tdt))
            cache.append(h)
    else:
        cache = [(torch.randn((T, 2, d), generator=g, device=dev) * 0.5).to(tdt) for _ in range(L)]
    x0 = torch.randn((T, d), generator=g, device=dev).to(tdt)
    yc0 = torch.randn((T, d), generator=g, device=dev).to(tdt)
    results = []
    for mb in [int(v) for v in args.batches.split(",")]:
        eng = ContinuousBatcher(shape, wc, mb, streamed=args.streamed)
        masks = [W.workload_mask(args.workload, shape.replace(batch=1), mask_id=i)[0] for i in range(args.requests)]
        pending = list(range(args.requests))
        steps_done, masked_rows, t_steps, lat = 0, 0, 0.0, []
        joined_at = {}
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while pending or eng.free() < mb:
            while pending and eng.free() > 0:
                i = pending.pop(0)
                eng.join(Request(masks[i], x0, yc0, cache, args.steps))
                joined_at[i] = steps_done
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(eng.stream)
            n_rows = sum(int(r.mask.sum()) + shape.n_text for r in
                         (eng.running + eng.joining if eng.streamed else
                          [r for r in eng.slot_req if r is not None] + eng.joining))
            eng.step()
            b.record(eng.stream)
            torch.cuda.synchronize()
            t_steps += a.elapsed_time(b)
            steps_done += 1
            masked_rows += n_rows
        wall = time.perf_counter() - t0
        results.append({"max_batch": mb, "steps": steps_done, "ms_per_step": round(t_steps / steps_done, 3),
                        "masked_tokens_per_s": round(masked_rows / (t_steps / 1e3), 1),
                        "requests_per_s": round(args.requests / (t_steps / 1e3), 3),
                        "wall_s": round(wall, 2)})
    print(json.dumps({"metric": "step-level continuous batching: throughput vs max batch",
                      "workload": args.workload, "layers": L, "steps_per_request": args.steps,
                      "requests": args.requests, "streamed": args.streamed, "results": results}))


if __name__ == "__main__":
    main()
