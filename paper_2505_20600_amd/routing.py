"""Cluster-level routing simulation with the mask-aware policy (Sec. 4.3, Alg. 2).

Host-only: worker replicas serve requests by step-level continuous batching
(a request joins its worker's running batch at the next denoising-step
boundary and leaves after its last step); the latency of one step of a batch
is the Alg. 1 pipeline latency of that batch under the fitted linear cost
models (``mask_batch_cost`` of the native library). New requests are routed
on arrival by Alg. 2 (``mask_route_request``): among the workers with room in
their batch, the least pipeline latency of the worker's batch with the
request added.

When no worker has room the request waits in a FIFO queue and is routed at
the next step boundary that frees a slot. Arrivals are Poisson; mask ratios
are drawn log-uniform (the heterogeneous batch workload's distribution).

Usage: python -m paper_2505_20600_amd.routing --comp 0.05 0.004 --load 0.2 0.02
       (per-block intercept ms and slope ms/GFLOP, ms/MB; from ``bench.py --fit``)
"""
from __future__ import annotations

import argparse
import heapq
import json
import math

import numpy as np

from . import maskstep as MS
from . import workloads as W

class _Worker:
    def __init__(self):
        self.running = []      # [masked, steps_left, arrival, rid]
        self.joining = []
        self.busy = False

    def load(self):
        return len(self.running) + len(self.joining)

    def masked(self):
        return [r[0] for r in self.running] + [r[0] for r in self.joining]


def draw_requests(n, rate_per_s, n_image, seed, ratio_lo=0.03, ratio_hi=0.80):
    """(arrival seconds, masked image tokens) of n Poisson arrivals with log-uniform mask ratios."""
    g = np.random.default_rng(np.random.SeedSequence([9, 0, seed]))
    t = np.cumsum(g.exponential(1.0 / rate_per_s, n))
    r = np.exp(g.uniform(math.log(ratio_lo), math.log(ratio_hi), n))
    return list(zip(t.tolist(), [max(1, int(round(x * n_image))) for x in r]))


def simulate(desc, model, requests, n_workers, max_batch, steps_per_request, decisions=None):
    """Latency (seconds) of every request, in arrival order. With a list in ``decisions``,
    every routing decision is appended as (request masked tokens, every worker's running
    and joining masked tokens, chosen worker)."""
    workers = [_Worker() for _ in range(n_workers)]
    lat = [None] * len(requests)
    queue = []           # request ids waiting for room
    events = []          # (time, kind, seq, payload): kind 0 = step end, 1 = arrival
    seq = 0
    for rid, (t, _) in enumerate(requests):
        events.append((t, 1, seq, rid))
        seq += 1
    heapq.heapify(events)

    def step_ms(masked):
        return MS.mask_batch_cost(desc, model, masked)[2]

    def pick(masked):
        return MS.mask_route_request(desc, model, [w.masked() for w in workers], max_batch, masked)[0]

    def start(i, now):
        nonlocal seq
        w = workers[i]
        w.running += w.joining
        w.joining = []
        if not w.running:
            w.busy = False
            return
        w.busy = True
        heapq.heappush(events, (now + step_ms([r[0] for r in w.running]) / 1e3, 0, seq, i))
        seq += 1

    def assign(rid, now):
        i = pick(requests[rid][1])
        if decisions is not None:
            decisions.append((requests[rid][1], [w.masked() for w in workers], i))
        if i < 0:
            return False
        workers[i].joining.append([requests[rid][1], steps_per_request, requests[rid][0], rid])
        if not workers[i].busy:
            start(i, now)
        return True

    while events:
        now, kind, _, x = heapq.heappop(events)
        if kind == 1:
            if not assign(x, now):
                queue.append(x)
            continue
        w = workers[x]
        keep = []
        for r in w.running:
            r[1] -= 1
            if r[1] == 0:
                lat[r[3]] = now - r[2]
            else:
                keep.append(r)
        w.running = keep
        while queue and assign(queue[0], now):
            queue.pop(0)
        start(x, now)
    return lat


def summarize(lat):
    a = np.asarray(lat, float)
    return {"mean_s": round(float(a.mean()), 4), "p50_s": round(float(np.percentile(a, 50)), 4),
            "p95_s": round(float(np.percentile(a, 95)), 4), "p99_s": round(float(np.percentile(a, 99)), 4)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="c4", choices=sorted(W.CONFIGS))
    ap.add_argument("--comp", nargs=2, type=float, required=True, metavar=("MS0", "MS_PER_GFLOP"))
    ap.add_argument("--load", nargs=2, type=float, required=True, metavar=("MS0", "MS_PER_MB"))
    ap.add_argument("--workers", type=int, default=8)
    ap.add_argument("--max-batch", type=int, default=8)
    ap.add_argument("--steps", type=int, default=20, help="denoising steps per request")
    ap.add_argument("--requests", type=int, default=2000)
    ap.add_argument("--load-factor", type=float, default=0.8,
                    help="arrival rate as a fraction of the cluster's estimated capacity")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    shape = W.CONFIGS[args.workload]
    desc = MS.model_desc(shape, max_batch=args.max_batch)
    elt = 2 if shape.dtype == "bf16" else 4
    model = MS.CostModel(args.comp[0], args.comp[1], args.load[0], args.load[1], 2.0 * shape.d_model * elt)
    # capacity estimate: full batches of mean-ratio requests
    mean_masked = int(round(0.2345 * shape.n_image))
    step_s = MS.mask_batch_cost(desc, model, [mean_masked] * args.max_batch)[2] / 1e3
    capacity = args.workers * args.max_batch / (step_s * args.steps)
    reqs = draw_requests(args.requests, args.load_factor * capacity, shape.n_image, args.seed)
    out = {"workload": args.workload, "workers": args.workers, "max_batch": args.max_batch, "steps": args.steps,
           "requests": args.requests, "arrival_per_s": round(args.load_factor * capacity, 3),
           "model": {"comp": args.comp, "load": args.load}}
    out["mask-aware"] = summarize(simulate(desc, model, reqs, args.workers, args.max_batch, args.steps))
    print(json.dumps(out))


if __name__ == "__main__":
    main()
