#!/usr/bin/env python3
"""Benchmark of the mask-aware K/V-cached denoising step on one MI355X.

One step = gather + every block of the stack (LN, QKV GEMM with the
fresh-K/V scatter, masked-query attention over all tokens, out-projection,
LN, MLP) + final scatter, over one synthetic request set (and, for the
streamed workloads, the per-layer cache loads from pinned host memory): one
mask_stack_forward. Steps cycle through seeded mask sets whose ratios follow
the workload's distribution; each mask set's step context (the mask
compaction, fixed over a request's denoising steps) is built once before the
timed steps and its cost reported separately.

Prints ONE JSON line on stdout. Default workload: the largest, a 19-block
dual-stream d=3072 bf16 stack over 4 requests of 4096 image + 512 text
tokens, each block's image K/V streamed from pinned host memory on a copy
stream, Gaussian-blob masks of ratio U[10%, 40%], and the Alg. 1 dense
prefix planned per mask set from per-block costs measured on this GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

METRIC = "masked-token step time (ms) & tokens/s vs mask ratio; % MFMA/HBM peak"
PEAK = {"bf16_mfma_tflops": 2500.0, "fp32_mfma_tflops": 157.3, "hbm_gbs": 8000.0}

DESCR = {
    "c1": "single pre-LN block, fp32, d=256, 4 heads, MLP 4x GELU, 32x32 grid = 1024 tokens, "
          "12x17 rectangle mask (19.9%)",
    "c2": "12-block stack, bf16, d=768, 12 heads, MLP 4x, 64x64 grid = 4096 tokens, HBM-resident "
          "per-layer K/V cache, union of 1-4 random ellipses, ratio U[5%,60%]",
    "c3": "28-block stack, bf16, d=1152, 16 heads (head_dim 72), MLP 4x, 4096 tokens, K/V cache "
          "streamed per layer from pinned host memory, ellipse masks 5/10/25/50/100%",
    "c4": "28-block d=1152 bf16 stack, heterogeneous batch of 8 x 4096 tokens, blob masks "
          "log-U[3%,80%], HBM-resident cache, varlen packing",
    "c5": "19-block dual-stream d=3072 bf16 stack, 24 heads (head_dim 128), batch 4, 4096 image "
          "+ 512 text tokens, image K/V streamed from pinned host memory, blob masks U[10%,40%]",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=40)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="c5", choices=sorted(DESCR))
    p.add_argument("--masks", type=int, default=8, help="distinct seeded mask sets cycled over the steps")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cache", default="kv", choices=("kv", "y"),
                   help="kv: per-layer K/V cache (Fig. 7); y: per-layer cached block inputs (Fig. 5 bottom)")
    p.add_argument("--no-profile-pass", action="store_true")
    p.add_argument("--trace-marks", action="store_true",
                   help="launch a marker kernel (torch's spin kernel) right before and after the profiled pass, "
                        "so that a rocprofv3 trace of this run can be cut to exactly the launches the roofline "
                        "averages (see --summarize-trace)")
    p.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                   help="only summarise a rocprofv3 kernel trace of a --trace-marks run: per kernel symbol over "
                        "the profiled pass, and the roofline kernel's family; with --pmc-fetch/--pmc-write/"
                        "--copy-fetch/--copy-write also its copy-calibrated HBM traffic per launch")
    p.add_argument("--family", help="with --summarize-trace: the bench kernel class to aggregate (e.g. gemm_up)")
    p.add_argument("--pmc-fetch")
    p.add_argument("--pmc-write")
    p.add_argument("--copy-fetch")
    p.add_argument("--copy-write")
    p.add_argument("--counters", action="append", default=[],
                   help="with --summarize-trace and --family: a rocprofv3 counter-collection CSV of a "
                        "--trace-marks run; per-dispatch averages of its counters over the family's launches")
    p.add_argument("--prefix", default="auto",
                   help="dense-prefix blocks for streamed caches: 'auto' (Alg. 1 planner on measured "
                        "per-block costs) or a fixed count")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device copy (HBM counter calibration) and exit")
    p.add_argument("--ceilings", action="store_true",
                   help="only measure this GPU's ceilings (a library bf16 GEMM at 8192^3, a device copy, "
                        "a pinned host-to-device copy), print one JSON line and exit")
    p.add_argument("--fit", type=int, default=0, metavar="K",
                   help="only fit the per-block cost models of Sec. 4.3 on K measured random batches of "
                        "the workload (compute vs FLOPs, cache load vs bytes), run the routing simulation "
                        "with them, print one JSON line and exit")
    return p.parse_args()


# ----------------------------------------------------------------------------- inputs


def make_inputs(key, shape, n_masks, torch, W, cache="kv"):
    cfg = W.CONFIG_IDS[key]
    dev = "cuda:0"
    tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    n_params = shape.n_layers * (12 * shape.d_model ** 2) * (2 if shape.dual_stream else 1)
    weights = []
    if n_params <= 300_000_000:
        for w in W.stack_weights(shape, cfg):
            sets = w if isinstance(w, tuple) else (w,)
            dev_sets = tuple({k: torch.as_tensor(v).to(dev).to(tdt) for k, v in s.items()} for s in sets)
            weights.append(dev_sets if shape.dual_stream else dev_sets[0])
    else:
        # large stacks: the same N(0, 0.02) recipe drawn by a seeded device generator
        g = torch.Generator(device=dev)
        g.manual_seed(1000 + cfg)
        d, f = shape.d_model, shape.mlp_mult * shape.d_model
        shapes = {"w_qkv": (3 * d, d), "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,), "w_1": (f, d),
                  "b_1": (f,), "w_2": (d, f), "b_2": (d,)}

        def one():
            w = {k: (torch.randn(s, generator=g, device=dev) * 0.02).to(tdt) for k, s in shapes.items()}
            for k in ("ln1_g", "ln2_g"):
                w[k] = torch.ones(d, device=dev, dtype=tdt)
            for k in ("ln1_b", "ln2_b"):
                w[k] = torch.zeros(d, device=dev, dtype=tdt)
            return w

        for _ in range(shape.n_layers):
            weights.append((one(), one()) if shape.dual_stream else one())
    masks, xs, ratios, unmasked = [], [], [], []
    xt = W.template_hidden(shape, cfg)
    for i in range(n_masks):
        if key == "c3":
            m = W.workload_mask(key, shape, mask_id=i, ratio=W.C3_RATIOS[i % len(W.C3_RATIOS)])
        else:
            m = W.workload_mask(key, shape, mask_id=i)
        masks.append(torch.as_tensor(m).to(dev))
        ratios.append(float(m.mean()))
        unmasked.append(int((np.asarray(m) == 0).sum()))
        xs.append(torch.as_tensor(W.edited_hidden(shape, cfg, xt, m)).to(dev).to(tdt))
    g = torch.Generator(device=dev)
    g.manual_seed(2000 + cfg)
    B, T, N, d = shape.batch, shape.n_tokens, shape.n_image, shape.d_model
    pinned = key in ("c3", "c5")
    kv_layers = []
    # K/V caching: per-layer K/V ([B][T][2][d] resident, [B][N][2][d] image rows in pinned host
    # memory); Y caching: per-layer block inputs of the image tokens, [B][N][d], hidden-state scale
    row_shape = (B, N, d) if cache == "y" else ((B, N, 2, d) if pinned else (B, T, 2, d))
    scale = 1.0 if cache == "y" else 0.5
    for _ in range(shape.n_layers):
        t = (torch.randn(row_shape, generator=g, device=dev) * scale).to(tdt)
        if pinned:
            h = torch.empty(t.shape, dtype=tdt, pin_memory=True)
            h.copy_(t)
            kv_layers.append(h)
            del t
        else:
            kv_layers.append(t)
    # one device slot per layer: every cached layer's load can start at once
    slot_shape = (B, N, d) if cache == "y" else (B, T, 2, d)
    slots = [torch.empty(slot_shape, dtype=tdt, device=dev) for _ in range(shape.n_layers)] if pinned else []
    ycache = torch.randn((B, T, d), generator=g, device=dev).to(tdt)
    return weights, masks, xs, ratios, kv_layers, slots, ycache, pinned, unmasked


# ----------------------------------------------------------------------------- measured HBM traffic

ROOT = os.path.dirname(os.path.abspath(__file__))

# Kernel symbols (as rocprofv3 names them) of each bench kernel class: the GEMM
# classes are told apart by their epilogue template argument (1 residual:
# out and down projections alike, 2 GELU, 3 QKV split).
FAMILY = {
    "attention": (r"attention_dma_kernel<(\d+), 2>", "paper_2505_20600_amd/csrc/attention.hip"),
    "gemm_up": (r"gemm_dl_kernel<\d+, \d+, \d, 2>", "paper_2505_20600_amd/csrc/gemm.hip"),
    "gemm_qkv": (r"gemm_dl_kernel<\d+, \d+, \d, 3>", "paper_2505_20600_amd/csrc/gemm.hip"),
    "gemm_out": (r"gemm_dl_kernel<\d+, \d+, \d, 1>", "paper_2505_20600_amd/csrc/gemm.hip"),
    "gemm_down": (r"gemm_dl_kernel<\d+, \d+, \d, 4>", "paper_2505_20600_amd/csrc/gemm.hip"),
    "gather": (r"::gather_kernel", "paper_2505_20600_amd/csrc/rows.hip"),
    "scatter": (r"::(scatter_masked|merge)_kernel", "paper_2505_20600_amd/csrc/rows.hip"),
}
MARKER = "spin_kernel"


def measured_traffic(kernel: str, workload: str | None = None):
    """Calibrated HBM bytes per launch of `kernel` on `workload` from a profiles/hbm_traffic_*.txt
    summary (rocprofv3 FETCH_SIZE / WRITE_SIZE passes scaled by a plain-copy calibration), or
    None when there is none or the kernel's source changed since it was taken."""
    import glob
    import hashlib
    for fn in sorted(glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.txt"))):
        kv = {}
        for line in open(fn):
            if "=" in line and not line.startswith("#"):
                k, v = line.strip().split("=", 1)
                kv[k] = v
        if kv.get("kernel") != kernel or kv.get("workload") != workload:
            continue
        src = os.path.join(ROOT, kv.get("source", ""))
        if not os.path.exists(src):
            continue
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        if sha != kv.get("source_sha256_16"):
            return None
        return {"bytes_per_launch": float(kv["hbm_bytes_per_launch"]), "file": os.path.relpath(fn, ROOT)}
    return None


# ----------------------------------------------------------------------------- rocprofv3 trace summaries


def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _window(rows):
    """The rows of dispatches that ran between the first two marker dispatches (--trace-marks);
    counter traces hold one row per counter and dispatch."""
    marks = sorted({(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in rows if MARKER in r["Kernel_Name"]})
    if len(marks) < 2:
        raise SystemExit("the trace has fewer than two marker dispatches: trace a bench.py --trace-marks run")
    t0, t1 = marks[0][1], marks[1][0]
    return sorted((r for r in rows if int(r["Start_Timestamp"]) >= t0 and int(r["End_Timestamp"]) <= t1
                   and MARKER not in r["Kernel_Name"]), key=lambda r: int(r["Start_Timestamp"]))


def _short(name):
    name = name.replace("void ", "").replace("ms::(anonymous namespace)::", "")
    return name.split("(")[0] if not name.startswith("__") else name


def summarize_trace(args):
    """Per-symbol statistics of a rocprofv3 kernel trace over the profiled pass of a
    --trace-marks run, the roofline kernel family's launch average, and (given the counter
    traces) its HBM bytes per launch scaled by a plain device copy's counter readings."""
    import re
    rows = _window(_read_csv(args.summarize_trace))
    per = {}
    for r in rows:
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        a = per.setdefault(_short(r["Kernel_Name"]), [0, 0.0, 1e30, 0.0])
        a[0] += 1
        a[1] += us
        a[2] = min(a[2], us)
        a[3] = max(a[3], us)
    tot = sum(a[1] for a in per.values())
    print(f"# {len(rows)} dispatches between the marker kernels (the profiled pass), {tot / 1e3:.3f} ms of kernel time")
    print(f"{'kernel':<64} {'calls':>6} {'total_ms':>10} {'avg_us':>9} {'min_us':>9} {'max_us':>9} {'pct':>6}")
    for name, (n, t, lo, hi) in sorted(per.items(), key=lambda kv: -kv[1][1]):
        print(f"{name[:64]:<64} {n:6d} {t / 1e3:10.3f} {t / n:9.2f} {lo:9.2f} {hi:9.2f} {100 * t / tot:6.2f}")
    if not args.family:
        return
    rx = re.compile(FAMILY[args.family][0])
    fam = [r for r in rows if rx.search(r["Kernel_Name"])]
    fus = sum((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in fam)
    print(f"family {args.family} ({FAMILY[args.family][0]}): {len(fam)} launches, {fus / 1e3:.3f} ms, "
          f"{fus / max(1, len(fam)):.2f} us per launch")
    for path in args.counters:
        vals = {}
        for r in _window(_read_csv(path)):
            if rx.search(r["Kernel_Name"]):
                vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        for c, v in sorted(vals.items()):
            print(f"counter {c}: {sum(v) / len(v):.6g} per dispatch over {len(v)} dispatches")
    if not (args.pmc_fetch and args.pmc_write and args.copy_fetch and args.copy_write):
        return

    def per_dispatch(path, window=True):
        rr = _read_csv(path)
        if window:
            rr = _window(rr)
        vals = [float(r["Counter_Value"]) for r in rr if rx.search(r["Kernel_Name"])]
        return sum(vals) / max(1, len(vals)), len(vals)

    def copy_kib(path):
        vals = [float(r["Counter_Value"]) for r in _read_csv(path) if "copy" in r["Kernel_Name"].lower()]
        return sum(vals) / max(1, len(vals))

    fetch, nf = per_dispatch(args.pmc_fetch)
    write, nw = per_dispatch(args.pmc_write)
    copy_bytes = float(1 << 30)
    ff = copy_bytes / (copy_kib(args.copy_fetch) * 1024)
    wf = copy_bytes / (copy_kib(args.copy_write) * 1024)
    import hashlib
    src = FAMILY[args.family][1]
    sha = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()[:16]
    print(f"# calibration: a plain 1 GiB device copy reads FETCH_SIZE {copy_bytes / ff / 1024:.1f} KiB and "
          f"WRITE_SIZE {copy_bytes / wf / 1024:.1f} KiB per dispatch")
    print(f"kernel={args.family}")
    print(f"symbols={FAMILY[args.family][0]}")
    print(f"source={src}")
    print(f"source_sha256_16={sha}")
    print(f"dispatches={nf},{nw}")
    print(f"fetch_kib_per_dispatch={fetch:.1f}")
    print(f"write_kib_per_dispatch={write:.1f}")
    print(f"fetch_factor={ff:.4f}")
    print(f"write_factor={wf:.4f}")
    print(f"hbm_bytes_per_launch={round((fetch * ff + write * wf) * 1024)}")


# ----------------------------------------------------------------------------- cost-model fit (Sec. 4.3)


def fit_cost_models(key, shape, n_points, torch, MS, W):
    """Measure per-block latencies of random batches and fit Comp(FLOPs) and Load(bytes).

    Each point is one batch of 1..B requests with log-uniform mask ratios in [3%, 80%]
    (blob masks): the per-block time of the cached blocks (resident K/V) and of blocks
    over every token (a dense prefix of all layers) against their Table 1 FLOPs, and
    the per-layer time of the pinned-host cache prefetch against its bytes. A stack of
    min(L, 4) layers of the workload's shape is enough: every quantity is per block.
    """
    import math
    from paper_2505_20600_amd import routing
    L = min(shape.n_layers, 4)
    fs = shape.replace(n_layers=L)
    cfg = W.CONFIG_IDS[key]
    dev = "cuda:0"
    tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    elt = 2 if shape.dtype == "bf16" else 4
    B, T, N, d = shape.batch, shape.n_tokens, shape.n_image, shape.d_model
    g = torch.Generator(device=dev)
    g.manual_seed(3000 + cfg)
    weights, _, _, _, _, _, _, _, _ = make_inputs(key, fs, 1, torch, W)
    wc = MS.weights_array(weights)
    kv_dev = [(torch.randn((B, T, 2, d), generator=g, device=dev) * 0.5).to(tdt) for _ in range(L)]
    kv_host = []
    for _ in range(L):
        h = torch.empty((B, N, 2, d), dtype=tdt, pin_memory=True)
        h.copy_((torch.randn((B, N, 2, d), generator=g, device=dev) * 0.5).to(tdt))
        kv_host.append(h)
    slots = [torch.empty((B, T, 2, d), dtype=tdt, device=dev) for _ in range(L)]
    x = torch.randn((B, T, d), generator=g, device=dev).to(tdt)
    yc = torch.randn((B, T, d), generator=g, device=dev).to(tdt)
    y = torch.empty_like(yc)
    desc = MS.model_desc(fs)
    ws = torch.empty(MS.mask_workspace_bytes(desc, B), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    copy_stream = torch.cuda.Stream()
    unit = MS.CostModel(0.0, 1.0, 0.0, 1.0, 2.0 * d * elt)     # mask_batch_cost in GFLOP and MB
    rng = np.random.default_rng(np.random.SeedSequence([cfg, 7, 0]))

    def timed(fn, reps=3):
        ts = []
        for _ in range(reps + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts[1:]))

    comp_pts, load_pts = [], []
    for i in range(n_points):
        b = 1 + i % B
        r = np.exp(rng.uniform(math.log(0.03), math.log(0.80), b))
        m = np.stack([W.blob_mask(shape.grid_h, shape.grid_w, float(rr), W.rng(cfg, 7, 64 * i + j))
                      for j, rr in enumerate(r)])
        counts = [int(v) for v in m.sum(1)]
        (mb, gf_c, gf_f), _, _ = MS.mask_batch_cost(desc, unit, counts)
        st = MS.MaskStep(desc, b, torch.as_tensor(m).to(dev), ws, stream)
        kvs = [t[:b] for t in kv_dev]
        run = lambda: st.stack_forward(wc, x[:b], yc[:b], kvs, y[:b], stream=stream)
        t_c = timed(run) / L
        st.set_dense_prefix(L, stream)
        t_f = timed(run) / L
        st.set_dense_prefix(0, stream)
        hs = [h[:b] for h in kv_host]
        ss = [sl[:b] for sl in slots]
        MS.profiler_start(("copy",))
        for _ in range(3):
            st.stack_forward(wc, x[:b], yc[:b], hs, y[:b], pinned=True, slots=ss, stream=stream,
                             copy_stream=copy_stream)
        torch.cuda.synchronize()
        prof = MS.profiler_stop()
        st.close()
        comp_pts += [[round(gf_c, 4), round(t_c, 5)], [round(gf_f, 4), round(t_f, 5)]]
        if "copy" in prof and prof["copy"][1] > 0 and mb > 0:
            load_pts.append([round(mb, 3), round(prof["copy"][0] / prof["copy"][1], 5)])
        log(f"[fit] batch {b} masked {counts}: cached {t_c:.4f} ms ({gf_c:.1f} GF), full {t_f:.4f} ms "
            f"({gf_f:.1f} GF), load {load_pts[-1] if load_pts else None}")
    def fit(pts):
        xs, ys = [p[0] for p in pts], [p[1] for p in pts]
        a, b, r2 = MS.mask_fit_linear(xs, ys)
        if b < 0 or a < 0:
            # a cost model has no negative part: a negative slope (latency flat in the amount,
            # e.g. copies that move nearly every row whatever the mask) keeps the mean, a negative
            # intercept the line through the origin
            if b < 0:
                a, b, r2 = float(np.mean(ys)), 0.0, 0.0
            else:
                b = float(np.dot(xs, ys) / np.dot(xs, xs))
                a = 0.0
                r2 = 1.0 - float(np.sum((np.asarray(ys) - b * np.asarray(xs)) ** 2) /
                                 np.sum((np.asarray(ys) - np.mean(ys)) ** 2))
        return a, b, r2

    c0, c1, c_r2 = fit(comp_pts)
    l0, l1, l_r2 = fit(load_pts)
    # routing simulation with the fitted models (host-only): caches streamed from pinned host
    # memory (the fitted load model) and HBM-resident (no loads)
    import contextlib
    import io
    sims = {}
    for name, load_args in (("streamed", [str(l0), str(l1)]), ("resident", ["0", "0"])):
        buf = io.StringIO()
        with contextlib.redirect_stdout(buf):
            routing.main(["--workload", key, "--comp", str(c0), str(c1), "--load", *load_args, "--requests", "2000"])
        sims[name] = json.loads(buf.getvalue())
    return {
        "comp": {"ms0": round(c0, 5), "ms_per_gflop": round(c1, 6), "r2": round(c_r2, 5), "points": comp_pts},
        "load": {"ms0": round(l0, 5), "ms_per_mb": round(l1, 6), "r2": round(l_r2, 5), "points": load_pts},
        "routing": sims,
    }


# ----------------------------------------------------------------------------- cache-load overlap


def _union(iv):
    out = []
    for a, b in sorted(iv):
        if out and a <= out[-1][1]:
            out[-1][1] = max(out[-1][1], b)
        else:
            out.append([a, b])
    return out


def _length(u):
    return sum(b - a for a, b in u)


def _intersection(u, v):
    i = j = 0
    tot = 0.0
    while i < len(u) and j < len(v):
        lo, hi = max(u[i][0], v[j][0]), min(u[i][1], v[j][1])
        if hi > lo:
            tot += hi - lo
        if u[i][1] < v[j][1]:
            i += 1
        else:
            j += 1
    return tot


def step_fit(per_ratio):
    """Least-squares line of the median step time against the masked rows (Table 1: the
    masked computation is linear in M), over the mask sets that share the most common
    dense prefix; None below three distinct row counts."""
    if not per_ratio:
        return None
    prefixes = [r[3] for r in per_ratio]
    pre = max(set(prefixes), key=prefixes.count)
    pts = [(r[1], r[2]) for r in per_ratio if r[3] == pre]
    x = np.array([p[0] for p in pts], float)
    y = np.array([p[1] for p in pts], float)
    if len(set(x.tolist())) < 3:
        return None
    slope, icpt = np.polyfit(x, y, 1)
    ss_tot = float(np.sum((y - y.mean()) ** 2))
    r2 = 1.0 - float(np.sum((y - (icpt + slope * x)) ** 2)) / ss_tot if ss_tot > 0 else 1.0
    return {"ms0": round(float(icpt), 4), "ms_per_1k_rows": round(1e3 * float(slope), 4),
            "r2": round(r2, 4), "points": len(pts), "dense_prefix": pre}


def stream_overlap(intervals, steps):
    """Per step: summed cache-load time, summed kernel time, the first layer's load, and the
    fraction of the shorter of the two that runs concurrently with the other."""
    copies = [(a, b) for c, a, b in intervals if c == "copy"]
    kern = [(a, b) for c, a, b in intervals if c != "copy"]
    uc, uk = _union(copies), _union(kern)
    lc, lk = _length(uc), _length(uk)
    both = _intersection(uc, uk)
    first = (sum(b - a for a, b in copies) / len(copies)) if copies else 0.0
    sc, sk = lc / steps, lk / steps
    return {"sum_copy_ms": round(sc, 4), "sum_kernel_ms": round(sk, 4),
            "first_layer_copy_ms": round(first, 4), "bound_ms": round(max(sc, sk) + first, 4),
            "overlap": round(both / min(lc, lk), 4) if min(lc, lk) > 0 else None}


def measure_ceilings(torch):
    """Reference rates of this GPU: hipBLASLt (torch.matmul) bf16 at 8192^3, a 1 GiB device
    copy (read + write bytes), and 256 MiB pinned host-to-device copies."""
    dev = "cuda:0"

    def best_ms(fn, reps=5):
        fn()
        best = 1e30
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b))
        return best

    n = 8192
    A = torch.randn(n, n, device=dev).bfloat16()
    Bm = torch.randn(n, n, device=dev).bfloat16()
    C = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
    t_mm = best_ms(lambda: torch.matmul(A, Bm, out=C))
    del A, Bm, C
    nb = 1 << 30
    x = torch.empty(nb, dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    x.fill_(1)
    t_cp = best_ms(lambda: y.copy_(x))
    del x, y
    from paper_2505_20600_amd import maskstep as MS
    return {"gemm_bf16_8192_tflops": round(2.0 * n ** 3 / (t_mm / 1e3) / 1e12, 1),
            "d2d_copy_gbs": round(2.0 * nb / (t_cp / 1e3) / 1e9, 1),
            "h2d_pinned_gbs": round(h2d_ceiling(torch, torch.cuda.current_stream()), 2),
            **MS.probe_ceilings(),
            "note": "best of 5 (GEMM, copy) or 3 (H2D) timed runs; copy counts bytes read + written; "
                    "mfma_* / lds_* / operand_stream_*: the library's diagnostic probes (second of two "
                    "launches), clock from the shader clock counter against the 100 MHz constant clock"}


def h2d_ceiling(torch, stream, nbytes=256 << 20):
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    h.fill_(1)
    best = 0.0
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        with torch.cuda.stream(stream):
            d.copy_(h, non_blocking=True)
        b.record(stream)
        torch.cuda.synchronize()
        best = max(best, nbytes / (a.elapsed_time(b) / 1e3) / 1e9)
    return best


# ----------------------------------------------------------------------------- CPU oracle


def cpu_baseline(key, shape, budget_s):
    """The oracle as it stands, timed on this host over a bounded sample of the workload: the
    masked path (request 0's recomputed rows through as many layers as half the budget allows)
    and, beside it, the dense path (one block over every token of request 0), each scaled to
    the full stack and batch."""
    import oracle
    from paper_2505_20600_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        cores = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:
        cores = len(os.sched_getaffinity(0))
    cfg = W.CONFIG_IDS[key]
    one = shape.replace(batch=1)
    mask = W.workload_mask(key, shape, mask_id=0,
                           ratio=(W.C3_RATIOS[0] if key == "c3" else None))[:1]
    xt = W.template_hidden(one, cfg)
    x = W.edited_hidden(one, cfg, xt, mask)
    toks = oracle.masked_tokens(mask[0], one.n_text)
    M = len(toks)
    rnd = oracle.rounder(one.dtype)

    def layer(l):
        w = W.layer_weights(one, cfg, l)
        return (w, W.layer_weights(one, cfg, l, text=True)) if one.dual_stream else w

    xm = np.asarray(x[0][toks], np.float64)
    t_layers, n = 0.0, 0
    for l in range(one.n_layers):
        w, kv = layer(l), W.synthetic_kv_cache(one, cfg, l)[0]
        t0 = time.perf_counter()
        xm, _ = oracle.block_rows(xm, toks, w, kv, one, rnd, round_p=True)
        t_layers += time.perf_counter() - t0
        n += 1
        if t_layers >= budget_s / 2:
            break
    per_layer = t_layers / n
    T = one.n_tokens
    t0 = time.perf_counter()
    oracle.block_rows(np.asarray(x[0], np.float64), np.arange(T), layer(0), np.zeros((T, 2, one.d_model)), one,
                      rnd, round_p=True)
    dense_layer = time.perf_counter() - t0
    # masked tokens of the whole step: the batch's expected M equals B x this request's M
    value = M / (per_layer * shape.n_layers)
    try:
        model = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name"))
    except Exception:
        model = "unknown"
    return {
        "value": value, "unit": "masked tokens/s", "cores": int(cores), "kind": "oracle",
        "sample": f"masked path: request 0 of mask set 0 (M={M} recomputed rows), {n} of {shape.n_layers} layers "
                  f"timed ({t_layers:.1f} s), scaled to the full stack; dense path: one block over all {T} tokens "
                  f"of request 0 ({dense_layer:.1f} s), scaled to the full stack; float64 NumPy, bf16 rounding "
                  f"points and round_p as in the parity tests; host: {model}",
        "ms_per_layer": per_layer * 1e3,
        "dense_ms_per_layer": dense_layer * 1e3,
        "dense_tokens_per_s": T / (dense_layer * shape.n_layers),
        "masked_vs_dense_step": (per_layer / dense_layer),
    }


# ----------------------------------------------------------------------------- main


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the method serves each request set on a single GPU); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2505_20600_amd import maskstep as MS
    from paper_2505_20600_amd import workloads as W
    import oracle

    if args.copy_calibration:
        n = 1 << 30
        a = torch.empty(n, dtype=torch.uint8, device="cuda:0")
        b = torch.empty_like(a)
        a.fill_(1)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 3}))
        return

    if args.ceilings:
        print(json.dumps(measure_ceilings(torch)), flush=True)
        return

    key = args.workload
    shape = W.CONFIGS[key]
    torch.cuda.set_device(0)
    if args.fit:
        t0 = time.perf_counter()
        res = fit_cost_models(key, shape, args.fit, torch, MS, W)
        print(json.dumps({"metric": "per-block cost models (Sec. 4.3): latency vs FLOPs and vs cached bytes",
                          "workload": f"{shape.name}: {DESCR[key]}", "points": args.fit,
                          "seconds": round(time.perf_counter() - t0, 1), **res}), flush=True)
        return
    t0 = time.perf_counter()
    weights, masks, xs, ratios, kv_layers, slots, ycache, pinned, unmasked = make_inputs(
        key, shape, args.masks, torch, W, args.cache)
    yc_mode = args.cache == "y"
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f} s; ratios {np.round(ratios, 3).tolist()}")
    wc = MS.weights_array(weights)
    desc = MS.model_desc(shape)
    ws_bytes = MS.mask_workspace_bytes(desc, shape.batch)
    y = torch.empty_like(ycache)
    stream = torch.cuda.current_stream()
    copy_stream = torch.cuda.Stream() if pinned else None
    prefix = [0] * args.masks
    plan_info = []

    # One step context per mask set, built before any timing: a request's mask is fixed over
    # its denoising steps, so the compaction (mask_step_init, one host sync) runs once per
    # mask set and is timed on its own; a step is mask_stack_forward.
    ctx, init_ms = [], []
    for i in range(args.masks):
        wsi = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
        torch.cuda.synchronize()
        t_init = time.perf_counter()
        ctx.append(MS.MaskStep(desc, shape.batch, masks[i], wsi, stream))
        torch.cuda.synchronize()
        init_ms.append((time.perf_counter() - t_init) * 1e3)
    Ms = [c.info().rows for c in ctx]
    log(f"[bench] step contexts: {args.masks} x {ws_bytes / 2**20:.0f} MiB workspace; "
        f"mask_step_init {np.round(init_ms, 3).tolist()} ms")

    def one_step(i):
        ctx[i].stack_forward(wc, xs[i], ycache, kv_layers, y, pinned=pinned, slots=slots, stream=stream,
                             copy_stream=copy_stream, inputs=yc_mode, loads_ahead=True)
        return Ms[i]

    def timed_once(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b)

    for i in range(args.masks):
        one_step(i)
    if pinned and args.prefix == "auto":
        # Alg. 1 inputs per mask set, measured on this GPU: one block over every token, one
        # block over the masked rows (cache resident), one block's cache load
        L = shape.n_layers
        for i in range(args.masks):
            st = ctx[i]
            run = lambda: st.stack_forward(wc, xs[i], ycache, slots, y, pinned=False, stream=stream,
                                           inputs=yc_mode)
            run()
            cached_ms = min(timed_once(run) for _ in range(2)) / L
            st.set_dense_prefix(L, stream)
            run()
            full_ms = min(timed_once(run) for _ in range(2)) / L
            st.set_dense_prefix(0, stream)
            MS.profiler_start(("copy",))
            st.stack_forward(wc, xs[i], ycache, kv_layers, y, pinned=True, slots=slots, stream=stream,
                             copy_stream=copy_stream, inputs=yc_mode)
            torch.cuda.synchronize()
            prof = MS.profiler_stop()
            load_ms = prof["copy"][0] / max(1, prof["copy"][1]) if "copy" in prof else 0.0
            k, model_ms = MS.mask_plan_dense_prefix(L, load_ms, cached_ms, full_ms)
            prefix[i] = k
            st.set_dense_prefix(k, stream)
            plan_info.append({"ratio": round(ratios[i], 4), "load_ms": round(load_ms, 4),
                              "cached_ms": round(cached_ms, 4), "full_ms": round(full_ms, 4),
                              "dense_prefix": k, "modelled_ms": round(model_ms, 3)})
        log(f"[bench] dense-prefix plan: {plan_info}")
    elif args.prefix != "auto":
        prefix = [int(args.prefix)] * args.masks
        for i in range(args.masks):
            if prefix[i]:
                ctx[i].set_dense_prefix(prefix[i], stream)
    for i in range(args.warmup):
        one_step(i % args.masks)
    torch.cuda.synchronize()

    def row_layers(i):
        # rows each block of the step computes in full: every token in the first k - 1 blocks
        # of a dense prefix, the masked rows (plus text rows) in the others (the prefix's last
        # block projects K/V over every token and computes the rest over the masked rows)
        k = prefix[i]
        full = max(k - 1, 0)
        return full * shape.batch * shape.n_tokens + (shape.n_layers - full) * Ms[i]

    def unmasked_layers(i):
        # rows whose K/V alone are projected: every token in a dense prefix's last block; with
        # Y caching, the unmasked rows of every cached block
        k = prefix[i]
        kv_rows = shape.batch * shape.n_tokens if k > 0 else 0
        return kv_rows + ((shape.n_layers - k) * unmasked[i] if yc_mode else 0)

    def timed(k, per_step=False):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(k + 1)]
        tot_m = 0
        tot_rl = 0
        tot_ul = 0
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        evs[0].record(stream)
        for s in range(k):
            tot_m += one_step(s % args.masks)
            tot_rl += row_layers(s % args.masks)
            tot_ul += unmasked_layers(s % args.masks)
            evs[s + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        ms = evs[0].elapsed_time(evs[k])
        steps = [evs[s].elapsed_time(evs[s + 1]) for s in range(k)] if per_step else None
        return ms, wall, tot_m, steps, tot_rl, tot_ul

    ms_total, wall, tot_m, step_ms, _, _ = timed(args.steps, per_step=True)
    log(f"[bench] timed {args.steps} steps: {ms_total:.3f} ms (events), {wall * 1e3:.3f} ms (wall)")
    ms_step = ms_total / args.steps
    value = tot_m / (ms_total / 1e3)
    per_mask = {}
    for s, t in enumerate(step_ms):
        per_mask.setdefault(s % args.masks, []).append(t)
    per_ratio = sorted([[round(ratios[i], 4), int(Ms[i]), round(float(np.median(v)), 4), prefix[i]]
                        for i, v in per_mask.items()])
    q10, q50, q90 = (round(float(v), 4) for v in np.percentile(step_ms, [10, 50, 90]))

    # profiled pass: per-kernel event timing over a second timed region
    kernels, roof = {}, None
    if not args.no_profile_pass:
        if args.trace_marks:
            torch.cuda._sleep(1000)
            torch.cuda.synchronize()
        MS.profiler_start(MS.KERNEL_CLASSES, capacity=1 << 16)
        ms_prof, _, tot_m_prof, _, tot_rl_prof, u_sum = timed(args.steps)
        prof = MS.profiler_stop()
        if args.trace_marks:
            torch.cuda._sleep(1000)
            torch.cuda.synchronize()
        log(f"[bench] profiled pass: {ms_prof / args.steps:.4f} ms/step; {prof}")
        d, T, L, f = shape.d_model, shape.n_tokens, shape.n_layers, shape.mlp_mult * shape.d_model
        e = 2 if shape.dtype == "bf16" else 4
        nset = 2 if shape.dual_stream else 1
        m_sum = tot_rl_prof                         # computed rows summed over the blocks of all steps
        work = {
            "attention": ("mfma", 4.0 * m_sum * T * d),
            "gemm_qkv": ("mfma", 2.0 * m_sum * d * 3 * d + 2.0 * u_sum * d * 2 * d),
            "gemm_out": ("mfma", 2.0 * m_sum * d * d),
            "gemm_up": ("mfma", 2.0 * m_sum * d * f),
            "gemm_down": ("mfma", 2.0 * m_sum * f * d),
            "gather": ("hbm", 2.0 * tot_m_prof * d * e),
        }
        prof.pop("_dropped", None)
        for c, (t_ms, n) in prof.items():
            kernels[c] = {"ms_total": round(t_ms, 4), "launches": n, "us_avg": round(1e3 * t_ms / max(n, 1), 3)}
            if c in work:
                kind, amount = work[c]
                if kind == "mfma":
                    kernels[c]["tflops"] = round(amount / (t_ms / 1e3) / 1e12, 2)
                else:
                    kernels[c]["gbs"] = round(amount / (t_ms / 1e3) / 1e9, 1)
        dom = max((c for c in kernels if c in work), key=lambda c: kernels[c]["ms_total"])
        kind, amount = work[dom]
        t_s = kernels[dom]["ms_total"] / 1e3
        # algorithmic HBM bytes per launch of the dominant kernel: attention reads every token's
        # K/V of the batch and the masked rows' Q, writes their O; a projection reads its rows
        # of A, its weights and (residual epilogues) the residual rows, writes its rows of C
        n_launch = kernels[dom]["launches"]
        m_avg = m_sum / n_launch
        gemm_dims = {"gemm_qkv": (d, 3 * d, 1), "gemm_out": (d, d, 2), "gemm_up": (d, f, 1), "gemm_down": (f, d, 2)}
        if dom == "attention":
            alg_bytes = (2 * shape.batch * T * d + 2 * m_avg * d) * e
        elif dom in gemm_dims:
            K_, N_, outs = gemm_dims[dom]
            alg_bytes = (m_avg * K_ + N_ * K_ + outs * m_avg * N_) * e
        else:
            alg_bytes = None
        tr = measured_traffic(dom, key)
        if kind == "mfma":
            peak = PEAK["bf16_mfma_tflops"] if shape.dtype == "bf16" else PEAK["fp32_mfma_tflops"]
            ach = amount / t_s / 1e12
            roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(ach / peak, 4)}
        else:
            ach = amount / t_s / 1e9
            roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK["hbm_gbs"], "unit": "GB/s",
                    "frac": round(ach / PEAK["hbm_gbs"], 4)}
        roof.update({"traffic": round(tr["bytes_per_launch"]) if tr else None,
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "traffic_source": tr["file"] if tr else None,
                     "algorithmic_bytes_per_launch": round(alg_bytes) if alg_bytes else None,
                     "kernel": dom, "kernel_symbols": FAMILY.get(dom, (None,))[0],
                     "per_launch_us": kernels[dom]["us_avg"],
                     "algorithmic_flops_per_launch": round(amount / n_launch) if kind == "mfma" else None})

    # streamed caches: how much of the per-layer load stream runs under the computation
    # (layer-wise pipelining, Sec. 3.2), against the loads issued in line (the naive loading
    # the paper measures) and the pinned host-to-device ceiling of this GPU's link
    stream_info = None
    if pinned and not args.no_profile_pass:
        stream_info = stream_overlap(MS.profiler_intervals(), args.steps)
        row_bytes = (1 if yc_mode else 2) * shape.d_model * (2 if shape.dtype == "bf16" else 4)
        copy_rows = [c.info().copy_rows_y if yc_mode else c.info().copy_rows for c in ctx]
        copied = sum((shape.n_layers - prefix[s % args.masks]) * copy_rows[s % args.masks]
                     for s in range(args.steps)) * row_bytes
        needed = sum((shape.n_layers - prefix[s % args.masks]) * unmasked[s % args.masks]
                     for s in range(args.steps)) * row_bytes
        os.environ["MS_SERIALIZE"] = "1"
        try:
            ms_ser = timed(args.steps)[0] / args.steps
        finally:
            del os.environ["MS_SERIALIZE"]
        ceil_gbs = h2d_ceiling(torch, copy_stream)
        sc = stream_info["sum_copy_ms"]
        stream_info.update({
            "step_ms": round(ms_step, 4),
            "profiled_step_ms": round(ms_prof / args.steps, 4),
            "serialized_step_ms": round(ms_ser, 4),
            "speedup_vs_serialized": round(ms_ser / ms_step, 3),
            "copied_mb_per_step": round(copied / args.steps / 1e6, 2),
            "needed_mb_per_step": round(needed / args.steps / 1e6, 2),
            "h2d_gbs": round(copied / args.steps / (sc / 1e3) / 1e9, 2) if sc > 0 else None,
            "h2d_ceiling_gbs": round(ceil_gbs, 2),
            "note": "overlap = |copy union & kernel union| / min(|copy union|, |kernel union|) over the "
                    "profiled pass; bound_ms = max(sum_copy_ms, sum_kernel_ms) + first_layer_copy_ms; "
                    "serialized = loads issued on the compute stream before each block (MS_SERIALIZE=1); "
                    "ceiling = best of three 256 MiB pinned host-to-device copies",
        })
        log(f"[bench] stream: {stream_info}")

    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        cpu = cpu_baseline(key, shape, args.cpu_seconds)
        log(f"[bench] cpu oracle sample took {time.perf_counter() - t0:.1f} s")

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "masked tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_ms_p10_p50_p90": [q10, q50, q90],
        "effective_tokens_per_s": round(shape.batch * shape.n_tokens / (ms_step / 1e3), 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic",
        "config": {"workload": f"{shape.name}: {DESCR[key]}", "global_batch": shape.batch,
                   "seq_len": shape.n_tokens, "parallelism": "none (1 GPU)",
                   "masks": args.masks, "mean_masked_rows": round(float(np.mean(Ms)), 1),
                   "cache": "per-layer K/V (Fig. 7)" if args.cache == "kv" else
                            "per-layer block inputs, K/V recomputed (Fig. 5 bottom)"},
        "per_mask": {"columns": ["ratio", "masked_rows", "median_ms", "dense_prefix"], "rows": per_ratio},
        "step_vs_rows_fit": step_fit(per_ratio),
        "prefix_plan": plan_info or None,
        "mask_step_init_ms": {"mean": round(float(np.mean(init_ms)), 3), "max": round(float(max(init_ms)), 3),
                              "note": "once per mask set (compaction + one host sync), outside the step"},
        "roofline": roof,
        "stream": stream_info,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    for c in ctx:
        c.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
