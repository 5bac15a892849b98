"""Benchmark of the path-compositional MoE layer on one MI355X.

A step is one forward pass of the whole layer (the fused indexing operation over the
layer's packed mask, expand, project and combine, plus the shared expert when the workload
has one) over one batch of synthetic, seeded inputs already resident in HBM (bf16 layers keep
their projection weights as float16, widened once before the steps by pcm_widen_f16, which
gives the same output bits as the bf16 weights; --down-weights bf16 times the bf16 weights,
widened by the kernels per fragment). Prints ONE JSON
line: the headline workload (Mixtral-shaped) at the top level with its ablation (the same
layer per path, with and without source reuse, and the vanilla top-k layer), and every
workload under "workloads".

  python bench.py [--steps K] [--warmup W] [--config NAME] [--only] [--router topk|scored]
                  [--indexing fused|separate] [--down-weights f16|bf16] [--no-cpu-baseline]
                  [--no-ablation] [--no-graph]
  python bench.py --trace-summary DIR     per-kernel durations (kernel traces) or counter
                                          means (--pmc runs) of the timed launches in the
                                          rocprofv3 output written under DIR
  python bench.py --vendor-compare [--config NAME]
                                          the two grouped GEMMs under uniform routing beside
                                          torch.bmm (the vendor library) of the same shapes

Per-kernel times come from HIP events recorded in the timed steps on the stream the kernels
run on: around each call, and inside pcm_project_combine between the mix, the projection GEMM
and the combine (pcm_tuning's stage events). A second pass over the same steps writes a 512 MB
buffer before each step, so that the memory-bound stages (indexing, mix, combine)
read from HBM rather than from the 256 MB MALL; their GB/s come from that pass. Then the
same step is captured as one HIP graph (LayerPlan.capture's capture_graph) and its replays are
timed the same way (ms_graph and tokens_per_s_graph per workload: the layer without the host's
per-call cost; the headline stays the eager figure).
The eager timed region and the graph replays are each fenced by two short spin kernels, which
--trace-summary uses to keep only the timed launches of a rocprofv3 trace (region 0 the eager
steps, region 1 the replays). The CPU baseline times the float64 oracle on
a bounded sample of the headline workload's tokens.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "path-MoE layer tokens/sec and grouped-GEMM TFLOP/s (% bf16 MFMA peak), 1 GPU"
FLUSH_BYTES = 512 << 20
FENCE = "spin_kernel"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=None, help="headline workload (default: mixtral)")
    ap.add_argument("--only", action="store_true",
                    help="measure the headline workload only (for profiler runs)")
    ap.add_argument("--router", choices=("topk", "scored"), default="topk",
                    help="topk: top-k experts, paths among them allowed by the mask; "
                         "scored: scored compositional routing over the active paths")
    ap.add_argument("--indexing", choices=("fused", "separate"), default="fused",
                    help="fused: route, path table and dispatch layout in one operation over the "
                         "layer's packed mask; separate: the route and the path build as two calls")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stack", type=int, default=0, metavar="L",
                    help="time a decode step through L layers of the workload's shape (router GEMM, "
                         "paths, experts, residual; the first two layers diagonal-only); "
                         "reported as a separate JSON line")
    ap.add_argument("--down-weights", choices=("f16", "bf16"), default="f16",
                    help="projection weights of bf16 layers: float16, widened once from the bf16 "
                         "weights by pcm_widen_f16 before the timed steps (the layer's output bits "
                         "are the same), or the bf16 weights, widened by the kernels per fragment")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the timing of each workload's step captured as one HIP graph "
                         "(ms_graph, tokens_per_s_graph beside the eager figures)")
    ap.add_argument("--no-ablation", action="store_true",
                    help="skip the headline workload's ablation (the same layer executed per path, "
                         "with and without source reuse, and the vanilla top-k layer)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--vendor-compare", action="store_true",
                    help="only time the workload's two grouped GEMMs under uniform routing (every "
                         "expert T*k/n rows) beside the vendor library's batched GEMM (torch.bmm) "
                         "of the same shapes, alternating per iteration; one JSON line")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized buffer 5 times (calibrates HBM byte counters)")
    ap.add_argument("--trace-summary", default=None, metavar="DIR",
                    help="summarise the timed launches of a rocprofv3 kernel trace under DIR")
    return ap.parse_args()


# ------------------------------------------------------------------ trace summary
def _fenced(rows):
    """Index ranges (a, b) of the fenced timed regions of time-ordered dispatch rows; the whole
    list when it has no fences (a plain program such as the copy probe)."""
    fences = [i for i, r in enumerate(rows) if FENCE in r["Kernel_Name"]]
    if len(fences) < 2:
        return [(-1, len(rows))]
    return list(zip(fences[0::2], fences[1::2]))


def _short(name: str) -> str:
    return name.replace("(anonymous namespace)::", "").replace("pcm::", "").split("(")[0] \
        .replace("void ", "")


def trace_summary(path: str):
    """Per-kernel launch durations (kernel traces) or counter averages (counter collections)
    inside each fenced timed region of the rocprofv3 output under `path` (markdown tables)."""
    traces = sorted(glob.glob(os.path.join(path, "**", "*kernel_trace.csv"), recursive=True))
    counters = sorted(glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True))
    if not traces and not counters:
        sys.exit(f"no kernel_trace.csv or counter_collection.csv under {path}")
    for f in traces:
        rows = sorted(csv.DictReader(open(f)), key=lambda r: int(r["Start_Timestamp"]))
        for reg, (a, b) in enumerate(_fenced(rows)):
            stats = {}
            for r in rows[a + 1:b]:
                d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
                stats.setdefault(r["Kernel_Name"], []).append(d)
            print(f"### kernel trace, timed region {reg} ({os.path.basename(f)})\n")
            print("| kernel | launches | avg us | min us | max us | total us |")
            print("|---|---|---|---|---|---|")
            for name, ds in sorted(stats.items(), key=lambda kv: -sum(kv[1])):
                print(f"| `{_short(name)}` | {len(ds)} | {np.mean(ds):.1f} | {min(ds):.1f} | "
                      f"{max(ds):.1f} | {sum(ds):.1f} |")
            print()
    for f in counters:
        disp = {}
        for r in csv.DictReader(open(f)):
            d = disp.setdefault(r["Dispatch_Id"], {"name": r["Kernel_Name"],
                                                  "start": int(r["Start_Timestamp"]),
                                                  "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"]),
                                                  "c": {}})
            d["c"][r["Counter_Name"]] = d["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        rows = sorted(({"Kernel_Name": v["name"], **v} for v in disp.values()), key=lambda v: v["start"])
        names = sorted({c for v in rows for c in v["c"]})
        for reg, (a, b) in enumerate(_fenced(rows)):
            agg = {}
            for v in rows[a + 1:b]:
                agg.setdefault(v["name"], []).append(v)
            print(f"### counters, timed region {reg} ({os.path.basename(f)}; mean per dispatch)\n")
            extra = []
            if "SQ_VALU_MFMA_BUSY_CYCLES" in names and "GRBM_GUI_ACTIVE" in names:
                extra = ["MFMA busy", "clock GHz"]
            print("| kernel | dispatches | avg us | " + " | ".join(names + extra) + " |")
            print("|---|---|---|" + "---|" * (len(names) + len(extra)))
            for name, vs in sorted(agg.items(), key=lambda kv: -sum(v["ns"] for v in kv[1])):
                m = {c: np.mean([v["c"].get(c, 0.0) for v in vs]) for c in names}
                ns = np.mean([v["ns"] for v in vs])
                cells = [f"{m[c]:.6g}" for c in names]
                if extra:
                    # 8 XCDs count GRBM_GUI_ACTIVE each; 1024 SIMDs count MFMA-busy cycles. The
                    # busy window of a dispatch includes a fixed start-up of a few microseconds,
                    # so the clock is shown for dispatches of 50 us or more only
                    gui = m["GRBM_GUI_ACTIVE"] / 8
                    cells += [f"{m['SQ_VALU_MFMA_BUSY_CYCLES'] / 1024 / max(gui, 1):.1%}",
                              f"{gui / max(ns, 1):.2f}" if ns >= 50e3 else "—"]
                print(f"| `{_short(name)}` | {len(vs)} | {ns / 1e3:.1f} | " + " | ".join(cells) + " |")
            print()


def vendor_compare(args):
    """The workload's expansion and projection GEMMs with uniform routing (token t takes experts
    (t + j) mod n, j < k, so that every expert has T*k/n rows: the case a batched GEMM handles)
    against torch.bmm over n experts of the same shapes: bf16 for the expansion (the plain
    products, without the gather, SwiGLU and float32 U), bf16 and float16 for the projection
    (operands contiguous). Iterations alternate between the kernels; medians are reported."""
    import torch
    import paper_2609_01024_amd as pcm
    from workloads import CONFIGS, HEADLINE
    name = args.config or HEADLINE
    cfg = CONFIGS[name]
    T, H, F, n, k = cfg.T, cfg.H, cfg.F, cfg.n, cfg.k
    if cfg.dtype != "bf16" or T % n or (T * k) % n:
        sys.exit(f"--vendor-compare needs a bf16 workload with T and T*k multiples of n ({name})")
    dev, rows = "cuda:0", T * k // n
    d = device_inputs(cfg, args.seed, host_weights=False)
    widen_down_weights(pcm, d)
    g = torch.Generator(device=dev).manual_seed(args.seed * 1000 + 29)
    logits = torch.empty((T, n), dtype=torch.float32, device=dev).uniform_(0.0, 0.5, generator=g)
    t = torch.arange(T, device=dev)
    for j in range(k):
        logits[t, (t + j) % n] = 10.0 - j
    plan = pcm.LayerPlan(T, H, F, n, k, torch.bfloat16, dev)
    plan.index(logits, pcm.pcm_mask_pack(d["mask"]))
    counts = torch.diff(plan.paths.expert_offsets).tolist()
    assert counts == [rows] * n, counts
    a_e = torch.empty((n, rows, H), device=dev).normal_(0.0, 1.0, generator=g).to(torch.bfloat16)
    b_e = torch.empty((n, H, 2 * F), device=dev).normal_(0.0, cfg.w_std, generator=g).to(torch.bfloat16)
    a_p = torch.empty((n, rows, F), device=dev).normal_(0.0, 1.0, generator=g).to(torch.bfloat16)
    b_p = torch.empty((n, F, H), device=dev).normal_(0.0, cfg.w_std, generator=g).to(torch.bfloat16)
    bmm = {"bmm_expand_bf16": (a_e, b_e), "bmm_project_bf16": (a_p, b_p),
           "bmm_project_f16": (a_p.to(torch.float16), b_p.to(torch.float16))}
    runs = {"ours_expand": [], "ours_project": [], **{key: [] for key in bmm}}
    for it in range(args.warmup + args.steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        inner = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        for e in inner:
            e.record()
        ev[0].record()
        pcm.pcm_expand(d["x"], d["wg"], d["wu"], plan.paths, u=plan.u)
        ev[1].record()
        pcm.pcm_project_combine(plan.u, d["wd"], plan.paths, y=plan.y, ws=plan.ws_proj,
                                tuning=pcm.Tuning(stage_events=inner))
        times = {}
        for key, (a, b) in bmm.items():
            e2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e2[0].record()
            torch.bmm(a, b)
            e2[1].record()
            times[key] = e2
        torch.cuda.synchronize()
        if it >= args.warmup:
            runs["ours_expand"].append(ev[0].elapsed_time(ev[1]))
            runs["ours_project"].append(inner[1].elapsed_time(inner[2]))
            for key, e2 in times.items():
                runs[key].append(e2[0].elapsed_time(e2[1]))
    flops = {"expand": 4.0 * T * k * H * F, "project": 2.0 * T * k * H * F}
    out = {}
    for key, v in runs.items():
        ms = float(np.median(v))
        f = flops["expand" if "expand" in key else "project"]
        out[key] = {"us": round(ms * 1e3, 1), "TFLOP/s": round(f / (ms * 1e-3) / 1e12, 1),
                    "frac_bf16_peak": round(f / (ms * 1e-3) / 2.5e15, 4)}
    print(json.dumps({"vendor_compare": out, "config": {
        "workload": f"{name}: T={T} H={H} n={n} F={F} k={k}, uniform routing ({rows} rows per expert)",
        "steps": args.steps, "warmup": args.warmup}}), flush=True)


def copy_probe(mib: int):
    """A plain device-to-device copy of known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_per_launch": n * 4, "launches": 5}), flush=True)


def measured_traffic(workload: str):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counters
    (profiles/traffic.json), or None when they were taken on a different kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = os.path.join(ROOT, rec["kernel_source"])
    if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["sha256"]:
        return None
    w = rec["workloads"].get(workload)
    return None if w is None else w["bytes_per_launch"]


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, target_s: float) -> dict:
    import oracle
    cfg = inp.cfg
    nt = oracle.num_threads()
    rng = np.random.default_rng(123)
    ntok = max(1, nt)
    spent = 0.0
    while True:
        toks = np.sort(rng.choice(cfg.T, min(ntok, cfg.T), replace=False))
        t0 = time.perf_counter()
        oracle.layer_inputs(inp, tokens=toks)
        spent = time.perf_counter() - t0
        if spent >= target_s / 4 or ntok >= cfg.T:
            break
        ntok = min(cfg.T, int(ntok * max(2.0, target_s / max(spent, 1e-3) * 0.9)))
    return {"value": round(toks.size / spent, 3), "unit": "tokens/s", "cores": nt, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{toks.size} of {cfg.T} tokens of the same workload (route, paths, per-path "
                      f"float64 evaluation), {spent:.1f} s wall on {nt} threads"}


# ------------------------------------------------------------------ inputs on the device
def device_inputs(cfg, seed: int, host_weights: bool):
    """The layer's inputs on cuda:0. x, logits and the mask always come from the seeded host
    generator (they decide the routing); the expert weights too when host_weights (the
    oracle needs them), otherwise they are drawn on the device with the same distribution
    (N(0, w_std), rounded to the layer's dtype), which keeps the decode-shaped layer's 22 GB
    of weights off the host."""
    import torch
    from workloads import make_inputs
    dev = "cuda:0"
    inp = make_inputs(cfg, seed=seed, with_weights=host_weights)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d = {"x": inp.x.to(dev), "logits": torch.from_numpy(inp.logits).to(dev),
         "mask": torch.from_numpy(inp.mask).to(dev), "dtype": dtype, "inp": inp}
    if host_weights:
        d["wg"], d["wu"], d["wd"] = inp.w_gate.to(dev), inp.w_up.to(dev), inp.w_down.to(dev)
        d["shared"] = ((inp.s_gate.to(dev), inp.s_up.to(dev), inp.s_down.to(dev))
                       if cfg.shared_F else None)
    else:
        g = torch.Generator(device=dev).manual_seed(seed * 1000 + 17)

        def rnd(*shape):
            w = torch.empty(shape, dtype=torch.float32, device=dev)
            w.normal_(0.0, cfg.w_std, generator=g)
            return w.to(dtype)
        d["wg"], d["wu"], d["wd"] = rnd(cfg.n, cfg.F, cfg.H), rnd(cfg.n, cfg.F, cfg.H), rnd(cfg.n, cfg.H, cfg.F)
        d["shared"] = ((rnd(cfg.shared_F, cfg.H), rnd(cfg.shared_F, cfg.H), rnd(cfg.H, cfg.shared_F))
                       if cfg.shared_F else None)
    return d


def widen_down_weights(pcm, d):
    """Projection weights (routed and shared) as float16, widened once from the bf16 weights:
    a per-layer weight layout prepared before any step, like the packed mask. The bf16 copies
    are released."""
    d["wd"] = pcm.pcm_widen_f16(d["wd"])
    if d["shared"] is not None:
        g, u, dn = d["shared"]
        d["shared"] = (g, u, pcm.pcm_widen_f16(dn))


# ------------------------------------------------------------------ one workload
def measure(pcm, name, cfg, d, args, flush, scored):
    """Timed steps of one workload: wall time per step, per-stage times from HIP events, and
    the same stages again with the MALL flushed before each step."""
    import torch
    from paper_2609_01024_amd import binding
    dev = "cuda:0"
    stream = torch.cuda.current_stream()
    x, logits, mask, wg, wu, wd, shared = (d["x"], d["logits"], d["mask"], d["wg"], d["wu"],
                                           d["wd"], d["shared"])
    if scored:
        from workloads import make_scored_inputs
        sinp = make_scored_inputs(cfg, seed=args.seed)
        g_tgt = torch.from_numpy(sinp.g_tgt).to(dev)
        plan = pcm.ScoredLayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, d["dtype"], dev, cfg.shared_F)
        plan.build_layout(mask, torch.from_numpy(sinp.bias).to(dev))   # once per layer
        marks = (["shared"] if shared else []) + ["route", "expand"]
    else:
        sinp = None
        plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, d["dtype"], dev, cfg.shared_F)
        fused = args.indexing == "fused"
        packed = pcm.pcm_mask_pack(mask) if fused else None   # once per layer
        marks = (["shared"] if shared else []) + (["route_paths"] if fused else
                                                  ["route", "build_paths"]) + ["expand"]

    def new_events():
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(marks) + 1)]
        inner = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        for e in inner:           # created by a first record; the library records them again
            e.record(stream)
        t = binding.Tuning(stage_events=inner).struct()
        return ev, inner, t

    def step(slot=None):
        ev, _, tun = slot if slot is not None else (None, None, None)
        it = iter(range(len(marks) + 1))

        def mark():
            i = next(it)
            if ev is not None:
                ev[i].record(stream)
        mark()
        if shared:
            pcm.pcm_dense_swiglu(x, *shared, y=plan.y, accumulate=False, ws=plan.ws_shared)
            mark()
        if scored:
            pcm.pcm_route_scored(logits, g_tgt, sinp.lam, plan.layout, cfg.k, out=plan.paths,
                                 ws=plan.ws_route)
            mark()
            pcm.pcm_expand_scored(x, wg, wu, plan.paths, u=plan.u)
            mark()
            pcm.pcm_project_combine_scored(plan.u, wd, plan.paths, y=plan.y,
                                           accumulate=bool(shared), ws=plan.ws_proj, tuning=tun)
        else:
            if fused:
                pcm.pcm_route_paths(logits, packed, cfg.k, 0, plan.ids, plan.w, out=plan.paths,
                                    ws=plan.ws_index)
            else:
                pcm.pcm_route(logits, cfg.k, plan.ids, plan.w)
                mark()
                pcm.pcm_build_paths(plan.ids, plan.w, mask, 0, out=plan.paths, ws=plan.ws_paths)
            mark()
            pcm.pcm_expand(x, wg, wu, plan.paths, u=plan.u)
            mark()
            pcm.pcm_project_combine(plan.u, wd, plan.paths, y=plan.y, accumulate=bool(shared),
                                    ws=plan.ws_proj, tuning=tun)

    def stage_ms(slots):
        out = {}
        for i, st in enumerate(marks):
            out[st] = float(np.median([s[0][i].elapsed_time(s[0][i + 1]) for s in slots]))
        for i, st in enumerate(("mix", "project", "combine")):
            out[st] = float(np.median([s[1][i].elapsed_time(s[1][i + 1]) for s in slots]))
        out["project_combine"] = float(np.median([s[0][-1].elapsed_time(s[1][3]) for s in slots]))
        return out

    def fence():
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(1000)

    for _ in range(args.warmup):
        step()
    # the timed steps, with HIP events between the stages (the per-stage times and the roofline
    # come from the same launches as the step time and a profiler's fenced region; recording
    # the events costs no measurable time)
    slots = [new_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    fence()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(slots[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fence()
    torch.cuda.synchronize()
    timed = stage_ms(slots)
    # the same steps with the MALL flushed before each (outside the recorded stages)
    fslots = [new_events() for _ in range(args.steps)]
    for s in range(args.steps):
        flush.fill_(s & 0xFF)
        step(fslots[s])
    torch.cuda.synchronize()
    flushed = stage_ms(fslots)
    # the same step captured as one HIP graph (no per-call host cost), its replays timed like the
    # eager steps; kept beside the eager figure, which stays the headline
    graph_ms = None
    if not args.no_graph:
        try:
            graph = binding.capture_graph(lambda: step(None))
        except RuntimeError as err:   # an optional figure: the line is written without it
            print(f"[bench] {name}: no graph timing ({err})", file=sys.stderr, flush=True)
            torch.cuda.synchronize()
            return plan, sinp, wall * 1e3 / args.steps, timed, flushed, None
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        fence()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        fence()
        torch.cuda.synchronize()
        del graph
    return plan, sinp, wall * 1e3 / args.steps, timed, flushed, graph_ms


def workload_record(pcm, acc, name, cfg, plan, sinp, ms, st, fl, scored):
    """Throughput, GEMM rates against the bf16 peak and GB/s of the memory-bound stages."""
    bf16 = cfg.dtype == "bf16"
    K = cfg.k
    if scored:
        src_off = plan.paths.src_offsets.cpu().numpy()
        tgt_off = plan.paths.tgt_offsets.cpu().numpy()
        R, R_tgt = int(src_off[-1]), int(tgt_off[-1])
        touched_src = int(np.count_nonzero(np.diff(src_off)))
        touched_tgt = int(np.count_nonzero(np.diff(tgt_off)))
        touched = int(np.count_nonzero(np.diff(src_off) + np.diff(tgt_off)))
        R_bound = cfg.T * K
    else:
        off = plan.paths.expert_offsets.cpu().numpy()
        touched = touched_src = touched_tgt = int(np.count_nonzero(np.diff(off)))
        R = R_tgt = R_bound = cfg.R
    if scored:
        per_expert = np.diff(src_off)
        n_paths = int(R_bound)
    else:
        per_expert = np.diff(off)
        n_paths = int(np.unpackbits(plan.paths.path_bits.cpu().numpy().view(np.uint8)).sum())
    f = acc.gemm_flops(R, cfg.H, cfg.F, cfg.T, cfg.shared_F, R_tgt)
    peak = acc.BF16_PEAK_TFLOPS if bf16 else acc.FP32_PEAK_TFLOPS
    gemm_ms = st["expand"] + st["project_combine"] + st.get("shared", 0.0)
    ksplit = pcm.project_workspace_layout(cfg.T, cfg.H, cfg.F, cfg.n, K,
                                          pcm.PCM_BF16 if bf16 else pcm.PCM_F32)["ksplit"]
    u_elem, z_elem = 4, (2 if bf16 else 4)
    hbm = {"mix": acc.mix_bytes(R, R_tgt, cfg.F, cfg.T, K, u_elem, z_elem) / (fl["mix"] * 1e-3) / 1e9,
           "combine": acc.combine_bytes(R_bound, cfg.H, cfg.T, K, ksplit, bool(cfg.shared_F))
           / (fl["combine"] * 1e-3) / 1e9}
    if "route_paths" in fl:
        hbm["route_paths"] = acc.route_paths_bytes(cfg.T, cfg.n, K) / (fl["route_paths"] * 1e-3) / 1e9
    elif not scored:
        hbm["route"] = acc.route_bytes(cfg.T, cfg.n, K) / (fl["route"] * 1e-3) / 1e9
        hbm["build_paths"] = acc.paths_bytes(cfg.T, cfg.n, K) / (fl["build_paths"] * 1e-3) / 1e9
    rec = {"ms": round(ms, 4), "tokens_per_s": round(cfg.T / (ms * 1e-3), 1),
           "rows": R, "touched_experts": touched,
           "rows_per_expert_min": int(per_expert.min()), "rows_per_expert_max": int(per_expert.max()),
           "paths": n_paths,
           "gemm_tflops": round(f["total"] / (gemm_ms * 1e-3) / 1e12, 1),
           "gemm_frac_peak": round(f["total"] / (gemm_ms * 1e-3) / 1e12 / peak, 4),
           "stages_ms": {k: round(v, 4) for k, v in st.items()},
           "stages_flushed_ms": {k: round(v, 4) for k, v in fl.items()},
           "hbm_GBps": {k: round(v, 1) for k, v in hbm.items()},
           "hbm_frac": {k: round(v / acc.HBM_PEAK_GBS, 4) for k, v in hbm.items()}}
    if scored:
        rec["projection_rows"] = R_tgt
    if name == "decode":
        # weight streaming: every touched expert's matrices are read once per step
        eb = touched_src * 2 * cfg.H * cfg.F * 2
        pb = touched_tgt * cfg.H * cfg.F * 2
        rec.update({"expand_GBps": round(eb / (st["expand"] * 1e-3) / 1e9, 1),
                    "expand_frac": round(eb / (st["expand"] * 1e-3) / 1e9 / acc.HBM_PEAK_GBS, 4),
                    "project_GBps": round(pb / (st["project"] * 1e-3) / 1e9, 1),
                    "project_frac": round(pb / (st["project"] * 1e-3) / 1e9 / acc.HBM_PEAK_GBS, 4),
                    "layer_weight_GBps": round((eb + pb) / (ms * 1e-3) / 1e9, 1)})
    else:
        et = f["expand"] / (st["expand"] * 1e-3) / 1e12
        pt = f["project"] / (st["project"] * 1e-3) / 1e12
        rec.update({"expand_tflops": round(et, 1), "expand_frac": round(et / peak, 4),
                    "project_tflops": round(pt, 1), "project_frac": round(pt / peak, 4)})
        if cfg.shared_F:
            rec["shared_tflops"] = round((f["shared_expand"] + f["shared_project"])
                                         / (st["shared"] * 1e-3) / 1e12, 1)
    return rec, f, R, touched_src


# ------------------------------------------------------------------ other modes
def stack_bench(args):
    """A decode step through a stack of L MoE layers of the workload's shape, weights drawn
    on the device (resident in HBM before timing)."""
    import torch
    from paper_2609_01024_amd.stack import random_stack
    from workloads import CONFIGS
    name = args.config or "decode"
    cfg = CONFIGS[name]
    dev = "cuda:0"
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    t0 = time.time()
    st = random_stack(args.stack, cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, cfg.density, args.seed, dev,
                      dtype, w_std=cfg.w_std)
    g = torch.Generator(device=dev).manual_seed(args.seed + 1)
    x0 = (torch.randn((cfg.T, cfg.H), generator=g, device=dev) * cfg.x_std).to(dtype)
    h = x0.clone()
    torch.cuda.synchronize()
    print(f"[bench] stack of {args.stack}: weights in {time.time() - t0:.1f} s", file=sys.stderr,
          flush=True)
    for _ in range(args.warmup):
        h.copy_(x0)
        st.forward(h)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        h.copy_(x0)
        st.forward(h)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ms_graph = None
    if not args.no_graph:   # the step's layers as one HIP graph (the reset of h stays eager)
        graph = st.capture(h)
        for _ in range(args.warmup):
            h.copy_(x0)
            graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            h.copy_(x0)
            graph.replay()
        torch.cuda.synchronize()
        ms_graph = (time.perf_counter() - t0) * 1e3 / args.steps
        del graph
    wbytes = args.stack * 3 * cfg.n * cfg.H * cfg.F * (2 if dtype == torch.bfloat16 else 4)
    line = {"metric": "decode step through a stack of path-MoE layers, tokens/sec, 1 GPU",
            "value": round(cfg.T / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16" if dtype == torch.bfloat16 else "f32", "data": "synthetic",
            "config": {"workload": f"{args.stack} x {name}: T={cfg.T} H={cfg.H} n={cfg.n} "
                                   f"F={cfg.F} k={cfg.k}, layers 0-1 diagonal-only, then mask "
                                   f"density {cfg.density}", "layers": args.stack},
            "ms_per_layer": round(ms / args.stack, 4),
            "all_expert_weight_GB": round(wbytes / 1e9, 1)}
    if ms_graph is not None:
        line["ms_per_step_graph"] = round(ms_graph, 4)
        line["tokens_per_s_graph"] = round(cfg.T / (ms_graph * 1e-3), 1)
    print(json.dumps(line), flush=True)


def router_gemm(pcm, cfg, x, args):
    """The router's own GEMM fused with the top-k (pcm_route_logits) on this workload's x and
    a seeded router matrix of shape [n, H]; reported beside the layer, not inside it (the
    workloads' logits are drawn directly)."""
    import torch
    from workloads import make_router_weights
    wr = make_router_weights(cfg, seed=args.seed).to(x.device)
    ids = torch.empty((cfg.T, cfg.k), dtype=torch.int32, device=x.device)
    w = torch.empty((cfg.T, cfg.k), dtype=torch.float32, device=x.device)
    nws = pcm.workspace_bytes(6, cfg.T, cfg.H, 0, cfg.n, cfg.k, 1 if cfg.dtype == "bf16" else 0)
    ws = torch.empty((max(nws, 1),), dtype=torch.uint8, device=x.device) if nws else None
    for _ in range(max(1, args.warmup)):
        pcm.pcm_route_logits(x, wr, cfg.k, topk_ids=ids, topk_w=w, ws=ws)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        pcm.pcm_route_logits(x, wr, cfg.k, topk_ids=ids, topk_w=w, ws=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    elem = 2 if cfg.dtype == "bf16" else 4
    nbytes = (cfg.T * cfg.H + cfg.n * cfg.H) * elem + cfg.T * cfg.k * 8
    return {"ms": round(ms, 4), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "TFLOPs": round(2 * cfg.T * cfg.H * cfg.n / (ms * 1e-3) / 1e12, 2)}


def ablation(pcm, plan, cfg, d, args):
    """Layer time of the same routing and paths executed three other ways (Table 3's
    question on this hardware): one projection per path reusing U per source; one expansion
    and one projection per path; and the vanilla top-k layer (diagonal-only mask)."""
    import torch
    x, logits, mask, wg, wu, wd, shared = (d["x"], d["logits"], d["mask"], d["wg"], d["wu"],
                                           d["wd"], d["shared"])
    n_paths = int(np.unpackbits(plan.paths.path_bits.cpu().numpy().view(np.uint8)).sum())

    def timed(fn):
        for _ in range(max(1, args.warmup)):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps

    ws = torch.empty((pcm.workspace_bytes(5, cfg.T, cfg.H, cfg.F, cfg.n, cfg.k,
                                          1 if cfg.dtype == "bf16" else 0),), dtype=torch.uint8,
                     device=x.device)
    y = torch.empty_like(plan.y)

    packed = pcm.pcm_mask_pack(mask)   # every variant indexes through the fused operation

    def per_path(reuse):
        def fn():
            if shared:
                pcm.pcm_dense_swiglu(x, *shared, y=y, accumulate=False, ws=plan.ws_shared)
            plan.index(logits, packed)
            pcm.pcm_layer_per_path(x, wg, wu, wd, plan.paths, reuse=reuse, y=y,
                                   accumulate=bool(shared), ws=ws)
        return fn

    eye = pcm.pcm_mask_pack(torch.eye(cfg.n, dtype=torch.uint8, device=x.device))

    def mixed(m):
        def fn():
            plan.forward(x, logits, m, wg, wu, wd, shared)
        return fn

    out = {"paths": n_paths, "expansion_rows_reused": cfg.R,
           "ms_target_mix": round(timed(mixed(packed)), 4),
           "ms_per_path_reuse": round(timed(per_path(True)), 4),
           "ms_per_path_no_reuse": round(timed(per_path(False)), 4),
           "ms_vanilla_topk": round(timed(mixed(eye)), 4)}
    del ws
    return out


def main():
    args = parse()
    if args.trace_summary:
        trace_summary(args.trace_summary)
        return
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer is sharded by design, not measured, across GPUs)", file=sys.stderr)
        sys.exit(2)
    if args.stack:
        stack_bench(args)
        return
    if args.vendor_compare:
        vendor_compare(args)
        return

    import torch

    import paper_2609_01024_amd as pcm
    from paper_2609_01024_amd import accounting as acc
    from workloads import CONFIGS, HEADLINE

    head = args.config or HEADLINE
    scored = args.router == "scored"
    order = [head] + ([] if args.only else [w for w in CONFIGS if w != head])
    flush = torch.empty((FLUSH_BYTES,), dtype=torch.uint8, device="cuda:0")
    records, line = {}, None
    for name in order:
        cfg = CONFIGS[name]
        t0 = time.time()
        d = device_inputs(cfg, args.seed, host_weights=(name == head))
        if cfg.dtype == "bf16" and args.down_weights == "f16":
            widen_down_weights(pcm, d)
        print(f"[bench] {name}: inputs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
        plan, sinp, ms, st, fl, graph_ms = measure(pcm, name, cfg, d, args, flush, scored)
        rec, f, R, touched_src = workload_record(pcm, acc, name, cfg, plan, sinp, ms, st, fl, scored)
        if graph_ms is not None:
            rec["ms_graph"] = round(graph_ms, 4)
            rec["tokens_per_s_graph"] = round(cfg.T / (graph_ms * 1e-3), 1)
        records[name] = rec
        print(f"[bench] {name}: {ms:.3f} ms per layer", file=sys.stderr, flush=True)
        if name == head:
            bf16 = cfg.dtype == "bf16"
            peak = acc.BF16_PEAK_TFLOPS if bf16 else acc.FP32_PEAK_TFLOPS
            traffic = measured_traffic(name)
            if name == "decode":
                exp_bytes = touched_src * 2 * cfg.H * cfg.F * 2
                achieved = exp_bytes / (st["expand"] * 1e-3) / 1e9
                roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": acc.HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(achieved / acc.HBM_PEAK_GBS, 4),
                        "traffic": traffic, "kernel": "expand (grouped gate/up GEMM + SwiGLU)",
                        "per_launch": f"{touched_src} source experts x 2*H*F*2 B of gate/up weights"}
            else:
                achieved = f["expand"] / (st["expand"] * 1e-3) / 1e12
                roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak,
                        "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": traffic,
                        "kernel": "expand (grouped gate/up GEMM + SwiGLU)",
                        "per_launch": f"4*H*F flop x R={R} rows"}
            line = {
                "metric": METRIC, "value": round(cfg.T / (ms * 1e-3), 1), "unit": "tokens/s",
                "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
                "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                "dtype": "bf16" if bf16 else "f32", "data": "synthetic",
                "config": {"workload": f"{name}: T={cfg.T} H={cfg.H} n={cfg.n} F={cfg.F} k={cfg.k} "
                                       f"mask density {cfg.density}"
                                       + (f" shared F={cfg.shared_F}" if cfg.shared_F else ""),
                           "tokens": cfg.T, "rows": R, "touched_experts": rec["touched_experts"],
                           "router": args.router,
                           "down_weights": ("float16, widened once from the bf16 weights"
                                            if bf16 and args.down_weights == "f16" else cfg.dtype),
                           **({"projection_rows": rec["projection_rows"], "lambda": sinp.lam}
                              if scored else {})},
                "gemm_tflops": rec["gemm_tflops"], "gemm_frac_peak": rec["gemm_frac_peak"],
                "stages_ms": rec["stages_ms"], "hbm_GBps": rec["hbm_GBps"], "roofline": roof,
            }
            line["router_gemm"] = router_gemm(pcm, cfg, d["x"], args)
            if not args.no_ablation and not scored:
                line["ablation"] = ablation(pcm, plan, cfg, d, args)
            if not args.no_cpu_baseline:
                print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
                line["cpu_baseline"] = cpu_baseline(d["inp"], args.cpu_seconds)
        del plan, d
        torch.cuda.empty_cache()
    line["workloads"] = records
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
