#!/usr/bin/env python3
"""Benchmark of the fused routed-MoE decode operator on one MI355X.

One step = one forward of the operator for each decode token count T in {1, 2, 4, 8} on
the small-expert layer shape (H=2048, E=128, I=768, top-8, renormalised softmax), each
forward on its own synthetic layer.  Layers rotate over `--layers` distinct weight sets
so that successive launches stream weights from HBM rather than from the 256 MB
last-level cache (as consecutive MoE layers of a decode step do).

Each launch's duration comes from HIP events that its own dispatch stamps (hipExtLaunchKernel
through monomoe_forward_timed): the kernel's begin and end, as a kernel trace reports them.

Printed (one JSON line): value = algorithmic bytes of the step / summed launch time (GB/s);
per-T latency (mean and p50, microseconds), achieved GB/s and fraction of the 8 TB/s peak;
a roofline object for the kernel; and the CPU oracle timed on a bounded sample.

Other layers and token counts (up to 64, where the multi-tile kernel runs) are a flag away:
`--workload coarse --tokens 16,32,64`; the workload's routing policy (softmax, or sigmoid
with a selection bias) is applied to every plan.  The roofline's measured traffic is the
committed FETCH_SIZE/WRITE_SIZE record of each T's kernel on that workload, when there is
one and its kernel sources are unchanged.

Algorithmic bytes of one launch: every selected expert's weights read once,
U * 3*H*I fp8 bytes plus their fp32 block scales U * 3*H*I/4096, plus the router
weight E*H*2, the input T*H*2 and the output T*H*2 bytes.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
TS = (1, 2, 4, 8)
# HBM counter records (rocprofv3 FETCH_SIZE / WRITE_SIZE passes over the C++ profiling
# driver, calibrated on a plain copy kernel), one per kernel and workload; a record is used
# only while its kernel's sources still hash to the value it was taken on.
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="small_expert")
    ap.add_argument("--tokens", default="1,2,4,8",
                    help="decode token counts of one step (up to 64; the metric is quoted on 1,2,4,8)")
    ap.add_argument("--layers", type=int, default=16)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    return ap.parse_args()


def algorithmic_bytes(U, T, H, E, I):
    """Bytes one launch must move at least once: the U selected experts' fp8 weights and
    fp32 block scales, the bf16 router weight, input and output."""
    weights = U * 3 * H * I
    scales = U * 3 * (H // 128) * (I // 128) * 4
    return weights + scales + E * H * 2 + 2 * T * H * 2


def measured_traffic(workload, kinds):
    """HBM bytes per launch (read + write, mean over the step's token counts) from the
    committed counter records, or None unless every token count T has a record of this
    workload, taken on the kernel that runs at T (kinds[T], "single" or "multi") whose
    sources have not changed since."""
    import glob
    from paper_2609_04244_amd.profile_layer import kernel_kind, kernel_source_hash
    per = {}
    for path in sorted(glob.glob(os.path.join(PROFILES, "*_counters.json"))):
        with open(path) as fh:
            rec = json.load(fh)
        kind = kernel_kind(rec.get("kernel", ""))
        if rec.get("workload") != workload or rec.get("kernel_source_sha256") != kernel_source_hash(kind):
            continue
        for T, v in rec.get("per_T", {}).items():
            if "fetch_bytes" in v and kinds.get(int(T)) == kind:
                per.setdefault(int(T), v["fetch_bytes"] + v["write_bytes"])
    if any(T not in per for T in TS):
        return None
    return sum(per[T] for T in TS) / len(TS)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this operator build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2609_04244_amd import monomoe as mm
    from paper_2609_04244_amd import workloads as wl

    global TS
    TS = tuple(int(t) for t in args.tokens.split(","))
    cfg = wl.config(args.workload)
    H, E, I, k, renorm = cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print("bench: generating %d layers of %s" % (args.layers, args.workload), file=sys.stderr, flush=True)
    layers = [wl.generate(cfg, T=max(TS), seed=args.seed + 1000 * l, device=dev) for l in range(args.layers)]
    plans = {T: mm.Plan(T, H, E, I, k, renorm) for T in TS}
    outs = {T: torch.empty((T, H), dtype=torch.bfloat16, device=dev) for T in TS}
    xs = {(l, T): layers[l]["x"][:T].contiguous() for l in range(args.layers) for T in TS}

    def route(p, L):   # the layer's routing inputs (logit bias; sigmoid selection bias)
        if L["bias"] is not None:
            p.set_router_bias(L["bias"])
        if L["policy"] == "sigmoid_bias":
            p.set_routing(mm.ROUTING_SIGMOID_BIAS, L["sel_bias"], L["route_scale"])

    def launch(l, T, timer):
        L = layers[l]
        p = plans[T]
        route(p, L)
        p.forward_timed(xs[(l, T)], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], outs[T], timer)

    # unique experts of every (layer, T), from the operator's own selection (untimed)
    U = {}
    for l in range(args.layers):
        for T in TS:
            L = layers[l]
            route(plans[T], L)
            _, d = plans[T].forward_debug(xs[(l, T)], L["router_w"], L["w13"], L["w13_scale"], L["w2"],
                                          L["w2_scale"])
            torch.cuda.synchronize()
            U[(l, T)] = len(set(d["ids"].cpu().numpy().reshape(-1).tolist()))
    for T in TS:
        if plans[T].status() != mm.MONOMOE_OK:
            raise RuntimeError("device status after the selection pass: %s" % mm.status_string(plans[T].status()))

    stream = torch.cuda.current_stream()
    order = [(s, T) for s in range(args.warmup + args.steps) for T in TS]
    n_launch = len(order)
    # each launch's dispatch stamps its own begin and end (hipExtLaunchKernel events)
    timers = [mm.DispatchTimer() for _ in range(n_launch)]
    layer_of = []
    li = 0
    for i in range(n_launch):
        layer_of.append(li % args.layers)
        li += 1

    torch.cuda.synchronize()
    t_start = None
    w_start = torch.cuda.Event(enable_timing=True)
    w_end = torch.cuda.Event(enable_timing=True)
    for i, (s, T) in enumerate(order):
        if s == args.warmup and t_start is None:
            torch.cuda.synchronize()
            t_start = time.perf_counter()
            w_start.record(stream)
        launch(layer_of[i], T, timers[i])
    w_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    for T in TS:
        st = plans[T].status()
        if st != mm.MONOMOE_OK:
            raise RuntimeError("device status after timing: %s" % mm.status_string(st))

    per_T = {}
    tot_bytes = 0.0
    tot_ms = 0.0
    wbytes_tot = 0.0
    for T in TS:
        ms, by, wb = [], [], []
        for i, (s, TT) in enumerate(order):
            if s < args.warmup or TT != T:
                continue
            ms.append(timers[i].elapsed_ms())
            u = U[(layer_of[i], T)]
            by.append(algorithmic_bytes(u, T, H, E, I))
            wb.append(u * 3 * H * I)
        ms = np.array(ms)
        by = np.array(by, dtype=np.float64)
        gbps = by.sum() / (ms.sum() * 1e-3) / 1e9
        per_T[str(T)] = {
            "us_mean": round(float(ms.mean() * 1e3), 2), "us_p50": round(float(np.median(ms) * 1e3), 2),
            "us_p10": round(float(np.percentile(ms, 10) * 1e3), 2),
            "us_p90": round(float(np.percentile(ms, 90) * 1e3), 2),
            "unique_experts_mean": round(float(np.mean([U[(l, T)] for l in range(args.layers)])), 2),
            "unique_experts_uniform_estimate": round(wl.expected_unique_experts(E, k, T), 2),
            "GBps": round(float(gbps), 1), "frac_of_peak": round(float(gbps / PEAK_HBM_GBPS), 4),
            "expert_weight_GBps": round(float(np.sum(wb) / (ms.sum() * 1e-3) / 1e9), 1),
        }
        tot_bytes += by.sum()
        tot_ms += ms.sum()
        wbytes_tot += float(np.sum(wb))
    value = tot_bytes / (tot_ms * 1e-3) / 1e9
    ms_per_step = w_start.elapsed_time(w_end) / args.steps
    kinds = {T: "multi" if plans[T].info()["multi_tile"] else "single" for T in TS}
    traffic = measured_traffic(args.workload, kinds)

    res = {
        "metric": "routed-MoE op latency us + achieved HBM GB/s (% of peak) at T=" + ",".join(map(str, TS)) + " tokens",
        "value": round(float(value), 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(float(ms_per_step), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {
            "workload": "%s: H=%d E=%d I=%d top-%d %s, block-FP8 128x128 weights, T in %s, "
                        "%d rotated layers" % (args.workload, H, E, I, k,
                                               "sigmoid routing with selection bias"
                                               if cfg.get("policy") == "sigmoid_bias" else
                                               ("renormalised" if renorm else "plain") + " softmax",
                                               list(TS), args.layers),
            "launches_per_step": len(TS), "grid": plans[TS[0]].info()["grid"],
            "block": plans[TS[0]].info()["block"],
        },
        "per_T": per_T,
        "roofline": {
            "bound": "hbm", "achieved": round(float(value), 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(float(value / PEAK_HBM_GBPS), 4),
            "traffic": None if traffic is None else round(float(traffic)),
            "traffic_unit": "HBM bytes per launch (read + write, mean over T)",
            "algorithmic_bytes_per_launch": round(float(tot_bytes / (args.steps * len(TS)))),
            "kernel": ", ".join(sorted({"monomoe_fused%s<%d,%d>" % ("_mt" if plans[T].info()["multi_tile"] else "", H, I)
                                        for T in TS})),
            "launch_us_mean": round(float(tot_ms / (args.steps * len(TS)) * 1e3), 2),
        },
        "wall_s_timed": round(wall, 3),
    }

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(args, layers, U, plans, outs, xs, cfg, wbytes_tot / args.steps,
                                           tot_bytes / args.steps)
    for p in plans.values():
        p.close()
    print(json.dumps(res), flush=True)


def cpu_baseline(args, layers, U, plans, outs, xs, cfg, wbytes_step, bytes_step):
    """The fp64 oracle on the host cores, on a bounded sample of the same workload: the
    step's forwards (one per token count) on layer 0, repeated while under the time budget.
    Also checks the operator's outputs on those forwards against the oracle."""
    import numpy as np
    import torch
    from oracle import oracle
    from paper_2609_04244_amd import monomoe as mm
    from paper_2609_04244_amd import workloads as wl

    H, E, I, k, renorm = cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"]
    L = layers[0]
    rw = wl.bf16_bits(L["router_w"])
    bias = None if L["bias"] is None else L["bias"].cpu().numpy()
    sigmoid = L["policy"] == "sigmoid_bias"
    sel_bias = None if not sigmoid or L["sel_bias"] is None else L["sel_bias"].cpu().numpy()
    route = dict(policy=oracle.SIGMOID_BIAS, sel_bias=sel_bias, scale=L["route_scale"]) if sigmoid else {}
    logits = oracle.router_logits(wl.bf16_bits(L["x"]), rw, bias)
    if sigmoid:
        ids, _ = oracle.select_sigmoid(logits, k, sel_bias, L["route_scale"])
    else:
        ids, _ = oracle.select(logits, k, renorm)
    ex = sorted(set(ids.reshape(-1).tolist()))
    idx = torch.tensor(ex, device=L["w13"].device)
    host = [t.index_select(0, idx).cpu().numpy() for t in (L["w13"], L["w13_scale"], L["w2"], L["w2_scale"])]
    tabs = [{e: a[i] for i, e in enumerate(ex)} for a in host]
    worst = 0.0
    mre_worst = 0.0
    t0 = time.perf_counter()
    reps = 0
    while True:
        for T in TS:
            ref = oracle.forward(wl.bf16_bits(xs[(0, T)]), rw, *tabs, k, renorm, bias=bias, **route)
            if reps == 0:
                p = plans[T]
                if L["bias"] is not None:
                    p.set_router_bias(L["bias"])
                if sigmoid:
                    p.set_routing(mm.ROUTING_SIGMOID_BIAS, L["sel_bias"], L["route_scale"])
                out = p.forward(xs[(0, T)], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"])
                torch.cuda.synchronize()
                got = out.float().cpu().numpy().astype(np.float64)
                rms = float(np.sqrt(np.mean(ref ** 2)))
                worst = max(worst, float(np.abs(got - ref).max()) / rms)
                mre_worst = max(mre_worst, float(np.abs(got - ref).sum() / np.abs(ref).sum()))
        reps += 1
        if time.perf_counter() - t0 >= args.cpu_seconds:
            break
    dt = (time.perf_counter() - t0) / reps
    u0 = sum(U[(0, T)] for T in TS)
    wb0 = sum(U[(0, T)] * 3 * H * I for T in TS)
    by0 = sum(algorithmic_bytes(U[(0, T)], T, H, E, I) for T in TS)
    return {
        "value": round(by0 / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
        "sample": "the step's %d forwards (T=%s) on layer 0, %d repetition(s), %.2f s each; "
                  "%d selected experts in total" % (len(TS), ",".join(map(str, TS)), reps, dt, u0),
        "ms_per_step": round(dt * 1e3, 1),
        "gpu_vs_oracle_max_err_over_rms": round(worst, 5), "gpu_vs_oracle_mean_rel_err": round(mre_worst, 6),
    }


if __name__ == "__main__":
    main()
