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
# HBM counter record of this workload (rocprofv3 FETCH_SIZE / WRITE_SIZE passes over the
# C++ profiling driver, calibrated on a plain copy kernel); used only while the kernel
# sources still hash to the value it was taken on.
COUNTERS = os.path.join(ROOT, "profiles", "monomoe_fused_small_expert_counters.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="small_expert")
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


def measured_traffic(workload):
    """HBM bytes per launch (read + write, mean over the step's token counts) from the
    committed counter record, or None when there is none for this workload or the kernel
    sources changed since it was taken."""
    try:
        with open(COUNTERS) as fh:
            rec = json.load(fh)
    except OSError:
        return None
    from paper_2609_04244_amd.profile_layer import kernel_kind, kernel_source_hash
    if (rec.get("workload") != workload or
            rec.get("kernel_source_sha256") != kernel_source_hash(kernel_kind(rec.get("kernel", "")))):
        return None
    per = rec["per_T"]
    if any(str(T) not in per or "fetch_bytes" not in per[str(T)] for T in TS):
        return None
    return sum(per[str(T)]["fetch_bytes"] + per[str(T)]["write_bytes"] for T in TS) / len(TS)


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

    cfg = wl.config(args.workload)
    H, E, I, k, renorm = cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print("bench: generating %d layers of %s" % (args.layers, args.workload), file=sys.stderr, flush=True)
    layers = [wl.generate(cfg, T=max(TS), seed=args.seed + 1000 * l, device=dev) for l in range(args.layers)]
    plans = {T: mm.Plan(T, H, E, I, k, renorm) for T in TS}
    outs = {T: torch.empty((T, H), dtype=torch.bfloat16, device=dev) for T in TS}
    xs = {(l, T): layers[l]["x"][:T].contiguous() for l in range(args.layers) for T in TS}

    def launch(l, T, timer):
        L = layers[l]
        p = plans[T]
        if L["bias"] is not None:
            p.set_router_bias(L["bias"])
        p.forward_timed(xs[(l, T)], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], outs[T], timer)

    # unique experts of every (layer, T), from the operator's own selection (untimed)
    U = {}
    for l in range(args.layers):
        for T in TS:
            L = layers[l]
            if L["bias"] is not None:
                plans[T].set_router_bias(L["bias"])
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
    traffic = measured_traffic(args.workload)

    res = {
        "metric": "routed-MoE op latency us + achieved HBM GB/s (% of peak) at T=1,2,4,8 tokens",
        "value": round(float(value), 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(float(ms_per_step), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {
            "workload": "%s: H=%d E=%d I=%d top-%d %s softmax, block-FP8 128x128 weights, T in %s, "
                        "%d rotated layers" % (args.workload, H, E, I, k, "renormalised" if renorm else "plain",
                                               list(TS), args.layers),
            "launches_per_step": len(TS), "grid": plans[1].info()["grid"], "block": plans[1].info()["block"],
        },
        "per_T": per_T,
        "roofline": {
            "bound": "hbm", "achieved": round(float(value), 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(float(value / PEAK_HBM_GBPS), 4),
            "traffic": None if traffic is None else round(float(traffic)),
            "traffic_unit": "HBM bytes per launch (read + write, mean over T)",
            "algorithmic_bytes_per_launch": round(float(tot_bytes / (args.steps * len(TS)))),
            "kernel": "monomoe_fused<%d,%d>" % (H, I),
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
    step's four forwards (T = 1, 2, 4, 8) on layer 0, repeated while under the time budget.
    Also checks the operator's outputs on those forwards against the oracle."""
    import numpy as np
    import torch
    from oracle import oracle
    from paper_2609_04244_amd import workloads as wl

    H, E, I, k, renorm = cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"]
    L = layers[0]
    rw = wl.bf16_bits(L["router_w"])
    bias = None if L["bias"] is None else L["bias"].cpu().numpy()
    logits = oracle.router_logits(wl.bf16_bits(L["x"]), rw, bias)
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
            ref = oracle.forward(wl.bf16_bits(xs[(0, T)]), rw, *tabs, k, renorm, bias=bias)
            if reps == 0:
                p = plans[T]
                if L["bias"] is not None:
                    p.set_router_bias(L["bias"])
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
        "sample": "the step's 4 forwards (T=1,2,4,8) on layer 0, %d repetition(s), %.2f s each; "
                  "%d selected experts in total" % (reps, dt, u0),
        "ms_per_step": round(dt * 1e3, 1),
        "gpu_vs_oracle_max_err_over_rms": round(worst, 5), "gpu_vs_oracle_mean_rel_err": round(mre_worst, 6),
    }


if __name__ == "__main__":
    main()
