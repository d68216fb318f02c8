#!/usr/bin/env python3
"""Benchmark of the fused routed-MoE decode operator on one MI355X.

One step = one forward of the operator for each decode token count T in {1, 2, 4, 8}; each
(layer, T) is timed over its own block of consecutive launches (the paper's isolated-operator
protocol, repeated launches of one operator configuration, as the MoE layers of one decode step
at one batch size run; `--order interleaved` cycles T within every step instead).  The layers:
  wide_fine         H=7168 E=256 I=2048 top-8, renormalised softmax (the headline: the largest
                    evaluated layer that fits one GPU, ~11 GB of FP8 expert weights),
  small_expert      H=2048 E=128 I=768  top-8, renormalised softmax,
  many_tiny_expert  H=2048 E=256 I=512  top-8, renormalised softmax with a per-expert logit
                    bias (the paper's Qwen3.5-35B-A3B per-GPU shape).
Every layer rotates over enough distinct synthetic weight sets that the weights a launch reads
were last read more than 512 MB of weight traffic earlier (twice the 256 MB last-level cache),
so every launch streams its weights from HBM, as consecutive MoE layers of a decode step do.

Each launch's duration comes from HIP events that its own dispatch stamps (hipExtLaunchKernel
through monomoe_forward_timed): the kernel's begin and end, as a kernel trace reports them.
The forwards of every weight set at one T are also captured into one HIP graph (as a decode
step's graph holds a model's MoE layers) and its replays are event-timed on the stream (the
paper's protocol: graph replays after warm-ups); replay time over the graph's launches is
reported beside the kernel time.

Printed (one JSON line): value = algorithmic bytes / summed launch time (GB/s) of the headline
layer over its token counts; per-T latency (mean, p10/p50/p90, graph replay p50), achieved GB/s
and fraction of the 8 TB/s peak; the same block for every layer under "workloads"; a roofline
object for the headline kernel, which also carries the device's achievable HBM read rate
measured in the same run (a plain streaming-read kernel over 2 GiB) and the value's fraction of
it; the CPU oracle on a bounded sample of the headline layer, on one host core and on all of
them.

Other layers and token counts (up to 64, where the multi-tile kernel runs) are a flag away:
`--workloads coarse --tokens 16,32,64`; each layer's routing policy (softmax, or sigmoid with a
selection bias) is applied to its plans.  A workload's measured traffic is the committed
FETCH_SIZE/WRITE_SIZE record of each T's kernel on that workload, when there is one and its
kernel sources are unchanged.

Algorithmic bytes of one launch: every selected expert's weights read once,
U * 3*H*I fp8 bytes plus their fp32 block scales U * 3*H*I/4096, plus the router
weight E*H*2, the input T*H*2 and the output T*H*2 bytes.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
DEFAULT_WORKLOADS = "wide_fine,small_expert,many_tiny_expert"
REUSE_BYTES = 512e6       # weight bytes between two reads of the same weights, at least
LAYER_BUDGET = 40e9       # device bytes of generated layers per workload, at most
# HBM counter records (rocprofv3 FETCH_SIZE / WRITE_SIZE passes over the C++ profiling
# driver, calibrated on a plain copy kernel), one per kernel and workload; a record is used
# only while its kernel's sources still hash to the value it was taken on.
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workloads", default=DEFAULT_WORKLOADS,
                    help="comma-separated layers; the first is the headline")
    ap.add_argument("--workload", help="a single layer (same as --workloads NAME)")
    ap.add_argument("--tokens", default="1,2,4,8",
                    help="decode token counts of one step (up to 64; the metric is quoted on 1,2,4,8)")
    ap.add_argument("--layers", type=int, default=0, help="weight sets per workload (0: as the reuse bound needs)")
    ap.add_argument("--replays", type=int, default=100,
                    help="timed launches per T in graph replays (a replay launches every weight set once); 0: none")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--order", choices=("blocked", "interleaved"), default="blocked",
                    help="blocked: each (layer, T) timed over consecutive launches; interleaved: T cycles "
                         "within every step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="per oracle mode (one core, all cores)")
    return ap.parse_args()


def algorithmic_bytes(U, T, H, E, I):
    """Bytes one launch must move at least once: the U selected experts' fp8 weights and
    fp32 block scales, the bf16 router weight, input and output."""
    weights = U * 3 * H * I
    scales = U * 3 * (H // 128) * (I // 128) * 4
    return weights + scales + E * H * 2 + 2 * T * H * 2


def layers_needed(cfg, TS, expected_unique):
    """Distinct weight sets so that, with the launches of all token counts rotating over them,
    a launch's weights were last read at least REUSE_BYTES of weight traffic earlier."""
    H, E, I, k = cfg["H"], cfg["E"], cfg["I"], cfg["k"]
    smallest = min(expected_unique(E, k, T) for T in TS) * 3 * H * I
    n = int(math.ceil(REUSE_BYTES / smallest)) + 1
    layer_bytes = E * 3 * H * I
    return max(2, min(n, int(LAYER_BUDGET // layer_bytes)))


def measured_traffic(workload, kinds, TS):
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
        if rec.get("workload") != workload:
            continue
        for T, v in rec.get("per_T", {}).items():
            kind = kernel_kind(v.get("kernel", rec.get("kernel", "")))
            hashes = rec.get("kernel_source_sha256_by_kind", {kernel_kind(rec.get("kernel", "")):
                                                               rec.get("kernel_source_sha256")})
            if "fetch_bytes" in v and kinds.get(int(T)) == kind and hashes.get(kind) == kernel_source_hash(kind):
                per.setdefault(int(T), v["fetch_bytes"] + v["write_bytes"])
    if any(T not in per for T in TS):
        return None
    return sum(per[T] for T in TS) / len(TS)


class Workload:
    """The generated layers, plans, outputs and per-launch records of one layer shape."""

    def __init__(self, name, TS, n_layers, seed, dev):
        import torch
        from paper_2609_04244_amd import monomoe as mm
        from paper_2609_04244_amd import workloads as wl
        self.name, self.TS = name, TS
        self.cfg = cfg = wl.config(name)
        self.H, self.E, self.I, self.k, self.renorm = cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"]
        self.n = n_layers or layers_needed(cfg, TS, wl.expected_unique_experts)
        print("bench: generating %d layers of %s" % (self.n, name), file=sys.stderr, flush=True)
        self.layers = [wl.generate(cfg, T=max(TS), seed=seed + 1000 * l, device=dev) for l in range(self.n)]
        self.plans = {T: mm.Plan(T, self.H, self.E, self.I, self.k, self.renorm) for T in TS}
        self.outs = {T: torch.empty((T, self.H), dtype=torch.bfloat16, device=dev) for T in TS}
        self.xs = {(l, T): self.layers[l]["x"][:T].contiguous() for l in range(self.n) for T in TS}
        # one rotation per workload over all of its launches, so that consecutive launches (of
        # any T) read different weight sets
        self.next_layer = 0
        self.records = {T: [] for T in TS}   # (layer, timer, timed?)
        self.graph_ms = {T: [] for T in TS}
        self.U = {}

    def route(self, T, L):   # the layer's routing inputs (logit bias; sigmoid selection bias)
        from paper_2609_04244_amd import monomoe as mm
        p = self.plans[T]
        if L["bias"] is not None:
            p.set_router_bias(L["bias"])
        if L["policy"] == "sigmoid_bias":
            p.set_routing(mm.ROUTING_SIGMOID_BIAS, L["sel_bias"], L["route_scale"])

    def args(self, l, T):
        L = self.layers[l]
        return (self.xs[(l, T)], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"])

    def select(self):
        """Unique experts of every (layer, T), from the operator's own selection (untimed)."""
        import torch
        from paper_2609_04244_amd import monomoe as mm
        for l in range(self.n):
            for T in self.TS:
                self.route(T, self.layers[l])
                _, d = self.plans[T].forward_debug(*self.args(l, T))
                torch.cuda.synchronize()
                self.U[(l, T)] = len(set(d["ids"].cpu().numpy().reshape(-1).tolist()))
        for T in self.TS:
            if self.plans[T].status() != mm.MONOMOE_OK:
                raise RuntimeError("%s: device status after the selection pass: %s"
                                   % (self.name, mm.status_string(self.plans[T].status())))

    def launch(self, T, timed):
        from paper_2609_04244_amd import monomoe as mm
        l = self.next_layer
        self.next_layer = (l + 1) % self.n
        self.route(T, self.layers[l])
        timer = mm.DispatchTimer()
        self.plans[T].forward_timed(*self.args(l, T), self.outs[T], timer)
        self.records[T].append((l, timer, timed))

    def capture_graphs(self):
        """One HIP graph per T holding a forward of every weight set in turn (as a decode step's
        graph holds the MoE layers of a model), so a replay is n consecutive operator launches."""
        import torch
        self.graphs = {}
        side = torch.cuda.Stream()
        for T in self.TS:
            for l in range(self.n):
                self.route(T, self.layers[l])
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    self.plans[T].forward(*self.args(l, T), out=self.outs[T])
                torch.cuda.current_stream().wait_stream(side)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for l in range(self.n):
                    self.route(T, self.layers[l])   # the routing inputs are read from the plan at capture
                    self.plans[T].forward(*self.args(l, T), out=self.outs[T], check=False)
            self.graphs[T] = g
        torch.cuda.synchronize()

    def replay(self, T, timed):
        """One replay of T's graph; with `timed`, events around it (the replay time over the
        graph's n launches is the per-launch figure)."""
        import torch
        if not timed:
            self.graphs[T].replay()
            return None
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        self.graphs[T].replay()
        b.record()
        return (a, b)

    def status_ok(self):
        from paper_2609_04244_amd import monomoe as mm
        for T in self.TS:
            st = self.plans[T].status()
            if st != mm.MONOMOE_OK:
                raise RuntimeError("%s: device status after timing: %s" % (self.name, mm.status_string(st)))

    def summary(self, steps):
        import numpy as np
        from paper_2609_04244_amd import workloads as wl
        H, E, I, k = self.H, self.E, self.I, self.k
        per_T = {}
        tot_bytes = tot_ms = 0.0
        for T in self.TS:
            ms, by, wb = [], [], []
            for l, timer, timed in self.records[T]:
                if not timed:
                    continue
                ms.append(timer.elapsed_ms())
                u = self.U[(l, T)]
                by.append(algorithmic_bytes(u, T, H, E, I))
                wb.append(u * 3 * H * I)
            ms = np.array(ms)
            by = np.array(by, dtype=np.float64)
            gbps = by.sum() / (ms.sum() * 1e-3) / 1e9
            e = {
                "us_mean": round(float(ms.mean() * 1e3), 2), "us_p50": round(float(np.median(ms) * 1e3), 2),
                "us_p10": round(float(np.percentile(ms, 10) * 1e3), 2),
                "us_p90": round(float(np.percentile(ms, 90) * 1e3), 2),
                "unique_experts_mean": round(float(np.mean([self.U[(l, T)] for l in range(self.n)])), 2),
                "unique_experts_uniform_estimate": round(wl.expected_unique_experts(E, k, T), 2),
                "GBps": round(float(gbps), 1), "frac_of_peak": round(float(gbps / PEAK_HBM_GBPS), 4),
                "expert_weight_GBps": round(float(np.sum(wb) / (ms.sum() * 1e-3) / 1e9), 1),
            }
            if self.graph_ms[T]:
                g = np.array(self.graph_ms[T])
                e["graph_replay_us_p50"] = round(float(np.median(g) * 1e3), 2)
                e["graph_replay_us_p10"] = round(float(np.percentile(g, 10) * 1e3), 2)
                e["graph_replay_us_p90"] = round(float(np.percentile(g, 90) * 1e3), 2)
            per_T[str(T)] = e
            tot_bytes += by.sum()
            tot_ms += ms.sum()
        value = tot_bytes / (tot_ms * 1e-3) / 1e9
        kinds = {T: "multi" if self.plans[T].info()["multi_tile"] else "single" for T in self.TS}
        traffic = measured_traffic(self.name, kinds, self.TS)
        cfg = self.cfg
        routing = ("sigmoid routing with selection bias" if cfg.get("policy") == "sigmoid_bias" else
                   ("renormalised" if self.renorm else "plain") + " softmax") + \
            (" + per-expert logit bias" if cfg.get("bias_std") else "")
        n_launch = steps * len(self.TS)
        return {
            "layer": "%s: H=%d E=%d I=%d top-%d %s, block-FP8 128x128 weights, T in %s, %d rotated weight sets" % (
                self.name, H, E, I, k, routing, list(self.TS), self.n),
            "weight_sets": self.n,
            "value_GBps": round(float(value), 1), "frac_of_peak": round(float(value / PEAK_HBM_GBPS), 4),
            "launch_us_mean": round(float(tot_ms / n_launch * 1e3), 2),
            "ms_per_step": round(float(self.ms_per_step), 4),
            "algorithmic_bytes_per_launch": round(float(tot_bytes / n_launch)),
            "traffic": None if traffic is None else round(float(traffic)),
            "kernel": ", ".join(sorted({"monomoe_fused%s<%d,%d>" % ("_mt" if self.plans[T].info()["multi_tile"] else "",
                                                                    H, I) for T in self.TS})),
            "per_T": per_T,
        }, value, tot_bytes, tot_ms

    def close(self):
        for p in self.plans.values():
            p.close()


def read_ceiling(dev, gib=2, reps=10):
    """Achievable HBM read rate of this device: monomoe_stream_read (each workgroup reads one
    contiguous chunk, sixteen 16-byte loads in flight per thread) over a fresh `gib` GiB
    buffer, event-timed; the median of `reps` launches after three warm-ups, in GB/s."""
    import torch
    from paper_2609_04244_amd import monomoe as mm
    n = gib << 30
    src = torch.ones(n, dtype=torch.uint8, device=dev)
    sink = torch.zeros(16, dtype=torch.uint8, device=dev)
    evs = []
    for r in range(3 + reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        mm.stream_read(src, sink, n)
        b.record()
        if r >= 3:
            evs.append((a, b))
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    del src
    torch.cuda.empty_cache()
    return n / (ms[len(ms) // 2] * 1e6)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this operator build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr, flush=True)
        sys.exit(2)

    import torch

    TS = tuple(int(t) for t in args.tokens.split(","))
    names = [args.workload] if args.workload else args.workloads.split(",")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wls = [Workload(n, TS, args.layers, args.seed, dev) for n in names]
    for w in wls:
        w.select()

    # dispatch-stamped kernel times, one layer after the other (the paper's isolated-operator
    # protocol: consecutive launches of one operator configuration).  Blocked order (default):
    # each (layer, T) runs warmup + steps consecutive launches, as the MoE layers of a decode
    # step at one batch size do; interleaved order: every step launches T = 1, 2, 4, 8 in turn.
    # A step is one launch per T either way.
    stream = torch.cuda.current_stream()
    wall = 0.0
    ms_per_step = 0.0
    blocks = [[T] for T in TS] if args.order == "blocked" else [list(TS)]
    for w in wls:
        w.ms_per_step = 0.0
        for blk in blocks:
            torch.cuda.synchronize()
            w_start = torch.cuda.Event(enable_timing=True)
            w_end = torch.cuda.Event(enable_timing=True)
            t_start = None
            for s in range(args.warmup + args.steps):
                if s == args.warmup:
                    torch.cuda.synchronize()
                    t_start = time.perf_counter()
                    w_start.record(stream)
                for T in blk:
                    w.launch(T, s >= args.warmup)
            w_end.record(stream)
            torch.cuda.synchronize()
            wall += time.perf_counter() - t_start
            w.ms_per_step += w_start.elapsed_time(w_end) / args.steps
        w.status_ok()
        ms_per_step += w.ms_per_step

    # graph replays, event-timed on the stream, same order and layer rotation
    if args.replays > 0:
        for w in wls:
            w.capture_graphs()
            pending = []
            reps = max(1, args.replays // w.n)   # graph replays of n launches each
            for blk in blocks:
                for r in range(5 + reps):
                    for T in blk:
                        ev = w.replay(T, r >= 5)
                        if ev is not None:
                            pending.append((T, ev))
            torch.cuda.synchronize()
            for T, (a, b) in pending:
                w.graph_ms[T].append(a.elapsed_time(b) / w.n)
            w.status_ok()

    ceiling = read_ceiling(dev)

    blocks = {}
    head = None
    for w in wls:
        blk, value, tot_bytes, tot_ms = w.summary(args.steps)
        blocks[w.name] = blk
        if head is None:
            head = (w, blk, value)
    w0, blk0, value = head
    res = {
        "metric": "routed-MoE op latency us + achieved HBM GB/s (% of peak) at T=" + ",".join(map(str, TS)) + " tokens",
        "value": round(float(value), 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(float(ms_per_step), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8_e4m3 operands (gate/up: exact fp16 MFMA, down: e4m3 MFMA), fp32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": blk0["layer"],
            "other_workloads": [b["layer"] for n, b in blocks.items() if n != w0.name],
            "launches_per_step": len(TS) * len(wls), "grid": w0.plans[TS[0]].info()["grid"],
            "block": w0.plans[TS[0]].info()["block"], "order": args.order,
            "step": "one forward per token count; each (layer, T) is timed over its own block of consecutive "
                    "launches (order %s); value, per_T and roofline are the headline layer's; ms_per_step sums "
                    "one launch of every T of every layer" % args.order,
        },
        "per_T": blk0["per_T"],
        "workloads": blocks,
        "roofline": {
            "bound": "hbm", "achieved": round(float(value), 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(float(value / PEAK_HBM_GBPS), 4),
            "traffic": blk0["traffic"],
            "traffic_unit": "HBM bytes per launch (read + write, mean over T)",
            "algorithmic_bytes_per_launch": blk0["algorithmic_bytes_per_launch"],
            "kernel": blk0["kernel"],
            "launch_us_mean": blk0["launch_us_mean"],
            "read_ceiling": round(float(ceiling), 1),
            "frac_of_read_ceiling": round(float(value / ceiling), 4),
            "read_ceiling_note": "achievable HBM read rate measured in the same run: monomoe_stream_read, "
                                 "2 GiB, per-workgroup contiguous chunks, median of 10",
        },
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(args, w0, TS)
    for w in wls:
        w.close()
    print(json.dumps(res), flush=True)


def cpu_info():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return model, os.cpu_count() or 1, avail


def cpu_baseline(args, w, TS):
    """The fp64 oracle on the host cores, on a bounded sample of the headline workload: the
    step's forwards (one per token count) on layer 0, timed on one core and with one token per
    thread over all available cores (the oracle's tokens are independent; the C oracle runs
    without the interpreter lock), each repeated while under the time budget.  Also checks the
    operator's outputs on those forwards against the oracle."""
    import numpy as np
    import torch
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle
    from paper_2609_04244_amd import workloads as wl

    H, E, I, k, renorm = w.H, w.E, w.I, w.k, w.renorm
    L = w.layers[0]
    rw = wl.bf16_bits(L["router_w"])
    bias = None if L["bias"] is None else L["bias"].cpu().numpy()
    sigmoid = L["policy"] == "sigmoid_bias"
    sel_bias = None if not sigmoid or L["sel_bias"] is None else L["sel_bias"].cpu().numpy()
    route = dict(policy=oracle.SIGMOID_BIAS, sel_bias=sel_bias, scale=L["route_scale"]) if sigmoid else {}
    xb = {T: wl.bf16_bits(w.xs[(0, T)]) for T in TS}
    logits = oracle.router_logits(xb[max(TS)], rw, bias)
    ids = (oracle.select_sigmoid(logits, k, sel_bias, L["route_scale"])[0] if sigmoid
           else oracle.select(logits, k, renorm)[0])
    ex = sorted(set(ids.reshape(-1).tolist()))
    idx = torch.tensor(ex, device=L["w13"].device)
    host = [t.index_select(0, idx).cpu().numpy() for t in (L["w13"], L["w13_scale"], L["w2"], L["w2_scale"])]
    tabs = [{e: a[i] for i, e in enumerate(ex)} for a in host]

    def one_token(T, t):
        return oracle.forward(xb[T][t:t + 1], rw, *tabs, k, renorm, bias=bias, **route)

    jobs = [(T, t) for T in TS for t in range(T)]
    # GPU outputs of the sample's forwards, checked against the oracle once
    worst = mre_worst = 0.0
    refs = {}
    for T, t in jobs:
        refs[(T, t)] = one_token(T, t)
    for T in TS:
        w.route(T, L)
        out = w.plans[T].forward(*w.args(0, T))
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().astype(np.float64)
        ref = np.concatenate([refs[(T, t)] for t in range(T)], axis=0)
        rms = float(np.sqrt(np.mean(ref ** 2)))
        worst = max(worst, float(np.abs(got - ref).max()) / rms)
        mre_worst = max(mre_worst, float(np.abs(got - ref).sum() / np.abs(ref).sum()))

    model, nproc, avail = cpu_info()
    threads = max(1, min(avail, 16))

    def timed(run):
        reps = 0
        t0 = time.perf_counter()
        while True:
            run()
            reps += 1
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        return (time.perf_counter() - t0) / reps, reps

    dt1, reps1 = timed(lambda: [one_token(T, t) for T, t in jobs])
    with ThreadPoolExecutor(max_workers=threads) as pool:
        dtn, repsn = timed(lambda: list(pool.map(lambda j: one_token(*j), jobs)))
    by0 = sum(algorithmic_bytes(w.U[(0, T)], T, H, E, I) for T in TS)
    return {
        "value": round(by0 / dtn / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
        "sample": "the headline layer's step on weight set 0: %d forwards (T=%s, %d tokens, %d selected experts "
                  "in total), one token per oracle call; %d repetition(s) on %d threads, %.3f s each; on one core "
                  "%d repetition(s), %.3f s each" % (len(TS), ",".join(map(str, TS)), len(jobs),
                                                      sum(w.U[(0, T)] for T in TS), repsn, threads, dtn, reps1, dt1),
        "single_core": {"value": round(by0 / dt1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                        "ms_per_step": round(dt1 * 1e3, 1)},
        "all_cores": {"value": round(by0 / dtn / 1e9, 4), "unit": "GB/s", "cores": threads,
                      "ms_per_step": round(dtn * 1e3, 1)},
        "cpu_model": model, "nproc": nproc, "cpus_available": avail,
        "gpu_vs_oracle_max_err_over_rms": round(worst, 5), "gpu_vs_oracle_mean_rel_err": round(mre_worst, 6),
    }


if __name__ == "__main__":
    main()
