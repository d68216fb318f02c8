"""Input files for profiling runs of the fused operator.

Hardware-counter runs profile a process that loads only the system HIP runtime and the
operator library (the C++ driver built from csrc/monomoe_profile.cpp), so the layers
are generated here beforehand and saved as raw little-endian binaries:

  generate:  draw `--layers` synthetic layers of a workload on the GPU and save
             DIR/l<l>_<field>.bin plus DIR/meta.txt ("H E I k renorm layers tmax has_bias");
  run:       the same launches from Python through the ctypes binding (no profiler needed);
  bench:     summarise a --kernel-trace --stats run of bench.py itself: the headline layer's
             timed launches per token count against bench.py's own event timing;
  timeline:  per-workgroup phase stamps of cold-cache launches (median and slowest
             workgroup per phase) beside the dispatch-stamped launch time;
  compare:   two summarize records of one workload side by side (launch time and counters);
  summarize: turn the CSV output of one --kernel-trace run and two --pmc runs (FETCH_SIZE,
             WRITE_SIZE) of the C++ driver into a markdown summary and a JSON record: mean
             launch duration per token count, HBM bytes per launch from the counters scaled by
             what they read for the driver's plain copy kernel of known size, and the hash of
             the kernel sources the counters belong to.

Example:
  python3 -m paper_2609_04244_amd.profile_layer generate --workload small_expert --dir /tmp/moe
  rocprofv3 --kernel-trace --stats -d out -- paper_2609_04244_amd/monomoe_profile /tmp/moe 1,8 16 1024
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import sys

import numpy as np

FIELDS = ("x", "router_w", "bias", "w13", "w13_scale", "w2", "w2_scale")


def generate(args):
    import torch
    from . import workloads as wl
    cfg = wl.config(args.workload)
    os.makedirs(args.dir, exist_ok=True)
    for l in range(args.layers):
        inp = wl.generate(cfg, T=args.tmax, seed=args.seed + 1000 * l, device="cuda:0")
        for f in FIELDS:
            t = inp[f]
            if t is None:
                continue
            a = t.detach().cpu()
            a = a.view(torch.int16).numpy().view(np.uint16) if a.dtype == torch.bfloat16 else a.numpy()
            np.ascontiguousarray(a).tofile(os.path.join(args.dir, "l%d_%s.bin" % (l, f)))
    meta = {k: cfg[k] for k in ("H", "E", "I", "k", "renorm")}
    meta.update(layers=args.layers, tmax=args.tmax, workload=args.workload, has_bias=cfg.get("bias_std") is not None)
    with open(os.path.join(args.dir, "meta.json"), "w") as fh:
        json.dump(meta, fh)
    with open(os.path.join(args.dir, "meta.txt"), "w") as fh:
        fh.write("%d %d %d %d %d %d %d %d\n" % (cfg["H"], cfg["E"], cfg["I"], cfg["k"], int(cfg["renorm"]),
                                               args.layers, args.tmax, int(meta["has_bias"])))
    print("saved %d layers of %s to %s" % (args.layers, args.workload, args.dir), flush=True)


def run(args):
    import torch
    from . import monomoe as mm
    with open(os.path.join(args.dir, "meta.json")) as fh:
        meta = json.load(fh)
    dev = torch.device("cuda:0")
    H, E, I, tmax = meta["H"], meta["E"], meta["I"], meta["tmax"]
    shapes = {"x": ((tmax, H), np.uint16), "router_w": ((E, H), np.uint16), "bias": ((E,), np.float32),
              "w13": ((E, 2 * I, H), np.uint8), "w13_scale": ((E, 2 * I // 128, H // 128), np.float32),
              "w2": ((E, H, I), np.uint8), "w2_scale": ((E, H // 128, I // 128), np.float32)}
    layers = []
    for l in range(meta["layers"]):
        L = {}
        for f in FIELDS:
            path = os.path.join(args.dir, "l%d_%s.bin" % (l, f))
            if not os.path.exists(path):
                L[f] = None
                continue
            shape, dt = shapes[f]
            a = np.fromfile(path, dtype=dt).reshape(shape)
            if f in ("x", "router_w"):
                L[f] = torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
            else:
                L[f] = torch.from_numpy(a).to(dev)
        layers.append(L)
    Ts = [int(t) for t in args.T.split(",")]
    for T in Ts:
        plan = mm.Plan(T, meta["H"], meta["E"], meta["I"], meta["k"], meta["renorm"])
        out = torch.empty((T, meta["H"]), dtype=torch.bfloat16, device=dev)
        xs = [L["x"][:T].contiguous() for L in layers]
        for i in range(args.iters):
            l = i % len(layers)
            L = layers[l]
            if L["bias"] is not None:
                plan.set_router_bias(L["bias"])
            plan.forward(xs[l], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], out=out, check=False)
        torch.cuda.synchronize()
        st = plan.status()
        plan.close()
        print("T=%d: %d launches, device status %s" % (T, args.iters, mm.status_string(st)), flush=True)
        if st != mm.MONOMOE_OK:
            sys.exit(1)
    if args.copy_mib:
        n = args.copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        sink = torch.empty(16, dtype=torch.uint8, device=dev)
        for _ in range(3):
            mm.stream_copy(dst, src, n)
        for _ in range(3):
            mm.stream_read(src, sink, n)
        torch.cuda.synchronize()
        print("reference copy and read kernels: %d MiB each, 3 launches" % args.copy_mib, flush=True)


# sources of each kernel (counters and traces are only valid for this code)
KERNEL_SOURCES = {
    "single": ("csrc/monomoe_kernel.hip", "csrc/monomoe_kernel_one.hip", "csrc/monomoe_fused.h",
               "csrc/monomoe_device.h", "csrc/monomoe_internal.h", "csrc/monomoe_partition.h"),
    "multi": ("csrc/monomoe_kernel_mt.hip", "csrc/monomoe_device.h", "csrc/monomoe_internal.h",
              "csrc/monomoe_partition.h"),
}


def kernel_kind(kernel_name):
    """'multi' for the multi-tile kernel's symbol, else 'single'."""
    return "multi" if "monomoe_fused_mt" in kernel_name else "single"


def kernel_source_hash(kind="single", root=None):
    """sha256 over one kernel's sources in this package, or over those of them that exist in
    the package directory `root` of another checkout (an older one may have fewer files)."""
    h = hashlib.sha256()
    here = root or os.path.dirname(os.path.abspath(__file__))
    for f in KERNEL_SOURCES[kind]:
        if root and not os.path.exists(os.path.join(here, f)):
            continue
        with open(os.path.join(here, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _rows(path):
    files = glob.glob(os.path.join(path, "**", "*.csv"), recursive=True) if os.path.isdir(path) else [path]
    return files


def _find(path, suffix):
    for f in _rows(path):
        if f.endswith(suffix):
            return f
    raise FileNotFoundError("no *%s under %s" % (suffix, path))


def _counter_by_dispatch(path, name):
    """{dispatch_id: (kernel_name, value)} for counter `name` (summed over rows)."""
    out = {}
    with open(_find(path, "counter_collection.csv")) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != name:
                continue
            d = int(r["Dispatch_Id"])
            k, v = out.get(d, (r["Kernel_Name"], 0.0))
            out[d] = (k, v + float(r["Counter_Value"]))
    return out


def summarize(args):
    Ts = [int(t) for t in args.T.split(",")]
    n = args.iters
    # kernel trace: durations of the fused launches in dispatch order
    with open(_find(args.trace, "kernel_trace.csv")) as fh:
        tr = [r for r in csv.DictReader(fh)]
    tr.sort(key=lambda r: int(r["Dispatch_Id"]))
    fused = [r for r in tr if "monomoe_fused" in r["Kernel_Name"]]
    copies = [r for r in tr if "stream_copy" in r["Kernel_Name"]]
    reads = [r for r in tr if "stream_read" in r["Kernel_Name"]]
    if len(fused) != n * len(Ts):
        raise SystemExit("expected %d fused launches in the trace, found %d" % (n * len(Ts), len(fused)))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3   # us
    per_T, names = {}, []
    for i, T in enumerate(Ts):
        rs = fused[i * n:(i + 1) * n]
        if len({r["Kernel_Name"] for r in rs}) != 1:
            raise SystemExit("T=%d: launches of more than one kernel" % T)
        d = [dur(r) for r in rs]
        per_T[T] = {"launches": n, "us_mean": sum(d) / n, "us_min": min(d), "us_max": max(d),
                    "kernel": rs[0]["Kernel_Name"]}
        names += [rs[0]["Kernel_Name"]] if rs[0]["Kernel_Name"] not in names else []
    # the kernel of the largest T names the record; a plan's forwards of one token may run
    # another one (the one-token specialisation), named per T
    kname = per_T[Ts[-1]]["kernel"]
    nbytes = args.copy_mib << 20
    copy_us = min(dur(r) for r in copies) if copies else None
    read_us = min(dur(r) for r in reads) if reads else None
    rec = {
        "kernel": kname, "workload": args.workload, "token_counts": Ts, "launches_per_T": n,
        "kernel_source_sha256": kernel_source_hash(kernel_kind(kname), args.sources),
        "kernel_source_sha256_by_kind": {k: kernel_source_hash(k, args.sources)
                                         for k in sorted({kernel_kind(m) for m in names})},
        "per_T": {},
        "copy_kernel": {"bytes_each_way": nbytes, "us_min": copy_us,
                        "GBps_read_plus_write": (2 * nbytes / copy_us / 1e3) if copy_us else None},
        "read_kernel": {"bytes": nbytes, "us_min": read_us,
                        "GBps": (nbytes / read_us / 1e3) if read_us else None},
    }
    if args.fetch and args.write:
        fetch = _counter_by_dispatch(args.fetch, "FETCH_SIZE")
        write = _counter_by_dispatch(args.write, "WRITE_SIZE")
        for name, tab in (("fetch", fetch), ("write", write)):
            ids = sorted(tab)
            f_ids = [d for d in ids if "monomoe_fused" in tab[d][0]]
            c_ids = [d for d in ids if "stream_copy" in tab[d][0]]
            if len(f_ids) != n * len(Ts) or not c_ids:
                raise SystemExit("%s pass: expected %d fused dispatches and the copy kernel" % (name, n * len(Ts)))
            copy_kib = sum(tab[d][1] for d in c_ids) / len(c_ids)
            factor = nbytes / (copy_kib * 1024.0)   # true bytes per counted byte
            rec[name + "_calibration"] = {"copy_counter_KiB": copy_kib, "expected_KiB": nbytes / 1024.0,
                                          "factor": factor}
            for i, T in enumerate(Ts):
                v = [tab[d][1] for d in f_ids[i * n:(i + 1) * n]]
                kib = sum(v) / n
                rec["per_T"].setdefault(str(T), {})[name + "_KiB_raw"] = kib
                rec["per_T"][str(T)][name + "_bytes"] = kib * 1024.0 * factor
    if args.mfma:
        busy = _counter_by_dispatch(args.mfma, "SQ_VALU_MFMA_BUSY_CYCLES")
        gui = _counter_by_dispatch(args.mfma, "GRBM_GUI_ACTIVE")
        f_ids = [d for d in sorted(busy) if "monomoe_fused" in busy[d][0]]
        if len(f_ids) == n * len(Ts):
            for i, T in enumerate(Ts):
                ids = f_ids[i * n:(i + 1) * n]
                b = sum(busy[d][1] for d in ids) / n
                g = sum(gui[d][1] for d in ids) / n
                # GRBM_GUI_ACTIVE sums the XCDs' clocks; SQ_VALU_MFMA_BUSY_CYCLES sums the CUs
                rec["per_T"].setdefault(str(T), {}).update(
                    {"mfma_busy_cycles": b, "gui_active_cycles": g,
                     "mfma_busy_frac": b / (g / args.xcds * args.cus) if g > 0 else None})
    extra = []   # counter names of the --pmc runs, in order
    for d in args.pmc:
        with open(_find(d, "counter_collection.csv")) as fh:
            names = sorted({r["Counter_Name"] for r in csv.DictReader(fh)})
        for name in names:
            tab = _counter_by_dispatch(d, name)
            f_ids = [i for i in sorted(tab) if "monomoe_fused" in tab[i][0]]
            if len(f_ids) != n * len(Ts):
                raise SystemExit("%s: expected %d fused dispatches, found %d" % (name, n * len(Ts), len(f_ids)))
            extra.append(name)
            for i, T in enumerate(Ts):
                v = [tab[k][1] for k in f_ids[i * n:(i + 1) * n]]
                rec["per_T"].setdefault(str(T), {}).setdefault("counters", {})[name] = sum(v) / n
    for T in Ts:
        rec["per_T"].setdefault(str(T), {}).update(per_T[T])
    stats = [f for f in _rows(args.trace) if f.endswith("kernel_stats.csv")]
    if stats:
        with open(stats[0]) as fh:
            rec["kernel_stats"] = [r for r in csv.DictReader(fh)]
    os.makedirs(os.path.dirname(os.path.abspath(args.out_json)), exist_ok=True)
    with open(args.out_json, "w") as fh:
        json.dump(rec, fh, indent=1)
    short = lambda m: m.split("(")[0].replace("void ", "")
    lines = ["# %s on the %s workload" % (", ".join(short(m) for m in names), args.workload), "",
             "Command (from the repository root; DIR and OUT are scratch directories):", "", "```",
             args.command.strip(), "```", "",
             "Kernel source sha256: " + ", ".join("%s `%s`" % (k, h) for k, h in
                                                  rec["kernel_source_sha256_by_kind"].items()), "",
             "| T | kernel | launches | mean us | min us | max us | HBM read (calibrated) | HBM write (calibrated) "
             "| HBM GB/s (read+write / mean) | % of 8 TB/s |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for T in Ts:
        q = rec["per_T"][str(T)]
        rd = "%.1f MB" % (q["fetch_bytes"] / 1e6) if "fetch_bytes" in q else "-"
        wr = "%.2f MB" % (q["write_bytes"] / 1e6) if "write_bytes" in q else "-"
        bw, frac = "-", "-"
        if "fetch_bytes" in q and "write_bytes" in q:
            g = (q["fetch_bytes"] + q["write_bytes"]) / (q["us_mean"] * 1e-6) / 1e9
            bw, frac = "%.0f" % g, "%.1f" % (100.0 * g / 8000.0)
        lines.append("| %d | %s | %d | %.2f | %.2f | %.2f | %s | %s | %s | %s |" %
                     (T, short(q["kernel"]).replace("monomoe::", ""), n, q["us_mean"], q["us_min"], q["us_max"],
                      rd, wr, bw, frac))
    lines.append("")
    if copy_us:
        lines.append("Plain copy kernel, %d MiB each way: %.1f us (%.0f GB/s read+write)." %
                     (args.copy_mib, copy_us, rec["copy_kernel"]["GBps_read_plus_write"]))
    if read_us:
        lines.append("Plain read kernel, %d MiB: %.1f us (%.0f GB/s)." % (args.copy_mib, read_us, rec["read_kernel"]["GBps"]))
    for name in ("fetch", "write"):
        c = rec.get(name + "_calibration")
        if c:
            lines.append("%s counter on the copy kernel: %.0f KiB for %.0f KiB moved (factor %.4f)." %
                         ("FETCH_SIZE" if name == "fetch" else "WRITE_SIZE", c["copy_counter_KiB"], c["expected_KiB"],
                          c["factor"]))
    if any("mfma_busy_frac" in rec["per_T"][str(T)] for T in Ts):
        lines.append("MFMA busy per CU (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / %d XCDs x %d CUs)): %s." % (
            args.xcds, args.cus, ", ".join("T=%d %.1f%%" % (T, 100 * rec["per_T"][str(T)]["mfma_busy_frac"]) for T in Ts
                                if rec["per_T"][str(T)].get("mfma_busy_frac") is not None)))
    if extra:
        lines += ["", "Further counters, mean per launch (rocprofv3 sums them over the device):", "",
                  "| counter | " + " | ".join("T=%d" % T for T in Ts) + " |",
                  "|---|" + "---|" * len(Ts)]
        for name in extra:
            lines.append("| %s | " % name + " | ".join("%.4g" % rec["per_T"][str(T)]["counters"][name] for T in Ts)
                         + " |")
    if rec.get("kernel_stats"):
        lines += ["", "rocprofv3 --stats (all launches of the run):", "",
                  "| kernel | calls | average ns | min ns | max ns |", "|---|---|---|---|---|"]
        for r in rec["kernel_stats"]:
            lines.append("| %s | %s | %s | %s | %s |" % (r.get("Name", "")[:60], r.get("Calls", ""),
                         r.get("AverageNs", ""), r.get("MinNs", ""), r.get("MaxNs", "")))
    with open(args.out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def bench_trace(args):
    """The headline layer's timed launches in a kernel trace of bench.py, per token count,
    beside bench.py's own dispatch-stamped times of the same launches.  The trace holds, in
    dispatch order, every layer's selection pass (one forward per weight set and T), then the
    headline layer's warm-up and timed launches per T in blocked order; the other layers'
    launches and the graph replays come after."""
    with open(_find(args.trace, "kernel_trace.csv")) as fh:
        tr = [r for r in csv.DictReader(fh) if "monomoe_fused" in r["Kernel_Name"]]
    tr.sort(key=lambda r: int(r["Dispatch_Id"]))
    with open(args.bench_json) as fh:
        b = json.loads(fh.read().strip().splitlines()[-1])
    head = next(iter(b["workloads"].values()))
    Ts = [int(t) for t in b["per_T"]]
    steps, warmup, n = b["steps"], b["warmup"], head["weight_sets"]
    if b["config"].get("order", "blocked") != "blocked":
        raise SystemExit("the trace summary reads bench.py's blocked launch order")
    H, I = (int(v) for v in head["kernel"].split("<")[1].rstrip(">").split(","))
    sel = sum(w["weight_sets"] for w in b["workloads"].values()) * len(Ts)   # every layer's selection pass
    per_T, names = {}, []
    for i, T in enumerate(Ts):
        start = sel + i * (warmup + steps) + warmup
        rs = tr[start:start + steps]
        if len(rs) != steps or any("<%d, %d," % (H, I) not in r["Kernel_Name"] for r in rs):
            raise SystemExit("T=%d: the trace does not hold the headline layer's timed launches where "
                             "bench.py's launch order puts them" % T)
        d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rs]
        per_T[T] = sum(d) / len(d)
        names += [rs[0]["Kernel_Name"]] if rs[0]["Kernel_Name"] not in names else []
    kinds = sorted({kernel_kind(m) for m in names})
    short = lambda m: m.split("(")[0].replace("void ", "").replace("monomoe::", "")
    lines = ["# bench.py under rocprofv3 --kernel-trace --stats", "",
             "Command (from the repository root; OUT is a scratch directory):", "", "```", args.command.strip(), "```", "",
             "Kernel source sha256: " + ", ".join("%s `%s`" % (k, kernel_source_hash(k)) for k in kinds), "",
             "Headline layer: %s." % head["layer"], "",
             "Fused-kernel launches in the trace: %d (selection pass, warm-up, timed launches of every layer, graph "
             "replays); per T the headline layer's %d timed launches sit after the selection passes (%d launches) "
             "and, per T, %d warm-up launches." % (len(tr), steps, sel, warmup), ""]
    un = None
    if args.untraced_json:
        with open(args.untraced_json) as fh:
            un = json.loads(fh.read().strip().splitlines()[-1])
    lines += ["| T | kernel | trace mean us | bench.py events, traced run, us | bench.py events, untraced run, us |",
              "|---|---|---|---|---|"]
    for i, T in enumerate(Ts):
        start = sel + i * (warmup + steps) + warmup
        lines.append("| %d | %s | %.2f | %.2f | %s |" % (
            T, short(tr[start]["Kernel_Name"]), per_T[T], b["per_T"][str(T)]["us_mean"],
            "%.2f" % un["per_T"][str(T)]["us_mean"] if un else "-"))
    mean = sum(per_T.values()) / len(per_T)
    lines.append("| mean | | %.2f | %.2f | %s |" % (mean, b["roofline"]["launch_us_mean"],
                                                   "%.2f" % un["roofline"]["launch_us_mean"] if un else "-"))
    lines += ["", "(Under the tracer the event stamps include its own per-dispatch work; without it the "
              "dispatch-stamped events and the kernel trace agree.)", ""]

    def line(r):
        return "value %.1f GB/s (%.1f%% of 8 TB/s); per T: %s" % (
            r["value"], 100 * r["roofline"]["frac"],
            ", ".join("T=%s %.2f us" % (k, v["us_mean"]) for k, v in r["per_T"].items()))
    lines.append("bench.py line under the tracer: %s." % line(b))
    if un:
        lines += ["", "bench.py line without the tracer: %s." % line(un)]
    stats = [f for f in _rows(args.trace) if f.endswith("kernel_stats.csv")]
    if stats:
        with open(stats[0]) as fh:
            rows = [r for r in csv.DictReader(fh)]
        lines += ["", "rocprofv3 --stats (every launch of the process, the fused kernels first):", "",
                  "| kernel | calls | average ns | min ns | max ns |", "|---|---|---|---|---|"]
        rows.sort(key=lambda r: "monomoe_fused" not in r.get("Name", ""))
        for r in rows[:10]:
            lines.append("| %s | %s | %s | %s | %s |" % (short(r.get("Name", ""))[:60], r.get("Calls", ""),
                         r.get("AverageNs", ""), r.get("MinNs", ""), r.get("MaxNs", "")))
    with open(args.out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def compare(args):
    """Two summarize records of one workload side by side: mean launch time and every
    counter both hold, per token count both hold, with the relative change."""
    recs = []
    for path in (args.before, args.after):
        with open(path) as fh:
            recs.append(json.load(fh))
    a, b = recs
    Ts = [T for T in a["per_T"] if T in b["per_T"]]
    names = [n for n in a["per_T"][Ts[0]].get("counters", {}) if n in b["per_T"][Ts[0]].get("counters", {})]
    short = lambda m: m.split("(")[0].replace("void ", "").replace("monomoe::", "")
    lines = ["# %s: %s against %s" % (a["workload"], args.label_after, args.label_before), "",
             "Commands (from the repository root):", "", "```", args.command.strip(), "```", ""]
    for label, r in ((args.label_before, a), (args.label_after, b)):
        lines.append("- %s: kernel source sha256 %s." % (label, ", ".join(
            "%s `%s`" % kv for kv in r.get("kernel_source_sha256_by_kind",
                                           {kernel_kind(r["kernel"]): r["kernel_source_sha256"]}).items())))
    lines += ["", "Mean per launch (rocprofv3 sums counters over the device); change = after / before - 1.", ""]
    if args.note:
        lines += [args.note, ""]
    for T in Ts:
        qa, qb = a["per_T"][T], b["per_T"][T]
        lines += ["## T=%s" % T, "",
                  "| quantity | %s | %s | change |" % (args.label_before, args.label_after), "|---|---|---|---|",
                  "| kernel | %s | %s | |" % (short(qa.get("kernel", a["kernel"])), short(qb.get("kernel", b["kernel"]))),
                  "| launch us (kernel trace mean) | %.2f | %.2f | %+.1f%% |" % (
                      qa["us_mean"], qb["us_mean"], 100 * (qb["us_mean"] / qa["us_mean"] - 1))]
        for n in names:
            va, vb = qa["counters"][n], qb["counters"][n]
            lines.append("| %s | %.4g | %.4g | %s |" % (n, va, vb, "%+.1f%%" % (100 * (vb / va - 1)) if va else "-"))
        lines.append("")
    text = "\n".join(lines)
    with open(args.out_md, "w") as fh:
        fh.write(text)
    print(text)


# Phase stamps of the kernels (the kSt* indices of csrc/monomoe_internal.h), in the order
# the phases happen; the label says which wavefront stamps it.
STAMPS = [
    (11, "router rows stored"),
    (12, "input quantised (LDS)"),
    (15, "all logits of token 0 seen (wave 0)"),
    (16, "token 0 selected (wave 0)"),
    (13, "top-k done (barrier passed; one-token kernel: last expert ranked)"),
    (19, "expert token masks built"),
    (3, "routing metadata built"),
    (17, "work partition found (wave 0)"),
    (18, "first task addresses (wave 0)"),
    (1, "weight ring filled (wave 0)"),
    (2, "first weights used (wave 0)"),
    (9, "first partial tile handed off (wave 0)"),
    (4, "gate/up stream done (wave 0)"),
    (5, "gate/up epilogues stored (helper)"),
    (6, "first down activation requantised (helper)"),
    (10, "down stream done (wave 0)"),
    (7, "down epilogues stored (helper)"),
    (14, "output chunks reduced"),
    (8, "exit"),
]


def timeline(args):
    """Per-workgroup phase stamps of cold-cache launches: for every phase, the median and
    the slowest workgroup's time since the first workgroup started (medians over launches),
    next to the dispatch-stamped launch time."""
    import torch
    from . import monomoe as mm
    from . import workloads as wl
    dev = torch.device("cuda:0")
    Ts = [int(t) for t in args.T.split(",")]
    cfg = wl.config(args.workload)
    inp = wl.generate(cfg, T=max(Ts), seed=args.seed, device=dev)
    flush_src = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev)
    sink = torch.empty(16, dtype=torch.uint8, device=dev)
    cols = {}
    for T in Ts:
        plan = mm.Plan(T, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
        if inp["bias"] is not None:
            plan.set_router_bias(inp["bias"])
        if inp["policy"] == "sigmoid_bias":
            plan.set_routing(mm.ROUTING_SIGMOID_BIAS, inp["sel_bias"], inp["route_scale"])
        G = plan.info()["grid"]
        x = inp["x"][:T].contiguous()
        out = torch.empty((T, inp["H"]), dtype=torch.bfloat16, device=dev)
        w = (x, inp["router_w"], inp["w13"], inp["w13_scale"], inp["w2"], inp["w2_scale"])
        stamps = torch.zeros((G, 24), dtype=torch.int64, device=dev)
        per_phase = {i: ([], []) for i, _ in STAMPS}
        launch_us, timed_us = [], []
        timer = mm.DispatchTimer()
        for it in range(args.warmup + args.iters):
            mm.stream_read(flush_src, sink)            # evict the weights: a cold-cache launch
            plan.forward_timed(*w, out, timer)
            mm.stream_read(flush_src, sink)
            stamps.zero_()
            plan.forward_stamped(*w, out, stamps)
            torch.cuda.synchronize()
            if it < args.warmup:
                continue
            timed_us.append(timer.elapsed_ms() * 1e3)
            s = stamps.cpu().numpy().astype(np.int64)
            t0 = s[:, 0].min()
            launch_us.append((s[:, 8].max() - t0) / 100.0)
            for i, _ in STAMPS:
                v = s[:, i]
                v = v[v > 0]
                if len(v):
                    per_phase[i][0].append(float(np.median(v - t0)) / 100.0)
                    per_phase[i][1].append(float(np.max(v - t0)) / 100.0)
        if plan.status() != mm.MONOMOE_OK:
            raise SystemExit("device status %s at T=%d" % (mm.status_string(plan.status()), T))
        plan.close()
        cols[T] = dict(launch=float(np.median(launch_us)), timed=float(np.median(timed_us)),
                       phases={i: (float(np.median(a)), float(np.median(b))) if a else None
                               for i, (a, b) in per_phase.items()})
        print("T=%d: %d launches, stamped first entry to last exit %.2f us, untraced launch %.2f us"
              % (T, args.iters, cols[T]["launch"], cols[T]["timed"]), flush=True)
    lines = ["# Phase timeline: %s" % args.workload, ""]
    if args.command:
        lines += ["Command: `%s`" % args.command, ""]
    lines += ["Per-workgroup phase stamps (s_memrealtime, 10 ns) of %d cold-cache launches per T (a %d MiB "
              "streaming read before each), in us since the first workgroup started: median workgroup / "
              "slowest workgroup, medians over the launches. Stamps come from the stamps-only debug forward; "
              "the untraced launch time is the dispatch-stamped duration of the same launch without stamps."
              % (args.iters, args.flush_mib), ""]
    lines.append("| phase | " + " | ".join("T=%d" % T for T in Ts) + " |")
    lines.append("|---|" + "---|" * len(Ts))
    for i, label in STAMPS:
        cells = []
        for T in Ts:
            v = cols[T]["phases"][i]
            cells.append("—" if v is None else "%.2f / %.2f" % v)
        lines.append("| %s | %s |" % (label, " | ".join(cells)))
    lines.append("| first entry to last exit (stamped) | %s |" % " | ".join("%.2f" % cols[T]["launch"] for T in Ts))
    lines.append("| untraced launch (dispatch-stamped events) | %s |" % " | ".join("%.2f" % cols[T]["timed"] for T in Ts))
    text = "\n".join(lines) + "\n"
    if args.out_md:
        with open(args.out_md, "w") as fh:
            fh.write(text)
    print(text, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    g = sub.add_parser("generate")
    g.add_argument("--workload", default="small_expert")
    g.add_argument("--layers", type=int, default=4)
    g.add_argument("--tmax", type=int, default=8)
    g.add_argument("--seed", type=int, default=0)
    g.add_argument("--dir", required=True)
    r = sub.add_parser("run")
    r.add_argument("--dir", required=True)
    r.add_argument("--T", default="1,8")
    r.add_argument("--iters", type=int, default=16)
    r.add_argument("--copy-mib", type=int, default=0)
    m = sub.add_parser("summarize")
    m.add_argument("--trace", required=True, help="output directory of the --kernel-trace run")
    m.add_argument("--fetch", help="output directory of the --pmc FETCH_SIZE run")
    m.add_argument("--write", help="output directory of the --pmc WRITE_SIZE run")
    m.add_argument("--mfma", help="output directory of a --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE run")
    m.add_argument("--pmc", action="append", default=[],
                   help="output directory of any further --pmc run: every counter it holds is reported "
                        "as a mean per fused launch (repeatable)")
    m.add_argument("--cus", type=int, default=256)
    m.add_argument("--xcds", type=int, default=8)
    m.add_argument("--T", default="1,2,4,8")
    m.add_argument("--iters", type=int, required=True)
    m.add_argument("--copy-mib", type=int, default=1024)
    m.add_argument("--workload", default="small_expert")
    m.add_argument("--command", default="", help="the command lines that produced the runs")
    m.add_argument("--out-md", required=True)
    m.add_argument("--out-json", required=True)
    m.add_argument("--sources", help="package directory whose kernel sources the runs were built from "
                                     "(default: this package)")
    c = sub.add_parser("compare")
    c.add_argument("--before", required=True, help="summarize record (JSON)")
    c.add_argument("--after", required=True, help="summarize record (JSON)")
    c.add_argument("--label-before", default="before")
    c.add_argument("--label-after", default="after")
    c.add_argument("--command", default="")
    c.add_argument("--note", default="", help="a paragraph printed above the tables")
    c.add_argument("--out-md", required=True)
    bt = sub.add_parser("bench")
    bt.add_argument("--trace", required=True)
    bt.add_argument("--bench-json", required=True, help="bench.py's output line")
    bt.add_argument("--untraced-json", help="bench.py's output line from a run without the tracer")
    bt.add_argument("--command", default="")
    bt.add_argument("--out-md", required=True)
    tl = sub.add_parser("timeline")
    tl.add_argument("--workload", default="small_expert")
    tl.add_argument("--T", default="1,8")
    tl.add_argument("--iters", type=int, default=20)
    tl.add_argument("--warmup", type=int, default=3)
    tl.add_argument("--seed", type=int, default=0)
    tl.add_argument("--flush-mib", type=int, default=1024)
    tl.add_argument("--command", default="")
    tl.add_argument("--out-md")
    args = ap.parse_args()
    if args.cmd == "timeline":
        timeline(args)
    elif args.cmd == "bench":
        bench_trace(args)
    elif args.cmd == "compare":
        compare(args)
    elif args.cmd == "generate":
        generate(args)
    elif args.cmd == "run":
        run(args)
    else:
        summarize(args)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    main()
