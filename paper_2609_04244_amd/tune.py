"""Schedule enumerator and offline tuner (paper Sec. 3.4: every shape's kernels are
precompiled for a set of schedules; candidates that fail numerical validation are
rejected and the rest ranked by latency over the target token-count range).

A schedule here is (kernel, grid, ring): the single-tile or multi-tile kernel, the
persistent workgroup count and the weight-ring depth (see monomoe_plan_set_schedule).  For
one workload and a list of token counts:

  1. enumerate kernel x grid x ring candidates (combinations the plan rejects are dropped:
     the multi-tile kernel has ring depth 2 only, grids must be resident);
  2. validation gate, against the default schedule's output on the same inputs (the default
     is what the parity tests check against the fp64 oracle), with the device status OK: a
     candidate that runs the same kernel must be bit-identical (grid and ring change when and
     where the work runs, never the arithmetic); one that runs the other kernel sums in
     another order and must be within the operator's output bound (max |diff| <= 2e-2 rms,
     mean relative difference <= 5e-3);
  3. rank the survivors by the sum over the token counts of the mean dispatch-stamped
     launch time, with layers rotated so every launch streams its weights from HBM.

Writes a markdown summary (the command, every candidate's per-T latency, the ranking).

Example:
  python3 -m paper_2609_04244_amd.tune --workload small_expert --T 1,2,4,8 \\
      --grids 0,192,128 --rings 2,4 --kernels single,multi \\
      --out profiles/schedule_tuning_small_expert.md
"""
import argparse
import sys

import numpy as np
import torch

from . import monomoe as mm
from . import workloads as wl


def run(plan, L, T, out):
    return plan.forward(L["x"][:T].contiguous(), L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"],
                        out=out, check=False)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="small_expert")
    ap.add_argument("--T", default="1,2,4,8")
    ap.add_argument("--grids", default="0,192,128", help="persistent grids (0 = one workgroup per CU)")
    ap.add_argument("--rings", default="2,4")
    ap.add_argument("--kernels", default="single", help="single, multi or both (comma-separated)")
    ap.add_argument("--layers", type=int, default=8)
    ap.add_argument("--iters", type=int, default=48)
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--out", default=None)
    ap.add_argument("--command", default=None, help="command text recorded in the summary")
    args = ap.parse_args(argv)
    Ts = [int(t) for t in args.T.split(",")]
    cfg = wl.config(args.workload)
    dev = "cuda:0"
    layers = [wl.generate(cfg, T=max(Ts), seed=500 + l, device=dev) for l in range(args.layers)]
    print("generated %d layers of %s" % (args.layers, args.workload), flush=True)

    def make_plan(T, L):
        plan = mm.Plan(T, cfg["H"], cfg["E"], cfg["I"], cfg["k"], cfg["renorm"])
        if L["bias"] is not None:
            plan.set_router_bias(L["bias"])
        if L["policy"] == "sigmoid_bias":
            plan.set_routing(mm.ROUTING_SIGMOID_BIAS, L["sel_bias"], L["route_scale"])
        return plan

    kmode = {"single": mm.KERNEL_SINGLE, "multi": mm.KERNEL_MULTI}
    probe = make_plan(Ts[0], layers[0])
    info = probe.info()
    probe.close()
    cands = []
    for kn in args.kernels.split(","):
        for g in (int(x) for x in args.grids.split(",")):
            for r in (int(x) for x in args.rings.split(",")):
                if kn == "multi" and r != 2:
                    continue   # the multi-tile kernel has ring depth 2 only
                cands.append((kn, g if g else info["num_cus"], r))

    # 1-2. enumeration and validation gate
    valid, rejected, defaults = [], {}, {}
    for T in Ts:
        plan = make_plan(T, layers[0])
        dinfo = plan.info()
        dk = "multi" if dinfo["multi_tile"] else "single"
        defaults[T] = (dk, dinfo["grid"], dinfo["ring"])
        out = torch.empty((T, cfg["H"]), dtype=torch.bfloat16, device=dev)
        ref = run(plan, layers[0], T, out).clone()
        reff = ref.float()
        rms = float(reff.pow(2).mean().sqrt())
        for c in cands:
            if c in rejected:
                continue
            try:
                plan.set_schedule(kernel=kmode[c[0]], grid=c[1], ring=c[2])
            except mm.MonoMoEError as e:
                rejected[c] = "not accepted: %s" % e
                continue
            o = run(plan, layers[0], T, out)
            torch.cuda.synchronize()
            if plan.status() != mm.MONOMOE_OK:
                rejected[c] = "device status %s at T=%d" % (mm.status_string(plan.status()), T)
                plan.reset()
            elif c[0] == dk:
                if not torch.equal(o.view(torch.int16), ref.view(torch.int16)):
                    rejected[c] = "output differs from the default schedule at T=%d" % T
            else:
                d = (o.float() - reff).abs()
                if float(d.max()) > 2e-2 * rms or float(d.sum() / reff.abs().sum()) > 5e-3:
                    rejected[c] = "output outside the bound of the default schedule's at T=%d" % T
        plan.close()
    valid = [c for c in cands if c not in rejected]
    print("candidates %d, valid %d" % (len(cands), len(valid)), flush=True)

    # 3. ranking by latency over the token-count range
    lat = {}
    for rep in range(args.reps):
        for T in Ts:
            plan = make_plan(T, layers[0])
            out = torch.empty((T, cfg["H"]), dtype=torch.bfloat16, device=dev)
            xs = [L["x"][:T].contiguous() for L in layers]
            for c in valid:
                plan.set_schedule(kernel=kmode[c[0]], grid=c[1], ring=c[2])
                for i in range(len(layers)):   # warm-up
                    L = layers[i]
                    plan.forward(xs[i], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], out=out,
                                 check=False)
                timers = [mm.DispatchTimer() for _ in range(args.iters)]
                for i in range(args.iters):
                    L = layers[i % len(layers)]
                    plan.forward_timed(xs[i % len(layers)], L["router_w"], L["w13"], L["w13_scale"], L["w2"],
                                       L["w2_scale"], out, timers[i])
                torch.cuda.synchronize()
                assert plan.status() == mm.MONOMOE_OK
                us = float(np.mean([t.elapsed_ms() * 1e3 for t in timers]))
                lat.setdefault((c, T), []).append(us)
            plan.close()
    best_us = {k: min(v) for k, v in lat.items()}
    ranked = sorted(valid, key=lambda c: sum(best_us[(c, T)] for T in Ts))

    lines = ["# Schedule tuning: %s" % args.workload, ""]
    if args.command:
        lines += ["Command (from the repository root):", "", "```", args.command.strip(), "```", ""]
    lines += ["Shape H=%d E=%d I=%d k=%d; %d CUs; default schedule per T (kernel, grid, ring): %s. Latency: "
              "mean of %d dispatch-stamped launches over %d rotated layers, best of %d repetitions." %
              (cfg["H"], cfg["E"], cfg["I"], cfg["k"], info["num_cus"],
               ", ".join("T=%d %s/%d/%d" % ((T,) + defaults[T]) for T in Ts), args.iters, args.layers, args.reps), "",
              "| rank | kernel | grid | ring | " + " | ".join("T=%d us" % T for T in Ts) + " | sum us |",
              "|---|---|---|---|" + "---|" * len(Ts) + "---|"]
    for i, c in enumerate(ranked):
        lines.append("| %d | %s | %d | %d | " % (i + 1, c[0], c[1], c[2]) +
                     " | ".join("%.2f%s" % (best_us[(c, T)], "*" if defaults[T] == c else "") for T in Ts) +
                     " | %.2f |" % sum(best_us[(c, T)] for T in Ts))
    for c, why in rejected.items():
        lines.append("| rejected | %s | %d | %d | %s |" % (c[0], c[1], c[2], why))
    best_T = {T: min(valid, key=lambda c: best_us[(c, T)]) for T in Ts} if valid else {}
    lines += ["", "(* = the default schedule at that T.)", "",
              "Best by sum: %s, grid %d, ring %d." % ranked[0] if ranked else "No valid schedule."]
    if best_T:
        lines.append("Best per T: " + ", ".join("T=%d %s/%d/%d" % ((T,) + best_T[T]) for T in Ts) + ".")
    text = "\n".join(lines) + "\n"
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
