"""Token-count sweep of the two kernels (the crossover study of more tokens than one tile).

For one workload and a list of token counts, times the single-tile kernel (token passes of
one tile beyond its tile) and the multi-tile kernel (one launch), each forced through
monomoe_plan_set_schedule, with dispatch-stamped events over layers rotated so every
launch streams its weights from HBM; reports the mean launch time per (kernel, T), the
speed-up, and the rate of unique expert-weight bytes (experts selected at least once per
launch, counted from the selection) for the multi-tile kernel.

Example:
  python3 -m paper_2609_04244_amd.crossover --workload coarse --T 1,8,16,32,64 --layers 2 \\
      --out profiles/crossover_coarse.md
"""
import argparse
import sys

import numpy as np
import torch

from . import monomoe as mm
from . import workloads as wl

KERNELS = (("single-tile", mm.KERNEL_SINGLE), ("multi-tile", mm.KERNEL_MULTI))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="coarse")
    ap.add_argument("--T", default="1,8,16,32,64")
    ap.add_argument("--layers", type=int, default=2)
    ap.add_argument("--iters", type=int, default=12)
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--out", default=None)
    ap.add_argument("--command", default=None, help="command text recorded in the summary")
    args = ap.parse_args(argv)
    Ts = [int(t) for t in args.T.split(",")]
    cfg = wl.config(args.workload)
    H, E, I, k = cfg["H"], cfg["E"], cfg["I"], cfg["k"]
    dev = "cuda:0"
    layers = [wl.generate(cfg, T=max(Ts), seed=100 + l, device=dev) for l in range(args.layers)]
    print("generated %d layers of %s" % (args.layers, args.workload), flush=True)
    expert_bytes = 3 * H * I + 3 * (H // 128) * (I // 128) * 4

    lat, info, unique = {}, {}, {}
    for rep in range(args.reps):
        for name, kernel in KERNELS:
            for T in Ts:
                plan = mm.Plan(T, H, E, I, k, cfg["renorm"])
                L0 = layers[0]
                if L0["bias"] is not None:
                    plan.set_router_bias(L0["bias"])
                if L0["policy"] == "sigmoid_bias":
                    plan.set_routing(mm.ROUTING_SIGMOID_BIAS, L0["sel_bias"], L0["route_scale"])
                plan.set_schedule(kernel=kernel)
                info[(name, T)] = plan.info()
                out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
                xs = [L["x"][:T].contiguous() for L in layers]
                if (T not in unique) and kernel == mm.KERNEL_MULTI:
                    cnt = []
                    for i, L in enumerate(layers):
                        _, d = plan.forward_debug(xs[i], L["router_w"], L["w13"], L["w13_scale"], L["w2"],
                                                  L["w2_scale"])
                        cnt.append(len(np.unique(d["ids"].cpu().numpy())))
                    unique[T] = float(np.mean(cnt))
                for i, L in enumerate(layers):   # warm-up
                    plan.forward(xs[i], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], out=out,
                                 check=False)
                timers = [mm.DispatchTimer() for _ in range(args.iters)]
                for i in range(args.iters):
                    l = i % len(layers)
                    L = layers[l]
                    plan.forward_timed(xs[l], L["router_w"], L["w13"], L["w13_scale"], L["w2"], L["w2_scale"], out,
                                       timers[i])
                torch.cuda.synchronize()
                st = plan.status()
                plan.close()
                if st != mm.MONOMOE_OK:
                    raise SystemExit("device status %s (%s, T=%d)" % (mm.status_string(st), name, T))
                lat.setdefault((name, T), []).append(float(np.mean([t.elapsed_ms() * 1e3 for t in timers])))
                print("%s T=%d %.1f us" % (name, T, lat[(name, T)][-1]), flush=True)
    best = {key: min(v) for key, v in lat.items()}

    lines = ["# Token-count sweep, single-tile vs multi-tile kernel: %s" % args.workload, ""]
    if args.command:
        lines += ["Command (from the repository root):", "", "```", args.command.strip(), "```", ""]
    lines += ["Shape H=%d E=%d I=%d k=%d. Mean of %d dispatch-stamped launches over %d rotated layers, best of "
              "%d repetitions. Unique expert bytes: experts selected at least once (mean over the layers) x "
              "%.1f MB of FP8 weights and scales." % (H, E, I, k, args.iters, args.layers, args.reps,
                                                      expert_bytes / 1e6), "",
              "| T | single-tile us (passes) | multi-tile us (R, slices) | speed-up | active experts | "
              "multi-tile unique-weight GB/s | % of 8 TB/s |",
              "|---|---|---|---|---|---|---|"]
    for T in Ts:
        s, m = best[("single-tile", T)], best[("multi-tile", T)]
        si, mi = info[("single-tile", T)], info[("multi-tile", T)]
        passes = -(-T // si["tokens_per_pass"])
        gbps = unique[T] * expert_bytes / (m * 1e-6) / 1e9
        lines.append("| %d | %.1f (%d) | %.1f (%d, %d) | %.2fx | %.1f | %.0f | %.1f |" %
                     (T, s, passes, m, mi["group_tokens"], mi["down_slices"], s / m, unique[T], gbps,
                      100.0 * gbps / 8000.0))
    text = "\n".join(lines) + "\n"
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
