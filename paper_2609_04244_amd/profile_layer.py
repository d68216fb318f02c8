"""Input files for profiling runs of the fused operator.

Hardware-counter runs profile a process that loads only the system HIP runtime and the
operator library (the C++ driver built from csrc/monomoe_profile.cpp), so the layers
are generated here beforehand and saved as raw little-endian binaries:

  generate: draw `--layers` synthetic layers of a workload on the GPU and save
            DIR/l<l>_<field>.bin plus DIR/meta.txt ("H E I k renorm layers tmax has_bias");
  run:      the same launches from Python through the ctypes binding (no profiler needed).

Example:
  python3 -m paper_2609_04244_amd.profile_layer generate --workload small_expert --dir /tmp/moe
  rocprofv3 --kernel-trace --stats -d out -- paper_2609_04244_amd/monomoe_profile /tmp/moe 1,8 16 1024
"""
import argparse
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
    args = ap.parse_args()
    if args.cmd == "generate":
        generate(args)
    else:
        run(args)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    main()
