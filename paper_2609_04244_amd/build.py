"""Build the HIP kernels + C ABI for gfx950 with hipcc, in-tree:

  * ``libmonomoe.so``: the product library;
  * ``libmonomoe_perturb.so``: the race-perturbation build, the same sources compiled with
    MONOMOE_RACE_PERTURB (a pseudo-random pause at every hand-off point of the kernels,
    taken when monomoe_forward_debug's jitter_seed is nonzero), for the robustness tests;
  * ``monomoe_profile``: the torch-free driver the counter profiles run.

Each source is compiled to an object of its own (under ``_build/``, all jobs of both
libraries in parallel), then linked.  Flags: -O3; -munsafe-fp-atomics so fp32 atomic adds
use the hardware instruction; packed fp32 arithmetic disabled (-packed-fp32-ops target
feature); no fast-math (the quantiser needs IEEE division).
"""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libmonomoe.so")
LIB_PERTURB = os.path.join(HERE, "libmonomoe_perturb.so")
SOURCES = ["monomoe_kernel.hip", "monomoe_kernel_one.hip", "monomoe_kernel_mt.hip", "monomoe_api.hip",
           "monomoe_stream.hip", "monomoe_schedule.hip"]
ARCH = "gfx950"
LIBRARIES = {LIB: [], LIB_PERTURB: ["-DMONOMOE_RACE_PERTURB"]}   # library -> extra defines


def _hipcc():
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
            "-munsafe-fp-atomics", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-command-line-argument", "-I", os.path.join(os.path.dirname(HERE), "include")]


def library_commands(lib):
    """(compile commands, link command) of one library."""
    objdir = os.path.join(BUILD_DIR, os.path.splitext(os.path.basename(lib))[0])
    objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    compiles = [[_hipcc()] + _flags() + LIBRARIES[lib] + ["-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
    link = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", lib] + objs
    return compiles, link


PROFILER = os.path.join(HERE, "monomoe_profile")


def profiler_command():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return [_hipcc(), "--offload-arch=" + ARCH, "-O2", "-std=c++17", "-Wno-unused-command-line-argument",
            os.path.join(CSRC, "monomoe_profile.cpp"), "-L" + HERE, "-l:libmonomoe.so",
            "-L" + os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath,$ORIGIN", "-o", PROFILER]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout)


def _jobs():
    n = int(os.environ.get("MAX_JOBS", "0") or 0) or (os.cpu_count() or 1)
    return max(1, min(n, 16))


def build(verbose=False):
    plans = {lib: library_commands(lib) for lib in LIBRARIES}
    for compiles, _ in plans.values():
        for c in compiles:
            os.makedirs(os.path.dirname(c[-1]), exist_ok=True)
    with ThreadPoolExecutor(max_workers=_jobs()) as pool:
        list(pool.map(lambda c: _run(c, verbose), [c for compiles, _ in plans.values() for c in compiles]))
    for _, link in plans.values():
        _run(link, verbose)
    _run(profiler_command(), verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
