"""Build ``libmonomoe.so`` (the HIP kernel + C ABI) for gfx950 with hipcc, in-tree.

Flags: -O3; -munsafe-fp-atomics so fp32 atomic adds use the hardware instruction;
packed fp32 arithmetic disabled (-packed-fp32-ops target feature); no fast-math (the
quantiser needs IEEE division).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmonomoe.so")
SOURCES = ["monomoe_kernel.hip", "monomoe_kernel_one.hip", "monomoe_kernel_mt.hip", "monomoe_api.hip",
           "monomoe_stream.hip"]
ARCH = "gfx950"


def command():
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return [hipcc, "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
            "-munsafe-fp-atomics", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-command-line-argument",
            "-I", os.path.join(os.path.dirname(HERE), "include"),
            "-o", LIB] + [os.path.join(CSRC, s) for s in SOURCES]


PROFILER = os.path.join(HERE, "monomoe_profile")


def profiler_command():
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return [hipcc, "--offload-arch=" + ARCH, "-O2", "-std=c++17", "-Wno-unused-command-line-argument",
            os.path.join(CSRC, "monomoe_profile.cpp"), "-L" + HERE, "-l:libmonomoe.so",
            "-L" + os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath,$ORIGIN", "-o", PROFILER]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout)


def build(verbose=False):
    _run(command(), verbose)
    _run(profiler_command(), verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
