"""The C-ABI library on the host: it loads, exports every entry point include/monomoe.h
declares, and rejects bad arguments before touching the GPU (no kernel is launched)."""
import ctypes
import os
import re

import pytest

from paper_2609_04244_amd import monomoe as mm

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "monomoe.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(monomoe_[a-z_]+)\s*\(", src)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(mm.EXPORTS)


@pytest.mark.parametrize("which", ["product", "perturbation"])
def test_library_loads_and_exports_every_declared_symbol(which):
    L = mm.lib() if which == "product" else mm.lib_perturb()
    for name in declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert mm.status_string(code) != "unknown status"
    assert mm.status_string(42) == "unknown status"


def test_supported_shapes():
    for H, I in ((256, 256), (2048, 768), (2048, 512), (7168, 2048), (4096, 14336), (7168, 256), (3072, 1024),
                 (6144, 256)):
        assert mm.supported_shape(H, I)
    assert not mm.supported_shape(2048, 1024)
    assert not mm.supported_shape(100, 256)


def _plan_rc(T, H, E, I, topk, renorm=1):
    h = ctypes.c_void_p()
    rc = mm.lib().monomoe_plan(ctypes.byref(mm.Shape(T, H, E, I)), topk, renorm, ctypes.byref(h))
    assert not h.value   # no plan handed out on failure
    return rc


@pytest.mark.parametrize("args,code", [
    ((1, 2048, 128, 700, 8), mm.MONOMOE_ERR_INVALID),       # I not a multiple of 128
    ((1, 2000, 128, 768, 8), mm.MONOMOE_ERR_INVALID),       # H not a multiple of 128
    ((1, 2048, 128, 768, 0), mm.MONOMOE_ERR_INVALID),       # topk < 1
    ((1, 2048, 4, 768, 5), mm.MONOMOE_ERR_INVALID),         # topk > E
    ((-1, 2048, 128, 768, 8), mm.MONOMOE_ERR_INVALID),      # negative T
    ((1, 2048, 0, 768, 1), mm.MONOMOE_ERR_INVALID),         # no experts
    ((65, 2048, 128, 768, 8), mm.MONOMOE_ERR_UNSUPPORTED),  # beyond 64 tokens per forward
    ((1, 2048, 600, 768, 8), mm.MONOMOE_ERR_UNSUPPORTED),   # E beyond 512
    ((1, 2048, 128, 768, 17), mm.MONOMOE_ERR_UNSUPPORTED),  # topk beyond 16
    ((1, 2048, 128, 1024, 8), mm.MONOMOE_ERR_UNSUPPORTED),  # (H, I) not compiled
])
def test_plan_rejects_bad_shapes_before_any_device_work(args, code):
    assert _plan_rc(*args) == code


def test_null_arguments():
    L = mm.lib()
    assert L.monomoe_plan(None, 1, 1, ctypes.byref(ctypes.c_void_p())) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_plan(ctypes.byref(mm.Shape(1, 256, 8, 256)), 2, 1, None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_forward(None, None, None, None, None, None, None, None, None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_forward_debug(None, None, None, None, None, None, None, None, None, None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_plan_set_router_bias(None, None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_plan_status(None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_plan_reset(None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_plan_info(None, None) == mm.MONOMOE_ERR_INVALID
    assert L.monomoe_layout(None, 8, 1, 163840, 8192, 1, 0, 256, None) == mm.MONOMOE_ERR_INVALID
    L.monomoe_plan_destroy(None)


def test_binding_structs_match_the_header_layout(tmp_path):
    # offsetof/sizeof of every field of the header's structs, from a C program compiled
    # against include/monomoe.h, against the ctypes layouts the binding passes
    if not os.path.isfile("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("HIP headers not installed")
    structs = [("monomoe_shape_t", mm.Shape), ("monomoe_debug_t", mm.Debug), ("monomoe_plan_info_t", mm.PlanInfo),
               ("monomoe_schedule_t", mm.Schedule), ("monomoe_layout_t", mm.Layout)]
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "monomoe.h"', "int main(void) {"]
    for cname, py in structs:
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in py._fields_:
            cf = "as" if f == "as_" else f
            lines.append('printf("%s.%s %%zu %%zu\\n", offsetof(%s, %s), sizeof(((%s*)0)->%s));'
                         % (cname, f, cname, cf, cname, cf))
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    import subprocess
    cc = subprocess.run(["gcc", "-std=c99", "-D__HIP_PLATFORM_AMD__", "-I", os.path.dirname(HEADER),
                         "-I", "/opt/rocm/include", "-o", str(exe), str(src)], capture_output=True, text=True)
    assert cc.returncode == 0, cc.stderr
    got = {}
    for line in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines():
        key, *vals = line.split()
        got[key] = tuple(int(v) for v in vals)
    for cname, py in structs:
        assert got[cname] == (ctypes.sizeof(py),), cname
        for f, _ in py._fields_:
            desc = getattr(py, f)
            assert got["%s.%s" % (cname, f)] == (desc.offset, desc.size), (cname, f)
