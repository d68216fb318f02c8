"""ctypes binding of the C oracle (``monomoe_oracle.c``), numpy in / numpy out.

Test infrastructure only: see the package docstring.  Every function marshals arrays
and calls the C code; none of the operator's arithmetic lives here.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        L.mo_e4m3_decode.restype = ctypes.c_double
        L.mo_e4m3_decode.argtypes = [ctypes.c_uint8]
        L.mo_e4m3_encode.restype = ctypes.c_uint8
        L.mo_e4m3_encode.argtypes = [ctypes.c_float]
        L.mo_bf16_decode.restype = ctypes.c_double
        L.mo_bf16_decode.argtypes = [ctypes.c_uint16]
        L.mo_quantize_group.restype = None
        L.mo_quantize_group.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        L.mo_router_logits.restype = None
        L.mo_router_logits.argtypes = [ctypes.c_int] * 3 + [ctypes.c_void_p] * 4
        L.mo_select.restype = None
        L.mo_select.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p] * 3
        L.mo_forward.restype = ctypes.c_int
        L.mo_forward.argtypes = [ctypes.c_int] * 6 + [ctypes.c_void_p] * 11
        L.mo_select_sigmoid.restype = None
        L.mo_select_sigmoid.argtypes = [ctypes.c_int] * 3 + [ctypes.c_void_p] * 2 + [ctypes.c_double] + \
            [ctypes.c_void_p] * 2
        L.mo_forward_policy.restype = ctypes.c_int
        L.mo_forward_policy.argtypes = [ctypes.c_int] * 7 + [ctypes.c_void_p, ctypes.c_double] + [ctypes.c_void_p] * 11
        _lib = L
    return _lib


class _Debug(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("ids", "w", "xq", "xs", "h", "act", "aq", "as_", "y")]


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def e4m3_decode(code):
    return lib().mo_e4m3_decode(int(code))


def e4m3_encode(v):
    return lib().mo_e4m3_encode(float(np.float32(v)))


def bf16_decode(bits):
    return lib().mo_bf16_decode(int(bits))


def quantize_group(v):
    """v: fp32 vector -> (codes uint8, scale float32)."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    q = np.zeros(v.shape[0], dtype=np.uint8)
    s = np.zeros(1, dtype=np.float32)
    lib().mo_quantize_group(_p(v), v.shape[0], _p(q), _p(s))
    return q, s[0]


def router_logits(x_bf16, rw_bf16, bias=None):
    """x_bf16 uint16 [T,H], rw_bf16 uint16 [E,H], bias float32 [E] -> float64 [T,E]."""
    x = np.ascontiguousarray(x_bf16, dtype=np.uint16)
    rw = np.ascontiguousarray(rw_bf16, dtype=np.uint16)
    T, H = x.shape
    E = rw.shape[0]
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    out = np.zeros((T, E), dtype=np.float64)
    lib().mo_router_logits(T, H, E, _p(x), _p(rw), _p(b), _p(out))
    return out


def select(logits, k, renorm):
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = logits.shape
    ids = np.zeros((T, k), dtype=np.int32)
    w = np.zeros((T, k), dtype=np.float64)
    lib().mo_select(T, E, k, int(bool(renorm)), _p(logits), _p(ids), _p(w))
    return ids, w


SOFTMAX, SIGMOID_BIAS = 0, 1


def select_sigmoid(logits, k, sel_bias=None, scale=2.5):
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = logits.shape
    b = None if sel_bias is None else np.ascontiguousarray(sel_bias, dtype=np.float32)
    ids = np.zeros((T, k), dtype=np.int32)
    w = np.zeros((T, k), dtype=np.float64)
    lib().mo_select_sigmoid(T, E, k, _p(logits), _p(b), float(scale), _p(ids), _p(w))
    return ids, w


def forward(x_bf16, rw_bf16, w13, w13s, w2, w2s, k, renorm, bias=None, ids_in=None, w_in=None,
            debug=False, experts=None, policy=SOFTMAX, sel_bias=None, scale=1.0):
    """The whole operator.

    x_bf16 uint16 [T,H]; rw_bf16 uint16 [E,H]; w13 uint8 [E,2I,H] (or a dict expert ->
    [2I,H] array); w13s float32 [E,2I/128,H/128] (or dict); w2 / w2s likewise.
    policy SOFTMAX (renorm as given) or SIGMOID_BIAS (sel_bias float32 [E] or None, scale).
    Returns ref float64 [T,H] and, with debug=True, a dict of intermediates.
    """
    x = np.ascontiguousarray(x_bf16, dtype=np.uint16)
    rw = np.ascontiguousarray(rw_bf16, dtype=np.uint16)
    T, H = x.shape
    E = rw.shape[0]
    if isinstance(w13, dict):
        any_e = next(iter(w13))
        I = w13[any_e].shape[0] // 2
    else:
        I = w13.shape[1] // 2
    keep = []

    def table(src, dtype):
        arr = (ctypes.c_void_p * E)()
        for e in range(E):
            if isinstance(src, dict):
                if e not in src:
                    continue
                a = np.ascontiguousarray(src[e], dtype=dtype)
            else:
                a = np.ascontiguousarray(src[e], dtype=dtype)
            keep.append(a)
            arr[e] = a.ctypes.data
        return arr

    t13 = table(w13, np.uint8)
    t13s = table(w13s, np.float32)
    t2 = table(w2, np.uint8)
    t2s = table(w2s, np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    ii = None if ids_in is None else np.ascontiguousarray(ids_in, dtype=np.int32)
    wi = None if w_in is None else np.ascontiguousarray(w_in, dtype=np.float64)
    ref = np.zeros((T, H), dtype=np.float64)
    dbg = None
    d = None
    if debug:
        d = {
            "ids": np.zeros((T, k), np.int32), "w": np.zeros((T, k), np.float64),
            "xq": np.zeros((T, H), np.uint8), "xs": np.zeros((T, H // 128), np.float32),
            "h": np.zeros((T * k, 2 * I), np.float64), "act": np.zeros((T * k, I), np.float64),
            "aq": np.zeros((T * k, I), np.uint8), "as": np.zeros((T * k, I // 128), np.float32),
            "y": np.zeros((T * k, H), np.float64),
        }
        dbg = _Debug(_p(d["ids"]), _p(d["w"]), _p(d["xq"]), _p(d["xs"]), _p(d["h"]), _p(d["act"]),
                     _p(d["aq"]), _p(d["as"]), _p(d["y"]))
    sb = None if sel_bias is None else np.ascontiguousarray(sel_bias, dtype=np.float32)
    rc = lib().mo_forward_policy(T, H, E, I, k, int(bool(renorm)), int(policy), _p(sb), float(scale),
                          _p(x), _p(rw), _p(b),
                          ctypes.cast(t13, ctypes.c_void_p), ctypes.cast(t13s, ctypes.c_void_p),
                          ctypes.cast(t2, ctypes.c_void_p), ctypes.cast(t2s, ctypes.c_void_p),
                          _p(ii), _p(wi), _p(ref), ctypes.byref(dbg) if dbg is not None else None)
    if rc != 0:
        raise ValueError("oracle mo_forward rejected its arguments (rc=%d)" % rc)
    return (ref, d) if debug else ref
