"""Thin ctypes binding of ``libmonomoe.so`` (the C ABI declared in include/monomoe.h).

Argument marshalling only: tensors are passed as device pointers and the current torch
stream as the ``hipStream_t``; every step of the operator runs in the HIP kernel.  There
is no fallback: if the library is missing this module raises.
"""
import ctypes
import os

import torch  # loads torch's HIP runtime first, so the library binds to the same one

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmonomoe.so")
# the race-perturbation build: the same sources with a pseudo-random pause at every hand-off
# point, taken when monomoe_forward_debug's jitter_seed is nonzero (test use only)
LIB_PERTURB_PATH = os.path.join(_HERE, "libmonomoe_perturb.so")

MONOMOE_OK = 0
MONOMOE_ERR_INVALID = -1
MONOMOE_ERR_UNSUPPORTED = -2
MONOMOE_ERR_OCCUPANCY = -3
MONOMOE_ERR_HIP = -4
MONOMOE_ERR_TIMEOUT = -5
ROUTING_SOFTMAX = 0
ROUTING_SIGMOID_BIAS = 1
KERNEL_AUTO = 0
KERNEL_SINGLE = 1
KERNEL_MULTI = 2

# Every symbol include/monomoe.h declares.
EXPORTS = (
    "monomoe_plan", "monomoe_plan_destroy", "monomoe_plan_set_router_bias", "monomoe_plan_set_routing",
    "monomoe_plan_set_schedule", "monomoe_layout", "monomoe_schedule_check",
    "monomoe_forward", "monomoe_forward_tokens", "monomoe_forward_noalloc",
    "monomoe_forward_debug", "monomoe_forward_timed", "monomoe_plan_status", "monomoe_plan_reset", "monomoe_plan_info",
    "monomoe_supported_shape", "monomoe_status_string", "monomoe_stream_copy", "monomoe_stream_read",
)


class MonoMoEError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__("%s failed: %s (%d)" % (what, status_string(code), code))


class Shape(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("E", ctypes.c_int32), ("I", ctypes.c_int32)]


class Debug(ctypes.Structure):
    _fields_ = [
        ("topk_ids", ctypes.c_void_p), ("topk_w", ctypes.c_void_p), ("xq", ctypes.c_void_p),
        ("xs", ctypes.c_void_p), ("act", ctypes.c_void_p), ("aq", ctypes.c_void_p), ("as_", ctypes.c_void_p),
        ("out_f32", ctypes.c_void_p), ("topk_ids_in", ctypes.c_void_p), ("topk_w_in", ctypes.c_void_p),
        ("stamps", ctypes.c_void_p), ("spin_limit_ticks", ctypes.c_uint64), ("fail_flag", ctypes.c_int32),
        ("jitter_seed", ctypes.c_uint32),
    ]


class PlanInfo(ctypes.Structure):
    _fields_ = [("grid", ctypes.c_int32), ("block", ctypes.c_int32), ("lds_bytes", ctypes.c_int32),
                ("occupancy", ctypes.c_int32), ("num_cus", ctypes.c_int32), ("workspace_bytes", ctypes.c_int64),
                ("scratch_bytes", ctypes.c_int32), ("ring", ctypes.c_int32), ("tokens_per_pass", ctypes.c_int32),
                ("multi_tile", ctypes.c_int32), ("group_tokens", ctypes.c_int32), ("down_slices", ctypes.c_int32),
                ("up_block", ctypes.c_int32), ("down_grid", ctypes.c_int32)]


class Schedule(ctypes.Structure):
    _fields_ = [("grid", ctypes.c_int32), ("ring", ctypes.c_int32), ("kernel", ctypes.c_int32),
                ("group_tokens", ctypes.c_int32), ("general_only", ctypes.c_int32), ("up_block", ctypes.c_int32),
                ("down_grid", ctypes.c_int32)]


class ScheduleReport(ctypes.Structure):
    _fields_ = [("complete", ctypes.c_int32), ("violations", ctypes.c_int32), ("first_violation", ctypes.c_int32),
                ("active_experts", ctypes.c_int32), ("events", ctypes.c_int64), ("blocked_wg", ctypes.c_int32),
                ("blocked_wave", ctypes.c_int32), ("blocked_event", ctypes.c_int32), ("reserved", ctypes.c_int32)]


SCHEDULE_MUTATE_NO_SLOT_WAIT = 1
SCHEDULE_MUTATE_NO_ACT_WAIT = 2
SCHEDULE_MUTATE_PREFETCH_ONE_BUFFER = 4


class Layout(ctypes.Structure):
    _fields_ = [("tokens_per_pass", ctypes.c_int32), ("group_tokens", ctypes.c_int32),
                ("act_buffers", ctypes.c_int32), ("handoff_slots", ctypes.c_int32), ("lds_bytes", ctypes.c_int32)]


_libs = {}


def lib():
    """Load libmonomoe.so (built by __graft_entry__.build()); raise if it is missing."""
    return _load(LIB_PATH)


def lib_perturb():
    """Load libmonomoe_perturb.so, the race-perturbation build (test use only)."""
    return _load(LIB_PERTURB_PATH)


def _load(path):
    if path not in _libs:
        if not os.path.exists(path):
            raise RuntimeError("%s is not built; run __graft_entry__.build()" % path)
        # RTLD_LOCAL (ctypes' default): both builds can be loaded side by side
        L = ctypes.CDLL(path, mode=os.RTLD_LOCAL)
        vp = ctypes.c_void_p
        L.monomoe_plan.argtypes = [ctypes.POINTER(Shape), ctypes.c_int, ctypes.c_int, ctypes.POINTER(vp)]
        L.monomoe_plan.restype = ctypes.c_int
        L.monomoe_plan_destroy.argtypes = [vp]
        L.monomoe_plan_destroy.restype = None
        L.monomoe_plan_set_router_bias.argtypes = [vp, vp]
        L.monomoe_plan_set_router_bias.restype = ctypes.c_int
        L.monomoe_plan_set_routing.argtypes = [vp, ctypes.c_int, vp, ctypes.c_float]
        L.monomoe_plan_set_routing.restype = ctypes.c_int
        L.monomoe_plan_set_schedule.argtypes = [vp, ctypes.POINTER(Schedule)]
        L.monomoe_plan_set_schedule.restype = ctypes.c_int
        L.monomoe_layout.argtypes = [ctypes.POINTER(Shape)] + [ctypes.c_int] * 7 + [ctypes.POINTER(Layout)]
        L.monomoe_layout.restype = ctypes.c_int
        L.monomoe_schedule_check.argtypes = [ctypes.POINTER(Shape), ctypes.c_int, vp] + [ctypes.c_int] * 8 + \
            [ctypes.c_uint32, ctypes.c_uint32, ctypes.POINTER(ScheduleReport)]
        L.monomoe_schedule_check.restype = ctypes.c_int
        L.monomoe_forward.argtypes = [vp] * 9
        L.monomoe_forward.restype = ctypes.c_int
        L.monomoe_forward_tokens.argtypes = [vp, ctypes.c_int32] + [vp] * 8
        L.monomoe_forward_tokens.restype = ctypes.c_int
        L.monomoe_forward_noalloc.argtypes = [ctypes.POINTER(Shape), ctypes.c_int, ctypes.c_int] + [vp] * 10
        L.monomoe_forward_noalloc.restype = ctypes.c_int
        L.monomoe_forward_debug.argtypes = [vp] * 8 + [ctypes.POINTER(Debug), vp]
        L.monomoe_forward_debug.restype = ctypes.c_int
        L.monomoe_forward_timed.argtypes = [vp] * 11
        L.monomoe_forward_timed.restype = ctypes.c_int
        L.monomoe_plan_status.argtypes = [vp]
        L.monomoe_plan_status.restype = ctypes.c_int
        L.monomoe_plan_reset.argtypes = [vp]
        L.monomoe_plan_reset.restype = ctypes.c_int
        L.monomoe_plan_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
        L.monomoe_plan_info.restype = ctypes.c_int
        L.monomoe_supported_shape.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.monomoe_supported_shape.restype = ctypes.c_int
        L.monomoe_status_string.argtypes = [ctypes.c_int]
        L.monomoe_status_string.restype = ctypes.c_char_p
        L.monomoe_stream_copy.argtypes = [vp, vp, ctypes.c_size_t, vp]
        L.monomoe_stream_copy.restype = ctypes.c_int
        L.monomoe_stream_read.argtypes = [vp, ctypes.c_size_t, vp, vp]
        L.monomoe_stream_read.restype = ctypes.c_int
        _libs[path] = L
    return _libs[path]


def status_string(code):
    return lib().monomoe_status_string(int(code)).decode()


def layout(T, H, E, I, topk, kernel, lds_total, lds_static, occupancy, grid=0, num_cus=256):
    """monomoe_layout (host arithmetic, no device): (status code, layout dict or None)."""
    out = Layout()
    rc = lib().monomoe_layout(ctypes.byref(Shape(T, H, E, I)), topk, kernel, lds_total, lds_static, occupancy,
                              grid, num_cus, ctypes.byref(out))
    fields = {f: getattr(out, f) for f, _ in Layout._fields_}
    return rc, (fields if rc in (MONOMOE_OK, MONOMOE_ERR_OCCUPANCY) else None)


def schedule_check(ids, H, E, I, one_token, grid, ring, handoff_slots, act_buffers, resident=None, seed=0,
                   mutate=0, up_block=0, down_grid=0):
    """monomoe_schedule_check (host model of the single-tile kernel's hand-offs, no device) for
    the selection `ids` (int array [T, topk]): (status code, report dict or None)."""
    import numpy as np
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    T, k = ids.shape
    out = ScheduleReport()
    rc = lib().monomoe_schedule_check(ctypes.byref(Shape(T, H, E, I)), k, ids.ctypes.data_as(ctypes.c_void_p),
                                      int(one_token), int(grid), int(ring), int(up_block), int(down_grid),
                                      int(handoff_slots), int(act_buffers),
                                      int(grid if resident is None else resident), int(seed), int(mutate),
                                      ctypes.byref(out))
    return rc, ({f: getattr(out, f) for f, _ in ScheduleReport._fields_} if rc == MONOMOE_OK else None)


def supported_shape(H, I):
    return bool(lib().monomoe_supported_shape(int(H), int(I)))


def stream_copy(dst, src, nbytes=None, stream=None):
    """Reference copy kernel: dst[:nbytes] = src[:nbytes] (device tensors)."""
    n = int(src.numel() * src.element_size() if nbytes is None else nbytes)
    rc = lib().monomoe_stream_copy(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), n, _stream(stream))
    if rc != MONOMOE_OK:
        raise MonoMoEError(rc, "monomoe_stream_copy")


def stream_read(src, sink, nbytes=None, stream=None):
    """Reference read-only streaming kernel over src[:nbytes]; sink is a 16-byte device tensor."""
    n = int(src.numel() * src.element_size() if nbytes is None else nbytes)
    rc = lib().monomoe_stream_read(ctypes.c_void_p(src.data_ptr()), n, ctypes.c_void_p(sink.data_ptr()), _stream(stream))
    if rc != MONOMOE_OK:
        raise MonoMoEError(rc, "monomoe_stream_read")


def forward_noalloc(T, H, E, I, topk, renorm, x, router_w, w13, w13_scale, w2, w2_scale, out, bias=None,
                    status=None, stream=None):
    """monomoe_forward_noalloc: the operator without a plan (the library's static scratch as
    workspace).  out: bf16 [T,H] device tensor; status: int32 [1] device tensor or None."""
    rc = lib().monomoe_forward_noalloc(ctypes.byref(Shape(int(T), int(H), int(E), int(I))), int(topk), int(bool(renorm)),
                                       _ptr(bias), _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale), _ptr(w2),
                                       _ptr(w2_scale), _ptr(out), _ptr(status), _stream(stream))
    if rc != MONOMOE_OK:
        raise MonoMoEError(rc, "monomoe_forward_noalloc")
    return out


_hip = None


def _hip_runtime():
    """The HIP runtime already loaded by torch (events for monomoe_forward_timed)."""
    global _hip
    if _hip is None:
        import torch  # noqa: F401  (loads the runtime first)
        h = None
        for name in ("libamdhip64.so.7", "libamdhip64.so"):
            try:
                h = ctypes.CDLL(name)
                break
            except OSError:
                continue
        if h is None:
            raise RuntimeError("HIP runtime library not found")
        vp = ctypes.c_void_p
        h.hipEventCreate.argtypes = [ctypes.POINTER(vp)]
        h.hipEventCreate.restype = ctypes.c_int
        h.hipEventDestroy.argtypes = [vp]
        h.hipEventDestroy.restype = ctypes.c_int
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        h.hipEventElapsedTime.restype = ctypes.c_int
        _hip = h
    return _hip


class DispatchTimer:
    """A pair of HIP events that monomoe_forward_timed stamps with the kernel dispatch's own
    begin and end."""

    def __init__(self):
        h = _hip_runtime()
        self.start, self.stop = ctypes.c_void_p(), ctypes.c_void_p()
        if h.hipEventCreate(ctypes.byref(self.start)) or h.hipEventCreate(ctypes.byref(self.stop)):
            raise RuntimeError("hipEventCreate failed")

    def elapsed_ms(self):
        ms = ctypes.c_float()
        if _hip_runtime().hipEventElapsedTime(ctypes.byref(ms), self.start, self.stop):
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def __del__(self):
        try:
            h = _hip_runtime()
            h.hipEventDestroy(self.start)
            h.hipEventDestroy(self.stop)
        except Exception:
            pass


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Plan:
    """A plan for one shape (T, H, E, I) with top-k and renormalisation fixed."""

    def __init__(self, T, H, E, I, topk, renorm=True, perturb=False):
        """perturb: make the plan with the race-perturbation build of the library (its
        launches pause at hand-off points when forward_debug gets a nonzero jitter_seed)."""
        self.T, self.H, self.E, self.I, self.topk, self.renorm = int(T), int(H), int(E), int(I), int(topk), bool(renorm)
        self._L = lib_perturb() if perturb else lib()
        self._h = ctypes.c_void_p()
        self._bias = None
        rc = self._L.monomoe_plan(ctypes.byref(Shape(self.T, self.H, self.E, self.I)), self.topk, int(self.renorm),
                                ctypes.byref(self._h))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan")

    def close(self):
        if self._h:
            self._L.monomoe_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_router_bias(self, bias):
        self._bias = bias  # keep the tensor alive while the plan refers to it
        rc = self._L.monomoe_plan_set_router_bias(self._h, _ptr(bias))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan_set_router_bias")

    def set_routing(self, policy, sel_bias=None, scale=1.0):
        """ROUTING_SOFTMAX, or ROUTING_SIGMOID_BIAS with an fp32 [E] selection bias (or None)
        and the routed scaling factor."""
        rc = self._L.monomoe_plan_set_routing(self._h, int(policy), _ptr(sel_bias), float(scale))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan_set_routing")
        self._sel_bias = sel_bias  # keep the tensor alive while the plan refers to it

    def set_schedule(self, grid=0, ring=0, kernel=KERNEL_AUTO, group_tokens=0, general_only=0, up_block=0,
                     down_grid=0):
        """Persistent grid (0 = one workgroup per CU), weight-ring depth (0 = default), kernel
        (KERNEL_AUTO / KERNEL_SINGLE / KERNEL_MULTI), the multi-tile segment cap (0 = none),
        general_only (1: passes of one token on the general single-tile kernel, not its
        one-token specialisation), and the single-tile kernel's work partition: gate/up units
        per deal (up_block: 0 = 1, 2, 4, 8) and the workgroups with down units (down_grid:
        0 = the whole grid)."""
        sch = Schedule(int(grid), int(ring), int(kernel), int(group_tokens), int(general_only), int(up_block),
                       int(down_grid))
        rc = self._L.monomoe_plan_set_schedule(self._h, ctypes.byref(sch))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan_set_schedule")

    def info(self):
        inf = PlanInfo()
        rc = self._L.monomoe_plan_info(self._h, ctypes.byref(inf))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan_info")
        return {f: getattr(inf, f) for f, _ in PlanInfo._fields_}

    def _check(self, x, router_w, w13, w13_scale, w2, w2_scale, out):
        T, H, E, I = self.T, self.H, self.E, self.I
        want = [
            (x, (T, H), torch.bfloat16), (router_w, (E, H), torch.bfloat16),
            (w13, (E, 2 * I, H), torch.uint8), (w13_scale, (E, 2 * I // 128, H // 128), torch.float32),
            (w2, (E, H, I), torch.uint8), (w2_scale, (E, H // 128, I // 128), torch.float32),
            (out, (T, H), torch.bfloat16),
        ]
        for t, shape, dtype in want:
            if tuple(t.shape) != shape or t.dtype != dtype or not t.is_contiguous() or not t.is_cuda:
                raise ValueError("expected a contiguous device tensor %s of %s, got %s %s"
                                 % (shape, dtype, tuple(t.shape), t.dtype))

    def forward(self, x, router_w, w13, w13_scale, w2, w2_scale, out=None, stream=None, check=True):
        """Enqueue the fused operator; returns out (bf16 [T,H])."""
        if out is None:
            out = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=x.device)
        if check:
            self._check(x, router_w, w13, w13_scale, w2, w2_scale, out)
        rc = self._L.monomoe_forward(self._h, _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale), _ptr(w2),
                                   _ptr(w2_scale), _ptr(out), _stream(stream))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_forward")
        return out

    def forward_tokens(self, T, x, router_w, w13, w13_scale, w2, w2_scale, out=None, stream=None, check=True):
        """The operator on the first T tokens of the plan's bound (0 <= T <= plan T): x and out
        are [T,H]; no re-planning.  Returns out."""
        T = int(T)
        if out is None:
            out = torch.empty((T, self.H), dtype=torch.bfloat16, device=x.device)
        if check:
            if not 0 <= T <= self.T:
                raise ValueError("T=%d outside [0, %d]" % (T, self.T))
            saved = self.T
            self.T = T
            try:
                self._check(x, router_w, w13, w13_scale, w2, w2_scale, out)
            finally:
                self.T = saved
        rc = self._L.monomoe_forward_tokens(self._h, T, _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale),
                                          _ptr(w2), _ptr(w2_scale), _ptr(out), _stream(stream))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_forward_tokens")
        return out

    def forward_timed(self, x, router_w, w13, w13_scale, w2, w2_scale, out, timer, stream=None):
        """monomoe_forward whose dispatch stamps `timer` (a DispatchTimer) with its own begin/end."""
        rc = self._L.monomoe_forward_timed(self._h, _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale), _ptr(w2),
                                         _ptr(w2_scale), _ptr(out), timer.start, timer.stop, _stream(stream))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_forward_timed")
        return out

    def forward_debug(self, x, router_w, w13, w13_scale, w2, w2_scale, out=None, ids_in=None, w_in=None,
                      spin_limit_ticks=0, fail_flag=False, jitter_seed=0, stream=None):
        """Forward with every test hook enabled; returns (out, dict of device tensors).
        `jitter_seed` nonzero (<= 65535) perturbs the hand-off timing (race perturbation)."""
        T, H, I, k = self.T, self.H, self.I, self.topk
        dev = x.device
        if out is None:
            out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        self._check(x, router_w, w13, w13_scale, w2, w2_scale, out)
        d = {
            "ids": torch.full((T, k), -1, dtype=torch.int32, device=dev),
            "w": torch.zeros((T, k), dtype=torch.float32, device=dev),
            "xq": torch.zeros((T, H), dtype=torch.uint8, device=dev),
            "xs": torch.zeros((T, H // 128), dtype=torch.float32, device=dev),
            "act": torch.zeros((T * k, I), dtype=torch.float32, device=dev),
            "aq": torch.zeros((T * k, I), dtype=torch.uint8, device=dev),
            "as": torch.zeros((T * k, I // 128), dtype=torch.float32, device=dev),
            "out_f32": torch.zeros((T, H), dtype=torch.float32, device=dev),
            "stamps": torch.zeros((self.info()["grid"], 24), dtype=torch.int64, device=dev),
        }
        if (ids_in is None) != (w_in is None):
            raise ValueError("ids_in and w_in go together")
        if ids_in is not None:
            ids_in = ids_in.to(device=dev, dtype=torch.int32).contiguous()
            w_in = w_in.to(device=dev, dtype=torch.float32).contiguous()
        dbg = Debug(d["ids"].data_ptr(), d["w"].data_ptr(), d["xq"].data_ptr(), d["xs"].data_ptr(),
                    d["act"].data_ptr(), d["aq"].data_ptr(), d["as"].data_ptr(), d["out_f32"].data_ptr(),
                    ids_in.data_ptr() if ids_in is not None else None,
                    w_in.data_ptr() if w_in is not None else None,
                    d["stamps"].data_ptr(), int(spin_limit_ticks), int(bool(fail_flag)), int(jitter_seed))
        rc = self._L.monomoe_forward_debug(self._h, _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale), _ptr(w2),
                                         _ptr(w2_scale), _ptr(out), ctypes.byref(dbg), _stream(stream))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_forward_debug")
        d["_keep"] = (ids_in, w_in)
        return out, d

    def forward_stamped(self, x, router_w, w13, w13_scale, w2, w2_scale, out, stamps, stream=None):
        """Forward with only the phase-stamp hook enabled: `stamps` is an int64 device tensor
        [grid, 24] that receives each workgroup's s_memrealtime (100 MHz) stamps."""
        dbg = Debug(None, None, None, None, None, None, None, None, None, None, stamps.data_ptr(), 0, 0, 0)
        rc = self._L.monomoe_forward_debug(self._h, _ptr(x), _ptr(router_w), _ptr(w13), _ptr(w13_scale), _ptr(w2),
                                         _ptr(w2_scale), _ptr(out), ctypes.byref(dbg), _stream(stream))
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_forward_debug")
        return out

    def status(self):
        return self._L.monomoe_plan_status(self._h)

    def reset(self):
        rc = self._L.monomoe_plan_reset(self._h)
        if rc != MONOMOE_OK:
            raise MonoMoEError(rc, "monomoe_plan_reset")
