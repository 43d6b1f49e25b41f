"""Thin ctypes binding of ``libooc.so`` (see ``include/ooc.h``).

The functions carry the C names and only marshal arguments; every step of the
training step runs inside the library.  ``Context`` wraps one ``ooc_ctx``.
Loading fails loudly when the library has not been built: there is no
fallback path.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libooc.so")

OK, E_INVALID, E_STATE, E_INFEASIBLE, E_HOST_OOM, E_DEVICE, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
INPUT, PARAM, STATE, OUTPUT, TEMP = 0, 1, 2, 3, 4
R, W, RW = 1, 2, 3
POLICY_CANCEL, POLICY_LITERAL = 0, 1
WAIT_OLDEST, WAIT_FURTHEST = 0, 1
LAYOUT_POOL, LAYOUT_BESTFIT = 0, 1
SWAPIN, ALLOC, CANCEL, WAIT_OUT, SWAPOUT, FREE = 0, 1, 2, 3, 4, 5
PRE, POST, END = 0, 1, 2
UNLIMITED = 2 ** 64 - 1

OPS = {
    "noop": 0, "linear_fwd": 1, "linear_bwd_w": 2, "linear_bwd_x": 3, "relu_fwd": 4,
    "relu_bwd": 5, "add": 6, "softmax_ce": 7, "sgd": 8, "conv_fwd": 9, "conv_bwd_w": 10,
    "conv_bwd_x": 11, "bn_fwd": 12, "bn_bwd": 13, "maxpool_fwd": 14, "maxpool_bwd": 15,
    "avgpool_fwd": 16, "avgpool_bwd": 17, "mix": 18, "embed_fwd": 19, "embed_bwd": 20,
    "layernorm_fwd": 21, "layernorm_bwd": 22, "gelu_fwd": 23, "gelu_bwd": 24,
    "attention_fwd": 25, "attention_bwd": 26, "concat_fwd": 27, "concat_bwd": 28,
    "upsample_fwd": 29, "upsample_bwd": 30, "acc": 31,
}

#: every symbol ``include/ooc.h`` declares
EXPORTS = [
    "ooc_create", "ooc_destroy", "ooc_last_error", "ooc_add_var", "ooc_add_fn", "ooc_set_budget",
    "ooc_set_window", "ooc_set_chunk", "ooc_set_policy", "ooc_build_schedule",
    "ooc_schedule_get", "ooc_schedule_windows", "ooc_incore_peak", "ooc_working_set_max",
    "ooc_plan_intervals", "ooc_plan_chunks", "ooc_prepare", "ooc_host_ptr", "ooc_upload",
    "ooc_download", "ooc_step", "ooc_get_stats", "ooc_fn_times", "ooc_link_probe",
    "ooc_timeline", "ooc_set_swapout_depth", "ooc_set_fixed_distance", "ooc_bestfit_extent",
    "ooc_set_wait_order", "ooc_set_host_limit", "ooc_wgrad_slices", "ooc_set_layout",
]


class ooc_op(ctypes.Structure):
    _fields_ = [("fn", ctypes.c_int32), ("phase", ctypes.c_uint8), ("kind", ctypes.c_uint8),
                ("reserved", ctypes.c_uint16), ("var", ctypes.c_int64), ("held", ctypes.c_uint64)]


class ooc_interval(ctypes.Structure):
    _fields_ = [("var", ctypes.c_int64), ("open", ctypes.c_int64), ("close", ctypes.c_int64),
                ("first_chunk", ctypes.c_int64), ("n_chunks", ctypes.c_int64)]


class ooc_span(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("fn", ctypes.c_int32), ("var", ctypes.c_int64),
                ("bytes", ctypes.c_uint64), ("start_ms", ctypes.c_double), ("ms", ctypes.c_double)]


class ooc_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "budget", "chunk", "peak_accounted", "pool_chunks", "pool_bytes", "max_chunks_used",
        "device_bytes_delta", "host_bytes", "sched_h2d_bytes", "sched_d2h_bytes", "h2d_bytes",
        "d2h_bytes", "n_intervals", "n_mappings")] + [(n, ctypes.c_double) for n in (
        "prepare_ms", "step_ms", "step_gpu_ms", "h2d_busy_ms", "d2h_busy_ms",
        "compute_busy_ms")] + [("incore", ctypes.c_int32), ("policy", ctypes.c_int32)] + [
        (n, ctypes.c_uint64) for n in ("spill_bytes", "staged_h2d_bytes", "staged_d2h_bytes")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class OocError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"ooc status {status}: {message}")
        self.status = status
        self.message = message


_lib = None


def load(path=LIB_PATH):
    """Loads libooc.so once; raises if it is missing (build it with ``build()`` first)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2010_14109_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(path)
    c = ctypes
    P = c.c_void_p
    sig = {
        "ooc_create": ([c.c_int32, c.POINTER(P)], c.c_int32),
        "ooc_destroy": ([P], None),
        "ooc_last_error": ([P], c.c_char_p),
        "ooc_add_var": ([P, c.c_uint64, c.c_int32, c.POINTER(c.c_int64)], c.c_int32),
        "ooc_add_fn": ([P, c.c_int32, c.POINTER(c.c_int64), c.POINTER(c.c_uint8), c.c_int32,
                        c.POINTER(c.c_int64), c.c_int32, c.POINTER(c.c_int64)], c.c_int32),
        "ooc_set_budget": ([P, c.c_uint64], c.c_int32),
        "ooc_set_window": ([P, c.c_uint64], c.c_int32),
        "ooc_set_chunk": ([P, c.c_uint64], c.c_int32),
        "ooc_set_policy": ([P, c.c_int32], c.c_int32),
        "ooc_set_swapout_depth": ([P, c.c_int64], c.c_int32),
        "ooc_set_fixed_distance": ([P, c.c_int64, c.c_int64], c.c_int32),
        "ooc_set_wait_order": ([P, c.c_int32], c.c_int32),
        "ooc_set_host_limit": ([P, c.c_uint64], c.c_int32),
        "ooc_set_layout": ([P, c.c_int32], c.c_int32),
        "ooc_bestfit_extent": ([P, c.c_uint64, c.POINTER(c.c_uint64), c.POINTER(c.c_uint64)],
                               c.c_int32),
        "ooc_build_schedule": ([P], c.c_int32),
        "ooc_schedule_get": ([P, c.POINTER(ooc_op), c.c_uint64, c.POINTER(c.c_uint64)], c.c_int32),
        "ooc_schedule_windows": ([P, c.POINTER(c.c_int64), c.c_uint64, c.POINTER(c.c_uint64)],
                                 c.c_int32),
        "ooc_incore_peak": ([P, c.POINTER(c.c_uint64)], c.c_int32),
        "ooc_working_set_max": ([P, c.POINTER(c.c_uint64)], c.c_int32),
        "ooc_plan_intervals": ([P, c.POINTER(ooc_interval), c.c_uint64, c.POINTER(c.c_uint64)],
                               c.c_int32),
        "ooc_plan_chunks": ([P, c.POINTER(c.c_int32), c.c_uint64, c.POINTER(c.c_uint64)],
                            c.c_int32),
        "ooc_prepare": ([P], c.c_int32),
        "ooc_host_ptr": ([P, c.c_int64, c.POINTER(P)], c.c_int32),
        "ooc_upload": ([P], c.c_int32),
        "ooc_download": ([P], c.c_int32),
        "ooc_step": ([P, c.c_float, c.c_float, c.POINTER(c.c_float)], c.c_int32),
        "ooc_get_stats": ([P, c.POINTER(ooc_stats)], c.c_int32),
        "ooc_fn_times": ([P, c.POINTER(c.c_double), c.c_uint64, c.POINTER(c.c_uint64)],
                         c.c_int32),
        "ooc_link_probe": ([c.c_int32, c.c_uint64, c.c_int32, c.POINTER(c.c_double),
                            c.POINTER(c.c_double), c.POINTER(c.c_double)], c.c_int32),
        "ooc_timeline": ([P, c.POINTER(ooc_span), c.c_uint64, c.POINTER(c.c_uint64)], c.c_int32),
        "ooc_wgrad_slices": ([c.c_int32, c.POINTER(c.c_int64), c.c_int32, c.POINTER(c.c_int64)],
                             c.c_int32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _check(status, ctx=None):
    if status != OK:
        msg = load().ooc_last_error(ctx)
        raise OocError(status, msg.decode() if msg else "")
    return status


def link_probe(device=0, nbytes=1 << 30, reps=3):
    """Best host-to-device, device-to-host and bidirectional rates in GB/s."""
    lib = load()
    h, d, b = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib.ooc_link_probe(device, nbytes, reps, ctypes.byref(h), ctypes.byref(d),
                              ctypes.byref(b)), None)
    return {"h2d": h.value, "d2h": d.value, "both": b.value}


def wgrad_slices(op, attrs):
    """Split-K slice count of a weight-gradient function (``conv_bwd_w`` with its 11 shape
    attributes or ``linear_bwd_w`` with M, K, N), as the library's kernels want it."""
    lib = load()
    a = (ctypes.c_int64 * len(attrs))(*attrs)
    out = ctypes.c_int64()
    _check(lib.ooc_wgrad_slices(OPS[op] if isinstance(op, str) else op, a, len(attrs),
                                ctypes.byref(out)), None)
    return out.value


_NP = {"f32": np.float32, "i32": np.int32, "u8": np.uint8, "u32": np.uint32}


class Context:
    """One ``ooc_ctx``.  Methods mirror the C calls without the ``ooc_`` prefix."""

    def __init__(self, device=0):
        self.h = None
        lib = load()
        h = ctypes.c_void_p()
        _check(lib.ooc_create(device, ctypes.byref(h)), None)
        self.h = h
        self.lib = lib
        self.var_bytes = []

    def close(self):
        if self.h:
            self.lib.ooc_destroy(self.h)
            self.h = None

    __del__ = close

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def add_var(self, nbytes, kind):
        out = ctypes.c_int64()
        _check(self.lib.ooc_add_var(self.h, nbytes, kind, ctypes.byref(out)), self.h)
        self.var_bytes.append(nbytes)
        return out.value

    def add_fn(self, op, vars_, access, attrs=()):
        n = len(vars_)
        v = (ctypes.c_int64 * n)(*vars_)
        a = (ctypes.c_uint8 * n)(*access)
        at = (ctypes.c_int64 * max(1, len(attrs)))(*attrs)
        out = ctypes.c_int64()
        op = OPS[op] if isinstance(op, str) else op
        _check(self.lib.ooc_add_fn(self.h, op, v, a, n, at, len(attrs), ctypes.byref(out)), self.h)
        return out.value

    def set_budget(self, b):
        _check(self.lib.ooc_set_budget(self.h, b), self.h)

    def set_window(self, w):
        _check(self.lib.ooc_set_window(self.h, w), self.h)

    def set_chunk(self, c):
        _check(self.lib.ooc_set_chunk(self.h, c), self.h)

    def set_policy(self, p):
        _check(self.lib.ooc_set_policy(self.h, {"C": 0, "L": 1}.get(p, p)), self.h)

    def bestfit_extent(self, align=256):
        """(extent, peak_live) of a contiguous best-fit heap serving this schedule."""
        e, p = ctypes.c_uint64(), ctypes.c_uint64()
        _check(self.lib.ooc_bestfit_extent(self.h, align, ctypes.byref(e), ctypes.byref(p)),
               self.h)
        return e.value, p.value

    def set_wait_order(self, order):
        """``"oldest"`` / WAIT_OLDEST or ``"furthest"`` / WAIT_FURTHEST (see ooc_set_wait_order)."""
        order = {"oldest": WAIT_OLDEST, "furthest": WAIT_FURTHEST}.get(order, order)
        _check(self.lib.ooc_set_wait_order(self.h, order), self.h)

    def set_layout(self, layout):
        """``"pool"`` / LAYOUT_POOL or ``"bestfit"`` / LAYOUT_BESTFIT (see ooc_set_layout)."""
        layout = {"pool": LAYOUT_POOL, "bestfit": LAYOUT_BESTFIT}.get(layout, layout)
        _check(self.lib.ooc_set_layout(self.h, layout), self.h)

    def set_fixed_distance(self, swapin_ahead, swapout_threshold):
        _check(self.lib.ooc_set_fixed_distance(self.h, swapin_ahead, swapout_threshold), self.h)

    def set_host_limit(self, nbytes):
        """Most pinned host bytes for the arena (see ooc_set_host_limit)."""
        _check(self.lib.ooc_set_host_limit(self.h, nbytes), self.h)

    def set_swapout_depth(self, depth):
        _check(self.lib.ooc_set_swapout_depth(self.h, depth), self.h)

    def build_schedule(self):
        _check(self.lib.ooc_build_schedule(self.h), self.h)

    def schedule(self):
        """Op list as tuples (fn, phase, kind, var) and the held trace."""
        n = ctypes.c_uint64()
        _check(self.lib.ooc_schedule_get(self.h, None, 0, ctypes.byref(n)), self.h)
        buf = (ooc_op * max(1, n.value))()
        _check(self.lib.ooc_schedule_get(self.h, buf, n.value, ctypes.byref(n)), self.h)
        ops = [(o.fn, o.phase, o.kind, o.var) for o in buf[:n.value]]
        return ops, [o.held for o in buf[:n.value]]

    def windows(self):
        n = ctypes.c_uint64()
        _check(self.lib.ooc_schedule_windows(self.h, None, 0, ctypes.byref(n)), self.h)
        buf = (ctypes.c_int64 * max(1, n.value))()
        _check(self.lib.ooc_schedule_windows(self.h, buf, n.value, ctypes.byref(n)), self.h)
        return list(buf[:n.value])

    def incore_peak(self):
        out = ctypes.c_uint64()
        _check(self.lib.ooc_incore_peak(self.h, ctypes.byref(out)), self.h)
        return out.value

    def working_set_max(self):
        out = ctypes.c_uint64()
        _check(self.lib.ooc_working_set_max(self.h, ctypes.byref(out)), self.h)
        return out.value

    def plan(self):
        """Intervals as dicts {var, open, close, chunks}."""
        n = ctypes.c_uint64()
        _check(self.lib.ooc_plan_intervals(self.h, None, 0, ctypes.byref(n)), self.h)
        ivs = (ooc_interval * max(1, n.value))()
        _check(self.lib.ooc_plan_intervals(self.h, ivs, n.value, ctypes.byref(n)), self.h)
        m = ctypes.c_uint64()
        _check(self.lib.ooc_plan_chunks(self.h, None, 0, ctypes.byref(m)), self.h)
        cs = (ctypes.c_int32 * max(1, m.value))()
        _check(self.lib.ooc_plan_chunks(self.h, cs, m.value, ctypes.byref(m)), self.h)
        out = []
        for iv in ivs[:n.value]:
            out.append({"var": iv.var, "open": iv.open, "close": iv.close,
                        "chunks": list(cs[iv.first_chunk:iv.first_chunk + iv.n_chunks])})
        return out

    def plan_counts(self):
        """(physical chunks the pool needs, chunk mappings over all intervals)."""
        m = ctypes.c_uint64()
        _check(self.lib.ooc_plan_chunks(self.h, None, 0, ctypes.byref(m)), self.h)
        return self.stats()["max_chunks_used"], m.value

    def prepare(self):
        _check(self.lib.ooc_prepare(self.h), self.h)

    def host_ptr(self, var):
        p = ctypes.c_void_p()
        _check(self.lib.ooc_host_ptr(self.h, var, ctypes.byref(p)), self.h)
        return p.value

    def host_view(self, var, dtype="f32", shape=None):
        """NumPy view of a variable's pinned host slot (valid while the context lives)."""
        t = np.dtype(_NP.get(dtype, dtype))
        nbytes = self.var_bytes[var]
        buf = (ctypes.c_char * nbytes).from_address(self.host_ptr(var))
        arr = np.frombuffer(buf, dtype=t, count=nbytes // t.itemsize)
        return arr.reshape(shape) if shape is not None else arr

    def upload(self):
        _check(self.lib.ooc_upload(self.h), self.h)

    def download(self):
        _check(self.lib.ooc_download(self.h), self.h)

    def step(self, lr, momentum=0.0):
        loss = ctypes.c_float()
        _check(self.lib.ooc_step(self.h, lr, momentum, ctypes.byref(loss)), self.h)
        return loss.value

    def fn_times(self):
        """Per-function kernel milliseconds of the last step."""
        n = ctypes.c_uint64()
        _check(self.lib.ooc_fn_times(self.h, None, 0, ctypes.byref(n)), self.h)
        buf = (ctypes.c_double * max(1, n.value))()
        _check(self.lib.ooc_fn_times(self.h, buf, n.value, ctypes.byref(n)), self.h)
        return list(buf[:n.value])

    def timeline(self):
        """The last step's spans: (kind, fn, var, bytes, start_ms, ms), kind 0 kernels,
        1 swap-in, 2 swap-out."""
        n = ctypes.c_uint64()
        _check(self.lib.ooc_timeline(self.h, None, 0, ctypes.byref(n)), self.h)
        buf = (ooc_span * max(1, n.value))()
        _check(self.lib.ooc_timeline(self.h, buf, n.value, ctypes.byref(n)), self.h)
        return [(b.kind, b.fn, b.var, b.bytes, b.start_ms, b.ms) for b in buf[:n.value]]

    def stats(self):
        st = ooc_stats()
        _check(self.lib.ooc_get_stats(self.h, ctypes.byref(st)), self.h)
        return st.as_dict()
