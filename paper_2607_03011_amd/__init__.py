"""IsoLoCo outer aggregation step on AMD MI355X (gfx950).

Thin ctypes binding of ``libisoloco.so`` (C ABI declared in
``include/isoloco.h``).  Every function below has the name and the argument
order of the C function it marshals; ``IsoLoCoPlan`` bundles them with a
torch-allocated workspace.  All arithmetic runs in the HIP kernels of the
library: if the library is missing, importing the binding raises.
"""
import ctypes
import os

__all__ = [
    "ISOLOCO_F32", "ISOLOCO_BF16", "ISOLOCO_KIND_ISO", "ISOLOCO_KIND_AVG",
    "IsoLoCoError", "isoloco_tensor", "isoloco_options", "isoloco_tensor_stats",
    "isoloco_plan", "isoloco_workspace_size", "isoloco_set_workspace", "isoloco_aggregate",
    "isoloco_get_stats", "isoloco_schedule", "isoloco_schedule_phases", "isoloco_plan_destroy",
    "isoloco_status_string", "isoloco_last_error", "isoloco_enable_timing", "isoloco_get_timing",
    "isoloco_timing", "isoloco_aggregate_static", "ISOLOCO_STATIC_WORKSPACE_BYTES",
    "isoloco_factored_steps",
    "IsoLoCoPlan", "LIB_PATH", "EXPORTED_SYMBOLS",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libisoloco.so")

ISOLOCO_F32 = 0
ISOLOCO_BF16 = 1
ISOLOCO_KIND_ISO = 0
ISOLOCO_KIND_AVG = 1
ISOLOCO_PREC_MIXED = 0
ISOLOCO_PREC_FP32 = 1
ISOLOCO_PREC_BF16X3 = 2
ISOLOCO_PREC_BF16X6 = 3
ISOLOCO_ORTH_POLAR = 0
ISOLOCO_ORTH_NS5 = 1
ISOLOCO_SCALE_MEAN = 0
ISOLOCO_SCALE_RMS = 1
ISOLOCO_SCALE_SPECTRAL = 2
ISOLOCO_MOMENTUM_NESTEROV = 0
ISOLOCO_MOMENTUM_HEAVY_BALL = 1
ISOLOCO_TARGET_DELTA = 0
ISOLOCO_TARGET_UPDATE = 1
ISOLOCO_CLIP_NONE = 0
ISOLOCO_CLIP_HIGH = 1
ISOLOCO_CLIP_LOW = 2
ISOLOCO_FLAG_NONFINITE = 1
ISOLOCO_FLAG_ZERO = 2
ISOLOCO_FLAG_NOT_CONVERGED = 4
ISOLOCO_FLAG_BELOW_RESOLUTION = 8
ISOLOCO_STATIC_WORKSPACE_BYTES = 128 * 1024 * 1024

EXPORTED_SYMBOLS = (
    "isoloco_plan", "isoloco_workspace_size", "isoloco_set_workspace", "isoloco_aggregate",
    "isoloco_get_stats", "isoloco_schedule", "isoloco_schedule_phases", "isoloco_plan_destroy",
    "isoloco_status_string", "isoloco_last_error", "isoloco_enable_timing", "isoloco_get_timing",
    "isoloco_aggregate_static", "isoloco_factored_steps",
)


class isoloco_tensor(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("kind", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class isoloco_options(ctypes.Structure):
    _fields_ = [("max_steps", ctypes.c_int32), ("ell0", ctypes.c_float), ("tol", ctypes.c_float),
                ("check", ctypes.c_int32), ("precision", ctypes.c_int32),
                ("orth", ctypes.c_int32), ("scale", ctypes.c_int32), ("momentum", ctypes.c_int32),
                ("target", ctypes.c_int32), ("clip", ctypes.c_int32), ("phase_tall", ctypes.c_float * 3),
                ("phase_square", ctypes.c_float * 3), ("streams", ctypes.c_int32),
                ("factored", ctypes.c_int32)]


class isoloco_tensor_stats(ctypes.Structure):
    _fields_ = [("sigma_bar", ctypes.c_float), ("fro_norm", ctypes.c_float),
                ("orth_resid", ctypes.c_float), ("steps", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class isoloco_timing(ctypes.Structure):
    _fields_ = [("total_ms", ctypes.c_float), ("reduce_ms", ctypes.c_float), ("gram_ms", ctypes.c_float),
                ("poly_ms", ctypes.c_float), ("update_ms", ctypes.c_float), ("finish_ms", ctypes.c_float),
                ("other_ms", ctypes.c_float), ("gram_launches", ctypes.c_int32),
                ("poly_launches", ctypes.c_int32), ("update_launches", ctypes.c_int32),
                ("launches", ctypes.c_int32), ("products_busy_ms", ctypes.c_float),
                ("streams", ctypes.c_int32)]


# torch brings its own copy of the HIP runtime (same SONAME as ROCm's).  Load it
# first so that libisoloco.so binds to that one runtime instead of loading a
# second copy from /opt/rocm into the same process.
import torch  # noqa: E402,F401

if not os.path.exists(LIB_PATH):
    raise ImportError("libisoloco.so is not built: run `python paper_2607_03011_amd/build.py` "
                      "(or __graft_entry__.build()) first")
_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_sig = {
    "isoloco_plan": (ctypes.c_int, [ctypes.POINTER(isoloco_tensor), ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_int32, ctypes.c_int, ctypes.POINTER(isoloco_options),
                                    ctypes.POINTER(_P)]),
    "isoloco_workspace_size": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "isoloco_set_workspace": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "isoloco_aggregate": (ctypes.c_int, [_P, _P, ctypes.POINTER(_P), _P, ctypes.c_float,
                                         ctypes.c_float, ctypes.c_float, _P]),
    "isoloco_aggregate_static": (ctypes.c_int, [_P, _P, ctypes.POINTER(_P), _P, ctypes.c_float,
                                                ctypes.c_float, ctypes.c_float, _P]),
    "isoloco_get_stats": (ctypes.c_int, [_P, ctypes.POINTER(isoloco_tensor_stats), ctypes.c_int32]),
    "isoloco_schedule": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_double), ctypes.c_int32,
                                        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
    "isoloco_schedule_phases": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                               ctypes.POINTER(ctypes.c_int32)]),
    "isoloco_factored_steps": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
    "isoloco_plan_destroy": (ctypes.c_int, [_P]),
    "isoloco_enable_timing": (ctypes.c_int, [_P, ctypes.c_int32]),
    "isoloco_get_timing": (ctypes.c_int, [_P, ctypes.POINTER(isoloco_timing)]),
    "isoloco_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "isoloco_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _sig.items():
    if not hasattr(_lib, _name):
        raise ImportError("libisoloco.so does not export %s: it predates its sources; rebuild it" % _name)
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class IsoLoCoError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = _lib.isoloco_last_error().decode()
        super().__init__("%s: %s (%d)%s" % (where, _lib.isoloco_status_string(status).decode(), status,
                                            (": " + msg) if msg else ""))


def _check(status, where):
    if status != 0:
        raise IsoLoCoError(status, where)


def isoloco_status_string(status):
    return _lib.isoloco_status_string(status).decode()


def isoloco_last_error():
    return _lib.isoloco_last_error().decode()


def isoloco_plan(layout, n_elems, K, worker_dtype=ISOLOCO_F32, opts=None):
    """layout: sequence of (offset, rows, cols, kind).  Returns an opaque plan handle."""
    arr = (isoloco_tensor * max(len(layout), 1))()
    for i, (off, rows, cols, kind) in enumerate(layout):
        arr[i] = isoloco_tensor(int(off), int(rows), int(cols), int(kind), 0)
    o = None
    if opts is not None:
        o = ctypes.byref(opts if isinstance(opts, isoloco_options) else isoloco_options(**opts))
    h = _P()
    _check(_lib.isoloco_plan(arr, len(layout), int(n_elems), int(K), int(worker_dtype), o,
                             ctypes.byref(h)), "isoloco_plan")
    return h


def isoloco_workspace_size(plan):
    n = ctypes.c_size_t()
    _check(_lib.isoloco_workspace_size(plan, ctypes.byref(n)), "isoloco_workspace_size")
    return n.value


def isoloco_set_workspace(plan, dev_ptr, nbytes):
    _check(_lib.isoloco_set_workspace(plan, _P(int(dev_ptr)), int(nbytes)), "isoloco_set_workspace")


def isoloco_aggregate(plan, global_ptr, worker_ptrs, momentum_ptr, alpha, outer_lr, mu, stream=0):
    arr = (_P * max(len(worker_ptrs), 1))(*[_P(int(p)) for p in worker_ptrs])
    _check(_lib.isoloco_aggregate(plan, _P(int(global_ptr)), arr, _P(int(momentum_ptr)),
                                  float(alpha), float(outer_lr), float(mu), _P(int(stream))),
           "isoloco_aggregate")


def isoloco_aggregate_static(plan, global_ptr, worker_ptrs, momentum_ptr, alpha, outer_lr, mu, stream=0):
    arr = (_P * max(len(worker_ptrs), 1))(*[_P(int(p)) for p in worker_ptrs])
    _check(_lib.isoloco_aggregate_static(plan, _P(int(global_ptr)), arr, _P(int(momentum_ptr)),
                                         float(alpha), float(outer_lr), float(mu), _P(int(stream))),
           "isoloco_aggregate_static")


def isoloco_get_stats(plan, n_tensors):
    arr = (isoloco_tensor_stats * max(n_tensors, 1))()
    _check(_lib.isoloco_get_stats(plan, arr, n_tensors), "isoloco_get_stats")
    return [arr[i] for i in range(n_tensors)]


def isoloco_schedule(plan, max_steps=256, with_split=False, tall=0):
    """List of (a, b, c) per step of the square-ish (tall=0) or tall (tall=1)
    matrices' schedule; with_split=True also returns the length of the short
    first phase."""
    buf = (ctypes.c_double * (3 * max_steps))()
    n = ctypes.c_int32()
    ns = ctypes.c_int32()
    _check(_lib.isoloco_schedule(plan, int(tall), buf, max_steps, ctypes.byref(n), ctypes.byref(ns)),
           "isoloco_schedule")
    sched = [tuple(buf[3 * k: 3 * k + 3]) for k in range(min(n.value, max_steps))]
    return (sched, ns.value) if with_split else sched


def isoloco_schedule_phases(plan, max_phases=16, tall=0):
    """Steps done at the end of each phase of a class's schedule (the last is its length)."""
    buf = (ctypes.c_int32 * max_phases)()
    n = ctypes.c_int32()
    _check(_lib.isoloco_schedule_phases(plan, int(tall), buf, max_phases, ctypes.byref(n)),
           "isoloco_schedule_phases")
    return [buf[i] for i in range(min(n.value, max_phases))]


def isoloco_factored_steps(plan):
    """The steps [first, end) that the tall matrices take on n x n factors ((0, 0): none)."""
    a = ctypes.c_int32()
    b = ctypes.c_int32()
    _check(_lib.isoloco_factored_steps(plan, ctypes.byref(a), ctypes.byref(b)), "isoloco_factored_steps")
    return a.value, b.value


def isoloco_enable_timing(plan, enable=True):
    _check(_lib.isoloco_enable_timing(plan, 1 if enable else 0), "isoloco_enable_timing")


def isoloco_get_timing(plan):
    t = isoloco_timing()
    _check(_lib.isoloco_get_timing(plan, ctypes.byref(t)), "isoloco_get_timing")
    return t


def isoloco_plan_destroy(plan):
    _check(_lib.isoloco_plan_destroy(plan), "isoloco_plan_destroy")


class IsoLoCoPlan:
    """A plan plus its workspace, allocated as a torch uint8 tensor on the
    current device (``workspace=False``: none, for ``aggregate_static`` only).
    ``aggregate`` and ``aggregate_static`` marshal torch tensors to the C calls
    and enqueue on the current torch stream (or ``stream``)."""

    def __init__(self, layout, n_elems, K, worker_dtype=ISOLOCO_F32, opts=None, device=None, workspace=True):
        import torch
        self.layout = [tuple(int(v) for v in t) for t in layout]
        self.n_elems = int(n_elems)
        self.K = int(K)
        self.worker_dtype = worker_dtype
        self.handle = isoloco_plan(self.layout, n_elems, K, worker_dtype, opts)
        self.ws_bytes = isoloco_workspace_size(self.handle)
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.workspace = None
        if not workspace:
            return
        with torch.cuda.device(dev):
            self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
            base = self.workspace.data_ptr()
            self._ws_ptr = (base + 255) // 256 * 256
            isoloco_set_workspace(self.handle, self._ws_ptr, self.ws_bytes)

    def aggregate(self, theta, workers, momentum, alpha=1.0, outer_lr=0.7, mu=0.9, stream=None):
        ptrs, stream = self._marshal(theta, workers, momentum, stream)
        isoloco_aggregate(self.handle, theta.data_ptr(), ptrs, momentum.data_ptr(), alpha, outer_lr,
                          mu, stream)

    def aggregate_static(self, theta, workers, momentum, alpha=1.0, outer_lr=0.7, mu=0.9, stream=None):
        ptrs, stream = self._marshal(theta, workers, momentum, stream)
        isoloco_aggregate_static(self.handle, theta.data_ptr(), ptrs, momentum.data_ptr(), alpha, outer_lr,
                                 mu, stream)

    def _marshal(self, theta, workers, momentum, stream):
        import torch
        for t in (theta, momentum):
            if t.dtype != torch.float32 or not t.is_contiguous() or t.numel() != self.n_elems:
                raise ValueError("theta and momentum must be contiguous float32 of n_elems")
        wdt = torch.float32 if self.worker_dtype == ISOLOCO_F32 else torch.bfloat16
        if isinstance(workers, torch.Tensor):
            if workers.dim() != 2 or workers.shape[0] != self.K or workers.shape[1] != self.n_elems:
                raise ValueError("workers tensor must be [K, n_elems]")
            if workers.dtype != wdt or workers.stride(1) != 1:
                raise ValueError("workers must be %s with contiguous rows" % wdt)
            ptrs = [workers[k].data_ptr() for k in range(self.K)]
        else:
            ws = list(workers)
            if len(ws) != self.K:
                raise ValueError("expected %d workers" % self.K)
            for w in ws:
                if w.dtype != wdt or not w.is_contiguous() or w.numel() != self.n_elems:
                    raise ValueError("each worker must be contiguous %s of n_elems" % wdt)
            ptrs = [w.data_ptr() for w in ws]
        if stream is None:
            stream = torch.cuda.current_stream(self.device).cuda_stream
        return ptrs, stream

    def stats(self):
        return isoloco_get_stats(self.handle, len(self.layout))

    def enable_timing(self, enable=True):
        isoloco_enable_timing(self.handle, enable)

    def timing(self):
        return isoloco_get_timing(self.handle)

    def schedule(self, tall=0):
        return isoloco_schedule(self.handle, tall=tall)

    def schedule_split(self, tall=0):
        return isoloco_schedule(self.handle, with_split=True, tall=tall)

    def schedule_phases(self, tall=0):
        return isoloco_schedule_phases(self.handle, tall=tall)

    def factored_steps(self):
        return isoloco_factored_steps(self.handle)

    def close(self):
        if self.handle is not None:
            isoloco_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
