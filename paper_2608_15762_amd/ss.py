"""Python binding of libss.so (the C ABI in include/ss.h).

Argument marshalling only: every step of the simulation runs in the HIP
kernels behind the C ABI.  PyTorch provides device memory and streams.  There
is no fallback: if the library is missing or cannot load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libss.so")

SS_OK = 0
SS_ERR_INVALID_ARG, SS_ERR_INVALID_GMG, SS_ERR_OOM, SS_ERR_DEVICE, SS_ERR_UNSUPPORTED = -1, -2, -3, -4, -5
ERRORS = {-1: "SS_ERR_INVALID_ARG", -2: "SS_ERR_INVALID_GMG", -3: "SS_ERR_OOM", -4: "SS_ERR_DEVICE",
          -5: "SS_ERR_UNSUPPORTED"}
SS_LAYOUT_ROW_MAJOR = 0
SS_LAYOUT_OP_MAJOR = 1
LAYOUTS = {"row": SS_LAYOUT_ROW_MAJOR, "op": SS_LAYOUT_OP_MAJOR}
SS_DISPATCH_READY = 0x100
SS_LINK_PORTS = 0x200
DISPATCH = {"index": 0, "ready": SS_DISPATCH_READY}
LINKS = {"latency": 0, "ports": SS_LINK_PORTS}
SS_VIOLATION_MEMORY = 0x1
SS_VIOLATION_INVALID = 0x4
SS_SELECT_REQUIRE_SLA = 0x1
SS_SCHED_PREFIX_REUSE = 0x2
EXPORTED = ("ss_gmg_load", "ss_gmg_free", "ss_gmg_info", "ss_simulate_batch", "ss_select_best", "ss_kernel_timing",
            "ss_kernel_time", "ss_last_error", "ss_est_create", "ss_est_free", "ss_est_add", "ss_est_solve",
            "ss_est_predict", "ss_sched_create", "ss_sched_free", "ss_sched_round", "ss_sched_complete",
            "ss_sched_state", "ss_state_create", "ss_state_free", "ss_state_info", "ss_simulate_batch_resume",
            "ss_state_capture", "ss_release_cached_memory", "ss_simulate_workspace_size", "ss_simulate_batch_ws",
            "ss_simulate_batch_noalloc", "ss_simulate_chunking", "ss_simulate_time_bits")
SS_OP_UNSCHEDULED, SS_OP_ISSUED, SS_OP_DONE = 0, 1, 2
SS_ROUND_ISSUED, SS_ROUND_BUDGET, SS_ROUND_IDLE, SS_ROUND_INFEASIBLE = 0, 1, 2, 3
SS_KERNEL_SCHEDULE, SS_KERNEL_MEMORY, SS_KERNEL_SELECT, SS_KERNEL_INTERVALS, SS_KERNEL_TRANSPOSE = 0, 1, 2, 3, 4
SS_KERNEL_ESTIMATOR = 6
KERNEL_NAMES = {0: "schedule_kernel", 1: "memory_kernel", 2: "select", 3: "intervals_kernel", 4: "transpose",
                6: "estimator"}
SS_EST_MAX_FEAT = 8
SS_EST_FITTED, SS_EST_UNDERDETERMINED, SS_EST_SINGULAR = 0, 1, 2

_lib = None
_lock = threading.Lock()


class SSError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class _Desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("n_ops", "n_edges", "n_dev", "n_class", "n_link", "n_req")] + \
               [(n, ctypes.c_void_p) for n in ("pred_ptr", "pred_idx", "op_req", "dur", "out_bytes", "dev_class",
                                               "link_class", "bw", "lat", "slice_ptr", "slice_begin", "slice_end",
                                               "cap", "release", "deadline", "done_fin", "issue_at")] + \
               [("t_now", ctypes.c_int64)]


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            # SS_LIBRARY: another build of the same sources (the host sanitizer run)
            path = os.environ.get("SS_LIBRARY") or LIB_PATH
            if not os.path.exists(path):
                raise RuntimeError(f"{path} is missing: build it with paper_2608_15762_amd/build.py")
            L = ctypes.CDLL(path)
            P, I64 = ctypes.c_void_p, ctypes.c_int64
            L.ss_gmg_load.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(ctypes.c_void_p)]
            L.ss_gmg_load.restype = ctypes.c_int
            L.ss_gmg_free.argtypes = [P]
            L.ss_gmg_free.restype = None
            L.ss_gmg_info.argtypes = [P, P, P, P]
            L.ss_simulate_batch.argtypes = [P, P, I64, ctypes.c_int, P, P, P, P, P, P]
            L.ss_simulate_batch.restype = ctypes.c_int
            L.ss_simulate_workspace_size.argtypes = [P, I64, ctypes.c_int, P, P]
            L.ss_simulate_workspace_size.restype = ctypes.c_int
            L.ss_simulate_batch_ws.argtypes = [P, P, I64, ctypes.c_int, P, P, P, P, P, P, I64, P]
            L.ss_simulate_batch_ws.restype = ctypes.c_int
            L.ss_simulate_batch_noalloc.argtypes = [P, P, I64, ctypes.c_int, P, P, P, P, P, P]
            L.ss_simulate_batch_noalloc.restype = ctypes.c_int
            L.ss_simulate_chunking.argtypes = [P, I64, ctypes.c_int, P, P]
            L.ss_simulate_chunking.restype = ctypes.c_int
            L.ss_simulate_time_bits.argtypes = [P, ctypes.c_int, P]
            L.ss_simulate_time_bits.restype = ctypes.c_int
            L.ss_select_best.argtypes = [P, P, P, P, I64, ctypes.c_int, P, P]
            L.ss_select_best.restype = ctypes.c_int
            L.ss_kernel_timing.argtypes = [ctypes.c_int]
            L.ss_kernel_timing.restype = ctypes.c_int
            L.ss_kernel_time.argtypes = [ctypes.c_int, P, P]
            L.ss_kernel_time.restype = ctypes.c_int
            L.ss_last_error.argtypes = []
            L.ss_last_error.restype = ctypes.c_char_p
            L.ss_est_create.argtypes = [I64, I64, ctypes.POINTER(ctypes.c_void_p)]
            L.ss_est_create.restype = ctypes.c_int
            L.ss_est_free.argtypes = [P]
            L.ss_est_free.restype = None
            L.ss_est_add.argtypes = [P, P, I64, P, P, P]
            L.ss_est_add.restype = ctypes.c_int
            L.ss_est_solve.argtypes = [P, P, P, P]
            L.ss_est_solve.restype = ctypes.c_int
            L.ss_est_predict.argtypes = [P, I64, I64, P, P, I64, P, P]
            L.ss_est_predict.restype = ctypes.c_int
            L.ss_sched_create.argtypes = [ctypes.POINTER(_SchedDesc), ctypes.POINTER(ctypes.c_void_p)]
            L.ss_sched_create.restype = ctypes.c_int
            L.ss_sched_free.argtypes = [P]
            L.ss_sched_free.restype = None
            L.ss_sched_round.argtypes = [P, I64, P, P, P, P, P]
            L.ss_sched_round.restype = ctypes.c_int
            L.ss_sched_complete.argtypes = [P, I64, I64]
            L.ss_sched_complete.restype = ctypes.c_int
            L.ss_sched_state.argtypes = [P, P, P, P, P]
            L.ss_sched_state.restype = ctypes.c_int
            L.ss_state_create.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            L.ss_state_create.restype = ctypes.c_int
            L.ss_state_free.argtypes = [P]
            L.ss_state_free.restype = None
            L.ss_state_info.argtypes = [P, P]
            L.ss_state_info.restype = ctypes.c_int
            L.ss_simulate_batch_resume.argtypes = [P, P, P, I64, P, P, P, P, P, P]
            L.ss_simulate_batch_resume.restype = ctypes.c_int
            L.ss_state_capture.argtypes = [P, P, P, P, P]
            L.ss_state_capture.restype = ctypes.c_int
            L.ss_release_cached_memory.argtypes = []
            L.ss_release_cached_memory.restype = ctypes.c_int
            _lib = L
    return _lib


def _check(rc):
    if rc != SS_OK:
        raise SSError(rc, lib().ss_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _gmg_desc(g, keep):
    """An ss_gmg_desc over contiguous copies of g's arrays (kept alive in `keep`)."""

    def arr(name, dtype):
        a = np.ascontiguousarray(getattr(g, name), dtype)
        keep[name] = a
        return a.ctypes.data

    def opt(name):  # the running schedule's state: NULL when absent
        return arr(name, np.int64) if getattr(g, name, None) is not None else None

    return _Desc(int(g.n_ops), int(g.pred_ptr[-1]), int(g.n_dev), int(g.n_class), int(g.n_link), int(g.n_req),
                 arr("pred_ptr", np.int32), arr("pred_idx", np.int32), arr("op_req", np.int32),
                 arr("dur", np.int64), arr("out_bytes", np.int64), arr("dev_class", np.int32),
                 arr("link_class", np.uint8), arr("bw", np.int64), arr("lat", np.int64),
                 arr("slice_ptr", np.int64), arr("slice_begin", np.int64), arr("slice_end", np.int64),
                 arr("cap", np.int64), arr("release", np.int64), arr("deadline", np.int64),
                 opt("done_fin"), opt("issue_at"), int(getattr(g, "t_now", 0) or 0))


class Gmg:
    """A GMG snapshot staged on the current HIP device (ss_gmg_load)."""

    def __init__(self, g):
        keep = {}
        d = _gmg_desc(g, keep)
        h = ctypes.c_void_p()
        _check(lib().ss_gmg_load(ctypes.byref(d), ctypes.byref(h)))
        self.handle = h
        self.n_ops, self.n_dev, self.n_req = int(g.n_ops), int(g.n_dev), int(g.n_req)

    def info(self):
        n = [ctypes.c_int64() for _ in range(3)]
        _check(lib().ss_gmg_info(self.handle, *[ctypes.byref(x) for x in n]))
        return tuple(x.value for x in n)

    def free(self):
        if self.handle:
            lib().ss_gmg_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class _SchedDesc(ctypes.Structure):
    _fields_ = [("gmg", ctypes.POINTER(_Desc)), ("n_part", ctypes.c_int64), ("part_dev", ctypes.c_void_p),
                ("priority", ctypes.c_void_p), ("issue_budget", ctypes.c_int64), ("batch_cap", ctypes.c_int64),
                ("flags", ctypes.c_int)]


class Scheduler:
    """The incremental scheduling loop of Alg. 1 (ss_sched_*) over a run's GMG,
    its pre-defined partitions part_dev[n_part][n_ops] and request priorities."""

    def __init__(self, g, part_dev, priority, budget, cap, require_sla=False, prefix_reuse=False):
        keep = {}
        desc = _gmg_desc(g, keep)
        part = np.ascontiguousarray(part_dev, np.uint8)
        prio = np.ascontiguousarray(priority, np.int64)
        assert part.ndim == 2 and part.shape[1] == g.n_ops and prio.shape == (g.n_req,)
        flags = (SS_SELECT_REQUIRE_SLA if require_sla else 0) | (SS_SCHED_PREFIX_REUSE if prefix_reuse else 0)
        d = _SchedDesc(ctypes.pointer(desc), part.shape[0], part.ctypes.data, prio.ctypes.data, int(budget),
                       int(cap), flags)
        h = ctypes.c_void_p()
        _check(lib().ss_sched_create(ctypes.byref(d), ctypes.byref(h)))
        self.handle = h
        self.n_ops, self.cap = int(g.n_ops), int(cap)
        self._ops = np.zeros(max(1, int(cap)), np.int64)
        # reused per call: a run makes one round and one completion call per op
        self._st, self._n, self._p = ctypes.c_int(), ctypes.c_int64(), ctypes.c_int64()
        self._args = (ctypes.byref(self._st), self._ops.ctypes.data, ctypes.byref(self._n), ctypes.byref(self._p))
        self._round, self._complete = lib().ss_sched_round, lib().ss_sched_complete

    def round(self, now, stream=None):
        """One round at time `now`: (status, batch ops, partition or -1)."""
        st, ops, n, p = self._args
        _check(self._round(self.handle, int(now), st, ops, n, p, _stream_ptr(stream)))
        k = self._n.value
        return self._st.value, (self._ops[:k].tolist() if k else []), self._p.value

    def complete(self, op, t_done):
        _check(self._complete(self.handle, int(op), int(t_done)))

    def state(self):
        """(state[n_ops] of SS_OP_*, place[n_ops], issue time[n_ops], completion time[n_ops])."""
        st = np.zeros(self.n_ops, np.uint8)
        pl = np.zeros(self.n_ops, np.uint8)
        it = np.zeros(self.n_ops, np.int64)
        dt = np.zeros(self.n_ops, np.int64)
        _check(lib().ss_sched_state(self.handle, st.ctypes.data, pl.ctypes.data, it.ctypes.data, dt.ctypes.data))
        return st, pl, it, dt

    def free(self):
        if self.handle:
            lib().ss_sched_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def _layout(g: Gmg, placements, layout: str, dispatch: str, links: str) -> tuple[int, int]:
    """Batch size and layout flags of a placement tensor (uint8, contiguous):
    layout "row" is [B, n_ops], "op" is [n_ops, B]."""
    assert placements.dtype.is_floating_point is False and placements.element_size() == 1
    assert placements.is_contiguous() and placements.dim() == 2
    if layout == "row":
        B = placements.shape[0]
        assert placements.shape == (B, g.n_ops)
    else:
        B = placements.shape[1]
        assert placements.shape == (g.n_ops, B)
    return B, LAYOUTS[layout] | DISPATCH[dispatch] | LINKS[links]


def workspace_size(g: Gmg, B: int, layout="row", dispatch="index", links="latency") -> tuple[int, int]:
    """ss_simulate_workspace_size: (smallest, preferred) workspace bytes of
    ss_simulate_batch_ws for B candidates."""
    lo, hi = ctypes.c_int64(), ctypes.c_int64()
    flags = LAYOUTS[layout] | DISPATCH[dispatch] | LINKS[links]
    _check(lib().ss_simulate_workspace_size(g.handle, B, flags, ctypes.byref(lo), ctypes.byref(hi)))
    return lo.value, hi.value


def chunking(g: Gmg, B: int, layout="row", dispatch="index") -> tuple[int, int]:
    """ss_simulate_chunking: (candidates per chunk, per memory-pass sub-chunk)
    of an ss_simulate_batch call of B candidates."""
    c, s_ = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().ss_simulate_chunking(g.handle, B, LAYOUTS[layout] | DISPATCH[dispatch], ctypes.byref(c),
                                      ctypes.byref(s_)))
    return c.value, s_.value


def time_bits(g: Gmg, dispatch="index", links="latency") -> int:
    """ss_simulate_time_bits: 32 or 64, the width of the integers a
    simulation of g with this dispatch rule and link model computes its
    times in."""
    b = ctypes.c_int()
    _check(lib().ss_simulate_time_bits(g.handle, DISPATCH[dispatch] | LINKS[links], ctypes.byref(b)))
    return b.value


def simulate_batch_into(g: Gmg, placements, makespan, violation, peak=None, slack=None, sumfin=None,
                        stream=None, dispatch="index", links="latency", layout="row", workspace=None):
    """ss_simulate_batch on caller-provided torch CUDA tensors.

    layout: "row" (placements [B, n_ops]) or "op" (placements [n_ops, B]).
    dispatch: "index" (every device serves its ops in index order) or "ready"
    (earliest ready time first, SS_DISPATCH_READY).
    links: "latency" (a transfer takes its estimate from the producer's
    finish) or "ports" (SS_LINK_PORTS: transfers arbitrated event by event
    over each device's send and receive port; index-order dispatch only).
    workspace: None (the library's pool) or a device tensor whose memory
    becomes the call's scratch (ss_simulate_batch_ws)."""
    B, flags = _layout(g, placements, layout, dispatch, links)
    if workspace is None:
        _check(lib().ss_simulate_batch(g.handle, _ptr(placements), B, flags, _ptr(makespan), _ptr(peak),
                                       _ptr(violation), _ptr(slack), _ptr(sumfin), _stream_ptr(stream)))
    else:
        nbytes = workspace.numel() * workspace.element_size()
        _check(lib().ss_simulate_batch_ws(g.handle, _ptr(placements), B, flags, _ptr(makespan), _ptr(peak),
                                          _ptr(violation), _ptr(slack), _ptr(sumfin), _ptr(workspace), nbytes,
                                          _stream_ptr(stream)))


def simulate_batch_noalloc_into(g: Gmg, placements, makespan, violation, peak=None, slack=None, sumfin=None,
                                stream=None, dispatch="index", layout="row"):
    """ss_simulate_batch_noalloc: the library's fixed scratch array instead of
    any allocation (calls on one GPU must not overlap)."""
    B, flags = _layout(g, placements, layout, dispatch, "latency")
    _check(lib().ss_simulate_batch_noalloc(g.handle, _ptr(placements), B, flags, _ptr(makespan), _ptr(peak),
                                           _ptr(violation), _ptr(slack), _ptr(sumfin), _stream_ptr(stream)))


def simulate_batch(g: Gmg, placements, want_peak=True, want_slack=True, want_sumfin=True, stream=None,
                   dispatch="index", links="latency", layout="row", workspace=None) -> dict:
    """Allocate outputs on placements' device and run ss_simulate_batch (or
    ss_simulate_batch_ws with a workspace tensor)."""
    import torch
    B = placements.shape[0] if layout == "row" else placements.shape[1]
    dev = placements.device
    out = dict(makespan=torch.empty(B, dtype=torch.int64, device=dev),
               violation=torch.empty(B, dtype=torch.uint8, device=dev),
               peak=torch.empty((B, g.n_dev), dtype=torch.int64, device=dev) if want_peak else None,
               slack=torch.empty((B, g.n_req), dtype=torch.int64, device=dev) if want_slack else None,
               sumfin=torch.empty(B, dtype=torch.int64, device=dev) if want_sumfin else None)
    simulate_batch_into(g, placements, out["makespan"], out["violation"], out["peak"], out["slack"], out["sumfin"],
                        stream, dispatch, links, layout, workspace)
    return out


class State:
    """A captured simulation state (ss_state_*): one candidate after the first
    ops of a GMG, for resuming candidates that share those ops."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(lib().ss_state_create(ctypes.byref(h)))
        self.handle = h

    def n_ops(self):
        k = ctypes.c_int64()
        _check(lib().ss_state_info(self.handle, ctypes.byref(k)))
        return k.value

    def free(self):
        if self.handle:
            lib().ss_state_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def state_capture(g: Gmg, placement, capture, start=None, stream=None):
    """ss_state_capture: the schedule of one placement (device uint8 [n_ops]),
    resumed from State `start`, its state stored in State `capture`."""
    assert placement.is_contiguous() and placement.numel() == g.n_ops
    _check(lib().ss_state_capture(g.handle, None if start is None else start.handle, _ptr(placement),
                                  capture.handle, _stream_ptr(stream)))


def simulate_batch_resume(g: Gmg, placements, start=None, want_peak=True, want_slack=True, want_sumfin=True,
                          stream=None) -> dict:
    """ss_simulate_batch_resume: candidates resumed from State `start` (None:
    from op 0)."""
    import torch
    B = placements.shape[0]
    assert placements.dtype == torch.uint8 and placements.is_contiguous() and placements.shape == (B, g.n_ops)
    dev = placements.device
    out = dict(makespan=torch.empty(B, dtype=torch.int64, device=dev),
               violation=torch.empty(B, dtype=torch.uint8, device=dev),
               peak=torch.empty((B, g.n_dev), dtype=torch.int64, device=dev) if want_peak else None,
               slack=torch.empty((B, g.n_req), dtype=torch.int64, device=dev) if want_slack else None,
               sumfin=torch.empty(B, dtype=torch.int64, device=dev) if want_sumfin else None)
    _check(lib().ss_simulate_batch_resume(g.handle, None if start is None else start.handle, _ptr(placements), B,
                                          _ptr(out["makespan"]), _ptr(out["peak"]), _ptr(out["violation"]),
                                          _ptr(out["slack"]), _ptr(out["sumfin"]), _stream_ptr(stream)))
    return out


def release_cached_memory():
    """ss_release_cached_memory: hand the library pools' unused memory back."""
    _check(lib().ss_release_cached_memory())


def select_best(g: Gmg, violation, key, slack=None, require_sla=False, out=None, stream=None):
    """ss_select_best; returns a device int64[2] tensor {index or -1, key}."""
    import torch
    B = violation.shape[0]
    if out is None:
        out = torch.empty(2, dtype=torch.int64, device=violation.device)
    _check(lib().ss_select_best(g.handle, _ptr(violation), _ptr(key), _ptr(slack), B,
                                SS_SELECT_REQUIRE_SLA if require_sla else 0, _ptr(out), _stream_ptr(stream)))
    return out


def kernel_timing(enable: bool) -> None:
    """Turn per-kernel HIP event timing on or off (process-wide)."""
    _check(lib().ss_kernel_timing(1 if enable else 0))


def kernel_time(kernel: int) -> tuple[int, float]:
    """(launches, summed milliseconds) recorded for one kernel kind since the last read."""
    n, ms = ctypes.c_int64(), ctypes.c_double()
    _check(lib().ss_kernel_time(kernel, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


class Estimators:
    """An ss_est set: n_est online least-squares fits of n_feat features (Sec. 3.3.1)."""

    def __init__(self, n_est: int, n_feat: int):
        h = ctypes.c_void_p()
        _check(lib().ss_est_create(n_est, n_feat, ctypes.byref(h)))
        self.handle, self.n_est, self.n_feat = h, n_est, n_feat

    def add(self, sample_ptr, x, y, stream=None):
        """Samples grouped by estimator: int64 sample_ptr[n_est+1], float64 x[S][n_feat], y[S] (device)."""
        S = y.shape[0]
        assert sample_ptr.shape == (self.n_est + 1,) and x.shape == (S, self.n_feat)
        assert sample_ptr.is_contiguous() and x.is_contiguous() and y.is_contiguous()
        _check(lib().ss_est_add(self.handle, _ptr(sample_ptr), S, _ptr(x), _ptr(y), _stream_ptr(stream)))

    def solve(self, stream=None):
        """(coef float64[n_est][n_feat], status int32[n_est]) on the device."""
        import torch
        dev = torch.device("cuda", torch.cuda.current_device())
        coef = torch.empty((self.n_est, self.n_feat), dtype=torch.float64, device=dev)
        status = torch.empty(self.n_est, dtype=torch.int32, device=dev)
        _check(lib().ss_est_solve(self.handle, _ptr(coef), _ptr(status), _stream_ptr(stream)))
        return coef, status

    def free(self):
        if self.handle:
            lib().ss_est_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def est_predict(coef, est_of, x, stream=None):
    """Integer microseconds max(1, ceil(x . coef[est_of])) per query (0: invalid query)."""
    import torch
    M = est_of.shape[0]
    n_est, n_feat = coef.shape
    out = torch.empty(M, dtype=torch.int64, device=x.device)
    _check(lib().ss_est_predict(_ptr(coef), n_est, n_feat, _ptr(est_of), _ptr(x), M, _ptr(out),
                                _stream_ptr(stream)))
    return out
