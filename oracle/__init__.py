"""Oracle for the GMG what-if simulator -- TEST INFRASTRUCTURE ONLY.

A plain sequential C implementation (``ss_oracle.c``) of what the simulator
computes, written from the paper, with a thin ctypes wrapper.  Only the tests,
the smoke check and the benchmark's CPU-baseline leg use it; the product path
never imports it, and it imports nothing from the product package.

Every exported function is pinned by the CPU test-suite (closed forms, bounds,
brute force, hand-worked cases, metamorphic relations); see
tests/test_oracle_pins.py.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
INDEX_ORDER, READY_ORDER, LINK_PORTS = 0, 1, 2
_lib = None
_lock = threading.Lock()


def build(force: bool = False) -> str:
    """Compile ss_oracle.c with gcc (the checker is built, not used, by build())."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                               os.path.join(_HERE, "ss_oracle.c"), "-o", tmp])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


class _Gmg(ctypes.Structure):
    _fields_ = [("n_ops", ctypes.c_int64), ("n_dev", ctypes.c_int64), ("n_class", ctypes.c_int64),
                ("n_link", ctypes.c_int64), ("n_req", ctypes.c_int64)] + \
               [(n, ctypes.c_void_p) for n in ("pred_ptr", "pred_idx", "op_req", "dur", "out_bytes", "dev_class",
                                               "link_class", "bw", "lat", "slice_ptr", "slice_begin", "slice_end",
                                               "cap", "release", "deadline", "done_fin", "issue_at")] + \
               [("t_now", ctypes.c_int64)]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def _get():
    global _lib
    with _lock:
        if _lib is None:
            # SS_ORACLE_LIB: another build of the same source (the sanitizer run)
            lib = ctypes.CDLL(os.environ.get("SS_ORACLE_LIB") or build())
            lib.sso_simulate_one.argtypes = [ctypes.POINTER(_Gmg), _P, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P]
            lib.sso_simulate_batch.argtypes = [ctypes.POINTER(_Gmg), _P, _I64, ctypes.c_int, _P, _P, _P, _P, _P]
            lib.sso_peak_sweep.argtypes = [ctypes.POINTER(_Gmg), _P, _P, _P, _P]
            lib.sso_peak_pairwise.argtypes = [ctypes.POINTER(_Gmg), _P, _P, _P, _P]
            lib.sso_select_best.argtypes = [_I64, _I64, _P, _P, _P, ctypes.c_int, _P, _P]
            lib.sso_port_transfers.argtypes = [ctypes.POINTER(_Gmg), _P, _P, _P, _P, _P, _P, _P]
            lib.sso_select_best.restype = None
            _lib = lib
    return _lib


class OracleGmg:
    """Holds contiguous copies of a GMG's arrays and the C view onto them."""

    def __init__(self, g):
        self.g = g
        self._keep = {}

        def arr(name, dtype):
            a = np.ascontiguousarray(getattr(g, name), dtype)
            self._keep[name] = a
            return a.ctypes.data

        def opt(name):  # optional snapshot arrays: NULL when absent
            return arr(name, np.int64) if getattr(g, name, None) is not None else None

        self.c = _Gmg(g.n_ops, g.n_dev, g.n_class, g.n_link, g.n_req,
                      arr("pred_ptr", np.int32), arr("pred_idx", np.int32), arr("op_req", np.int32),
                      arr("dur", np.int64), arr("out_bytes", np.int64), arr("dev_class", np.int32),
                      arr("link_class", np.uint8), arr("bw", np.int64), arr("lat", np.int64),
                      arr("slice_ptr", np.int64), arr("slice_begin", np.int64), arr("slice_end", np.int64),
                      arr("cap", np.int64), arr("release", np.int64), arr("deadline", np.int64),
                      opt("done_fin"), opt("issue_at"), int(getattr(g, "t_now", 0) or 0))


def _og(g):
    return g if isinstance(g, OracleGmg) else OracleGmg(g)


def simulate_one(g, placement, dispatch: int = INDEX_ORDER) -> dict:
    """One candidate with its schedule: st, fin, makespan, peak, violation, slack, sumfin."""
    og = _og(g)
    G = og.g
    p = np.ascontiguousarray(placement, np.uint8)
    assert p.shape == (G.n_ops,)
    st = np.zeros(G.n_ops, np.int64)
    fin = np.zeros(G.n_ops, np.int64)
    ms, sf = np.zeros(1, np.int64), np.zeros(1, np.int64)
    peak = np.zeros(G.n_dev, np.int64)
    viol = np.zeros(1, np.uint8)
    slack = np.zeros(G.n_req, np.int64)
    rc = _get().sso_simulate_one(ctypes.byref(og.c), p.ctypes.data, dispatch, st.ctypes.data, fin.ctypes.data,
                                 ms.ctypes.data, peak.ctypes.data, viol.ctypes.data, slack.ctypes.data,
                                 sf.ctypes.data)
    if rc == -3:
        raise ValueError("a snapshot (done_fin, issue_at) takes index-order dispatch only")
    if rc != 0:
        raise MemoryError("oracle allocation failed")
    return dict(st=st, fin=fin, makespan=int(ms[0]), peak=peak, violation=int(viol[0]), slack=slack,
                sumfin=int(sf[0]))


def simulate_batch(g, placements, dispatch: int = INDEX_ORDER, n_threads: int = 1) -> dict:
    """Row-major placements [B, N] -> makespan[B], peak[B, D], violation[B], slack[B, R], sumfin[B].

    With n_threads > 1 the batch is split into contiguous ranges, each run by
    the same sequential C routine on its own Python thread (ctypes releases the
    GIL during the call)."""
    og = _og(g)
    G = og.g
    P = np.ascontiguousarray(placements, np.uint8)
    B = P.shape[0]
    assert P.shape == (B, G.n_ops)
    out = dict(makespan=np.zeros(B, np.int64), peak=np.zeros((B, G.n_dev), np.int64),
               violation=np.zeros(B, np.uint8), slack=np.zeros((B, G.n_req), np.int64),
               sumfin=np.zeros(B, np.int64))
    lib = _get()
    errors = []

    def run(lo, hi):
        if hi <= lo:
            return
        rc = lib.sso_simulate_batch(ctypes.byref(og.c), P[lo:hi].ctypes.data, hi - lo, dispatch,
                                    out["makespan"][lo:hi].ctypes.data, out["peak"][lo:hi].ctypes.data,
                                    out["violation"][lo:hi].ctypes.data, out["slack"][lo:hi].ctypes.data,
                                    out["sumfin"][lo:hi].ctypes.data)
        if rc != 0:
            errors.append(rc)

    n_threads = max(1, min(n_threads, B))
    if n_threads == 1:
        run(0, B)
    else:
        per = (B + n_threads - 1) // n_threads
        ths = [threading.Thread(target=run, args=(i * per, min(B, (i + 1) * per))) for i in range(n_threads)]
        for t in ths:
            t.start()
        for t in ths:
            t.join()
    if -3 in errors:
        raise ValueError("a snapshot (done_fin, issue_at) takes index-order dispatch only")
    if errors:
        raise MemoryError("oracle allocation failed")
    return out


def peak_sweep(g, placement, st, fin) -> np.ndarray:
    og = _og(g)
    peak = np.zeros(og.g.n_dev, np.int64)
    p = np.ascontiguousarray(placement, np.uint8)
    st = np.ascontiguousarray(st, np.int64)
    fin = np.ascontiguousarray(fin, np.int64)
    if _get().sso_peak_sweep(ctypes.byref(og.c), p.ctypes.data, st.ctypes.data, fin.ctypes.data, peak.ctypes.data):
        raise MemoryError
    return peak


def peak_pairwise(g, placement, st, fin) -> np.ndarray:
    og = _og(g)
    peak = np.zeros(og.g.n_dev, np.int64)
    p = np.ascontiguousarray(placement, np.uint8)
    st = np.ascontiguousarray(st, np.int64)
    fin = np.ascontiguousarray(fin, np.int64)
    if _get().sso_peak_pairwise(ctypes.byref(og.c), p.ctypes.data, st.ctypes.data, fin.ctypes.data,
                                peak.ctypes.data):
        raise MemoryError
    return peak


def port_transfers(g, placement) -> dict:
    """Transfers of one candidate under LINK_PORTS in admission order: producer
    op, source and destination device, start and arrival (Sec. 3.5.2)."""
    og = _og(g)
    p = np.ascontiguousarray(placement, dtype=np.uint8)
    E = max(int(og.g.pred_ptr[-1]), 1)
    out = {k: np.zeros(E, np.int64) for k in ("op", "src", "dst", "start", "arrive")}
    n = np.zeros(1, np.int64)
    rc = _get().sso_port_transfers(ctypes.byref(og.c), p.ctypes.data, *(out[k].ctypes.data for k in
                                   ("op", "src", "dst", "start", "arrive")), n.ctypes.data)
    if rc != 0:
        raise ValueError(f"sso_port_transfers returned {rc}")
    return {k: v[:int(n[0])] for k, v in out.items()}


def select_best(violation, key, slack=None, require_sla: bool = False) -> tuple[int, int]:
    v = np.ascontiguousarray(violation, np.uint8)
    k = np.ascontiguousarray(key, np.int64)
    B = v.shape[0]
    R = 0
    sp = None
    if slack is not None:
        s = np.ascontiguousarray(slack, np.int64)
        R = s.shape[1] if s.ndim == 2 else 0
        sp = s.ctypes.data
    bi, bk = np.zeros(1, np.int64), np.zeros(1, np.int64)
    _get().sso_select_best(B, R, v.ctypes.data, k.ctypes.data, sp, int(require_sla), bi.ctypes.data, bk.ctypes.data)
    return int(bi[0]), int(bk[0])


def time_batch(g, placements, n_threads: int) -> float:
    """Wall seconds for simulate_batch on the given placements (CPU baseline)."""
    og = _og(g)
    t0 = time.perf_counter()
    simulate_batch(og, placements, INDEX_ORDER, n_threads)
    return time.perf_counter() - t0
