"""The C-ABI library on a machine without a GPU: it loads, exports every
entry point include/ss.h declares, and its loader rejects malformed GMG
snapshots before touching the device."""
import copy
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(ss_[a-z_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_entry_point():
    L = ss.lib()
    names = declared_functions()
    assert names == set(ss.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_null_arguments():
    L = ss.lib()
    h = ctypes.c_void_p()
    assert L.ss_gmg_load(None, ctypes.byref(h)) == -1
    assert L.ss_simulate_batch(None, None, 0, 0, None, None, None, None, None, None) == -1
    assert L.ss_select_best(None, None, None, None, 0, 0, None, None) == -1
    assert L.ss_gmg_info(None, None, None, None) == -1
    assert b"NULL" in L.ss_last_error()
    L.ss_gmg_free(None)


def good():
    return make_gmg(2, ["op"] * 3, [(0, 1), (1, 2)], [0, 0, 0], [[2], [3], [4]], [10, 20, 30],
                    [[(0, 5), (9, TIME_INF)], [(0, TIME_INF)]], [100, 100], [0], [50], bw=[10], lat=[1])


def load_rc(g):
    try:
        h = ss.Gmg(g)
        h.free()
        return 0
    except ss.SSError as e:
        return e.code


def test_valid_snapshot_passes_validation():
    # without a GPU the loader gets as far as the device (SS_ERR_DEVICE); with one it loads
    assert load_rc(good()) in (0, -4)


def _mut(fn):
    g = copy.deepcopy(good())
    fn(g)
    return g


BAD = {
    "non_topological_edge": lambda g: g.pred_idx.__setitem__(1, 2),
    "duplicate_pred": lambda g: (setattr(g, "pred_ptr", np.array([0, 0, 1, 3], np.int32)),
                                 setattr(g, "pred_idx", np.array([0, 1, 1], np.int32))),
    "zero_duration": lambda g: g.dur.__setitem__((1, 0), 0),
    "negative_bytes": lambda g: g.out_bytes.__setitem__(0, -1),
    "zero_bandwidth": lambda g: g.bw.__setitem__(0, 0),
    "negative_latency": lambda g: g.lat.__setitem__(0, -1),
    "no_open_tail": lambda g: g.slice_end.__setitem__(2, 1000),
    "overlapping_slices": lambda g: g.slice_end.__setitem__(0, 10),
    "empty_slice": lambda g: g.slice_end.__setitem__(0, 0),
    "open_slice_not_last": lambda g: g.slice_end.__setitem__(0, TIME_INF),
    "negative_slice_start": lambda g: g.slice_begin.__setitem__(0, -3),
    "link_class_out_of_range": lambda g: g.link_class.__setitem__((0, 1), 1),
    "dev_class_out_of_range": lambda g: g.dev_class.__setitem__(1, 1),
    "op_req_out_of_range": lambda g: g.op_req.__setitem__(0, 1),
    "negative_release": lambda g: g.release.__setitem__(0, -1),
    "huge_deadline": lambda g: g.deadline.__setitem__(0, 1 << 62),
    "negative_cap": lambda g: g.cap.__setitem__(0, -1),
    "horizon_overflow": lambda g: g.slice_begin.__setitem__(1, 1 << 62),
    "bytes_overflow": lambda g: g.out_bytes.__setitem__(0, 1 << 62),
}


@pytest.mark.parametrize("name", sorted(BAD))
def test_loader_rejects_malformed_snapshot(name):
    g = _mut(BAD[name])
    assert load_rc(g) == -2, name


def snap(done=(-1, -1, -1), issue=(0, 0, 0), t_now=0):
    g = good()
    g.done_fin = np.asarray(done, np.int64)
    g.issue_at = None if issue is None else np.asarray(issue, np.int64)
    g.t_now = t_now
    return g


def test_valid_running_schedule_passes_validation():
    for g in (snap(), snap((10, 20, -1), (0, 5, 30), 25), snap((10, -1, -1), None, 7)):
        assert load_rc(g) in (0, -4)


BAD_SNAPSHOTS = {
    "done_pred_not_done": snap((-1, 20, -1)),
    "done_before_pred": snap((20, 20, -1)),
    "done_at_issue": snap((10, -1, -1), (10, 0, 0)),
    "done_below_minus_one": snap((-2, -1, -1)),
    "negative_issue": snap(issue=(0, -1, 0)),
    "negative_t_now": snap(t_now=-1),
    "huge_done": snap((1 << 62, -1, -1)),
    "huge_issue": snap(issue=(0, 1 << 62, 0)),
}


@pytest.mark.parametrize("name", sorted(BAD_SNAPSHOTS))
def test_loader_rejects_malformed_running_schedule(name):
    assert load_rc(BAD_SNAPSHOTS[name]) == -2, name


def test_loader_rejects_too_many_devices():
    g = synth.random_gmg(0, n_ops=4, n_dev=3)
    g.n_dev = 256
    assert load_rc(g) == -2


def test_last_error_is_per_call():
    assert load_rc(_mut(BAD["zero_duration"])) == -2
    assert b"duration" in ss.lib().ss_last_error()


def header_constants():
    text = open(os.path.join(ROOT, "include", "ss.h")).read()
    return {k: int(v, 0) for k, v in re.findall(r"#define\s+(SS_[A-Z_0-9]+)\s+\(?(-?(?:0x)?[0-9A-Fa-f]+)\)?", text)}


def test_binding_constants_match_the_header():
    c = header_constants()
    assert c["SS_LAYOUT_ROW_MAJOR"] == ss.SS_LAYOUT_ROW_MAJOR == ss.LAYOUTS["row"]
    assert c["SS_LAYOUT_OP_MAJOR"] == ss.SS_LAYOUT_OP_MAJOR == ss.LAYOUTS["op"]
    assert c["SS_LAYOUT_OP_MAJOR"] & (c["SS_DISPATCH_READY"] | c["SS_LINK_PORTS"]) == 0
    assert c["SS_DISPATCH_READY"] == ss.SS_DISPATCH_READY == ss.DISPATCH["ready"]
    assert c["SS_DISPATCH_READY"] & c["SS_LAYOUT_ROW_MAJOR"] == 0
    assert c["SS_LINK_PORTS"] == ss.SS_LINK_PORTS == ss.LINKS["ports"]
    assert c["SS_LINK_PORTS"] & (c["SS_DISPATCH_READY"] | c["SS_LAYOUT_ROW_MAJOR"]) == 0
    assert c["SS_VIOLATION_MEMORY"] == ss.SS_VIOLATION_MEMORY and c["SS_VIOLATION_INVALID"] == ss.SS_VIOLATION_INVALID
    assert c["SS_SELECT_REQUIRE_SLA"] == ss.SS_SELECT_REQUIRE_SLA
    assert c["SS_SCHED_PREFIX_REUSE"] == ss.SS_SCHED_PREFIX_REUSE
    for code, name in ss.ERRORS.items():
        assert c[name] == code


def test_unknown_layout_bits_are_rejected_before_the_device():
    L = ss.lib()
    # a non-null dummy handle is never dereferenced: the layout check comes first
    for layout in (2, 3, 0x400, 0x102, 0x203, 0x80):
        assert L.ss_simulate_batch(ctypes.c_void_p(8), None, 1, layout, None, None, None, None, None, None) == -1
        assert b"layout" in L.ss_last_error()
        assert L.ss_simulate_batch_ws(ctypes.c_void_p(8), None, 1, layout, None, None, None, None, None, None, 0,
                                      None) == -1
        assert L.ss_simulate_workspace_size(ctypes.c_void_p(8), 1, layout, ctypes.byref(ctypes.c_int64()),
                                            None) == -1
    # transfer ports with ready-time dispatch (either layout): refused as unsupported
    for layout in (0x300, 0x301):
        assert L.ss_simulate_batch(ctypes.c_void_p(8), None, 1, layout, None, None, None, None, None, None) == -5
        assert b"SS_LINK_PORTS" in L.ss_last_error()


def test_time_bits_checks_arguments_first():
    L = ss.lib()
    b = ctypes.c_int(9)
    assert L.ss_simulate_time_bits(None, 0, ctypes.byref(b)) == -1 and b.value == 0
    # a non-null dummy handle is never dereferenced: the argument and flag checks come first
    assert L.ss_simulate_time_bits(ctypes.c_void_p(8), 0, None) == -1
    for layout in (2, 0x400, 0x80):
        assert L.ss_simulate_time_bits(ctypes.c_void_p(8), layout, ctypes.byref(b)) == -1
        assert b"layout" in L.ss_last_error()
    assert L.ss_simulate_time_bits(ctypes.c_void_p(8), 0x300, ctypes.byref(b)) == -5


def test_workspace_entry_points_check_arguments_first():
    L = ss.lib()
    lo = ctypes.c_int64(7)
    assert L.ss_simulate_workspace_size(None, 1, 0, ctypes.byref(lo), None) == -1 and lo.value == 0
    assert L.ss_simulate_workspace_size(ctypes.c_void_p(8), 1, 0, None, None) == -1
    assert L.ss_simulate_workspace_size(ctypes.c_void_p(8), -1, 0, ctypes.byref(lo), None) == -1
    assert L.ss_simulate_batch_ws(None, None, 1, 0, None, None, None, None, None, None, 0, None) == -1
    assert L.ss_simulate_batch_ws(ctypes.c_void_p(8), None, -1, 0, None, None, None, None, None, None, 0, None) == -1


def test_estimator_arguments_are_checked_before_the_device():
    L = ss.lib()
    h = ctypes.c_void_p()
    assert L.ss_est_create(4, 0, ctypes.byref(h)) == -1
    assert L.ss_est_create(4, 9, ctypes.byref(h)) == -1
    assert L.ss_est_create(-1, 3, ctypes.byref(h)) == -1
    assert L.ss_est_create(4, 3, None) == -1
    assert L.ss_est_create(1 << 40, 1, ctypes.byref(h)) == -1
    assert L.ss_est_add(None, None, 0, None, None, None) == -1
    assert L.ss_est_solve(None, None, None, None) == -1
    assert L.ss_est_predict(None, 1, 0, None, None, 1, None, None) == -1
    assert L.ss_est_predict(None, 1, 2, None, None, -1, None, None) == -1
    assert L.ss_est_predict(None, 1, 2, None, None, 3, None, None) == -1
    assert L.ss_est_predict(None, 1, 2, None, None, 0, None, None) == 0  # nothing to do
    L.ss_est_free(None)


def test_scheduler_arguments_are_checked_before_the_device():
    L = ss.lib()
    h = ctypes.c_void_p()
    assert L.ss_sched_create(None, ctypes.byref(h)) == -1
    g = synth.build_gmg(0)
    keep = {}
    desc = ss._gmg_desc(g, keep)
    part = synth.partition_table(g, 0)
    prio = synth.request_priority(g)
    for n_part, budget, cap, flags, bad_dev in [(0, 4, 4, 0, False), (3, 0, 4, 0, False), (3, 4, 0, 0, False),
                                                (3, 4, 4, 4, False), (3, 4, 4, 0, True)]:
        pd = part.copy()
        if bad_dev:
            pd[1, 5] = g.n_dev
        d = ss._SchedDesc(ctypes.pointer(desc), n_part, pd.ctypes.data, prio.ctypes.data, budget, cap, flags)
        assert L.ss_sched_create(ctypes.byref(d), ctypes.byref(h)) == -1
    g.done_fin = np.full(g.n_ops, -1, np.int64)  # the run's GMG holds no running state
    desc2 = ss._gmg_desc(g, keep)
    d = ss._SchedDesc(ctypes.pointer(desc2), 3, part.ctypes.data, prio.ctypes.data, 4, 4, 0)
    assert L.ss_sched_create(ctypes.byref(d), ctypes.byref(h)) == -1
    assert b"running state" in L.ss_last_error()
    assert L.ss_sched_round(None, 0, None, None, None, None, None) == -1
    assert L.ss_sched_complete(None, 0, 1) == -1
    assert L.ss_sched_state(None, None, None, None, None) == -1
    L.ss_sched_free(None)
