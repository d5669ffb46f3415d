"""The seeded input generator: shapes, statistics and determinism."""
import numpy as np
import pytest

from paper_2608_15762_amd import synth
from paper_2608_15762_amd.synth import TIME_INF

COUNTS = {0: (32, 37, 2, 1), 1: (322, 385, 8, 1), 2: (2052, None, 32, 4), 3: (10000, None, 64, 8),
          4: (50000, None, 128, 16)}


@pytest.fixture(scope="module")
def gmgs():
    return {cid: synth.build_gmg(cid) for cid in range(5)}


@pytest.mark.parametrize("cid", range(5))
def test_config_shapes(gmgs, cid):
    g = gmgs[cid]
    N, E, D, R = COUNTS[cid]
    assert (g.n_ops, g.n_dev, g.n_req) == (N, D, R)
    if E is not None:
        assert g.n_edges == E
    for u, v in g.edges():
        assert 0 <= u < v
    assert g.dur.min() >= 1 and g.out_bytes.min() >= 0
    assert g.pred_ptr[0] == 0 and np.all(np.diff(g.pred_ptr) >= 0)
    # every device: sorted, disjoint, non-empty idle slices and an open tail
    S = synth.CONFIGS[cid].n_slices
    for d in range(D):
        lo, hi = g.slice_ptr[d], g.slice_ptr[d + 1]
        assert hi - lo == S + 1
        b, e = g.slice_begin[lo:hi], g.slice_end[lo:hi]
        assert e[-1] == TIME_INF and np.all(e[:-1] < TIME_INF)
        assert np.all(b < e) and np.all(e[:-1] <= b[1:]) and b[0] >= 0
    # deadlines: release + ceil(f * isolated makespan) with f in [1.2, 2.0]
    iso = np.bincount(g.op_req, weights=g.dur[:, 0], minlength=R).astype(np.int64)
    assert np.all(g.deadline >= g.release + (6 * iso) // 5) and np.all(g.deadline <= g.release + 2 * iso + 1)


def test_llama8b_decode_magnitudes(gmgs):
    g = gmgs[1]
    by_kind = {}
    for v, k in enumerate(g.kinds):
        by_kind.setdefault(k, set()).add(int(g.dur[v, 0]))
    assert by_kind["qkv"] == {7} and by_kind["attn"] == {17} and by_kind["o_proj"] == {5}
    assert by_kind["gate_up"] == {30} and by_kind["down"] == {15} and by_kind["lm_head"] == {132}
    assert int(g.dur.sum()) == 2661
    assert g.deadline[0] == (3 * 2661 + 1) // 2


def test_idle_slice_statistics(gmgs):
    """Idle-slice median near the trace's 2551 ms and about 64% utilisation."""
    g = gmgs[4]
    idle, busy = [], []
    for d in range(g.n_dev):
        lo, hi = g.slice_ptr[d], g.slice_ptr[d + 1]
        b, e = g.slice_begin[lo:hi], g.slice_end[lo:hi]
        idle += (e[1:-1] - b[1:-1]).tolist()
        busy += (b[1:] - e[:-1]).tolist()
    idle, busy = np.array(idle), np.array(busy)
    assert idle.min() >= 10_000 and idle.max() <= 20_000_000
    assert abs(np.median(idle) / 2_551_110 - 1) < 0.05
    util = busy.sum() / (busy.sum() + idle.sum())
    assert 0.58 < util < 0.70


@pytest.mark.parametrize("cid", range(5))
def test_placements_deterministic_and_in_range(gmgs, cid):
    g = gmgs[cid]
    b0, nb = 5, 40
    a = synth.placements(g, cid, b0, nb)
    b = synth.placements(g, cid, 0, b0 + nb)[b0:]
    assert np.array_equal(a, b)
    assert a.max() < g.n_dev
    one_thread = synth.placements(g, cid, b0, nb, n_threads=1)
    assert np.array_equal(a, one_thread)


@pytest.mark.parametrize("cid", [2, 3, 4])
def test_perturbations_move_few_ops(gmgs, cid):
    g = gmgs[cid]
    base = synth.base_placement(g, cid)
    rec = synth.CONFIGS[cid].placement
    P = synth.placements(g, cid, 0, 64)
    for b in range(64):
        if (b % 2 == 0 and rec["mode_even"] == 0) or (b % 2 == 1 and rec["mode_odd"] == 0):
            continue
        moved = int((P[b] != base).sum())
        assert moved <= rec["kmax"]
        if rec["distinct"]:
            assert moved >= 1


def test_base_placement_keeps_each_request_on_its_node(gmgs):
    for cid in (2, 3, 4):
        g = gmgs[cid]
        cfg = synth.CONFIGS[cid]
        dpn = g.n_dev // cfg.n_nodes
        base = synth.base_placement(g, cid)
        assert np.all(base // dpn == g.op_req % cfg.n_nodes)


def test_counter_based_draws_match_c_generator():
    lib = synth._get_lib()
    for key in (0, 1, 123456789, synth.M64):
        for n in (0, 1, 7, 10 ** 9):
            assert lib.synth_draw(key, n) == synth.draw(key, n)


@pytest.mark.slow
def test_tight_capacity_constant_reproduces():
    import importlib.util
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "calibrate_memory_cap.py")
    spec = importlib.util.spec_from_file_location("calib", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert mod.compute() == synth.TIGHT_CAP_BYTES


def test_random_gmg_outdeg_cap():
    g = synth.random_gmg(5, n_ops=400, n_dev=4, edge_p=0.6, max_span=10, max_outdeg=2)
    assert np.bincount(np.asarray(g.pred_idx), minlength=g.n_ops).max() <= 2
    base = synth.random_gmg(5, n_ops=400, n_dev=4, edge_p=0.6, max_span=10)
    assert base.n_edges > g.n_edges
    assert np.array_equal(base.dur, g.dur)  # the cap changes no draw
