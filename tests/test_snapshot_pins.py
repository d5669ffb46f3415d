"""Pins of the oracle's snapshot semantics (Sec. 3.2 scheduling metadata: the
issued and done timestamps of every op; Sec. 3.3.2: the simulator is built
from the snapshot).  A done op is not simulated: it finished at its recorded
time on its device, which is free from then on, and its output counts from
that time minus its estimate.  An op does not start before it was issued.
The transfer of an output to a device does not start before the first of
its consumers there was issued, because its Intent exists only from then on.

Expected values are hand derivations (each case states its arithmetic) and
properties that must hold for any GMG: a prefix of ops marked done at the
finish times the full simulation gives them changes nothing; issue times
equal to a release act as that release; raising an issue time never moves
a finish earlier.
"""
import copy

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd.synth import TIME_INF, make_gmg, random_gmg

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


def with_snapshot(g, done=None, issue=None):
    g = copy.deepcopy(g)
    N = g.n_ops
    g.done_fin = None if done is None else np.asarray(done, np.int64).reshape(N)
    g.issue_at = None if issue is None else np.asarray(issue, np.int64).reshape(N)
    return g


def test_done_op_frees_its_device_at_its_recorded_time():
    # op0 done on d0 at 100 (estimate 10); op1 on d0, issued at 50, no inputs:
    # it runs after the device is free, [100, 105)
    g = make_gmg(1, ["op"] * 2, [], [0, 0], [[10], [5]], [7, 3], [[(0, TIME_INF)]], [100], [0], [500])
    s = with_snapshot(g, done=[100, -1], issue=[0, 50])
    out = oracle.simulate_one(s, np.array([0, 0], np.uint8))
    assert out["fin"].tolist() == [100, 105] and out["st"].tolist() == [90, 100]
    # memory: own op0 [90, INF) 7 B (no consumer: retained), own op1 [100, INF) 3 B -> 10
    assert out["peak"].tolist() == [10]
    assert out["makespan"] == 105 and out["sumfin"] == 205


def test_issue_time_bounds_the_start():
    # op0 issued at 200 on an idle device: starts at 200, not 0
    g = make_gmg(1, ["op"], [], [0], [[4]], [1], [[(0, TIME_INF)]], [10], [0], [1000])
    out = oracle.simulate_one(with_snapshot(g, issue=[200]), np.array([0], np.uint8))
    assert out["st"].tolist() == [200] and out["fin"].tolist() == [204] and out["slack"].tolist() == [796]


def test_transfer_of_a_done_output_starts_at_the_consumers_issue():
    # op0 done on d0 at 10 (10 B); op1 on d1 consumes it, issued at 100;
    # X = ceil(10 / 2) = 5: the transfer starts at max(10, 100) = 100, op1 at 105
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[3], [4]], [10, 1], [[(0, TIME_INF)]] * 2, [100, 100], [0], [500],
                 bw=(2,), lat=(0,))
    s = with_snapshot(g, done=[10, -1], issue=[0, 100])
    out = oracle.simulate_one(s, np.array([0, 1], np.uint8))
    assert out["st"].tolist() == [7, 105] and out["fin"].tolist() == [10, 109]
    # memory: d0 own op0 [7, 105) (freed at the arrival) 10 B -> 10;
    # d1 copy of op0 [100, 109) 10 B + own op1 [105, INF) 1 B -> 11
    assert out["peak"].tolist() == [10, 11]
    # without the snapshot the same graph runs from 0: op1 starts at 3 + 5
    plain = oracle.simulate_one(g, np.array([0, 1], np.uint8))
    assert plain["st"].tolist() == [0, 8]


def test_shared_transfer_starts_with_the_first_issued_consumer():
    # op0 done on d0 at 20 (8 B, X = 4 at 2 B/us); op1 (issued at 30) and op2
    # (issued at 60) both on d1 read op0: one transfer, started at
    # max(20, min(30, 60)) = 30, arriving at 34; op1 [34, 35), op2 issued at 60:
    # [60, 61)
    g = make_gmg(2, ["op"] * 3, [(0, 1), (0, 2)], [0] * 3, [[5], [1], [1]], [8, 0, 0], [[(0, TIME_INF)]] * 2,
                 [100, 100], [0], [500], bw=(2,), lat=(0,))
    s = with_snapshot(g, done=[20, -1, -1], issue=[0, 30, 60])
    out = oracle.simulate_one(s, np.array([0, 1, 1], np.uint8))
    assert out["st"].tolist() == [15, 34, 60] and out["fin"].tolist() == [20, 35, 61]
    # d1: the copy [30, 61) 8 B -> 8; d0: own op0 [15, 34) 8 B -> 8
    assert out["peak"].tolist() == [8, 8]


def test_issued_op_waits_for_a_done_local_input_and_the_device():
    # d0: op0 done at 40; op1 done at 70 (the device ran it after op0); op2
    # issued at 0 reads op0 locally: ready 40, but the device is free only
    # from 70 -> [70, 72)
    g = make_gmg(1, ["op"] * 3, [(0, 2)], [0] * 3, [[10], [10], [2]], [5, 5, 5], [[(0, TIME_INF)]], [100], [0],
                 [500])
    s = with_snapshot(g, done=[40, 70, -1], issue=[0, 0, 0])
    out = oracle.simulate_one(s, np.array([0, 0, 0], np.uint8))
    assert out["fin"].tolist() == [40, 70, 72]
    # memory: own op0 [30, 72) 5, own op1 [60, INF) 5, own op2 [70, INF) 5 -> 15
    assert out["peak"].tolist() == [15]


def test_snapshot_is_refused_with_other_dispatch_rules():
    g = make_gmg(1, ["op"], [], [0], [[4]], [1], [[(0, TIME_INF)]], [10], [0], [1000])
    with pytest.raises(ValueError):
        oracle.simulate_one(with_snapshot(g, issue=[5]), np.array([0], np.uint8), oracle.READY_ORDER)


GRAPHS = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_class=C, n_link=K, rel_max=0)
          for n, D, R, S, C, K in [(12, 2, 1, 2, 1, 1), (40, 3, 2, 3, 2, 2), (90, 5, 3, 4, 1, 2), (150, 7, 2, 5, 2, 3)]]


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_done_prefix_at_simulated_times_changes_nothing(gi):
    """Marking the first k ops done at the finish times the full simulation
    gives them reproduces every output: the rest of the schedule, the peaks,
    the slack, the sums."""
    g = random_gmg(700 + gi, **GRAPHS[gi])
    rng = np.random.default_rng(gi)
    for b in range(12):
        p = rng.integers(0, g.n_dev, g.n_ops).astype(np.uint8)
        full = oracle.simulate_one(g, p)
        for k in (0, 1, g.n_ops // 3, g.n_ops - 1, g.n_ops):
            done = np.where(np.arange(g.n_ops) < k, full["fin"], -1)
            snap = oracle.simulate_one(with_snapshot(g, done=done), p)
            for f in ("st", "fin") + FIELDS:
                a, e = snap[f], full[f]
                assert np.array_equal(np.asarray(a), np.asarray(e)), (gi, b, k, f)


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_uniform_issue_time_acts_as_a_release(gi):
    """Every op issued at t with no release is the same as every request
    released at t: every transfer's producer finishes after t, so no transfer
    floor binds."""
    g = random_gmg(800 + gi, **GRAPHS[gi])
    t = 12345
    rel = copy.deepcopy(g)
    rel.release = np.full_like(g.release, t)
    snap = with_snapshot(g, issue=np.full(g.n_ops, t))
    P = np.random.default_rng(gi).integers(0, g.n_dev, (16, g.n_ops)).astype(np.uint8)
    a, b = oracle.simulate_batch(snap, P), oracle.simulate_batch(rel, P)
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_later_issue_never_finishes_earlier(gi):
    g = random_gmg(900 + gi, **GRAPHS[gi])
    rng = np.random.default_rng(50 + gi)
    for b in range(10):
        p = rng.integers(0, g.n_dev, g.n_ops).astype(np.uint8)
        iss = rng.integers(0, 3000, g.n_ops)
        lo = oracle.simulate_one(with_snapshot(g, issue=iss), p)
        iss2 = iss.copy()
        iss2[rng.integers(0, g.n_ops)] += int(rng.integers(1, 5000))
        hi = oracle.simulate_one(with_snapshot(g, issue=iss2), p)
        assert (hi["fin"] >= lo["fin"]).all()


def test_peak_counts_memory_from_the_snapshot_time():
    # d0 only.  op0 done at 10 (estimate 10, 7 B), read by op1 done at 20 (3 B,
    # no consumer: kept); op2 issued at 50 (4 B).  Residencies: op0 [0, 20),
    # op1 [10, inf), op2 [50, inf).  From t = 0 the peak is 7 + 3 = 10 (at 10);
    # from t_now = 30, op0 is gone and the peak is 3 + 4 = 7 (at 50).
    g = make_gmg(1, ["op"] * 3, [(0, 1)], [0] * 3, [[10], [10], [5]], [7, 3, 4], [[(0, TIME_INF)]], [100], [0],
                 [500])
    s = with_snapshot(g, done=[10, 20, -1], issue=[0, 0, 50])
    p = np.zeros(3, np.uint8)
    assert oracle.simulate_one(s, p)["peak"].tolist() == [10]
    s.t_now = 30
    out = oracle.simulate_one(s, p)
    assert out["peak"].tolist() == [7] and out["fin"].tolist() == [10, 20, 55]
    s.t_now = 10  # op0 still held at 10 (half-open [0, 20)): 10 again
    assert oracle.simulate_one(s, p)["peak"].tolist() == [10]
    s.t_now = 20  # op0 freed at 20 before anything else counts: 3, then 7 at 50
    assert oracle.simulate_one(s, p)["peak"].tolist() == [7]


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_snapshot_time_clips_only_the_peak(gi):
    """The snapshot time changes no schedule; the peak does not grow with it;
    beyond every finite residency end what remains is the outputs without
    consumers, on their devices."""
    g = random_gmg(1000 + gi, **GRAPHS[gi])
    rng = np.random.default_rng(70 + gi)
    has_succ = np.zeros(g.n_ops, bool)
    has_succ[g.pred_idx] = True
    for b in range(8):
        p = rng.integers(0, g.n_dev, g.n_ops).astype(np.uint8)
        base = oracle.simulate_one(g, p)
        prev = base["peak"]
        for t in sorted(rng.integers(0, int(base["makespan"]) + 1, 4).tolist()) + [1 << 40]:
            h = copy.deepcopy(g)
            h.t_now = t
            out = oracle.simulate_one(h, p)
            for f in ("st", "fin", "makespan", "slack", "sumfin"):
                assert np.array_equal(np.asarray(out[f]), np.asarray(base[f])), f
            assert (out["peak"] <= prev).all()
            prev = out["peak"]
        kept = np.zeros(g.n_dev, np.int64)
        np.add.at(kept, p[~has_succ], g.out_bytes[~has_succ])
        assert prev.tolist() == kept.tolist()
