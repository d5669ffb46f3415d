"""Pins of the incremental-loop oracle (Alg. 1, Sec. 3.4) against hand-derived
timed rounds and against the algorithm's definitions checked from scratch:
the budget and idle returns, the priority order, the batch rules (closure,
connection through successors, lowest-index growth, the cap), the snapshot a
round simulates (issued ops, done ops still feeding an op to run with their
recorded completions, the batch issued at the round's time; Sec. 3.2,
3.3.2), the choice of partition by brute force (every partition simulated on
its own with the C oracle's single-candidate call), the shared schedule of
the ops before the batch, the write-back, and the feedback rules.  Whole
runs are driven by the stand-in executor, which reports completions with
times.
"""
import numpy as np
import pytest

import oracle
from oracle import sched as osch
from paper_2608_15762_amd import synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

INF = TIME_INF


def two_device_chain(dev0_slices, dev1_slices, lat, bytes_):
    """Two instances of a 2-op chain (ops 0-1, then 2-3 after op 1) on two
    devices; partitions: 0 = every op on device 0, 1 = every op on device 1."""
    g = make_gmg(2, ["op"] * 4, [(0, 1), (1, 2), (2, 3)], [0] * 4, [[10]] * 4, [bytes_] * 4,
                 [dev0_slices, dev1_slices], [10 ** 9] * 2, [0], [10 ** 6], bw=(10,), lat=(lat,))
    part = np.array([[0, 0, 0, 0], [1, 1, 1, 1]], np.uint8)
    return g, part


def test_round_prefers_the_device_that_is_free():
    """Device 0 is busy until 30, device 1 is free: the first batch (cap 2,
    ops 0-1) finishes at 40, 50 on device 0 (sum 90) and 10, 20 on device 1
    (sum 30): partition 1."""
    g, part = two_device_chain([(30, INF)], [(0, INF)], 0, 0)
    S = osch.Scheduler(g, part, [0], budget=10, cap=2)
    assert S.round(0) == (osch.ROUND_ISSUED, [0, 1], 1)
    assert S.place[:2].tolist() == [1, 1] and S.state.tolist() == [1, 1, 0, 0]
    assert S.issue_t.tolist() == [0, 0, -1, -1]


@pytest.mark.parametrize("lat,expect", [(100, 1), (0, 0)])
def test_locality_against_a_busy_window(lat, expect):
    """Device 1 holds [0, 20) then is busy until 60; device 0 is idle from 30.
    Round 1 puts ops 0-1 on device 1 (finishes 10, 20 against 40, 50).
    Round 2 (ops 2-3, after op 1 at 20):
      - staying on device 1: [60, 70), [70, 80), sum of the batch 150;
      - moving to device 0: op 2 ready at 20 + X, X = lat + ceil(0/10) = lat;
        with lat = 100: [120, 130), [130, 140), sum 270 -> stay (locality);
        with lat = 0: [30, 40), [40, 50), sum 90 -> move."""
    g, part = two_device_chain([(30, INF)], [(0, 20), (60, INF)], lat, 0)
    S = osch.Scheduler(g, part, [0], budget=10, cap=2)
    assert S.round(0) == (osch.ROUND_ISSUED, [0, 1], 1)
    assert S.round(0) == (osch.ROUND_ISSUED, [2, 3], expect)


def late_op_graph():
    """Request 0: chain op 0 -> op 1 (10 us each); request 1: op 2 (10 us),
    after request 0 by priority.  No bytes, no latency.  Device 1 is idle in
    [0, 50) and from 300 on; device 0 always.  Partition 0 = device 0,
    partition 1 = device 1."""
    g = make_gmg(2, ["op"] * 3, [(0, 1)], [0, 0, 1], [[10]] * 3, [0] * 3, [[(0, INF)], [(0, 50), (300, INF)]],
                 [10 ** 6] * 2, [0, 0], [10 ** 6] * 2, bw=(10,), lat=(0,))
    return g, np.array([[0, 0, 0], [1, 1, 1]], np.uint8)


def test_a_late_completion_moves_the_next_batch():
    """Hand-derived timed rounds (budget 2, cap 1).
      round at 0: op 0; both partitions finish at 10 -> partition 0 (lower);
      round at 0: op 1 after op 0 on d0 [10, 20) (sum 30) or d1 [10, 20)
        (sum 30) -> partition 0;  round at 0: budget;
      op 0 completes at 100 (its estimate was 10);
      round at 100: op 2.  Snapshot: op 0 done at 100, op 1 issued at 0 on
        d0 -> [100, 110); op 2 issued at 100: on d0 [110, 120), sum 100 +
        110 + 120 = 330; on d1 the window [0, 50) has passed -> [300, 310),
        sum 520 -> partition 0.  (Simulated from t = 0 with estimates, as
        if nothing had run, op 2 would take d1 at [0, 10).)"""
    g, part = late_op_graph()
    S = osch.Scheduler(g, part, [0, 1], budget=2, cap=1)
    assert S.round(0) == (osch.ROUND_ISSUED, [0], 0)
    assert S.round(0) == (osch.ROUND_ISSUED, [1], 0)
    assert S.round(0) == (osch.ROUND_BUDGET, [], -1)
    S.complete(0, 100)
    sub, order = S.round_graph([2], 100)
    assert order == [0, 1, 2]
    assert sub.done_fin.tolist() == [100, -1, -1] and sub.issue_at.tolist() == [0, 0, 100] and sub.t_now == 100
    fins = [oracle.simulate_one(sub, np.array([0, 0, part[q, 2]], np.uint8))["fin"].tolist() for q in range(2)]
    assert fins == [[100, 110, 120], [100, 110, 310]]
    assert S.round(100) == (osch.ROUND_ISSUED, [2], 0)
    assert S.issue_t.tolist() == [0, 0, 100]


def test_done_history_leaves_the_snapshot():
    """Once op 0 and op 1 are done (op 0's only successor done, op 1 without
    successors), the next round's graph is its batch alone; a checkpoint
    producer (a done op with a successor still to run) stays."""
    g, part = late_op_graph()
    S = osch.Scheduler(g, part, [0, 1], budget=1, cap=1)
    assert S.round(0)[0] == osch.ROUND_ISSUED
    S.complete(0, 12)
    sub, order = S.round_graph([1], 12)
    assert order == [0, 1] and sub.done_fin.tolist() == [12, -1]  # op 0 feeds the batch: kept
    assert S.round(12) == (osch.ROUND_ISSUED, [1], 0)
    S.complete(1, 30)
    sub, order = S.round_graph([2], 40)
    assert order == [2] and sub.issue_at.tolist() == [40] and sub.done_fin.tolist() == [-1]
    # d0 from 40: [40, 50) sum 50; d1: [40, 50) fits the window [0, 50): sum 50 -> tie -> partition 0
    assert S.round(40) == (osch.ROUND_ISSUED, [2], 0)
    assert S.scheduled_frontier() == []


def test_budget_and_completion():
    g, part = two_device_chain([(0, INF)], [(0, INF)], 0, 0)
    S = osch.Scheduler(g, part, [0], budget=2, cap=2)
    st, batch, _ = S.round(0)
    assert st == osch.ROUND_ISSUED and batch == [0, 1]
    assert S.round(0) == (osch.ROUND_BUDGET, [], -1)       # 2 issued >= budget 2
    S.complete(0, 10)
    st, batch, _ = S.round(10)                              # 1 issued < 2: a full batch again
    assert st == osch.ROUND_ISSUED and batch == [2, 3]
    assert int((S.state == osch.ISSUED).sum()) == 3       # budget - 1 + cap at most
    S.complete(1, 20)
    S.complete(2, 30)
    S.complete(3, 40)
    assert S.round(40) == (osch.ROUND_IDLE, [], -1)


def test_feedback_and_time_rules():
    g, part = two_device_chain([(0, INF)], [(0, INF)], 0, 0)
    S = osch.Scheduler(g, part, [0], budget=4, cap=2)
    assert S.round(5)[1] == [0, 1]
    with pytest.raises(ValueError):
        S.round(4)  # time goes backwards
    with pytest.raises(ValueError):
        S.complete(2, 50)  # not issued
    with pytest.raises(ValueError):
        S.complete(1, 50)  # its predecessor is not done
    with pytest.raises(ValueError):
        S.complete(0, 5)  # not after its issue at 5
    S.complete(0, 6)
    with pytest.raises(ValueError):
        S.complete(1, 6)  # not after its predecessor
    S.complete(1, 7)


def test_round_graph_follows_issue_order():
    """Two independent requests issued high-priority first: the round graph
    lists the scheduled ops still in play in issue order (op 1, then op 0),
    then the batch."""
    g = make_gmg(2, ["op"] * 3, [(0, 2)], [0, 1, 0], [[5], [7], [3]], [1, 1, 1], [[(0, INF)]] * 2, [10 ** 6] * 2,
                 [0, 0], [100, 50], bw=(10,), lat=(0,))
    part = np.array([[0, 0, 0], [1, 1, 1]], np.uint8)
    S = osch.Scheduler(g, part, [100, 50], budget=10, cap=1)
    assert S.round(0) == (osch.ROUND_ISSUED, [1], 0)
    assert S.round(0) == (osch.ROUND_ISSUED, [0], 1)  # device 0 busy with op 1 until 7: device 1 finishes op 0 at 5
    sub, order = S.round_graph([2], 0)
    assert order == [1, 0, 2] and sub.dur[:, 0].tolist() == [7, 5, 3]
    # op 1 on d0 [0,7), op 0 on d1 [0,5); op 2 after op 0: on d1 [5,8) (sum 20) or d0 [7,10) (sum 22)
    assert S.round(0) == (osch.ROUND_ISSUED, [2], 1)


def test_infeasible_round_changes_nothing():
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[5], [5]], [100, 100], [[(0, INF)]] * 2, [150, 150], [0], [99],
                 bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1], [0, 1]], np.uint8)
    S = osch.Scheduler(g, part, [0], budget=10, cap=2)
    # on one device: op0 [0,5) kept until op1 ends (100 B) + op1's own output (100 B) = 200 > 150;
    # split: d0 holds op0 until its transfer arrives, d1 holds the copy and op1's output: 200 > 150
    st, batch, p = S.round(0)
    assert (st, batch, p) == (osch.ROUND_INFEASIBLE, [0, 1], -1)
    assert S.state.tolist() == [0, 0]


def test_priority_picks_the_request_first():
    """Two independent requests; request 1 has the smaller priority value and
    its op (index 1) goes first although op 0 has the lower index."""
    g = make_gmg(2, ["op"] * 2, [], [0, 1], [[5], [5]], [1, 1], [[(0, INF)]] * 2, [10 ** 6] * 2, [0, 0],
                 [100, 50], bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1]], np.uint8)
    S = osch.Scheduler(g, part, [100, 50], budget=10, cap=4)
    assert S.round(0)[1] == [1]
    assert S.round(0)[1] == [0]


def test_executor_feedback_is_causal():
    """The stand-in executor: completions in time order, each after its issue
    and its predecessors' completions; a run drains."""
    g = synth.build_gmg(0)
    X = synth.Executor(g, 3)
    X.issue(range(g.n_ops), np.zeros(g.n_ops, np.int64), 7)
    last, seen = 0, 0
    while (ev := X.next_completion()) is not None:
        t, v = ev
        assert t >= last and t > 7
        for e in range(g.pred_ptr[v], g.pred_ptr[v + 1]):
            assert 0 <= X.done_t[g.pred_idx[e]] < t
        last, seen = t, seen + 1
    assert seen == g.n_ops


# ------------------------------------------------------------------ whole runs, checked round by round
def run_checked(g, part, prio, budget, cap, key, require_sla=False, check_choice=True):
    S = osch.Scheduler(g, part, prio, budget, cap, require_sla)
    X = synth.Executor(g, key)
    preds = [[int(g.pred_idx[e]) for e in range(g.pred_ptr[v], g.pred_ptr[v + 1])] for v in range(g.n_ops)]
    succs = [[] for _ in range(g.n_ops)]
    for v in range(g.n_ops):
        for u in preds[v]:
            succs[u].append(v)
    issued_by = {}
    now = 0
    max_graph = 0
    while True:
        before = S.state.copy()
        n_issued = int((before == osch.ISSUED).sum())
        st, batch, p = S.round(now)
        if st == osch.ROUND_BUDGET:
            assert n_issued >= budget
        elif st == osch.ROUND_IDLE:
            assert (before != osch.UNSCHEDULED).all()
        else:
            assert n_issued < budget
            F = [v for v in range(g.n_ops) if before[v] == 0 and all(before[u] != 0 for u in preds[v])]
            top = min(F, key=lambda v: (int(prio[g.op_req[v]]), v))
            assert top in batch and len(batch) <= cap and batch == sorted(batch)
            inb = set(batch)
            for x in batch:  # closed, and reached through successors
                assert all(before[u] != 0 or u in inb for u in preds[x])
                assert x == top or any(u in inb for u in preds[x])
            if len(batch) < cap:  # nothing eligible was left out
                for b in batch:
                    for x in succs[b]:
                        if before[x] == 0 and x not in inb:
                            assert not all(before[u] != 0 or u in inb for u in preds[x])
            sub, order = S.round_graph(batch, now) if st == osch.ROUND_INFEASIBLE else \
                _graph_before(S, before, batch, now)
            # the snapshot: what is issued and not done, done ops still feeding
            # an op to run, the batch; bounded by the budget and the checkpoints
            npre = len(order) - len(batch)
            for v in order[:npre]:
                assert before[v] == osch.ISSUED or (before[v] == osch.DONE and
                                                    any(before[x] != osch.DONE for x in succs[v]))
            assert sum(before[v] == osch.ISSUED for v in order) == n_issued
            max_graph = max(max_graph, len(order))
            if check_choice:
                keys, fins = [], []
                for q in range(len(part)):
                    row = np.concatenate([S.place[order[:npre]], part[q, batch]]).astype(np.uint8)
                    r = oracle.simulate_one(sub, row)
                    ok = r["violation"] == 0 and (not require_sla or (r["slack"] >= 0).all())
                    keys.append(r["sumfin"] if ok else None)
                    fins.append(r["fin"][:npre])
                    assert (r["fin"][npre:] > now).all()  # the batch runs in the future
                for q in range(1, len(part)):  # the ops before the batch: one schedule for all
                    assert np.array_equal(fins[q], fins[0])
                feas = [(k, q) for q, k in enumerate(keys) if k is not None]
                if st == osch.ROUND_INFEASIBLE:
                    assert not feas
                else:
                    assert p == min(feas)[1]
            if st == osch.ROUND_ISSUED:
                assert (S.state[batch] == osch.ISSUED).all() and (S.issue_t[batch] == now).all()
                assert S.place[batch].tolist() == part[p, batch].tolist()
                for v in batch:
                    issued_by[v] = p
        if st == osch.ROUND_ISSUED:
            X.issue(batch, S.place[batch], now)
            continue
        ev = X.next_completion()
        if ev is None:
            break
        now, v = ev
        S.complete(v, now)
    assert (S.state == osch.DONE).sum() + (S.state == osch.ISSUED).sum() == g.n_ops or st == osch.ROUND_INFEASIBLE
    return S, issued_by, max_graph


def _graph_before(S, before, batch, now):
    """The round graph as it was before the write-back of an issued round."""
    saved, saved_order = S.state.copy(), list(S.issue_order)
    S.state[:] = before
    S.issue_order = saved_order[:len(saved_order) - len(batch)]
    try:
        return S.round_graph(batch, now)
    finally:
        S.state[:] = saved
        S.issue_order = saved_order


@pytest.mark.parametrize("cid,budget,cap", [(0, 8, 5), (1, 64, 40), (2, 600, 150)])
def test_workload_runs(cid, budget, cap):
    g = synth.build_gmg(cid)
    part = synth.partition_table(g, cid)
    S, issued_by, max_graph = run_checked(g, part, synth.request_priority(g), budget, cap, key=cid,
                                          check_choice=(cid < 2))
    assert (S.state == osch.DONE).sum() + (S.state == osch.ISSUED).sum() == g.n_ops
    assert len(issued_by) == g.n_ops
    assert max_graph < g.n_ops or g.n_ops <= budget + cap


@pytest.mark.parametrize("seed", range(4))
def test_random_runs(seed):
    g = synth.random_gmg(700 + seed, n_ops=60, n_dev=4, n_req=3, n_slices=3, n_link=2, cap_scale=4000)
    rng = np.random.default_rng(seed)
    part = rng.integers(0, g.n_dev, (5, g.n_ops)).astype(np.uint8)
    prio = rng.integers(0, 3, g.n_req)
    run_checked(g, part, prio, budget=12, cap=7, key=seed, require_sla=(seed == 3))
