"""Pins of the incremental-loop oracle (Alg. 1, Sec. 3.4) against hand-derived
rounds and against the algorithm's definitions checked from scratch: the
budget and idle returns, the priority order, the batch rules (closure,
connection through successors, lowest-index growth, the cap), the choice of
partition by brute force (every partition simulated on its own with the C
oracle's single-candidate call), the shared schedule of the ops before the
batch, and the write-back.
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
    assert S.round() == (osch.ROUND_ISSUED, [0, 1], 1)
    assert S.place[:2].tolist() == [1, 1] and S.state.tolist() == [1, 1, 0, 0]


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
    assert S.round() == (osch.ROUND_ISSUED, [0, 1], 1)
    assert S.round() == (osch.ROUND_ISSUED, [2, 3], expect)


def test_budget_and_completion():
    g, part = two_device_chain([(0, INF)], [(0, INF)], 0, 0)
    S = osch.Scheduler(g, part, [0], budget=2, cap=2)
    st, batch, _ = S.round()
    assert st == osch.ROUND_ISSUED and batch == [0, 1]
    assert S.round() == (osch.ROUND_BUDGET, [], -1)       # 2 issued >= budget 2
    S.complete(0)
    st, batch, _ = S.round()                              # 1 issued < 2: a full batch again
    assert st == osch.ROUND_ISSUED and batch == [2, 3]
    assert int((S.state == osch.ISSUED).sum()) == 3       # budget - 1 + cap at most
    S.complete(1)
    S.complete(2)
    S.complete(3)
    assert S.round() == (osch.ROUND_IDLE, [], -1)


def test_round_graph_follows_issue_order():
    """Two independent requests issued high-priority first: the round graph
    lists the scheduled ops in issue order (op 1, then op 0), which completion
    does not change, then the batch."""
    g = make_gmg(2, ["op"] * 3, [(0, 2)], [0, 1, 0], [[5], [7], [3]], [1, 1, 1], [[(0, INF)]] * 2, [10 ** 6] * 2,
                 [0, 0], [100, 50], bw=(10,), lat=(0,))
    part = np.array([[0, 0, 0], [1, 1, 1]], np.uint8)
    S = osch.Scheduler(g, part, [100, 50], budget=10, cap=1)
    assert S.round() == (osch.ROUND_ISSUED, [1], 0)
    assert S.round() == (osch.ROUND_ISSUED, [0], 1)  # device 0 busy with op 1 until 7: device 1 finishes op 0 at 5
    S.complete(1)
    sub, order = S.round_graph([2])
    assert order == [1, 0, 2] and sub.dur[:, 0].tolist() == [7, 5, 3]
    # op 1 on d0 [0,7), op 0 on d1 [0,5); op 2 after op 0: on d1 [5,8) (sum 20) or d0 [7,10) (sum 22)
    assert S.round() == (osch.ROUND_ISSUED, [2], 1)


def test_infeasible_round_changes_nothing():
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[5], [5]], [100, 100], [[(0, INF)]] * 2, [150, 150], [0], [99],
                 bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1], [0, 1]], np.uint8)
    S = osch.Scheduler(g, part, [0], budget=10, cap=2)
    # on one device: op0 [0,5) kept until op1 ends (100 B) + op1's own output (100 B) = 200 > 150;
    # split: d0 holds op0 until its transfer arrives, d1 holds the copy and op1's output: 200 > 150
    st, batch, p = S.round()
    assert (st, batch, p) == (osch.ROUND_INFEASIBLE, [0, 1], -1)
    assert S.state.tolist() == [0, 0]


def test_priority_picks_the_request_first():
    """Two independent requests; request 1 has the smaller priority value and
    its op (index 1) goes first although op 0 has the lower index."""
    g = make_gmg(2, ["op"] * 2, [], [0, 1], [[5], [5]], [1, 1], [[(0, INF)]] * 2, [10 ** 6] * 2, [0, 0],
                 [100, 50], bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1]], np.uint8)
    S = osch.Scheduler(g, part, [100, 50], budget=10, cap=4)
    assert S.round()[1] == [1]
    assert S.round()[1] == [0]


# ------------------------------------------------------------------ whole runs, checked round by round
def run_checked(g, part, prio, budget, cap, key, require_sla=False, check_choice=True):
    S = osch.Scheduler(g, part, prio, budget, cap, require_sla)
    preds = [[int(g.pred_idx[e]) for e in range(g.pred_ptr[v], g.pred_ptr[v + 1])] for v in range(g.n_ops)]
    succs = [[] for _ in range(g.n_ops)]
    for v in range(g.n_ops):
        for u in preds[v]:
            succs[u].append(v)
    step = 0
    issued_by = {}
    while True:
        before = S.state.copy()
        n_issued = int((before == osch.ISSUED).sum())
        st, batch, p = S.round()
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
            if check_choice:
                sub, order = S.round_graph(batch) if st == osch.ROUND_INFEASIBLE else _graph_before(S, before, batch)
                npre = len(order) - len(batch)
                keys, fins = [], []
                for q in range(len(part)):
                    row = np.concatenate([S.place[order[:npre]], part[q, batch]]).astype(np.uint8)
                    r = oracle.simulate_one(sub, row)
                    ok = r["violation"] == 0 and (not require_sla or (r["slack"] >= 0).all())
                    keys.append(r["sumfin"] if ok else None)
                    fins.append(r["fin"][:npre])
                for q in range(1, len(part)):  # the ops before the batch: one schedule for all
                    assert np.array_equal(fins[q], fins[0])
                feas = [(k, q) for q, k in enumerate(keys) if k is not None]
                if st == osch.ROUND_INFEASIBLE:
                    assert not feas
                else:
                    assert p == min(feas)[1]
            if st == osch.ROUND_ISSUED:
                assert (S.state[batch] == osch.ISSUED).all()
                assert S.place[batch].tolist() == part[p, batch].tolist()
                for v in batch:
                    issued_by[v] = p
        if st == osch.ROUND_ISSUED:
            continue
        issued = np.nonzero(S.state == osch.ISSUED)[0]
        if len(issued) == 0:
            break
        for v in synth.completion_feedback(issued, key, step):
            S.complete(v)
        step += 1
    assert (S.state == osch.DONE).sum() + (S.state == osch.ISSUED).sum() == g.n_ops or st == osch.ROUND_INFEASIBLE
    return S, issued_by


def _graph_before(S, before, batch):
    """The round graph as it was before the write-back of an issued round."""
    saved, saved_order = S.state.copy(), list(S.issue_order)
    S.state[:] = before
    S.issue_order = saved_order[:len(saved_order) - len(batch)]
    try:
        return S.round_graph(batch)
    finally:
        S.state[:] = saved
        S.issue_order = saved_order


@pytest.mark.parametrize("cid,budget,cap", [(0, 8, 5), (1, 64, 40), (2, 600, 150)])
def test_workload_runs(cid, budget, cap):
    g = synth.build_gmg(cid)
    part = synth.partition_table(g, cid)
    S, issued_by = run_checked(g, part, synth.request_priority(g), budget, cap, key=cid,
                               check_choice=(cid < 2))
    assert (S.state == osch.DONE).sum() + (S.state == osch.ISSUED).sum() == g.n_ops
    assert len(issued_by) == g.n_ops


@pytest.mark.parametrize("seed", range(4))
def test_random_runs(seed):
    g = synth.random_gmg(700 + seed, n_ops=60, n_dev=4, n_req=3, n_slices=3, n_link=2, cap_scale=4000)
    rng = np.random.default_rng(seed)
    part = rng.integers(0, g.n_dev, (5, g.n_ops)).astype(np.uint8)
    prio = rng.integers(0, 3, g.n_req)
    run_checked(g, part, prio, budget=12, cap=7, key=seed, require_sla=(seed == 3))
