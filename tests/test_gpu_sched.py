"""The incremental scheduling loop (ss_sched_*, Alg. 1, Sec. 3.4) on the GPU
against the oracle loop (oracle/sched.py): the same run is driven through
both, with the same timed executor feedback (rounds at the completion times,
snapshots with done ops and issue times), and every round must agree exactly
on its status, its batch and the chosen partition, and the op states,
devices, issue and completion times on the final state.  Cases: three workloads with their partition tables,
random graphs with random partitions and priorities, the SLA filter, an
infeasible batch, the budget, argument errors."""
import numpy as np
import pytest

from oracle import sched as osch
from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def drive_both(g, part, prio, budget, cap, key, require_sla=False, max_rounds=10_000, prefix_reuse=False):
    """Drive the library and the oracle through the same run, fed by the
    stand-in executor (completions with times), comparing every round."""
    O = osch.Scheduler(g, part, prio, budget, cap, require_sla)
    L = ss.Scheduler(g, part, prio, budget, cap, require_sla, prefix_reuse=prefix_reuse)
    X = synth.Executor(g, key)
    rounds = 0
    now = 0
    try:
        while rounds < max_rounds:
            rounds += 1
            a = O.round(now)
            b = L.round(now)
            assert b == a, f"round {rounds} at {now}: library {b[0], b[2], b[1][:8]} oracle {a[0], a[2], a[1][:8]}"
            if a[0] == osch.ROUND_ISSUED:
                X.issue(a[1], O.place[a[1]], now)
                continue
            ev = X.next_completion()
            if ev is None:
                break
            now, v = ev
            O.complete(v, now)
            L.complete(v, now)
        st, pl, it, dt = L.state()
        assert np.array_equal(st, O.state) and np.array_equal(pl, O.place)
        assert np.array_equal(it, O.issue_t) and np.array_equal(dt, O.done_t)
        return rounds
    finally:
        L.free()


@pytest.mark.parametrize("cid,budget,cap,reuse", [(0, 8, 5, False), (1, 64, 40, True), (2, 600, 150, False),
                                                  (2, 300, 400, True)])
def test_workload_runs_match_the_oracle(dev, cid, budget, cap, reuse):
    print(f"incremental loop, workload {cid}, budget {budget}, cap {cap}, prefix reuse {reuse}", flush=True)
    g = synth.build_gmg(cid)
    rounds = drive_both(g, synth.partition_table(g, cid), synth.request_priority(g), budget, cap, key=cid,
                        prefix_reuse=reuse)
    assert rounds > 2


@pytest.mark.parametrize("seed", range(6))
def test_random_runs_match_the_oracle(dev, seed):
    g = synth.random_gmg(800 + seed, n_ops=70 + 20 * seed, n_dev=3 + seed, n_req=1 + seed % 3, n_slices=3,
                         n_link=2, cap_scale=3000 + 1000 * seed)
    rng = np.random.default_rng(seed)
    part = rng.integers(0, g.n_dev, (1 + 3 * seed, g.n_ops)).astype(np.uint8)
    prio = rng.integers(0, 4, g.n_req)
    drive_both(g, part, prio, budget=5 + 3 * seed, cap=1 + 4 * seed, key=seed, require_sla=(seed % 2 == 1),
               prefix_reuse=(seed % 3 == 0))


def test_prefix_reuse_changes_no_decision(dev):
    """With and without prefix reuse the library takes the oracle's decisions."""
    g = synth.build_gmg(1)
    part, prio = synth.partition_table(g, 1), synth.request_priority(g)
    for reuse in (True, False):
        drive_both(g, part, prio, 64, 40, key=11, prefix_reuse=reuse)


def test_a_late_completion_moves_the_next_batch(dev):
    """The oracle's hand-derived timed rounds, on the library."""
    g = make_gmg(2, ["op"] * 3, [(0, 1)], [0, 0, 1], [[10]] * 3, [0] * 3, [[(0, TIME_INF)], [(0, 50), (300, TIME_INF)]],
                 [10 ** 6] * 2, [0, 0], [10 ** 6] * 2, bw=(10,), lat=(0,))
    part = np.array([[0, 0, 0], [1, 1, 1]], np.uint8)
    L = ss.Scheduler(g, part, [0, 1], 2, 1)
    try:
        assert L.round(0) == (ss.SS_ROUND_ISSUED, [0], 0)
        assert L.round(0) == (ss.SS_ROUND_ISSUED, [1], 0)
        assert L.round(0) == (ss.SS_ROUND_BUDGET, [], -1)
        L.complete(0, 100)
        assert L.round(100) == (ss.SS_ROUND_ISSUED, [2], 0)
        assert L.state()[2].tolist() == [0, 0, 100]
    finally:
        L.free()


def test_infeasible_batch(dev):
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[5], [5]], [100, 100], [[(0, TIME_INF)]] * 2, [150, 150], [0],
                 [99], bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1], [0, 1]], np.uint8)
    L = ss.Scheduler(g, part, [0], 10, 2)
    assert L.round(0) == (ss.SS_ROUND_INFEASIBLE, [0, 1], -1)
    assert L.state()[0].tolist() == [0, 0]
    L.free()


def test_argument_errors(dev):
    g = synth.build_gmg(0)
    part = synth.partition_table(g, 0)
    with pytest.raises(ss.SSError):
        ss.Scheduler(g, part, synth.request_priority(g), 0, 4)
    bad = part.copy()
    bad[0, 3] = g.n_dev
    with pytest.raises(ss.SSError):
        ss.Scheduler(g, bad, synth.request_priority(g), 4, 4)
    L = ss.Scheduler(g, part, synth.request_priority(g), 4, 4)
    try:
        with pytest.raises(ss.SSError):
            L.complete(0, 5)  # not issued
        st, batch, p = L.round(10)
        assert st == ss.SS_ROUND_ISSUED
        with pytest.raises(ss.SSError):
            L.round(9)  # time goes backwards
        with pytest.raises(ss.SSError):
            L.complete(batch[0], 10)  # not after its issue
        L.complete(batch[0], 11)
        with pytest.raises(ss.SSError):
            L.complete(batch[0], 12)  # already done
    finally:
        L.free()
