"""The incremental scheduling loop (ss_sched_*, Alg. 1, Sec. 3.4) on the GPU
against the oracle loop (oracle/sched.py): the same run is driven through
both, with the same executor feedback, and every round must agree exactly on
its status, its batch and the chosen partition, and the op states and devices
on the final state.  Cases: three workloads with their partition tables,
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


def drive_both(g, part, prio, budget, cap, key, require_sla=False, max_rounds=10_000):
    O = osch.Scheduler(g, part, prio, budget, cap, require_sla)
    L = ss.Scheduler(g, part, prio, budget, cap, require_sla)
    step = rounds = 0
    try:
        while rounds < max_rounds:
            rounds += 1
            a = O.round()
            b = L.round()
            assert b == a, f"round {rounds}: library {b[0], b[2], b[1][:8]} oracle {a[0], a[2], a[1][:8]}"
            if a[0] == osch.ROUND_ISSUED:
                continue
            issued = np.nonzero(O.state == osch.ISSUED)[0]
            if len(issued) == 0:
                break
            for v in synth.completion_feedback(issued, key, step):
                O.complete(v)
                L.complete(v)
            step += 1
        st, pl = L.state()
        assert np.array_equal(st, O.state) and np.array_equal(pl, O.place)
        return rounds
    finally:
        L.free()


@pytest.mark.parametrize("cid,budget,cap", [(0, 8, 5), (1, 64, 40), (2, 600, 150), (2, 300, 400)])
def test_workload_runs_match_the_oracle(dev, cid, budget, cap):
    print(f"incremental loop, workload {cid}, budget {budget}, cap {cap}", flush=True)
    g = synth.build_gmg(cid)
    rounds = drive_both(g, synth.partition_table(g, cid), synth.request_priority(g), budget, cap, key=cid)
    assert rounds > 2


@pytest.mark.parametrize("seed", range(6))
def test_random_runs_match_the_oracle(dev, seed):
    g = synth.random_gmg(800 + seed, n_ops=70 + 20 * seed, n_dev=3 + seed, n_req=1 + seed % 3, n_slices=3,
                         n_link=2, cap_scale=3000 + 1000 * seed)
    rng = np.random.default_rng(seed)
    part = rng.integers(0, g.n_dev, (1 + 3 * seed, g.n_ops)).astype(np.uint8)
    prio = rng.integers(0, 4, g.n_req)
    drive_both(g, part, prio, budget=5 + 3 * seed, cap=1 + 4 * seed, key=seed, require_sla=(seed % 2 == 1))


def test_infeasible_batch(dev):
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[5], [5]], [100, 100], [[(0, TIME_INF)]] * 2, [150, 150], [0],
                 [99], bw=(10,), lat=(0,))
    part = np.array([[0, 0], [1, 1], [0, 1]], np.uint8)
    L = ss.Scheduler(g, part, [0], 10, 2)
    assert L.round() == (ss.SS_ROUND_INFEASIBLE, [0, 1], -1)
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
    with pytest.raises(ss.SSError):
        L.complete(0)  # not issued
    st, batch, p = L.round()
    assert st == ss.SS_ROUND_ISSUED
    L.complete(batch[0])
    with pytest.raises(ss.SSError):
        L.complete(batch[0])  # already done
    L.free()
