"""Parity of the HIP path with the oracle on GMGs that hold a running
schedule's state (done ops with recorded finishes, issue times, the
snapshot's timestamp; Sec. 3.2, 3.3.2).  Such a GMG takes the general
index-order kernels; every output is compared bit for bit, over batches that
span several waves with a ragged tail, through the pooled, workspace and
op-major entry points and the resumed simulation; the dispatch and link
rules it does not take are refused."""
import copy

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def gpu_run(h, P, dev, **kw):
    Pt = torch.from_numpy(np.ascontiguousarray(P)).to(dev)
    out = ss.simulate_batch(h, Pt, **kw)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def assert_same(gpu, ref, label=""):
    for f in FIELDS:
        a, b = gpu.get(f), ref[f]
        if a is None:
            continue
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[:5]
            pytest.fail(f"{label}: {f} differs at {bad.tolist()}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}")


CASES = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_class=C, n_link=K, rel_max=rel, cap_scale=cs)
         for n, D, R, S, C, K, rel, cs in [(1, 1, 1, 0, 1, 1, 0, None), (12, 2, 1, 2, 1, 1, 0, 400),
                                           (60, 4, 2, 3, 2, 2, 30, 2000), (150, 7, 3, 5, 1, 3, 0, 4000),
                                           (301, 12, 4, 6, 2, 2, 80, 9000)]]
SNAPS = [dict(done_p=0.0), dict(done_p=0.5), dict(done_p=0.9, issue_span=50), dict(done_p=0.6, issue=False),
         dict(done_p=0.3, t_now=0), dict(done_p=1.0)]


@pytest.mark.parametrize("ci", range(len(CASES)))
@pytest.mark.parametrize("si", range(len(SNAPS)))
def test_running_schedule_parity(dev, ci, si):
    print(f"snapshot case {ci}, state {si}", flush=True)
    g = synth.random_gmg(1200 + ci, **CASES[ci])
    h = synth.random_snapshot(g, 31 * ci + si, **SNAPS[si])
    B = 197
    P = np.random.default_rng(ci * 10 + si).integers(0, g.n_dev, (B, g.n_ops)).astype(np.uint8)
    P[5, :] = g.n_dev - 1
    P[7, 0] = g.n_dev  # an invalid candidate
    ref = oracle.simulate_batch(h, P)
    hg = ss.Gmg(h)
    try:
        assert_same(gpu_run(hg, P, dev), ref, f"case {ci} state {si}")
        if si == 1:
            assert_same(gpu_run(hg, P.T.copy(), dev, layout="op"), ref, "op-major")
            n = ss.workspace_size(hg, B)[0]
            ws = torch.empty(n, dtype=torch.uint8, device=dev)
            assert_same(gpu_run(hg, P, dev, workspace=ws), ref, "workspace")
    finally:
        hg.free()


def test_hand_case_on_the_gpu(dev):
    # the transfer of a done output waits for its consumer's issue (the
    # oracle's hand-derived case): op1 starts at 105, finishes at 109
    g = make_gmg(2, ["op"] * 2, [(0, 1)], [0, 0], [[3], [4]], [10, 1], [[(0, TIME_INF)]] * 2, [100, 100], [0], [500],
                 bw=(2,), lat=(0,))
    g.done_fin = np.array([10, -1], np.int64)
    g.issue_at = np.array([0, 100], np.int64)
    P = np.array([[0, 1], [0, 0], [1, 1]], np.uint8)
    ref = oracle.simulate_batch(g, P)
    assert ref["makespan"].tolist()[0] == 109
    hg = ss.Gmg(g)
    try:
        assert_same(gpu_run(hg, P, dev), ref, "hand case")
    finally:
        hg.free()


def test_cluster_graph_with_a_running_schedule(dev):
    """The 4,000-op workload with half its ops done: sampled candidates of a
    1,024-candidate batch against the oracle, one by one."""
    print("workload 2 with a running schedule", flush=True)
    g = synth.build_gmg(2)
    h = synth.random_snapshot(g, 7, done_p=0.7, issue_span=2000)
    P = synth.placements(g, 2, 0, 1024)
    hg = ss.Gmg(h)
    try:
        got = gpu_run(hg, P, dev)
    finally:
        hg.free()
    idx = [0, 1, 63, 64, 65, 511, 1022, 1023]
    ref = oracle.simulate_batch(h, P[idx], n_threads=8)
    for f in FIELDS:
        assert np.array_equal(got[f][idx], ref[f]), f


def test_resume_from_a_running_schedule(dev):
    """Candidates that share the first k ops, resumed from the state captured
    after them, agree with the full simulation when the later ops are issued
    no earlier than the first k (the incremental loop's order)."""
    g = synth.random_gmg(1300, n_ops=120, n_dev=5, n_req=2, n_slices=3, n_link=2)
    k = 70
    h = synth.random_snapshot(g, 3, done_p=0.5, issue_span=400)
    h.done_fin[k:] = -1
    h.issue_at[k:] = 401 + np.random.default_rng(5).integers(0, 300, g.n_ops - k)
    rng = np.random.default_rng(4)
    P = rng.integers(0, g.n_dev, (150, g.n_ops)).astype(np.uint8)
    P[:, :k] = P[0, :k]
    ref = oracle.simulate_batch(h, P)
    pre = copy.deepcopy(h)
    keep = np.arange(k)
    pre.n_ops = k
    pre.pred_ptr = h.pred_ptr[:k + 1].copy()
    pre.pred_idx = h.pred_idx[:h.pred_ptr[k]].copy()
    pre.op_req, pre.dur, pre.out_bytes = h.op_req[keep], h.dur[keep], h.out_bytes[keep]
    pre.done_fin, pre.issue_at = h.done_fin[keep], h.issue_at[keep]
    gp, gf = ss.Gmg(pre), ss.Gmg(h)
    st = ss.State()
    try:
        ss.state_capture(gp, torch.from_numpy(P[0, :k].copy()).to(dev), st)
        Pt = torch.from_numpy(P).to(dev)
        out = ss.simulate_batch_resume(gf, Pt, start=st)
        torch.cuda.synchronize()
        assert_same({k_: (None if v is None else v.cpu().numpy()) for k_, v in out.items()}, ref, "resumed")
    finally:
        st.free()
        gp.free()
        gf.free()


def test_other_rules_are_refused(dev):
    g = synth.random_gmg(1400, n_ops=20, n_dev=3)
    h = synth.random_snapshot(g, 0)
    hg = ss.Gmg(h)
    P = torch.zeros((4, g.n_ops), dtype=torch.uint8, device=dev)
    try:
        for kw in (dict(dispatch="ready"), dict(links="ports")):
            with pytest.raises(ss.SSError) as e:
                ss.simulate_batch(hg, P, **kw)
            assert e.value.code == ss.SS_ERR_UNSUPPORTED
    finally:
        hg.free()
