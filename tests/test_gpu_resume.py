"""Prefix reuse (ss_simulate_batch_resume, ss_state_capture, ss_state_*):
candidates that share their first k ops resumed from the captured state of one
schedule of those ops must give exactly what ss_simulate_batch gives on the
whole GMG (and the oracle).  Cases: prefixes of every length class (0, inside, all ops) on the
workloads and random graphs, chains of captures that extend each other,
invalid devices inside and after the prefix, and the argument errors."""
import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def truncate(g, k):
    """The GMG of g's first k ops (their predecessors all lie among them)."""
    e = int(g.pred_ptr[k])
    return type(g)(k, g.n_dev, g.n_class, g.n_link, g.n_req, g.pred_ptr[:k + 1].copy(), g.pred_idx[:e].copy(),
                   g.op_req[:k].copy(), g.dur[:k].copy(), g.out_bytes[:k].copy(), g.dev_class, g.link_class, g.bw,
                   g.lat, g.slice_ptr, g.slice_begin, g.slice_end, g.cap, g.release, g.deadline)


def host(out):
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def same(a, b, label):
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f"{label}: {f}"


def shared_prefix_batch(g, k, B, seed):
    rng = np.random.default_rng(seed)
    P = rng.integers(0, g.n_dev, (B, g.n_ops)).astype(np.uint8)
    P[:, :k] = P[0, :k]
    return P


def capture_prefix(g, row, k, dev):
    st = ss.State()
    if k > 0:
        hk = ss.Gmg(truncate(g, k))
        ss.state_capture(hk, torch.from_numpy(row[:k].copy()).to(dev), st)
        torch.cuda.synchronize()
        assert st.n_ops() == k
        hk.free()
    return st


CASES = [("cfg", 0, None), ("cfg", 1, None), ("cfg", 2, None)] + [("rnd", s, dict(
    n_ops=n, n_dev=D, n_req=R, n_slices=S, n_link=K, cap_scale=cs, rel_max=rel))
    for s, (n, D, R, S, K, cs, rel) in enumerate([(60, 3, 2, 3, 1, 2000, 0), (150, 7, 3, 5, 2, 5000, 9),
                                                  (333, 12, 4, 8, 2, 20000, 30)])]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("frac", [0.0, 0.37, 0.9, 1.0])
def test_resume_equals_a_full_simulation(dev, case, frac):
    kind, key, kw = CASES[case]
    g = synth.build_gmg(key) if kind == "cfg" else synth.random_gmg(950 + key, **kw)
    k = int(round(frac * g.n_ops))
    print(f"resume: {kind} {key}, prefix {k} of {g.n_ops}", flush=True)
    P = shared_prefix_batch(g, k, 130, key * 10 + int(frac * 100))
    h = ss.Gmg(g)
    st = capture_prefix(g, P[0], k, dev)
    Pt = torch.from_numpy(P).to(dev)
    got = host(ss.simulate_batch_resume(h, Pt, start=st))
    full = host(ss.simulate_batch(h, Pt))
    same(got, full, "resume vs full")
    same(got, oracle.simulate_batch(g, P, n_threads=8), "resume vs oracle")
    st.free()
    h.free()


def test_captures_that_extend_each_other(dev):
    """Capture after k1 ops, resume the k2-op GMG from it with a capture, then
    resume the whole GMG: a chain of rounds as the incremental loop runs it."""
    g = synth.build_gmg(2)
    k1, k2 = 500, 1300
    P = shared_prefix_batch(g, k2, 64, 5)
    st1 = capture_prefix(g, P[0], k1, dev)
    st2 = ss.State()
    h2 = ss.Gmg(truncate(g, k2))
    ss.state_capture(h2, torch.from_numpy(P[0, :k2].copy()).to(dev), st2, start=st1)
    torch.cuda.synchronize()
    assert st2.n_ops() == k2
    h = ss.Gmg(g)
    Pt = torch.from_numpy(P).to(dev)
    same(host(ss.simulate_batch_resume(h, Pt, start=st2)), host(ss.simulate_batch(h, Pt)), "chained")
    for x in (st1, st2, h2, h):
        x.free()


def test_invalid_devices_inside_and_after_the_prefix(dev):
    g = synth.random_gmg(951, **CASES[4][2])
    k = 70
    P = shared_prefix_batch(g, k, 40, 9)
    st = capture_prefix(g, P[0], k, dev)
    P[3, 10] = g.n_dev + 1   # inside the shared prefix (this row breaks the contract on purpose: flagged anyway)
    P[7, 100] = 250          # after it
    h = ss.Gmg(g)
    Pt = torch.from_numpy(P).to(dev)
    got = host(ss.simulate_batch_resume(h, Pt, start=st))
    assert got["violation"][3] == 4 and got["violation"][7] == 4
    full = host(ss.simulate_batch(h, Pt))
    keep = np.ones(len(P), bool)
    keep[3] = False
    for f in FIELDS:
        assert np.array_equal(got[f][keep], full[f][keep]), f
    st.free()
    h.free()


def test_argument_errors(dev):
    g = synth.build_gmg(1)
    h = ss.Gmg(g)
    P = shared_prefix_batch(g, 100, 4, 3)
    st = capture_prefix(g, P[0], 100, dev)
    Pt = torch.from_numpy(P).to(dev)
    other = ss.State()
    with pytest.raises(ss.SSError):  # capture into the state resumed from
        ss.state_capture(h, Pt[0], st, start=st)
    g2 = synth.build_gmg(0)  # other device and request counts
    h2 = ss.Gmg(g2)
    with pytest.raises(ss.SSError):
        ss.simulate_batch_resume(h2, torch.zeros((2, g2.n_ops), dtype=torch.uint8, device=dev), start=st)
    small = ss.Gmg(truncate(g, 50))  # fewer ops than the state holds
    with pytest.raises(ss.SSError):
        ss.simulate_batch_resume(small, torch.zeros((2, 50), dtype=torch.uint8, device=dev), start=st)
    for x in (st, other, h, h2, small):
        x.free()
