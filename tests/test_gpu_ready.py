"""Parity of the ready-time dispatch rule (Sec. 3.3.2) on the GPU with the
oracle's READY_ORDER schedule, element by element through the C ABI.

Integer results: bit-exact on every output.  Cases: the seeded workloads,
random graphs of every shape class (several device and link classes, fan-in
and fan-out, zero-byte outputs), graphs inside the branch-free interval
writer's limits, a fan-out wide enough to overflow the ready set kept in
registers, empty inputs and placements naming unknown devices.
"""
import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


@pytest.fixture(params=["auto", "generic"])
def path(request, monkeypatch):
    """Run a case on the default path (the 32-bit path when the GMG qualifies)
    and on the general int64 path."""
    if request.param == "generic":
        monkeypatch.setenv("SS_PATH", "generic")
    else:
        monkeypatch.delenv("SS_PATH", raising=False)
    return request.param


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def gpu_run(h, P, dev, dispatch="ready", **kw):
    Pt = torch.from_numpy(np.ascontiguousarray(P)).to(dev)
    out = ss.simulate_batch(h, Pt, dispatch=dispatch, **kw)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def assert_same(gpu, ref, idx=None, label=""):
    for f in FIELDS:
        if gpu.get(f) is None:
            continue
        a = gpu[f] if idx is None else gpu[f][idx]
        b = ref[f]
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[:5]
            pytest.fail(f"{label}: {f} differs at {bad.tolist()}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}")


def random_placements(g, seed, B, invalid_every=0):
    st = synth.Stream(seed)
    P = np.array([[st.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)] for _ in range(B)], np.uint8)
    if invalid_every:
        for b in range(0, B, invalid_every):
            P[b, st.uniform_int(0, g.n_ops - 1)] = g.n_dev + st.uniform_int(0, 255 - g.n_dev)
    return P


@pytest.mark.parametrize("cid,nb", [(0, 256), (1, 600), (2, 200), (3, 100), (4, 12)])
def test_config_parity_ready(dev, path, cid, nb):
    print(f"ready dispatch, config {cid}: {nb} candidates", flush=True)
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 0, nb)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER, n_threads=8)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ready, config {cid}")


FUZZ = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_class=C, n_link=K, rel_max=rel, zero_bytes_p=zb,
             cap_scale=cs, slice_scale=ss_)
        for n, D, R, S, C, K, rel, zb, cs, ss_ in [
            (1, 1, 1, 0, 1, 1, 0, 0.0, None, 60), (7, 2, 1, 2, 1, 1, 0, 0.1, 500, 60),
            (30, 3, 2, 4, 2, 2, 5, 0.2, 2000, 40), (64, 5, 3, 3, 1, 3, 0, 0.0, 3000, 100),
            (65, 4, 4, 6, 3, 2, 20, 0.3, 1500, 30), (200, 7, 2, 8, 2, 3, 9, 0.1, 5000, 80),
            (129, 16, 5, 5, 1, 2, 0, 0.05, 4000, 50), (333, 9, 6, 12, 2, 2, 50, 0.1, 20000, 200)]]


@pytest.mark.parametrize("seed", range(len(FUZZ)))
def test_fuzz_parity_ready(dev, path, seed):
    kw = FUZZ[seed]
    print(f"ready dispatch, fuzz {seed}: {kw}", flush=True)
    g = synth.random_gmg(seed, **kw)
    P = random_placements(g, seed + 12345, 197, invalid_every=17)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ready, fuzz {seed}")
    assert (got["violation"] == 4).sum() >= 1


FAST_WRITER = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_link=K, zero_bytes_p=0.2, max_outdeg=2, cap_scale=cs,
                    max_span=sp, edge_p=ep, max_dur=md)
               for n, D, R, S, K, cs, sp, ep, md in [
                   (64, 3, 1, 3, 1, 3000, 6, 0.4, 40), (130, 5, 2, 4, 2, 3000, 6, 0.5, 3),
                   (257, 8, 3, 5, 2, 6000, 12, 0.3, 40), (700, 16, 4, 6, 2, 20000, 40, 0.1, 2),
                   (1500, 40, 4, 3, 2, 50000, 200, 0.02, 40), (1025, 2, 2, 8, 2, 20000, 4, 0.6, 1)]]


@pytest.mark.parametrize("seed", range(len(FAST_WRITER)))
def test_fast_writer_parity_ready(dev, path, seed):
    """Graphs the branch-free interval writer takes, whose consumers on one
    device need not finish in index order under this rule."""
    kw = FAST_WRITER[seed]
    print(f"ready dispatch, fast writer {seed}: {kw}", flush=True)
    g = synth.random_gmg(100 + seed, **kw)
    P = random_placements(g, seed + 777, 131, invalid_every=29)
    P[1::3] = P[0]
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ready, fast writer {seed}")


def test_ready_differs_from_index_order(dev, path):
    """The flag reaches the kernels: on random graphs the two rules give
    different schedules for some candidates, and each matches its oracle."""
    g = synth.random_gmg(5, **FUZZ[5])
    P = random_placements(g, 99, 64)
    h = ss.Gmg(g)
    ready = gpu_run(h, P, dev, dispatch="ready")
    index = gpu_run(h, P, dev, dispatch="index")
    assert_same(ready, oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER), label="ready")
    assert_same(index, oracle.simulate_batch(g, P, dispatch=oracle.INDEX_ORDER), label="index")
    assert (ready["sumfin"] != index["sumfin"]).any()


def fan_out_gmg(width, n_dev):
    """One root whose output feeds `width` consumers, each followed by one more
    op: `width` ops become ready at once, more than the registers hold."""
    N = 1 + 2 * width
    edges = [(0, 1 + i) for i in range(width)] + [(1 + i, 1 + width + i) for i in range(width)]
    dur = [[3]] + [[1 + (i * 7) % 5] for i in range(width)] + [[2]] * width
    slices = [[(0, 40), (45, 300), (310, TIME_INF)]] * n_dev
    return make_gmg(n_dev, ["op"] * N, edges, [i % 3 for i in range(N)], dur, [64 * (1 + i % 4) for i in range(N)],
                    slices, [10 ** 6] * n_dev, [0, 5, 9], [10 ** 6] * 3, bw=(16,), lat=(2,))


@pytest.mark.parametrize("width", [300, 1200])
def test_wide_ready_set_spills(dev, path, width):
    g = fan_out_gmg(width, 6)
    P = random_placements(g, width, 40)
    P[0] = 0  # everything on one device: the whole fan-out waits in the ready set
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ready, fan-out {width}")


def test_zero_ops_and_empty_batch_ready(dev, path):
    g = make_gmg(3, [], [], [], np.zeros((0, 1), np.int64), [], [[(0, TIME_INF)]] * 3, [5, 5, 5], [4], [10])
    P = np.zeros((5, 0), np.uint8)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER), label="ready, zero ops")
    g0 = synth.build_gmg(0)
    empty = gpu_run(ss.Gmg(g0), np.zeros((0, g0.n_ops), np.uint8), dev)
    assert empty["makespan"].shape == (0,)


def test_nullable_outputs_ready(dev, path):
    g = synth.build_gmg(1)
    P = synth.placements(g, 1, 3, 90)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER)
    got = gpu_run(ss.Gmg(g), P, dev, want_peak=False, want_slack=False, want_sumfin=False)
    assert np.array_equal(got["makespan"], ref["makespan"]) and np.array_equal(got["violation"], ref["violation"])


@pytest.mark.parametrize("cid,n_sample", [(1, 128)])
def test_full_batch_sampled_parity_ready(dev, path, cid, n_sample):
    """A workload's whole batch in one call, sampled against the oracle."""
    g = synth.build_gmg(cid)
    B = synth.CONFIGS[cid].n_cand
    print(f"ready dispatch, config {cid}: full batch of {B}", flush=True)
    P = synth.placements(g, cid, 0, B)
    got = gpu_run(ss.Gmg(g), P, dev)
    rng = np.random.default_rng(cid + 50)
    idx = np.unique(np.concatenate([[0, B - 1], rng.choice(B, n_sample, replace=False)]))
    ref = oracle.simulate_batch(g, P[idx], dispatch=oracle.READY_ORDER, n_threads=8)
    assert_same(got, ref, idx=idx, label=f"ready, config {cid} full")


def test_horizon_beyond_32_bits_ready(dev, monkeypatch):
    """Slices far beyond 2^32 us: the 32-bit path is refused and the general
    path's ready-time dispatch still matches the oracle."""
    g = synth.random_gmg(11, n_ops=90, n_dev=4, n_req=2, n_slices=4, n_link=2, cap_scale=2000)
    shift = 1 << 33
    g.slice_begin = g.slice_begin + shift
    g.slice_end = np.where(g.slice_end == TIME_INF, TIME_INF, g.slice_end + shift)
    P = random_placements(g, 5, 150)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.READY_ORDER)
    assert ref["makespan"].min() > shift
    h = ss.Gmg(g)
    monkeypatch.delenv("SS_PATH", raising=False)
    assert_same(gpu_run(h, P, dev), ref, label="ready, horizon 2^33")
    monkeypatch.setenv("SS_PATH", "fast")
    with pytest.raises(ss.SSError):
        gpu_run(h, P, dev)
