"""Parity of the HIP path (through the C ABI) with the oracle, element by element.

Integer results, so the bar is bit-exact on every output.  Inputs are the
seeded workloads and random small GMGs; the oracle never sees GPU output.
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
    """Run a case on the default path (the 32-bit fast path when the GMG
    qualifies) and on the general int64 path."""
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


def gpu_run(h, P, dev, **kw):
    Pt = torch.from_numpy(np.ascontiguousarray(P)).to(dev)
    out = ss.simulate_batch(h, Pt, **kw)
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


@pytest.mark.parametrize("cid,nb", [(0, 256), (1, 1000), (2, 300), (3, 130), (4, 20)])
def test_config_parity(dev, path, cid, nb):
    print(f"config {cid}: {nb} candidates", flush=True)
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 0, nb)
    ref = oracle.simulate_batch(g, P, n_threads=8)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"config {cid}")


FUZZ = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_class=C, n_link=K, rel_max=rel, zero_bytes_p=zb,
             cap_scale=cs, slice_scale=ss_)
        for n, D, R, S, C, K, rel, zb, cs, ss_ in [
            (1, 1, 1, 0, 1, 1, 0, 0.0, None, 60), (7, 2, 1, 2, 1, 1, 0, 0.1, 500, 60),
            (30, 3, 2, 4, 2, 2, 5, 0.2, 2000, 40), (64, 5, 3, 3, 1, 3, 0, 0.0, 3000, 100),
            (65, 4, 4, 6, 3, 2, 20, 0.3, 1500, 30), (200, 7, 2, 8, 2, 3, 9, 0.1, 5000, 80),
            (129, 16, 5, 5, 1, 2, 0, 0.05, 4000, 50), (333, 9, 6, 12, 2, 2, 50, 0.1, 20000, 200)]]


@pytest.mark.parametrize("seed", range(len(FUZZ)))
def test_fuzz_parity(dev, path, seed):
    kw = FUZZ[seed]
    print(f"fuzz {seed}: {kw}", flush=True)
    g = synth.random_gmg(seed, **kw)
    st = synth.Stream(seed + 12345)
    B = 197
    P = np.array([[st.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)] for _ in range(B)], np.uint8)
    for b in range(0, B, 17):  # some candidates name a device outside the set
        P[b, st.uniform_int(0, g.n_ops - 1)] = g.n_dev + st.uniform_int(0, 255 - g.n_dev)
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"fuzz {seed}")
    assert (got["violation"] == 4).sum() >= 1



@pytest.mark.parametrize("n_ops,B", [(260, 388), (132, 4), (516, 1020)])
def test_word_transpose_ragged_tiles(dev, path, n_ops, B):
    # op and candidate counts divisible by 4 but not by the 128-wide tiles of
    # the word transpose of the placements: several tiles and ragged edges
    print(f"word transpose: {n_ops} ops, {B} candidates", flush=True)
    g = synth.random_gmg(n_ops, n_ops=n_ops, n_dev=6, n_req=2, n_slices=4, n_link=2, zero_bytes_p=0.1,
                         max_outdeg=2, cap_scale=4000)
    st = synth.Stream(n_ops * 7 + B)
    P = np.array([[st.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)] for _ in range(B)], np.uint8)
    ref = oracle.simulate_batch(g, P, n_threads=8)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"word transpose {n_ops}x{B}")

# Graphs inside the limits of the branch-free interval writer (one device
# class, at most two link classes and two successors per op), with zero-byte
# outputs, zero transfer latencies, far-reaching edges and ragged op counts.
FAST_WRITER = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_link=K, zero_bytes_p=0.2, max_outdeg=2, cap_scale=cs,
                    max_span=sp, edge_p=ep, max_dur=md)
               for n, D, R, S, K, cs, sp, ep, md in [
                   (64, 3, 1, 3, 1, 3000, 6, 0.4, 40), (130, 5, 2, 4, 2, 3000, 6, 0.5, 3),
                   (257, 8, 3, 5, 2, 6000, 12, 0.3, 40), (700, 16, 4, 6, 2, 20000, 40, 0.1, 2),
                   (1500, 40, 4, 3, 2, 50000, 200, 0.02, 40), (1025, 2, 2, 8, 2, 20000, 4, 0.6, 1)]]


@pytest.mark.parametrize("seed", range(len(FAST_WRITER)))
def test_fast_writer_parity(dev, path, seed):
    kw = FAST_WRITER[seed]
    print(f"fast writer {seed}: {kw}", flush=True)
    g = synth.random_gmg(100 + seed, **kw)
    assert np.bincount(np.asarray(g.pred_idx), minlength=g.n_ops).max() <= 2
    st = synth.Stream(seed + 777)
    B = 131
    P = np.array([[st.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)] for _ in range(B)], np.uint8)
    P[1::3] = P[0]  # some candidates keep whole chains on one device
    for b in range(0, B, 29):
        P[b, st.uniform_int(0, g.n_ops - 1)] = g.n_dev + st.uniform_int(0, 255 - g.n_dev)
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"fast writer {seed}")


# Link classes that follow device groups, as the schedule kernel reads them:
# contiguous groups of 2^s devices (group = device >> s), contiguous groups of
# another size, interleaved groups (both from a per-device group table), groups
# whose same-group class is 1, and a single group.
GROUPS = [([0, 0, 0, 0, 1, 1, 1, 1], 0), ([0, 0, 0, 1, 1, 1], 0), ([0, 1, 0, 1, 0, 1, 0, 1], 0),
          ([0, 0, 1, 1, 2, 2, 3, 3], 1), ([0] * 8, 0)]


@pytest.mark.parametrize("case", range(len(GROUPS)))
def test_device_group_links(dev, path, case):
    grp, same = GROUPS[case]
    D = len(grp)
    print(f"device groups {grp}, same-group class {same}", flush=True)
    g = synth.random_gmg(300 + case, n_ops=150, n_dev=D, n_req=2, n_slices=3, n_link=2, cap_scale=3000, lat_max=9)
    g.link_class = np.array([[0 if a == b else (same if grp[a] == grp[b] else 1 - same) for b in range(D)]
                             for a in range(D)], np.uint8)
    st = synth.Stream(case + 4242)
    B = 200
    P = np.array([[st.uniform_int(0, D - 1) for _ in range(g.n_ops)] for _ in range(B)], np.uint8)
    P[1::5] = np.repeat(np.arange(D, dtype=np.uint8), (g.n_ops + D - 1) // D)[:g.n_ops]  # runs per device
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"device groups {case}")


def test_predecessor_distances(dev, path):
    """Predecessors 1 to 7 ops back, in pairs and alone.  The schedule takes
    the nearest predecessors of an op from its register history and older
    ones from rows it loaded steps before, so every distance meets each of
    those paths (and the slices, with gaps, make the lookups do work)."""
    n = 300
    st = synth.Stream(9001)
    edges = []
    for v in range(1, n):
        a = v - (1 + (v * 5) % 7)
        b = v - (1 + (v // 7) % 7)
        ps = {p for p in (a, b) if p >= 0}
        if v % 11 == 0:
            ps = {max(a, 0)}
        edges += [(p, v) for p in sorted(ps)]
    dur = [[st.uniform_int(1, 40)] for _ in range(n)]
    out_b = [st.uniform_int(0, 900) for _ in range(n)]
    slices = [[(0, 300 + 50 * d), (400 + 70 * d, 2000), (2100, TIME_INF)] for d in range(4)]
    g = make_gmg(4, ["op"] * n, edges, [v % 2 for v in range(n)], dur, out_b, slices, [4200] * 4, [0, 25],
                 [4000, 5000], bw=[7], lat=[3])
    assert np.diff(g.pred_ptr).max() <= 2  # both predecessors go through the pipeline
    P = np.array([[st.uniform_int(0, 3) for _ in range(n)] for _ in range(96)], np.uint8)
    P[0] = 0
    P[1] = np.arange(n) % 4
    P[2] = (np.arange(n) // 5) % 4
    ref = oracle.simulate_batch(g, P)
    assert_same(gpu_run(ss.Gmg(g), P, dev), ref, label="predecessor distances")


def test_scratch_reuse_across_streams(dev):
    """Calls on two streams with no host synchronisation between them: the
    smaller call on the second stream takes the first call's idle scratch
    block, and may use it only after that call's work (its stream waits for
    the block's last use); the third call reuses a block again."""
    g = synth.build_gmg(2)
    h = ss.Gmg(g)
    rows = [synth.placements(g, 2, 0, 300), synth.placements(g, 2, 300, 120), synth.placements(g, 2, 420, 300)]
    refs = [oracle.simulate_batch(g, P, n_threads=8) for P in rows]
    ins = [torch.from_numpy(np.ascontiguousarray(P)).to(dev) for P in rows]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    outs = [ss.simulate_batch(h, P, stream=s) for P, s in zip(ins, (s1, s2, s1))]
    torch.cuda.synchronize()
    for i, (o, r) in enumerate(zip(outs, refs)):
        assert_same({k: (None if v is None else v.cpu().numpy()) for k, v in o.items()}, r, label=f"call {i}")


def test_nullable_outputs_and_empty_batch(dev, path):
    g = synth.build_gmg(0)
    h = ss.Gmg(g)
    P = synth.placements(g, 0, 0, 70)
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(h, P, dev, want_peak=False, want_slack=False, want_sumfin=False)
    assert np.array_equal(got["makespan"], ref["makespan"]) and np.array_equal(got["violation"], ref["violation"])
    empty = gpu_run(h, np.zeros((0, g.n_ops), np.uint8), dev)
    assert empty["makespan"].shape == (0,)


def test_zero_ops_gmg(dev, path):
    g = make_gmg(3, [], [], [], np.zeros((0, 1), np.int64), [], [[(0, TIME_INF)]] * 3, [5, 5, 5], [4], [10])
    P = np.zeros((5, 0), np.uint8)
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label="zero ops")
    assert got["slack"].tolist() == [[6]] * 5


def test_max_devices(dev, path):
    g = synth.random_gmg(7, n_ops=300, n_dev=255, n_req=3, n_slices=3, n_link=2, cap_scale=3000)
    st = synth.Stream(99)
    P = np.array([[st.uniform_int(0, 255) for _ in range(g.n_ops)] for _ in range(130)], np.uint8)
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label="255 devices")


def test_crowded_device_uses_global_sort_buffer(dev, path):
    """All 2,052 ops of the 4-tenant workload on one device: > 2,048 endpoints."""
    g = synth.build_gmg(2)
    P = np.zeros((6, g.n_ops), np.uint8)
    P[1:] = synth.placements(g, 2, 0, 5)
    P[2, : g.n_ops // 2] = 3
    ref = oracle.simulate_batch(g, P)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label="crowded")


def test_fan_in_many_copies_in_one_gap(dev, path):
    """One op consuming 40 remote outputs: all 40 copies land on its device
    before its own allocation (exercises the sorted-gap fallback)."""
    n = 41
    st = synth.Stream(77)
    edges = [(u, n - 1) for u in range(n - 1)]
    g = make_gmg(4, ["op"] * n, edges, [0] * n, [[st.uniform_int(1, 30)] for _ in range(n)],
                 [st.uniform_int(1, 500) for _ in range(n)], [[(0, TIME_INF)]] * 4, [10 ** 6] * 4, [0], [10 ** 5],
                 bw=[3], lat=[2])
    P = np.array([[1 + st.uniform_int(0, 2) for _ in range(n - 1)] + [0] for _ in range(64)], np.uint8)
    P[1::2, : n - 1] = np.array([[st.uniform_int(0, 3) for _ in range(n - 1)] for _ in range(32)], np.uint8)
    ref = oracle.simulate_batch(g, P)
    assert_same(gpu_run(ss.Gmg(g), P, dev), ref, label="fan-in")


@pytest.mark.parametrize("k", [30, 70])
def test_copies_and_frees_crowding_one_gap(dev, path, k):
    """Device 0 runs op A, then op B; device 1 runs k producers consumed by A,
    then k producers consumed by B.  The copies for B arrive while A runs and
    the copies for A are freed when A finishes: 2k events interleave between
    the starts of A and B (with k = 70 more than the peak kernel collects
    per device for its exact in-gap sweep, so it must fall back)."""
    n = 2 * k + 2
    a, b = 2 * k, 2 * k + 1
    st = synth.Stream(k)
    edges = [(i, a) for i in range(k)] + [(k + i, b) for i in range(k)]
    dur = [[st.uniform_int(5, 15)] for _ in range(2 * k)] + [[10 * k], [7]]
    out_b = [st.uniform_int(1000, 5000) for _ in range(n)]
    g = make_gmg(2, ["op"] * n, edges, [0] * n, dur, out_b, [[(0, TIME_INF)]] * 2, [10 ** 9] * 2, [0], [10 ** 9],
                 bw=[1000], lat=[1])
    P = np.ones((4, n), np.uint8)
    P[:, a] = P[:, b] = 0
    P[1, : k // 2] = 0  # some producers local to A
    P[2, k: k + k // 3] = 0  # some producers local to B
    P[3] = np.array([st.uniform_int(0, 1) for _ in range(n)], np.uint8)
    ref = oracle.simulate_batch(g, P)
    assert_same(gpu_run(ss.Gmg(g), P, dev), ref, label=f"crowded gap k={k}")


def test_horizon_beyond_32_bits_takes_general_path(dev, monkeypatch):
    """Slices far beyond 2^32 us: the fast path must be refused and the general
    path must still match the oracle."""
    g = synth.random_gmg(11, n_ops=90, n_dev=4, n_req=2, n_slices=4, n_link=2, cap_scale=2000)
    shift = 1 << 33
    g.slice_begin = g.slice_begin + shift
    g.slice_end = np.where(g.slice_end == TIME_INF, TIME_INF, g.slice_end + shift)
    st = synth.Stream(5)
    P = np.array([[st.uniform_int(0, 3) for _ in range(g.n_ops)] for _ in range(150)], np.uint8)
    ref = oracle.simulate_batch(g, P)
    assert ref["makespan"].min() > shift
    h = ss.Gmg(g)
    monkeypatch.delenv("SS_PATH", raising=False)
    assert_same(gpu_run(h, P, dev), ref, label="horizon 2^33")
    monkeypatch.setenv("SS_PATH", "fast")
    with pytest.raises(ss.SSError):
        gpu_run(h, P, dev)


@pytest.mark.parametrize("dispatch", ["index", "ready"])
@pytest.mark.parametrize("case", ["wide", "scaled", "scaled_small", "mixed"])
def test_byte_sums_beyond_32_bits(dev, monkeypatch, case, dispatch):
    """Output sizes near 2^31 on the 32-bit time path.  "wide": odd sizes, so
    no common power of two divides them and their sums pass 2^32 (the peak
    pass keeps 64-bit sums); "scaled": multiples of 2^20 whose sums pass 2^32
    but whose sums divided by 2^20 do not (32-bit sums of the scaled sizes);
    "scaled_small": multiples of 2^11 whose raw sums stay below 2^32 too;
    "mixed": zero sizes beside sizes of 2^31 - 1 (64-bit sums).
    Capacities at each device's 90th-percentile peak leave some candidates
    feasible and make others overflow."""
    g = synth.random_gmg(40 + (case == "scaled"), n_ops=300, n_dev=6, n_req=3, n_slices=3, n_link=2)
    st = synth.Stream(41)
    if case == "wide":
        ob = [2 * st.uniform_int(1 << 29, (1 << 30) - 1) + 1 for _ in range(g.n_ops)]
    elif case == "scaled":
        ob = [st.uniform_int(1, 1 << 11) << 20 for _ in range(g.n_ops)]
    elif case == "scaled_small":
        ob = [st.uniform_int(1, 1 << 10) << 11 for _ in range(g.n_ops)]
    else:
        ob = [0 if st.uniform_int(0, 2) == 0 else (1 << 31) - 1 for _ in range(g.n_ops)]
    g.out_bytes = np.asarray(ob, np.int64)
    g.bw = np.asarray([1 << 20, 1 << 21], np.int64)  # transfers of about a millisecond keep times in 32 bits
    st2 = synth.Stream(43)
    P = np.array([[st2.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)] for _ in range(200)], np.uint8)
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    g.cap = np.full(g.n_dev, 1 << 62, np.int64)
    roomy = oracle.simulate_batch(g, P, dispatch=mode)
    assert case == "scaled_small" or roomy["peak"].max() > (1 << 32)
    g.cap = np.percentile(roomy["peak"], 90, axis=0).astype(np.int64)
    ref = oracle.simulate_batch(g, P, dispatch=mode)
    assert 0 < (ref["violation"] == 1).sum() < len(P)
    monkeypatch.setenv("SS_PATH", "fast")  # the 32-bit path must take this GMG
    assert_same(gpu_run(ss.Gmg(g), P, dev, dispatch=dispatch), ref, label=f"byte sums beyond 2^32 ({case}, {dispatch})")


# ------------------------------------------------------------------ selection
def gpu_select(h, viol, key, slack, require_sla, dev):
    out = ss.select_best(h, torch.from_numpy(viol).to(dev), torch.from_numpy(key).to(dev),
                         None if slack is None else torch.from_numpy(slack).to(dev), require_sla)
    torch.cuda.synchronize()
    return tuple(out.cpu().tolist())


@pytest.mark.parametrize("batch", ["own", "uniform"])
def test_select_best_on_tight_memory_workload(dev, batch):
    """The tight-memory workload's own candidates (a balanced base with a few
    ops moved: about 1% violate) and uniform random placements over its 64
    devices (about a quarter violate), simulated and then selected with both
    keys, with and without the SLA condition."""
    g = synth.build_gmg(3)
    h = ss.Gmg(g)
    if batch == "own":
        P = synth.placements(g, 3, 0, 2000)
    else:
        words = synth.draw_np(3003, np.arange(600 * g.n_ops)).reshape(600, g.n_ops)
        P = (words % np.uint64(g.n_dev)).astype(np.uint8)
    got = gpu_run(h, P, dev)
    ref = oracle.simulate_batch(g, P, n_threads=8)
    assert_same(got, ref, label=f"config 3, {batch} candidates")
    n_viol = int((ref["violation"] == 1).sum())
    assert 0 < n_viol < len(P)
    if batch == "uniform":
        assert n_viol > len(P) // 10
    for key in ("sumfin", "makespan"):
        for sla in (False, True):
            exp = oracle.select_best(ref["violation"], ref[key], ref["slack"], sla)
            assert gpu_select(h, got["violation"], got[key], got["slack"], sla, dev) == exp


@pytest.mark.parametrize("B", [0, 1, 255, 256, 257, 100_003, 3_000_001])
def test_select_best_ties_and_sizes(dev, B):
    g = synth.random_gmg(1, n_ops=4, n_dev=2, n_req=2)
    h = ss.Gmg(g)
    rng = np.random.default_rng(B)
    key = rng.integers(0, 50, B).astype(np.int64)  # many ties
    viol = (rng.random(B) < 0.3).astype(np.uint8) * rng.choice(np.array([1, 4], np.uint8), B)
    slack = rng.integers(-3, 100, (B, 2)).astype(np.int64)
    for sla in (False, True):
        exp = oracle.select_best(viol, key, slack, sla)
        assert gpu_select(h, viol, key, slack, sla, dev) == exp
    none = gpu_select(h, np.ones(B, np.uint8), key, slack, False, dev)
    assert none == (-1, 2 ** 63 - 1)
