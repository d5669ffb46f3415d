"""Parity of the transfer-port variant (SS_LINK_PORTS: the event-driven
arbitration of Sec. 3.5.2 read into the simulation) on the GPU with the
oracle's LINK_PORTS schedule, element by element through the C ABI.

Integer results: bit-exact on every output.  Cases: the hand-derived port
cases, the seeded workloads (a slice of each batch, and one whole batch
sampled), random graphs of every shape class (several link classes,
zero-byte outputs, fan-in and fan-out, releases), candidates naming unknown
devices, empty inputs, nullable outputs, and the refusals (ports with
ready-time dispatch, ports forced onto the 32-bit path).
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


@pytest.fixture(params=["auto", "generic"])
def path(request, monkeypatch):
    """The memory pass of a port run: the 32-bit passes reading the arrivals
    (default, when the GMG fits the branch-free interval writer) or the
    general int64 memory kernel (SS_PATH=generic)."""
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
    out = ss.simulate_batch(h, Pt, links="ports", **kw)
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


CASES = json.load(open(os.path.join(HERE, "golden", "port_cases.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_cases_on_gpu(dev, case):
    slices = [[(a, TIME_INF if e == "INF" else e) for a, e in d] for d in case["slices"]]
    ops = case["ops"]
    g = make_gmg(case["n_dev"], ["op"] * len(ops), [tuple(e) for e in case["edges"]], [o["req"] for o in ops],
                 [[o["dur"]] for o in ops], [o["bytes"] for o in ops], slices, case["cap"], case["release"],
                 case["deadline"], bw=case["link"]["bw"], lat=case["link"]["lat"])
    got = gpu_run(ss.Gmg(g), np.array([case["placement"]], np.uint8), dev)
    exp = case["expect_link_ports"]
    assert got["makespan"][0] == exp["makespan"] and got["sumfin"][0] == exp["sumfin"]
    assert got["peak"][0].tolist() == exp["peak"] and got["slack"][0].tolist() == exp["slack"]
    assert got["violation"][0] == exp["violation"]


@pytest.mark.parametrize("cid,nb", [(0, 256), (1, 300), (2, 150), (3, 64), (4, 8)])
def test_config_parity_ports(dev, path, cid, nb):
    print(f"transfer ports, config {cid}: {nb} candidates, {path} memory pass", flush=True)
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 0, nb)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS, n_threads=8)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ports, config {cid}")


FUZZ = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_class=C, n_link=K, rel_max=rel, zero_bytes_p=zb,
             cap_scale=cs, slice_scale=ss_, lat_max=lm, bw_max=bm)
        for n, D, R, S, C, K, rel, zb, cs, ss_, lm, bm in [
            (1, 1, 1, 0, 1, 1, 0, 0.0, None, 60, 3, 50), (7, 2, 1, 2, 1, 1, 0, 0.1, 500, 60, 0, 5),
            (30, 3, 2, 4, 2, 2, 5, 0.2, 2000, 40, 2, 9), (64, 5, 3, 3, 1, 3, 0, 0.0, 3000, 100, 0, 2),
            (65, 4, 4, 6, 3, 2, 20, 0.3, 1500, 30, 5, 20), (200, 7, 2, 8, 2, 3, 9, 0.1, 5000, 80, 1, 3),
            (129, 16, 5, 5, 1, 2, 0, 0.05, 4000, 50, 0, 4), (333, 9, 6, 12, 2, 2, 50, 0.1, 20000, 200, 3, 7)]]


@pytest.mark.parametrize("seed", range(len(FUZZ)))
def test_fuzz_parity_ports(dev, seed):
    kw = FUZZ[seed]
    print(f"transfer ports, fuzz {seed}: {kw}", flush=True)
    g = synth.random_gmg(seed + 900, **kw)
    P = random_placements(g, seed + 4242, 197, invalid_every=17)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ports, fuzz {seed}")
    assert (got["violation"] == 4).sum() >= 1


# Graphs inside the branch-free interval writer's limits (one device class, at
# most two link classes and two successors per op) with slow links, so that
# transfers queue on the ports: the 32-bit memory pass reads the arrivals.
PORT_WRITER = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_link=K, zero_bytes_p=0.2, max_outdeg=2, cap_scale=cs,
                    max_span=sp, edge_p=ep, lat_max=lm, bw_max=bm)
               for n, D, R, S, K, cs, sp, ep, lm, bm in [
                   (64, 3, 1, 3, 1, 3000, 6, 0.5, 3, 2), (130, 5, 2, 4, 2, 3000, 6, 0.5, 9, 3),
                   (257, 8, 3, 5, 2, 6000, 12, 0.3, 0, 1), (700, 16, 4, 6, 2, 20000, 40, 0.1, 5, 4),
                   (1025, 2, 2, 8, 2, 20000, 4, 0.6, 2, 1)]]


@pytest.mark.parametrize("seed", range(len(PORT_WRITER)))
def test_port_writer_parity(dev, path, seed):
    kw = PORT_WRITER[seed]
    print(f"transfer ports, branch-free writer {seed}: {kw}, {path} memory pass", flush=True)
    g = synth.random_gmg(600 + seed, **kw)
    assert np.bincount(np.asarray(g.pred_idx), minlength=g.n_ops).max() <= 2
    P = random_placements(g, seed + 5151, 131, invalid_every=29)
    P[1::4] = P[0]  # some candidates keep whole chains on one device
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    got = gpu_run(ss.Gmg(g), P, dev)
    assert_same(got, ref, label=f"ports, branch-free writer {seed}")


def test_ports_differ_from_latency_only(dev):
    """The flag reaches the kernels: on random graphs with slow links the two
    rules give different schedules for some candidates, each matching its
    oracle."""
    g = synth.random_gmg(5, **FUZZ[5])
    P = random_placements(g, 99, 64)
    h = ss.Gmg(g)
    ports = gpu_run(h, P, dev)
    Pt = torch.from_numpy(P).to(dev)
    lat = {k: (None if v is None else v.cpu().numpy()) for k, v in ss.simulate_batch(h, Pt).items()}
    assert_same(ports, oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS), label="ports")
    assert_same(lat, oracle.simulate_batch(g, P, dispatch=oracle.INDEX_ORDER), label="latency")
    assert (ports["sumfin"] != lat["sumfin"]).any()
    assert (ports["sumfin"] >= lat["sumfin"]).all()


def test_wide_fan_out_and_fan_in(dev):
    """One producer feeding every device, every device feeding one consumer:
    the send port of the first and the receive port of the last carry long
    queues of transfers."""
    D, width = 12, 40
    N = 2 + 2 * width
    edges = [(0, 1 + i) for i in range(width)] + [(1 + i, 1 + width + i) for i in range(width)]
    edges += [(1 + width + i, N - 1) for i in range(width)]
    dur = [[5]] + [[1 + (i * 7) % 9] for i in range(2 * width)] + [[3]]
    g = make_gmg(D, ["op"] * N, edges, [0] * N, dur, [1000 + 37 * i for i in range(N)],
                 [[(0, 200), (260, 900), (1000, TIME_INF)]] * D, [10 ** 6] * D, [0], [5000], bw=(64,), lat=(2,))
    P = random_placements(g, 31, 90)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    assert_same(gpu_run(ss.Gmg(g), P, dev), ref, label="ports, fan-out/fan-in")


def test_zero_ops_and_empty_batch_ports(dev):
    g = make_gmg(3, [], [], [], np.zeros((0, 1), np.int64), [], [[(0, TIME_INF)]] * 3, [5, 5, 5], [4], [10])
    P = np.zeros((5, 0), np.uint8)
    assert_same(gpu_run(ss.Gmg(g), P, dev), oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS),
                label="ports, zero ops")
    g0 = synth.build_gmg(0)
    assert gpu_run(ss.Gmg(g0), np.zeros((0, g0.n_ops), np.uint8), dev)["makespan"].shape == (0,)


def test_nullable_outputs_ports(dev):
    g = synth.build_gmg(1)
    P = synth.placements(g, 1, 3, 90)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    got = gpu_run(ss.Gmg(g), P, dev, want_peak=False, want_slack=False, want_sumfin=False)
    assert np.array_equal(got["makespan"], ref["makespan"]) and np.array_equal(got["violation"], ref["violation"])


def test_full_batch_parity_ports(dev):
    """The llama8b workload's whole batch in one call, every candidate against
    the oracle."""
    cid = 1
    g = synth.build_gmg(cid)
    B = synth.CONFIGS[cid].n_cand
    print(f"transfer ports, config {cid}: full batch of {B}", flush=True)
    P = synth.placements(g, cid, 0, B)
    got = gpu_run(ss.Gmg(g), P, dev)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS, n_threads=max(1, min(16, os.cpu_count() or 1)))
    assert_same(got, ref, label=f"ports, config {cid} full")


@pytest.mark.parametrize("cid,nb", [(2, 200), (3, 40)])
def test_ports_with_workspace_and_op_major(dev, cid, nb):
    """Transfer ports through a caller's workspace (smallest and preferred)
    and with op-major placements."""
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 11, nb)
    ref = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS, n_threads=8)
    h = ss.Gmg(g)
    lo, hi = ss.workspace_size(h, nb, links="ports")
    for nbytes in (lo, hi):
        ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        assert_same(gpu_run(h, P, dev, workspace=ws), ref, label=f"ports, workspace {nbytes}")
    out = ss.simulate_batch(h, torch.from_numpy(np.ascontiguousarray(P.T)).to(dev), links="ports", layout="op")
    torch.cuda.synchronize()
    assert_same({k: v.cpu().numpy() for k, v in out.items()}, ref, label="ports, op-major")


def test_refusals(dev, monkeypatch):
    g = synth.build_gmg(0)
    h = ss.Gmg(g)
    Pt = torch.from_numpy(synth.placements(g, 0, 0, 8)).to(dev)
    with pytest.raises(ss.SSError):
        ss.simulate_batch(h, Pt, dispatch="ready", links="ports")
    # transfer ports run on the general kernels only
    g3 = make_gmg(2, ["op"] * 4, [(0, 3), (1, 3), (2, 3)], [0] * 4, [[5]] * 4, [10] * 4, [[(0, TIME_INF)]] * 2,
                  [10 ** 6] * 2, [0], [10 ** 6], bw=(10,), lat=(1,))
    P3 = torch.zeros((2, 4), dtype=torch.uint8, device=dev)
    monkeypatch.setenv("SS_PATH", "fast")
    with pytest.raises(ss.SSError):
        ss.simulate_batch(ss.Gmg(g3), P3, links="ports")
