"""Pins of the oracle's transfer-port variant (LINK_PORTS): the event-driven
arbitration of Sec. 3.5.2 read into the what-if simulation.  A device sends at
most one tensor at a time and receives at most one at a time; the transfer of
an output to a remote device is requested (its Intent arrives) when the
producer finishes; at every Intent arrival and every transfer completion the
pending transfers are examined in order of request time, producer index and
destination device, and each one whose two ports are idle starts.

Expected values are hand derivations (tests/golden/port_cases.json), special
cases that reduce to the latency-only rule, a monotonicity bound against it,
and properties of the transfer list checked from scratch here (port
exclusivity, durations, arrival before use, no pending transfer with both
ports idle at any instant, starts only at a request or a completion, and the
examination order of pending transfers).
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd.synth import TIME_INF, make_gmg, random_gmg

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = json.load(open(os.path.join(HERE, "golden", "port_cases.json")))["cases"]
FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


def gmg_from_case(c):
    slices = [[(a, TIME_INF if e == "INF" else e) for a, e in dev] for dev in c["slices"]]
    ops = c["ops"]
    return make_gmg(c["n_dev"], ["op"] * len(ops), [tuple(e) for e in c["edges"]], [o["req"] for o in ops],
                    [[o["dur"]] for o in ops], [o["bytes"] for o in ops], slices, c["cap"], c["release"],
                    c["deadline"], bw=c["link"]["bw"], lat=c["link"]["lat"])


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_worked_port_cases(case):
    g = gmg_from_case(case)
    for key, dispatch in (("expect", oracle.INDEX_ORDER), ("expect_link_ports", oracle.LINK_PORTS)):
        exp = case[key]
        out = oracle.simulate_one(g, np.array(case["placement"], np.uint8), dispatch)
        assert out["st"].tolist() == exp["st"], key
        assert out["fin"].tolist() == exp["fin"], key
        assert out["makespan"] == exp["makespan"], key
        assert out["sumfin"] == exp["sumfin"], key
        assert out["peak"].tolist() == exp["peak"], key
        assert out["violation"] == exp["violation"], key
        assert out["slack"].tolist() == exp["slack"], key


def xfer(g, u, s, t):
    """Transfer estimate, written out here: lat + ceil(bytes / bw) of the link class."""
    if s == t:
        return 0
    k = int(g.link_class[s, t])
    return int(g.lat[k]) + -(-int(g.out_bytes[u]) // int(g.bw[k]))


def placements(g, seed, B):
    rng = np.random.default_rng(seed)
    return rng.integers(0, g.n_dev, (B, g.n_ops)).astype(np.uint8)


GRAPHS = [dict(n_ops=n, n_dev=D, n_req=R, n_slices=S, n_link=K, lat_max=lm, bw_max=bm)
          for n, D, R, S, K, lm, bm in [(12, 3, 1, 2, 1, 3, 50), (40, 4, 2, 3, 2, 5, 20), (90, 6, 3, 4, 2, 2, 9),
                                        (150, 8, 2, 5, 2, 0, 3)]]


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_one_device_placements_need_no_transfer(gi):
    """With every op of a candidate on one device nothing moves: the port rule
    gives the latency-only result exactly."""
    g = random_gmg(200 + gi, **GRAPHS[gi])
    P = np.repeat(np.arange(g.n_dev, dtype=np.uint8)[:, None], g.n_ops, 1)
    a = oracle.simulate_batch(g, P, dispatch=oracle.INDEX_ORDER)
    b = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_free_transfers_change_nothing(gi):
    """Zero-byte outputs over zero-latency links have a zero estimate: such a
    transfer moves nothing, neither waits for nor holds a port, and the result
    is the latency-only one for any placement."""
    g = random_gmg(300 + gi, **GRAPHS[gi])
    g.out_bytes = np.zeros_like(g.out_bytes)
    g.lat = np.zeros_like(g.lat)
    P = placements(g, gi, 64)
    a = oracle.simulate_batch(g, P, dispatch=oracle.INDEX_ORDER)
    b = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f


def test_chains_match_latency_only():
    """A single dependency chain moves one tensor at a time: each transfer
    starts after the previous one has arrived and its consumer has run, so
    ports never make a transfer wait."""
    N, D = 30, 4
    rng = np.random.default_rng(7)
    g = make_gmg(D, ["op"] * N, [(i, i + 1) for i in range(N - 1)], [0] * N,
                 [[int(x)] for x in rng.integers(1, 50, N)], [int(x) for x in rng.integers(0, 5000, N)],
                 [[(0, TIME_INF)]] * D, [10 ** 9] * D, [0], [10 ** 6], bw=(7,), lat=(3,))
    P = placements(g, 3, 50)
    a = oracle.simulate_batch(g, P, dispatch=oracle.INDEX_ORDER)
    b = oracle.simulate_batch(g, P, dispatch=oracle.LINK_PORTS)
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_ports_never_finish_an_op_earlier(gi):
    """Every transfer takes at least its estimate under ports, and with the
    dispatch order fixed raising transfer times never lowers a finish time
    (monotonicity of the index-order list schedule)."""
    g = random_gmg(400 + gi, **GRAPHS[gi])
    for b, p in enumerate(placements(g, 40 + gi, 24)):
        a = oracle.simulate_one(g, p, oracle.INDEX_ORDER)
        q = oracle.simulate_one(g, p, oracle.LINK_PORTS)
        assert (q["fin"] >= a["fin"]).all(), b
        assert q["makespan"] >= a["makespan"] and q["sumfin"] >= a["sumfin"]


@pytest.mark.parametrize("gi", range(len(GRAPHS)))
def test_transfer_list_properties(gi):
    g = random_gmg(500 + gi, **GRAPHS[gi])
    succ = [[] for _ in range(g.n_ops)]
    for v in range(g.n_ops):
        for e in range(g.pred_ptr[v], g.pred_ptr[v + 1]):
            succ[int(g.pred_idx[e])].append(v)
    for b, p in enumerate(placements(g, 60 + gi, 16)):
        sim = oracle.simulate_one(g, p, oracle.LINK_PORTS)
        tr = oracle.port_transfers(g, p)
        # exactly one transfer per (output, remote device that consumes it)
        want = sorted((u, int(p[x])) for u in range(g.n_ops) for x in set(succ[u]) if p[x] != p[u])
        want = sorted(set(want))
        got = sorted(zip(tr["op"].tolist(), tr["dst"].tolist()))
        assert got == want, b
        n = len(tr["op"])
        for i in range(n):
            u, s, d = int(tr["op"][i]), int(tr["src"][i]), int(tr["dst"][i])
            assert s == p[u] and d != s
            assert tr["arrive"][i] - tr["start"][i] == xfer(g, u, s, d)
            assert tr["start"][i] >= sim["fin"][u]
            for x in succ[u]:  # every consumer on d starts after the arrival
                if p[x] == d:
                    assert sim["st"][x] >= tr["arrive"][i]
            if tr["arrive"][i] == tr["start"][i]:
                assert tr["start"][i] == sim["fin"][u]
        check_arbitration(tr, sim["fin"])
        # a port carries one transfer at a time (non-empty intervals disjoint)
        for key in ("src", "dst"):
            for dev in range(g.n_dev):
                iv = sorted((int(tr["start"][i]), int(tr["arrive"][i])) for i in range(n)
                            if tr[key][i] == dev and tr["arrive"][i] > tr["start"][i])
                for (a0, a1), (b0, b1) in zip(iv, iv[1:]):
                    assert a1 <= b0, (key, dev)


def check_arbitration(tr, fin):
    """The arbitration rule, checked from the transfer list alone."""
    n = len(tr["op"])
    req = [int(fin[int(tr["op"][i])]) for i in range(n)]
    st = [int(x) for x in tr["start"]]
    ar = [int(x) for x in tr["arrive"]]
    src = [int(x) for x in tr["src"]]
    dst = [int(x) for x in tr["dst"]]
    busy = [i for i in range(n) if ar[i] > st[i]]  # zero-estimate transfers hold no port
    key = {i: (req[i], int(tr["op"][i]), dst[i]) for i in range(n)}

    def shares_port(i, j):
        return src[i] == src[j] or dst[i] == dst[j]

    for i in busy:
        # it starts at its request or when a transfer on one of its ports completes
        assert st[i] == req[i] or any(ar[j] == st[i] for j in busy if j != i and shares_port(i, j))
        # while it waits, one of its ports is always held (no idle pair of ports is left unused)
        cover = sorted((st[j], ar[j]) for j in busy if j != i and shares_port(i, j))
        t = req[i]
        for lo, hi in cover:
            if lo <= t < hi:
                t = hi
        assert t >= st[i], (i, req[i], st[i], cover)
        # pending transfers are examined in order: a later one (j) that starts
        # while i still waits found i blocked by a third transfer, started
        # earlier or examined before i
        for j in busy:
            if j == i or key[j] <= key[i] or not (req[i] <= st[j] < st[i]):
                continue
            t = st[j]
            assert any(k not in (i, j) and shares_port(i, k) and st[k] <= t < ar[k] and (st[k] < t or key[k] < key[i])
                       for k in busy), (i, j)


def test_invalid_placement_sentinels():
    g = random_gmg(9, **GRAPHS[1])
    p = placements(g, 9, 1)[0]
    p[3] = g.n_dev + 2
    out = oracle.simulate_one(g, p, oracle.LINK_PORTS)
    assert out["violation"] == 4 and out["makespan"] == np.iinfo(np.int64).max
    with pytest.raises(ValueError):
        oracle.port_transfers(g, p)
