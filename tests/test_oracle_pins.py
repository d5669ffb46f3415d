"""Pins of the oracle against facts fixed by the paper and by mathematics.

Nothing here compares the oracle with itself: the expected values are hand
derivations (tests/golden/hand_cases.json), closed forms, bounds, exhaustive
or tick-by-tick brute force written independently below, and metamorphic
relations that any correct implementation must satisfy.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import synth
from paper_2608_15762_amd.synth import TIME_INF, make_gmg, random_gmg

HERE = os.path.dirname(os.path.abspath(__file__))


def gmg_from_case(c):
    slices = [[(a, TIME_INF if e == "INF" else e) for a, e in dev] for dev in c["slices"]]
    ops = c["ops"]
    return make_gmg(c["n_dev"], ["op"] * len(ops), [tuple(e) for e in c["edges"]], [o["req"] for o in ops],
                    [[o["dur"]] for o in ops], [o["bytes"] for o in ops], slices, c["cap"], c["release"],
                    c["deadline"], bw=c["link"]["bw"], lat=c["link"]["lat"])


CASES = json.load(open(os.path.join(HERE, "golden", "hand_cases.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_worked_cases(case):
    g = gmg_from_case(case)
    for key, dispatch in (("expect", oracle.INDEX_ORDER), ("expect_ready_order", oracle.READY_ORDER)):
        if key not in case:
            continue
        exp = case[key]
        out = oracle.simulate_one(g, np.array(case["placement"], np.uint8), dispatch)
        for f in ("st", "fin"):
            if f in exp:
                assert out[f].tolist() == exp[f], (key, f)
        assert out["makespan"] == exp["makespan"]
        assert out["sumfin"] == exp["sumfin"]
        assert out["peak"].tolist() == exp["peak"]
        assert out["violation"] == exp["violation"]
        assert out["slack"].tolist() == exp["slack"]


# ---------------------------------------------------------------------------------- helpers
def xfer(g, u, s, t):
    """Transfer estimate written out for the closed forms below."""
    if s == t:
        return 0
    k = int(g.link_class[s, t])
    b, bw = int(g.out_bytes[u]), int(g.bw[k])
    return int(g.lat[k]) + -(-b // bw)


def open_slices(n_dev):
    return [[(0, TIME_INF)] for _ in range(n_dev)]


def chain_gmg(durs, bytes_, n_dev, bw=(7,), lat=(3,), link=None, release=0, slices=None, cap=None):
    n = len(durs)
    return make_gmg(n_dev, ["op"] * n, [(i, i + 1) for i in range(n - 1)], [0] * n, [[w] for w in durs], bytes_,
                    slices or open_slices(n_dev), cap or [1 << 40] * n_dev, [release], [release + 10 ** 9],
                    link_class=link, bw=bw, lat=lat)


def longest_path(g):
    lp = [0] * g.n_ops
    for v in range(g.n_ops):
        best = 0
        for e in range(g.pred_ptr[v], g.pred_ptr[v + 1]):
            best = max(best, lp[int(g.pred_idx[e])])
        lp[v] = best + int(g.dur[v, 0])
    return max(lp, default=0)


# ---------------------------------------------------------------------------------- P1
@pytest.mark.parametrize("seed", range(12))
def test_p1_single_device_makespan_is_total_work(seed):
    """Any DAG with every op on one device with an always-idle slice: makespan = sum w."""
    g = random_gmg(seed, n_ops=5 + seed * 3, n_dev=3, n_req=2, open_only=True, lat_max=5)
    for d in range(g.n_dev):
        p = np.full(g.n_ops, d, np.uint8)
        w = int(sum(g.dur[v, g.dev_class[d]] for v in range(g.n_ops)))
        for dispatch in (oracle.INDEX_ORDER, oracle.READY_ORDER):
            assert oracle.simulate_one(g, p, dispatch)["makespan"] == w


# ---------------------------------------------------------------------------------- P2 / P7
@pytest.mark.parametrize("seed", range(20))
def test_p2_chain_across_devices_adds_exactly_its_transfers(seed):
    st = synth.Stream(seed + 1000)
    n = st.uniform_int(2, 12)
    D = st.uniform_int(2, 4)
    K = st.uniform_int(1, 3)
    link = np.array([[st.uniform_int(0, K - 1) if s != t else 0 for t in range(D)] for s in range(D)], np.uint8)
    g = chain_gmg([st.uniform_int(1, 30) for _ in range(n)], [st.uniform_int(0, 500) for _ in range(n)], D,
                  bw=[st.uniform_int(1, 40) for _ in range(K)], lat=[st.uniform_int(0, 9) for _ in range(K)],
                  link=link)
    p = np.array([st.uniform_int(0, D - 1) for _ in range(n)], np.uint8)
    expect = int(g.dur[:, 0].sum()) + sum(xfer(g, i, int(p[i]), int(p[i + 1])) for i in range(n - 1))
    for dispatch in (oracle.INDEX_ORDER, oracle.READY_ORDER):
        assert oracle.simulate_one(g, p, dispatch)["makespan"] == expect


@pytest.mark.parametrize("k,extra,lat,bw", [(3, 0, 5, 7), (3, 1, 5, 7), (0, 0, 4, 9), (10, 0, 0, 1000),
                                             (10, 999, 0, 1000), (1, 0, 0, 1)])
def test_p7_transfer_ceiling(k, extra, lat, bw):
    """b = k*bw -> X = lat + k; b = k*bw + r (0 < r < bw) -> lat + k + 1; b = 0 -> lat."""
    b = k * bw + extra
    g = chain_gmg([2, 3], [b, 0], 2, bw=(bw,), lat=(lat,))
    out = oracle.simulate_one(g, np.array([0, 1], np.uint8))
    X = lat + k + (1 if extra else 0)
    assert out["makespan"] == 2 + X + 3
    assert out["st"].tolist() == [0, 2 + X]


# ---------------------------------------------------------------------------------- P3
@pytest.mark.parametrize("seed", range(25))
def test_p3_lower_bounds(seed):
    g = random_gmg(seed, n_ops=6 + seed, n_dev=3, n_req=3, lat_max=4)
    st = synth.Stream(seed)
    for _ in range(4):
        p = np.array([st.uniform_int(0, g.n_dev - 1) for _ in range(g.n_ops)], np.uint8)
        for dispatch in (oracle.INDEX_ORDER, oracle.READY_ORDER):
            ms = oracle.simulate_one(g, p, dispatch)["makespan"]
            loads = [sum(int(g.dur[v, g.dev_class[d]]) for v in range(g.n_ops) if p[v] == d) for d in range(g.n_dev)]
            assert ms >= max(loads)
            if np.all(g.dev_class == 0):
                assert ms >= longest_path(g)
                assert ms >= -(-int(g.dur[:, 0].sum()) // g.n_dev)


@pytest.mark.parametrize("seed", range(10))
def test_p3_no_edges_open_slices_makespan_is_max_load(seed):
    g = random_gmg(seed, n_ops=10, n_dev=3, edge_p=0.0, open_only=True)
    st = synth.Stream(seed + 7)
    p = np.array([st.uniform_int(0, 2) for _ in range(g.n_ops)], np.uint8)
    loads = [sum(int(g.dur[v, g.dev_class[d]]) for v in range(g.n_ops) if p[v] == d) for d in range(3)]
    assert oracle.simulate_one(g, p)["makespan"] == max(loads)


# ---------------------------------------------------------------------------------- P4
@pytest.mark.parametrize("seed", range(10))
def test_p4_chain_on_one_device_peak_is_adjacent_pair(seed):
    st = synth.Stream(seed + 50)
    n = st.uniform_int(1, 15)
    b = [st.uniform_int(0, 1000) for _ in range(n)]
    g = chain_gmg([st.uniform_int(1, 9) for _ in range(n)], b, 1)
    out = oracle.simulate_one(g, np.zeros(n, np.uint8))
    assert out["peak"][0] == max((b[i - 1] if i else 0) + b[i] for i in range(n))


def test_p4_two_ops_two_devices():
    g = chain_gmg([4, 6], [300, 70], 2)
    out = oracle.simulate_one(g, np.array([0, 1], np.uint8))
    assert out["peak"].tolist() == [300, 370]


@pytest.mark.parametrize("n", [1, 4, 9])
def test_p4_independent_ops_are_all_retained(n):
    g = make_gmg(1, ["op"] * n, [], [0] * n, [[3]] * n, [10 * (i + 1) for i in range(n)], open_slices(1),
                 [0], [0], [10 ** 6])
    assert oracle.simulate_one(g, np.zeros(n, np.uint8))["peak"][0] == sum(10 * (i + 1) for i in range(n))


# ---------------------------------------------------------------------------------- P5
@pytest.mark.parametrize("seed,n,D", [(0, 5, 2), (1, 6, 3), (2, 7, 2), (3, 6, 3), (4, 8, 2)])
def test_p5_exhaustive_argmin(seed, n, D):
    g = random_gmg(seed, n_ops=n, n_dev=D, n_req=2, cap_scale=1500)
    P = np.array(list(itertools.product(range(D), repeat=n)), np.uint8)
    out = oracle.simulate_batch(g, P)
    for key in ("sumfin", "makespan"):
        for sla in (False, True):
            feas = [b for b in range(len(P)) if out["violation"][b] == 0 and
                    (not sla or out["slack"][b].min(initial=0) >= 0)]
            exp = min(((int(out[key][b]), b) for b in feas), default=(None, -1))
            bi, bk = oracle.select_best(out["violation"], out[key], out["slack"], sla)
            assert bi == exp[1]
            if bi >= 0:
                assert bk == exp[0]


def test_p5_ties_go_to_lowest_index():
    v = np.zeros(6, np.uint8)
    v[0] = 1
    assert oracle.select_best(v, np.array([1, 5, 3, 3, 9, 3]))[0] == 2
    assert oracle.select_best(np.ones(3, np.uint8), np.zeros(3, np.int64))[0] == -1


# ---------------------------------------------------------------------------------- P6 (brute force)
def brute_fit(slices, t, w):
    """Smallest integer s >= t such that every tick of [s, s+w) lies in one idle slice,
    found by trying s = t, t+1, ...  (independent of the slice-walk formulation)."""
    s = t
    while True:
        for a, e in slices:
            if a <= s and s + w <= e:
                return s
        s += 1


def brute_schedule(g, p):
    """Contract A by enumeration of start times, for tiny inputs."""
    fin = [0] * g.n_ops
    st = [0] * g.n_ops
    clock = [0] * g.n_dev
    for v in range(g.n_ops):
        d = int(p[v])
        sl = [(int(g.slice_begin[k]), int(g.slice_end[k])) for k in range(g.slice_ptr[d], g.slice_ptr[d + 1])]
        ready = max(0, int(g.release[g.op_req[v]]))
        for e in range(g.pred_ptr[v], g.pred_ptr[v + 1]):
            u = int(g.pred_idx[e])
            ready = max(ready, fin[u] + xfer(g, u, int(p[u]), d))
        w = int(g.dur[v, g.dev_class[d]])
        st[v] = brute_fit(sl, max(ready, clock[d]), w)
        fin[v] = st[v] + w
        clock[d] = fin[v]
    return st, fin


@pytest.mark.parametrize("seed", range(30))
def test_p6_earliest_fit_matches_enumeration(seed):
    g = random_gmg(seed, n_ops=8, n_dev=2, n_req=2, n_slices=4, slice_scale=25, max_dur=20, n_class=2, n_link=2,
                   rel_max=30)
    st = synth.Stream(seed + 99)
    p = np.array([st.uniform_int(0, 1) for _ in range(g.n_ops)], np.uint8)
    out = oracle.simulate_one(g, p)
    s, f = brute_schedule(g, p)
    assert out["st"].tolist() == s and out["fin"].tolist() == f


# ---------------------------------------------------------------------------------- P8
def _bump(g, what, st):
    """Copy of g with one quantity made 'worse' (longer, bigger, later, slower)."""
    import copy
    h = copy.deepcopy(g)
    if what == "dur":
        v = st.uniform_int(0, h.n_ops - 1)
        h.dur[v, :] += st.uniform_int(1, 9)
    elif what == "bytes":
        v = st.uniform_int(0, h.n_ops - 1)
        h.out_bytes[v] += st.uniform_int(1, 300)
    elif what == "lat":
        h.lat[st.uniform_int(0, h.n_link - 1)] += st.uniform_int(1, 5)
    elif what == "bw":
        k = st.uniform_int(0, h.n_link - 1)
        h.bw[k] = max(1, h.bw[k] - st.uniform_int(1, 20))
    elif what == "release":
        h.release[st.uniform_int(0, h.n_req - 1)] += st.uniform_int(1, 20)
    elif what == "busy":  # shrink an idle slice from its end (keeps it non-empty) or delay its start
        finite = [k for k in range(len(h.slice_end)) if h.slice_end[k] != TIME_INF]
        if finite:
            k = finite[st.uniform_int(0, len(finite) - 1)]
            length = h.slice_end[k] - h.slice_begin[k]
            if length > 1:
                cut = st.uniform_int(1, length - 1)
                if st.unit() < 0.5:
                    h.slice_end[k] -= cut
                else:
                    h.slice_begin[k] += cut
    return h


@pytest.mark.parametrize("what", ["dur", "bytes", "lat", "bw", "release", "busy"])
@pytest.mark.parametrize("seed", range(8))
def test_p8_monotone_in_every_cost(what, seed):
    g = random_gmg(seed, n_ops=14, n_dev=3, n_req=2, n_slices=4, n_link=2, rel_max=10)
    st = synth.Stream(seed * 31 + 7)
    p = np.array([st.uniform_int(0, 2) for _ in range(g.n_ops)], np.uint8)
    base = oracle.simulate_one(g, p)
    for _ in range(3):
        h = _bump(g, what, st)
        worse = oracle.simulate_one(h, p)
        assert np.all(worse["fin"] >= base["fin"])


# ---------------------------------------------------------------------------------- P9
@pytest.mark.parametrize("seed", range(10))
def test_p9_device_relabelling_permutes_peaks(seed):
    import copy
    g = random_gmg(seed, n_ops=12, n_dev=4, n_req=2, n_slices=3, n_link=2, n_class=2)
    st = synth.Stream(seed + 5)
    sigma = list(range(4))
    for i in range(3, 0, -1):
        j = st.uniform_int(0, i)
        sigma[i], sigma[j] = sigma[j], sigma[i]
    inv = [sigma.index(d) for d in range(4)]
    h = copy.deepcopy(g)
    h.dev_class = g.dev_class[inv].copy()
    h.cap = g.cap[inv].copy()
    h.link_class = g.link_class[np.ix_(inv, inv)].copy()
    sb, se, sp = [], [], [0]
    for d in range(4):
        o = inv[d]
        sb += g.slice_begin[g.slice_ptr[o]:g.slice_ptr[o + 1]].tolist()
        se += g.slice_end[g.slice_ptr[o]:g.slice_ptr[o + 1]].tolist()
        sp.append(len(sb))
    h.slice_begin, h.slice_end, h.slice_ptr = np.array(sb, np.int64), np.array(se, np.int64), np.array(sp, np.int64)
    p = np.array([st.uniform_int(0, 3) for _ in range(g.n_ops)], np.uint8)
    q = np.array([sigma[d] for d in p], np.uint8)
    a, b = oracle.simulate_one(g, p), oracle.simulate_one(h, q)
    assert b["fin"].tolist() == a["fin"].tolist()
    assert [int(b["peak"][sigma[d]]) for d in range(4)] == a["peak"].tolist()
    assert (a["makespan"], a["sumfin"], a["violation"]) == (b["makespan"], b["sumfin"], b["violation"])
    assert a["slack"].tolist() == b["slack"].tolist()


@pytest.mark.parametrize("seed", range(10))
def test_p9_time_shift(seed):
    import copy
    g = random_gmg(seed, n_ops=12, n_dev=3, n_req=2, n_slices=3, rel_max=5)
    delta = 17 + seed
    h = copy.deepcopy(g)
    h.slice_begin = g.slice_begin + delta
    h.slice_end = np.where(g.slice_end == TIME_INF, TIME_INF, g.slice_end + delta)
    h.release = g.release + delta
    h.deadline = g.deadline + delta
    st = synth.Stream(seed)
    p = np.array([st.uniform_int(0, 2) for _ in range(g.n_ops)], np.uint8)
    for dispatch in (oracle.INDEX_ORDER, oracle.READY_ORDER):
        a, b = oracle.simulate_one(g, p, dispatch), oracle.simulate_one(h, p, dispatch)
        assert (b["fin"] - a["fin"]).tolist() == [delta] * g.n_ops
        assert b["makespan"] == a["makespan"] + delta
        assert b["sumfin"] == a["sumfin"] + g.n_ops * delta
        assert b["slack"].tolist() == a["slack"].tolist()
        assert b["peak"].tolist() == a["peak"].tolist()


# ---------------------------------------------------------------------------------- P10
@pytest.mark.parametrize("seed", range(10))
def test_p10_index_order_equals_ready_order_on_private_chains(seed):
    """Each request is a chain on its own devices: the two dispatch rules coincide."""
    st = synth.Stream(seed + 400)
    R = st.uniform_int(1, 3)
    lens = [st.uniform_int(1, 8) for _ in range(R)]
    chains = [[(r, i) for i in range(n)] for r, n in enumerate(lens)]
    order = sorted(sum(chains, []), key=lambda ri: (ri[1], ri[0]))  # interleave requests
    gid = {ri: k for k, ri in enumerate(order)}
    edges = [(gid[(r, i - 1)], gid[(r, i)]) for r, n in enumerate(lens) for i in range(1, n)]
    D = 2 * R
    N = len(order)
    g = make_gmg(D, ["op"] * N, edges, [r for r, _ in order], [[st.uniform_int(1, 20)] for _ in range(N)],
                 [st.uniform_int(0, 100) for _ in range(N)],
                 [[(st.uniform_int(0, 10), st.uniform_int(11, 40)), (st.uniform_int(41, 60), TIME_INF)] for _ in range(D)],
                 [10 ** 6] * D, [st.uniform_int(0, 9) for _ in range(R)], [500] * R, bw=[3], lat=[1])
    for _ in range(5):
        p = np.array([2 * r + st.uniform_int(0, 1) for r, _ in order], np.uint8)
        a = oracle.simulate_one(g, p, oracle.INDEX_ORDER)
        b = oracle.simulate_one(g, p, oracle.READY_ORDER)
        for f in ("st", "fin", "peak", "slack"):
            assert a[f].tolist() == b[f].tolist()


@pytest.mark.parametrize("cid,nb", [(0, 256), (1, 512)])
def test_p10_single_request_configs_agree_across_dispatch_rules(cid, nb):
    g = synth.build_gmg(cid)
    og = oracle.OracleGmg(g)
    P = synth.placements(g, cid, 0, nb)
    a = oracle.simulate_batch(og, P, oracle.INDEX_ORDER)
    b = oracle.simulate_batch(og, P, oracle.READY_ORDER)
    for f in a:
        assert np.array_equal(a[f], b[f]), f


# ---------------------------------------------------------------------------------- P11
def brute_peak_by_ticks(g, p, st, fin):
    """Live bytes on every device at every integer tick, from the residency
    reading taken literally per tensor (own output / one copy per remote device)."""
    succ = [[] for _ in range(g.n_ops)]
    for u, v in g.edges():
        succ[u].append(v)
    horizon = max(fin, default=0) + 200
    live = np.zeros((g.n_dev, horizon + 1), np.int64)
    for v in range(g.n_ops):
        d, b = int(p[v]), int(g.out_bytes[v])
        if succ[v]:
            end = max([fin[x] if p[x] == d else fin[v] + xfer(g, v, d, int(p[x])) for x in succ[v]] + [fin[v]])
        else:
            end = horizon + 1
        live[d, st[v]:end] += b
        for e in sorted({int(p[x]) for x in succ[v]} - {d}):
            live[e, fin[v]:max(fin[x] for x in succ[v] if p[x] == e)] += b
    return live.max(axis=1)


@pytest.mark.parametrize("seed", range(30))
def test_p11_peak_sweep_equals_pairwise_and_ticks(seed):
    g = random_gmg(seed, n_ops=10, n_dev=3, n_req=2, n_slices=2, slice_scale=30, max_dur=15, n_link=2, bw_max=30)
    st = synth.Stream(seed + 3)
    p = np.array([st.uniform_int(0, 2) for _ in range(g.n_ops)], np.uint8)
    out = oracle.simulate_one(g, p)
    sweep = oracle.peak_sweep(g, p, out["st"], out["fin"])
    pair = oracle.peak_pairwise(g, p, out["st"], out["fin"])
    ticks = brute_peak_by_ticks(g, p, out["st"].tolist(), out["fin"].tolist())
    assert sweep.tolist() == pair.tolist() == ticks.tolist() == out["peak"].tolist()
    assert out["violation"] == int(any(out["peak"][d] > g.cap[d] for d in range(g.n_dev)))


# ---------------------------------------------------------------------------------- P12
@pytest.mark.parametrize("seed", range(10))
def test_p12_sla_slack_closed_form(seed):
    st = synth.Stream(seed + 77)
    n = st.uniform_int(1, 12)
    durs = [st.uniform_int(1, 50) for _ in range(n)]
    total = sum(durs)
    g = chain_gmg(durs, [1] * n, 1)
    g.deadline[:] = (3 * total + 1) // 2  # ceil(1.5 * isolated makespan)
    out = oracle.simulate_one(g, np.zeros(n, np.uint8))
    assert out["slack"][0] == (3 * total + 1) // 2 - total


# ---------------------------------------------------------------------------------- batch == one
def test_batch_matches_single_calls_and_threads():
    g = random_gmg(3, n_ops=20, n_dev=3, n_req=3, n_slices=4, n_link=2)
    st = synth.Stream(1)
    P = np.array([[st.uniform_int(0, 3) for _ in range(g.n_ops)] for _ in range(40)], np.uint8)  # some invalid (3)
    one = [oracle.simulate_one(g, P[b]) for b in range(len(P))]
    for thr in (1, 4):
        bat = oracle.simulate_batch(g, P, n_threads=thr)
        for b, o in enumerate(one):
            assert bat["makespan"][b] == o["makespan"] and bat["sumfin"][b] == o["sumfin"]
            assert bat["violation"][b] == o["violation"]
            assert bat["peak"][b].tolist() == o["peak"].tolist()
            assert bat["slack"][b].tolist() == o["slack"].tolist()
    assert any(o["violation"] == 4 for o in one)
