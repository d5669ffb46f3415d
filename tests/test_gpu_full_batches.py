"""Every candidate of the full batches of the four workloads the oracle can
cover on the host in seconds (256, 65,536, 262,144 and 131,072 candidates),
compared with the oracle element by element, bit for bit, on every output:
both dispatch rules, the fast and the general path, and the op-major layout.
The oracle runs once per workload and rule, on the host's cores (at most 16,
the host share of one GPU), over contiguous ranges of the batch.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")
THREADS = max(1, min(16, os.cpu_count() or 1))
_cache = {}


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def batch(cid):
    if ("P", cid) not in _cache:
        g = synth.build_gmg(cid)
        _cache[("P", cid)] = (g, synth.placements(g, cid, 0, synth.CONFIGS[cid].n_cand))
    return _cache[("P", cid)]


def reference(cid, dispatch):
    key = ("ref", cid, dispatch)
    if key not in _cache:
        g, P = batch(cid)
        mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
        print(f"oracle: config {cid}, {len(P)} candidates, {dispatch}, {THREADS} threads", flush=True)
        _cache[key] = oracle.simulate_batch(g, P, dispatch=mode, n_threads=THREADS)
    return _cache[key]


def assert_same(got, ref, label):
    for f in FIELDS:
        a, b = got[f], ref[f]
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[:5]
            n_bad = int(np.any((a != b).reshape(len(a), -1), axis=1).sum())
            pytest.fail(f"{label}: {f} differs on {n_bad} candidates, first at {bad.tolist()}")


@pytest.mark.parametrize("dispatch", ["index", "ready"])
@pytest.mark.parametrize("path", ["auto", "generic"])
@pytest.mark.parametrize("cid", [0, 1, 2, 3])
def test_every_candidate(dev, cid, path, dispatch, monkeypatch):
    if path == "generic":
        monkeypatch.setenv("SS_PATH", "generic")
    else:
        monkeypatch.delenv("SS_PATH", raising=False)
    g, P = batch(cid)
    ref = reference(cid, dispatch)
    print(f"config {cid}: {len(P)} candidates, {path} path, {dispatch}", flush=True)
    h = ss.Gmg(g)
    out = ss.simulate_batch(h, torch.from_numpy(P).to(dev), dispatch=dispatch)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    assert_same(got, ref, f"config {cid} {path} {dispatch}")


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_every_candidate_op_major(dev, cid, monkeypatch):
    monkeypatch.delenv("SS_PATH", raising=False)
    g, P = batch(cid)
    ref = reference(cid, "index")
    print(f"config {cid}: {len(P)} candidates, op-major", flush=True)
    h = ss.Gmg(g)
    out = ss.simulate_batch(h, torch.from_numpy(np.ascontiguousarray(P.T)).to(dev), layout="op")
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    assert_same(got, ref, f"config {cid} op-major")
