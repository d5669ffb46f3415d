"""The boundary of the library on the GPU, through the C ABI: op-major
placements (SS_LAYOUT_OP_MAJOR) and a caller-owned workspace
(ss_simulate_workspace_size, ss_simulate_batch_ws).

Each case is compared element by element, bit for bit, with the oracle on
the same seeded inputs and with the row-major, library-scratch call.
"""
import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth
from paper_2608_15762_amd.synth import random_gmg

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")


@pytest.fixture(params=["auto", "generic"])
def path(request, monkeypatch):
    """The default path (the 32-bit fast path when the GMG qualifies) and the
    general int64 path."""
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


def run(h, P, dev, layout="row", **kw):
    A = np.ascontiguousarray(P if layout == "row" else P.T)
    out = ss.simulate_batch(h, torch.from_numpy(A).to(dev), layout=layout, **kw)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def assert_same(a, b, label):
    for f in FIELDS:
        if a.get(f) is None or b.get(f) is None:
            continue
        if not np.array_equal(a[f], b[f]):
            bad = np.argwhere(a[f] != b[f])[:5]
            pytest.fail(f"{label}: {f} differs at {bad.tolist()}")


def workspace(nbytes, dev):
    # torch's allocator hands out blocks aligned to at least 512 bytes
    return torch.empty(int(nbytes), dtype=torch.uint8, device=dev)


CASES = [(0, 256), (1, 700), (2, 300), (3, 130), (4, 12)]


@pytest.mark.parametrize("dispatch", ["index", "ready"])
@pytest.mark.parametrize("cid,nb", CASES)
def test_op_major_layout(dev, path, cid, nb, dispatch):
    print(f"config {cid}: {nb} candidates, op-major, {dispatch}", flush=True)
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 0, nb)
    P[nb // 2, 0] = g.n_dev + 1  # one candidate names an unknown device
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    ref = oracle.simulate_batch(g, P, dispatch=mode, n_threads=8)
    h = ss.Gmg(g)
    assert_same(run(h, P, dev, "op", dispatch=dispatch), ref, f"config {cid} op-major")


@pytest.mark.parametrize("seed", range(4))
def test_op_major_fuzz(dev, path, seed):
    g = random_gmg(900 + seed, n_ops=[5, 64, 97, 300][seed], n_dev=[2, 3, 7, 11][seed], n_req=2, n_slices=3,
                   n_class=1 + seed % 2, n_link=2)
    rng = np.random.default_rng(seed)
    P = rng.integers(0, g.n_dev, (333, g.n_ops)).astype(np.uint8)
    ref = oracle.simulate_batch(g, P)
    assert_same(run(ss.Gmg(g), P, dev, "op"), ref, f"fuzz {seed} op-major")


def test_workspace_sizes(dev):
    g = synth.build_gmg(2)
    h = ss.Gmg(g)
    for layout in ("row", "op"):
        for dispatch in ("index", "ready"):
            lo, hi = ss.workspace_size(h, 262144, layout=layout, dispatch=dispatch)
            assert 0 < lo <= hi, (layout, dispatch, lo, hi)
            lo1, hi1 = ss.workspace_size(h, 64, layout=layout, dispatch=dispatch)
            assert lo1 <= lo and hi1 <= hi
    assert ss.workspace_size(h, 0) == (0, 0)


@pytest.mark.parametrize("dispatch", ["index", "ready"])
@pytest.mark.parametrize("layout", ["row", "op"])
@pytest.mark.parametrize("cid,nb", [(0, 256), (2, 1000), (3, 300), (4, 8)])
def test_caller_workspace(dev, path, cid, nb, layout, dispatch):
    """Results with the caller's workspace, at its preferred size and at its
    smallest (many small chunks), equal the oracle's."""
    print(f"config {cid}: {nb} candidates, {layout}, {dispatch}, caller workspace", flush=True)
    g = synth.build_gmg(cid)
    P = synth.placements(g, cid, 0, nb)
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    ref = oracle.simulate_batch(g, P, dispatch=mode, n_threads=8)
    h = ss.Gmg(g)
    lo, hi = ss.workspace_size(h, nb, layout=layout, dispatch=dispatch)
    for nbytes in (hi, lo, (lo + hi) // 2):
        ws = workspace(nbytes, dev)
        assert_same(run(h, P, dev, layout, dispatch=dispatch, workspace=ws), ref,
                    f"config {cid} workspace {nbytes}")


def test_workspace_errors(dev):
    g = synth.build_gmg(1)
    h = ss.Gmg(g)
    P = torch.from_numpy(synth.placements(g, 1, 0, 128)).to(dev)
    lo, _ = ss.workspace_size(h, 128)
    with pytest.raises(ss.SSError) as e:  # too small
        ss.simulate_batch(h, P, workspace=workspace(lo - 256, dev))
    assert e.value.code == ss.SS_ERR_INVALID_ARG
    ws = workspace(lo + 512, dev)
    with pytest.raises(ss.SSError) as e:  # misaligned
        ss.simulate_batch(h, P, workspace=ws[8:])
    assert e.value.code == ss.SS_ERR_INVALID_ARG
    out = ss.simulate_batch(h, P, workspace=ws)  # the aligned one works
    torch.cuda.synchronize()
    assert out["violation"].shape == (128,)


def test_workspace_reused_across_calls_and_sizes(dev):
    """One workspace serves consecutive calls of different sizes on one
    stream; each result equals the oracle's."""
    g = synth.build_gmg(3)
    h = ss.Gmg(g)
    _, hi = ss.workspace_size(h, 500)
    ws = workspace(hi, dev)
    for nb, b0 in ((500, 0), (77, 1000), (311, 3000)):
        P = synth.placements(g, 3, b0, nb)
        ref = oracle.simulate_batch(g, P, n_threads=8)
        assert_same(run(h, P, dev, workspace=ws), ref, f"{nb} candidates")


@pytest.mark.parametrize("dispatch", ["index", "ready"])
def test_pool_scratch_fits_the_memory_left(dev, dispatch):
    """With most of the device's memory held by the caller, a call sizes its
    own scratch to what is left: ss_simulate_chunking reports smaller
    memory-pass sub-chunks than with the memory free, and the results, computed
    in those smaller pieces, still equal the oracle's."""
    g = synth.build_gmg(3)
    h = ss.Gmg(g)
    nb = 8192
    P = synth.placements(g, 3, 0, nb)
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    ref = oracle.simulate_batch(g, P, dispatch=mode, n_threads=8)
    ss.release_cached_memory()
    torch.cuda.empty_cache()
    roomy = ss.chunking(h, nb, dispatch=dispatch)
    _, pref = ss.workspace_size(h, nb, dispatch=dispatch)
    free, _ = torch.cuda.mem_get_info()
    left = pref // 2 + 3 * g.n_ops * nb  # about half the preferred scratch, plus the test's own tensors
    print(f"roomy chunking {roomy}, preferred scratch {pref / 1e9:.2f} GB, holding {(free - left) / 1e9:.1f} GB",
          flush=True)
    hold = torch.empty(free - left, dtype=torch.uint8, device=dev)
    try:
        tight = ss.chunking(h, nb, dispatch=dispatch)
        print(f"tight chunking {tight}", flush=True)
        assert tight[0] <= roomy[0] and tight[1] < roomy[1], (roomy, tight)
        assert_same(run(h, P, dev, dispatch=dispatch), ref, f"scratch fitted to the memory left ({dispatch})")
    finally:
        del hold
        torch.cuda.empty_cache()


def test_time_bits_follow_the_path(dev, monkeypatch):
    """ss_simulate_time_bits names the integers the call computes its times
    in: 32 on the 32-bit kernels, 64 on the general path."""
    monkeypatch.delenv("SS_PATH", raising=False)
    h = ss.Gmg(synth.build_gmg(4))
    assert ss.time_bits(h) == 32
    assert ss.time_bits(h, dispatch="ready") == 32
    assert ss.time_bits(h, links="ports") == 64
    monkeypatch.setenv("SS_PATH", "generic")
    assert ss.time_bits(h) == 64
    monkeypatch.delenv("SS_PATH")
    g = random_gmg(11, n_ops=90, n_dev=4, n_req=2, n_slices=4, n_link=2, cap_scale=2000)
    shift = 1 << 33  # slices beyond 2^32 us: the loader keeps the GMG off the 32-bit tables
    g.slice_begin = g.slice_begin + shift
    g.slice_end = np.where(g.slice_end == synth.TIME_INF, synth.TIME_INF, g.slice_end + shift)
    assert ss.time_bits(ss.Gmg(g)) == 64
