"""The no-allocation entry point (ss_simulate_batch_noalloc) on the GPU,
through the C ABI: two calls in a row, the second with a smaller batch, each
compared element by element with ss_simulate_batch on the same inputs (and
with the oracle); both dispatch rules and both layouts; a batch whose
smallest scratch exceeds the fixed array is refused before any launch."""
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


def outputs(h, B, dev):
    return dict(makespan=torch.empty(B, dtype=torch.int64, device=dev),
                violation=torch.empty(B, dtype=torch.uint8, device=dev),
                peak=torch.empty((B, h.n_dev), dtype=torch.int64, device=dev),
                slack=torch.empty((B, h.n_req), dtype=torch.int64, device=dev),
                sumfin=torch.empty(B, dtype=torch.int64, device=dev))


def host(o):
    return {k: v.cpu().numpy() for k, v in o.items()}


@pytest.mark.parametrize("dispatch", ["index", "ready"])
@pytest.mark.parametrize("layout", ["row", "op"])
@pytest.mark.parametrize("cid,sizes", [(0, (256, 100)), (2, (3000, 700)), (3, (1200, 130)), (4, (200, 24))])
def test_noalloc_matches_simulate_batch(dev, cid, sizes, layout, dispatch):
    g = synth.build_gmg(cid)
    h = ss.Gmg(g)
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    for call, (nb, b0) in enumerate(zip(sizes, (0, 5000))):
        print(f"config {cid}: call {call}, {nb} candidates, {layout}, {dispatch}", flush=True)
        P = synth.placements(g, cid, b0, nb)
        A = torch.from_numpy(np.ascontiguousarray(P if layout == "row" else P.T)).to(dev)
        o1, o2 = outputs(h, nb, dev), outputs(h, nb, dev)
        ss.simulate_batch_noalloc_into(h, A, o1["makespan"], o1["violation"], o1["peak"], o1["slack"],
                                       o1["sumfin"], dispatch=dispatch, layout=layout)
        ss.simulate_batch_into(h, A, o2["makespan"], o2["violation"], o2["peak"], o2["slack"], o2["sumfin"],
                               dispatch=dispatch, layout=layout)
        torch.cuda.synchronize()
        a, b = host(o1), host(o2)
        for f in FIELDS:
            assert np.array_equal(a[f], b[f]), (call, f)
        idx = np.unique(np.linspace(0, nb - 1, min(nb, 64)).astype(np.int64))
        ref = oracle.simulate_batch(g, P[idx], dispatch=mode, n_threads=8)
        for f in FIELDS:
            assert np.array_equal(a[f][idx], ref[f]), (call, f)


def test_noalloc_refuses_a_batch_beyond_its_scratch(dev):
    g = synth.build_gmg(4)
    h = ss.Gmg(g)
    B = 1 << 40
    lo, _ = ss.workspace_size(h, B)
    assert lo > 128 << 20
    tiny = torch.zeros(64, dtype=torch.uint8, device=dev)
    o = outputs(h, 1, dev)
    # the size check comes before anything touches the placements or outputs
    rc = ss.lib().ss_simulate_batch_noalloc(h.handle, ss._ptr(tiny), B, 0, ss._ptr(o["makespan"]), None,
                                            ss._ptr(o["violation"]), None, None, None)
    assert rc == ss.SS_ERR_INVALID_ARG
    assert b"fixed" in ss.lib().ss_last_error()
