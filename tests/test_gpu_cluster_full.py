"""The cluster-scale workload (50,000 ops, 128 devices, 16 requests) at its
full batch of 1,048,576 candidates, in the launch configuration the benchmark
times: one ss_simulate_batch call over the whole batch resident in HBM, split
by the library into chunks and memory-pass sub-chunks (three record sets on
two streams).  The oracle cannot cover a million candidates on the host in
seconds, so it checks a sample, each output bit for bit: evenly spaced
candidates and the first and last candidate of every chunk and of every
sub-chunk of the call.  Both dispatch rules: index order (the benchmark's)
and earliest ready time first.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2608_15762_amd import ss, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CID = 4
FIELDS = ("makespan", "peak", "violation", "slack", "sumfin")
THREADS = max(1, min(16, os.cpu_count() or 1))


def sample(B, chunk, sub, n_even):
    idx = set(np.linspace(0, B - 1, n_even).astype(np.int64).tolist())
    for b0 in range(0, B, chunk):
        b1 = min(b0 + chunk, B)
        idx.update((b0, b1 - 1))
        for s0 in range(b0, b1, max(1, sub)):
            idx.update((s0, min(s0 + sub, b1) - 1))
    return np.array(sorted(idx), np.int64)


@pytest.mark.parametrize("dispatch", ["index", "ready"])
def test_cluster_batch_sampled(dispatch):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.empty_cache()
    g = synth.build_gmg(CID)
    B, N, D, R = synth.CONFIGS[CID].n_cand, g.n_ops, g.n_dev, g.n_req
    rec = synth.CONFIGS[CID].placement
    base = synth.base_placement(g, CID) if (rec["mode_even"] == 1 or rec["mode_odd"] == 1) else None
    print(f"cluster workload: staging {B} candidates of {N} ops", flush=True)
    P = torch.empty((B, N), dtype=torch.uint8, device=dev)
    step = 32768
    buf = torch.empty((step, N), dtype=torch.uint8, pin_memory=True)
    for b0 in range(0, B, step):
        nb = min(step, B - b0)
        synth.placements(g, CID, b0, nb, out=buf.numpy()[:nb], base=base)
        P[b0:b0 + nb].copy_(buf[:nb])  # synchronous: the buffer is refilled next
    out = dict(makespan=torch.empty(B, dtype=torch.int64, device=dev),
               violation=torch.empty(B, dtype=torch.uint8, device=dev),
               peak=torch.empty((B, D), dtype=torch.int64, device=dev),
               slack=torch.empty((B, R), dtype=torch.int64, device=dev),
               sumfin=torch.empty(B, dtype=torch.int64, device=dev))
    h = ss.Gmg(g)
    chunk, sub = ss.chunking(h, B, dispatch=dispatch)
    print(f"one call over {B} candidates ({dispatch}): chunks of {chunk}, sub-chunks of {sub}", flush=True)
    ss.simulate_batch_into(h, P, out["makespan"], out["violation"], out["peak"], out["slack"], out["sumfin"],
                           dispatch=dispatch)
    torch.cuda.synchronize()
    idx = sample(B, chunk, sub, 400)
    got = {f: out[f][torch.from_numpy(idx).to(dev)].cpu().numpy() for f in FIELDS}
    del P, out
    torch.cuda.empty_cache()
    ss.release_cached_memory()
    print(f"oracle on {len(idx)} sampled candidates, {THREADS} threads", flush=True)
    Ps = np.empty((len(idx), N), np.uint8)
    for i, b in enumerate(idx):
        synth.placements(g, CID, int(b), 1, out=Ps[i:i + 1], base=base, n_threads=1)
    mode = oracle.INDEX_ORDER if dispatch == "index" else oracle.READY_ORDER
    ref = oracle.simulate_batch(g, Ps, dispatch=mode, n_threads=THREADS)
    for f in FIELDS:
        if not np.array_equal(got[f], ref[f]):
            bad = np.argwhere(got[f] != ref[f])[:5]
            pytest.fail(f"{f} differs at sampled rows {bad.tolist()} (candidates "
                        f"{idx[bad[:, 0]].tolist()}): gpu {got[f][tuple(bad[0])]} oracle {ref[f][tuple(bad[0])]}")
