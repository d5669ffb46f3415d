"""Benchmark of the batched what-if simulator on one MI355X.

One step = the whole hot path over one batch: ss_simulate_batch on every
candidate of the workload (schedule, memory peak, verdicts, slack) followed by
ss_select_best.  Placements are generated and staged in HBM before timing.

Prints one JSON line.  The default workload is the cluster-scale one (50,000
ops of 16 tenants on 128 simulated devices, 1,048,576 candidates).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate placements simulated/sec (+ op-evals/sec, % HBM roofline), 1 GPU"
HBM_PEAK_GBS = 8000.0
COPY_BYTES = 1 << 31  # device-to-device copy: achievable bandwidth, and the counter calibration kernel
# Measured HBM traffic of the kernels (rocprofv3 read requests by size and
# WRITE_SIZE), valid while the kernel sources hash as recorded there.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_16tenant-50kop-128dev.md")
KERNEL_SOURCES = ("paper_2608_15762_amd/csrc/sim_fast.hip", "paper_2608_15762_amd/csrc/gmg_load.cpp")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=4, help="workload id 0-4 (4 = cluster scale)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gen-chunk", type=int, default=32768, help="candidates generated per host chunk")
    ap.add_argument("--candidates", type=int, default=0, help="first N candidates only (default: the whole batch)")
    ap.add_argument("--dispatch", choices=("index", "ready"), default="index",
                    help="device queues in index order (default) or earliest ready time first")
    ap.add_argument("--links", choices=("latency", "ports"), default="latency",
                    help="transfers take their estimate (default) or contend for device send/receive ports")
    ap.add_argument("--part", choices=("simulate", "estimator", "sched"), default="simulate",
                    help="the what-if simulator (default), the online estimators, or the incremental loop")
    ap.add_argument("--pipeline", type=int, default=0, metavar="CHUNK",
                    help="also time the batch streamed through the GPU in CHUNK-candidate pieces (host generation, "
                         "host-to-device copy and simulation overlapped; reported beside value, not as it)")
    ap.add_argument("--batch-cap", type=int, default=400, help="incremental loop: ops per batch")
    ap.add_argument("--budget", type=int, default=1600, help="incremental loop: issued-op budget")
    ap.add_argument("--prefix-reuse", action="store_true",
                    help="incremental loop: resume candidates from the last issuing round's capture while no "
                         "completion came in between")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """{kernel: HBM bytes per candidate} from the committed counter summary, or
    {} when it is missing or was taken on other kernel sources."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return {}
    out, src = {}, None
    for line in text.splitlines():
        if line.startswith("source_hash:"):
            src = line.split(":", 1)[1].strip()
        elif line.startswith("bytes_per_candidate:"):
            name, val = line.split(":", 1)[1].split()
            out[name] = float(val)
    return out if src == kernel_source_hash() else {}


def copy_bandwidth(torch, dev):
    """Achievable HBM bandwidth: a device-to-device copy of COPY_BYTES (read + write)."""
    a = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 5
    del a, b
    return 2 * COPY_BYTES / (ms * 1e-3) / 1e9


def stage_placements(torch, synth, g, cid, B, dev, chunk):
    """Generate the candidate batch on the host in chunks and copy it into one
    device tensor [B, N] (row-major uint8)."""
    N = g.n_ops
    P = torch.empty((B, N), dtype=torch.uint8, device=dev)
    chunk = max(1, min(chunk, B))
    bufs = [torch.empty((chunk, N), dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    events = [None, None]
    base = None
    rec = synth.CONFIGS[cid].placement
    if rec["mode_even"] == 1 or rec["mode_odd"] == 1:
        base = synth.base_placement(g, cid)
    for i, b0 in enumerate(range(0, B, chunk)):
        nb = min(chunk, B - b0)
        k = i % 2
        if events[k] is not None:
            events[k].synchronize()
        synth.placements(g, cid, b0, nb, out=bufs[k].numpy()[:nb], base=base)
        P[b0:b0 + nb].copy_(bufs[k][:nb], non_blocking=True)
        events[k] = torch.cuda.Event()
        events[k].record()
    torch.cuda.synchronize()
    return P


def pipeline_rate(torch, ss, synth, g, cid, h, B, chunk, out, best):
    """The batch streamed through the GPU: the host generator fills a ring of
    three pinned chunk buffers, each chunk is copied to one of two device slots
    on a copy stream while the previous chunk is simulated.  Returns (candidates
    per second over the whole stream, host-to-device GB/s of the copies)."""
    N = g.n_ops
    rec = synth.CONFIGS[cid].placement
    base = synth.base_placement(g, cid) if (rec["mode_even"] == 1 or rec["mode_odd"] == 1) else None
    ring = [torch.empty((chunk, N), dtype=torch.uint8, pin_memory=True) for _ in range(3)]
    dev = out["makespan"].device
    slots = [torch.empty((chunk, N), dtype=torch.uint8, device=dev) for _ in range(2)]
    copy_stream = torch.cuda.Stream()
    comp = torch.cuda.current_stream()
    copied = [torch.cuda.Event() for _ in range(2)]
    freed = [torch.cuda.Event() for _ in range(2)]
    host_free = [None, None, None]
    n_chunks = (B + chunk - 1) // chunk
    c_start = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks)]
    c_stop = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks)]
    # untimed warm-up: one chunk through the library, so the scratch pool holds
    # this chunk size's buffers (the resident run left a block of another size)
    ss.release_cached_memory()
    n0 = min(chunk, B)
    synth.placements(g, cid, 0, n0, out=ring[0].numpy()[:n0], base=base)
    slots[0][:n0].copy_(ring[0][:n0])
    ss.simulate_batch_into(h, slots[0][:n0], out["makespan"][:n0], out["violation"][:n0], out["peak"][:n0],
                           out["slack"][:n0], out["sumfin"][:n0], stream=comp)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i, b0 in enumerate(range(0, B, chunk)):
        nb = min(chunk, B - b0)
        r, k = i % 3, i % 2
        if host_free[r] is not None:
            host_free[r].synchronize()  # the copy that read this host buffer has finished
        synth.placements(g, cid, b0, nb, out=ring[r].numpy()[:nb], base=base)
        with torch.cuda.stream(copy_stream):
            if i >= 2:
                copy_stream.wait_event(freed[k])
            c_start[i].record(copy_stream)
            slots[k][:nb].copy_(ring[r][:nb], non_blocking=True)
            c_stop[i].record(copy_stream)
            copied[k].record(copy_stream)
            host_free[r] = torch.cuda.Event()
            host_free[r].record(copy_stream)
        comp.wait_event(copied[k])
        ss.simulate_batch_into(h, slots[k][:nb], out["makespan"][b0:b0 + nb], out["violation"][b0:b0 + nb],
                               out["peak"][b0:b0 + nb], out["slack"][b0:b0 + nb], out["sumfin"][b0:b0 + nb],
                               stream=comp)
        freed[k].record(comp)
    ss.select_best(h, out["violation"], out["sumfin"], out=best, stream=comp)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    copy_ms = sum(c_start[i].elapsed_time(c_stop[i]) for i in range(n_chunks))
    return B / elapsed, B * N / (copy_ms * 1e-3) / 1e9


def sample_rows(synth, g, cid, idx):
    """Placements of the candidates idx (the same seeded rows the GPU batch holds)."""
    rec = synth.CONFIGS[cid].placement
    base = synth.base_placement(g, cid) if (rec["mode_even"] == 1 or rec["mode_odd"] == 1) else None
    out = np.empty((len(idx), g.n_ops), np.uint8)
    for i, b in enumerate(idx):
        synth.placements(g, cid, int(b), 1, out=out[i:i + 1], base=base, n_threads=1)
    return out


def host_cpu():
    """The host's CPU model (from /proc/cpuinfo, as lscpu reports it), the
    logical CPUs this process may run on, and the thread count the baseline
    uses: all of them, or the host share the environment states for this
    GPU (OMP_NUM_THREADS), whichever is smaller."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    avail = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    threads = min(avail, int(share)) if share.isdigit() and int(share) > 0 else avail
    return model, avail, threads


def parity_indices(B, chunk, sub, n_even):
    """Evenly spaced candidates plus the first and last candidate of every
    chunk and of every memory-pass sub-chunk of the call's split."""
    idx = set(np.linspace(0, B - 1, n_even).astype(np.int64).tolist())
    for b0 in range(0, B, chunk):
        b1 = min(b0 + chunk, B)
        idx.update((b0, b1 - 1))
        for s0 in range(b0, b1, max(1, sub)):
            idx.update((s0, min(s0 + sub, b1) - 1))
    return np.array(sorted(idx), np.int64)


def cpu_baseline(g, cid, B, seconds, got, dispatch, links="latency", split=None):
    """The oracle, as it stands, on the host's cores: a one-thread rate on the
    first 4,096 candidates of the batch, then a bounded sample of the batch
    (evenly spaced, plus every chunk's and sub-chunk's first and last
    candidate) on all the threads the host share allows; every candidate it
    evaluates is compared with the GPU's results."""
    import oracle
    from paper_2608_15762_amd import synth

    model, avail, threads = host_cpu()
    mode = oracle.READY_ORDER if dispatch == "ready" else oracle.LINK_PORTS if links == "ports" else oracle.INDEX_ORDER
    og = oracle.OracleGmg(g)
    fields = ("makespan", "peak", "violation", "slack", "sumfin")

    def mismatches(idx, ref):
        return int(sum((got[f][idx] != ref[f]).reshape(len(idx), -1).any(axis=1) for f in fields).astype(bool).sum())

    # one thread, the first 4,096 candidates
    first = np.arange(min(B, 4096), dtype=np.int64)
    P1 = sample_rows(synth, g, cid, first)
    oracle.simulate_batch(og, P1[:1], dispatch=mode, n_threads=1)  # first call pays one-time costs
    t0 = time.perf_counter()
    ref1 = oracle.simulate_batch(og, P1, dispatch=mode, n_threads=1)
    wall1 = time.perf_counter() - t0
    per = wall1 / len(first)
    mism = mismatches(first, ref1)
    log(f"oracle: {per * 1e3:.2f} ms per candidate on one thread over the first {len(first)}; {mism} differ")
    # all threads, a sample sized to about `seconds` of CPU work per thread
    n_even = int(max(threads, min(B, 65536, seconds * threads / max(per, 1e-9))))
    chunk, sub = split if split else (B, B)
    idx = parity_indices(B, chunk, sub, n_even)
    log(f"oracle: timing {len(idx)} candidates on {threads} threads ({avail} CPUs available, {model})")
    P = sample_rows(synth, g, cid, idx)
    t0 = time.perf_counter()
    ref = oracle.simulate_batch(og, P, dispatch=mode, n_threads=threads)
    wall = time.perf_counter() - t0
    mism_all = mismatches(idx, ref)
    log(f"oracle: {len(idx) / wall:.1f} candidates/s; {mism_all} candidates differ from the GPU")
    return dict(value=len(idx) / wall, unit="candidates/s", cores=threads, kind="oracle",
                sample=f"{len(idx)} candidates of the same batch (indices 0..{B - 1}: evenly spaced, and the first "
                       f"and last of every chunk of {chunk} and sub-chunk of {sub}), {threads} threads, "
                       f"{wall:.1f} s wall",
                op_evals_per_s=len(idx) * g.n_ops / wall, cpu_model=model, cpus_available=avail,
                one_thread={"value": len(first) / wall1, "unit": "candidates/s",
                            "sample": f"the first {len(first)} candidates, 1 thread, {wall1:.1f} s wall"}), \
        dict(checked=int(len(idx) + len(first)), mismatching_candidates=mism_all + mism,
             chunk=int(chunk), sub_chunk=int(sub))


EST_N, EST_F, EST_SAMPLES = 65536, 5, 1 << 23  # estimators, features, samples fed back per step


def estimator_workload(seed=0):
    """Samples of 65,536 operator estimators (8 accelerator types x 8,192
    template operators) with batched-matmul features (bmnk, bmk, bkn, bmn, 1),
    scaled, grouped by estimator; noisy times from per-estimator models."""
    rng = np.random.default_rng(seed)
    counts = rng.multinomial(EST_SAMPLES, np.full(EST_N, 1.0 / EST_N))
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    shp = rng.integers(1, 64, (EST_SAMPLES, 4)).astype(np.float64)
    b, m, n, k = shp.T
    x = np.stack([b * m * n * k / 1e5, b * m * k / 1e3, b * k * n / 1e3, b * m * n / 1e3, np.ones(EST_SAMPLES)], 1)
    beta = rng.uniform(0.1, 5.0, (EST_N, EST_F))
    ids = np.repeat(np.arange(EST_N), counts)
    y = np.einsum("sf,sf->s", x, beta[ids]) * (1 + rng.normal(0, 0.02, EST_SAMPLES))
    return ptr, x, y, ids


def estimator_main(args):
    """Online estimators: one step feeds back a batch of samples and solves
    every fit; throughput in samples per second."""
    import torch

    from paper_2608_15762_amd import ss

    dev = torch.device("cuda:0")
    ptr, x, y, ids = estimator_workload()
    P, X, Y = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (ptr, x, y))
    copy_gbs = copy_bandwidth(torch, dev)
    E = ss.Estimators(EST_N, EST_F)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        E.add(P, X, Y, stream=stream)
        E.solve(stream=stream)
    torch.cuda.synchronize()
    add_ms = solve_ms = 0.0
    t0 = time.perf_counter()
    for i in range(args.steps):
        ss.kernel_timing(True)
        E.add(P, X, Y, stream=stream)
        _, ms_a = ss.kernel_time(ss.SS_KERNEL_ESTIMATOR)
        coef, status = E.solve(stream=stream)
        _, ms_s = ss.kernel_time(ss.SS_KERNEL_ESTIMATOR)
        ss.kernel_timing(False)
        add_ms += ms_a
        solve_ms += ms_s
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    value = EST_SAMPLES * args.steps / elapsed
    # algorithmic bytes of the accumulation: features and time per sample,
    # offsets, and the statistics of every estimator read and written
    stat = (EST_F * EST_F + EST_F + 1) * 8
    acc_bytes = EST_SAMPLES * (EST_F + 1) * 8 + (EST_N + 1) * 8 + 2 * EST_N * stat
    achieved = acc_bytes / (add_ms / args.steps * 1e-3) / 1e9
    result = {
        "metric": "estimator samples fitted/sec (online least squares, 1 GPU)", "value": round(value, 1),
        "unit": "samples/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"estimators-{EST_N}x{EST_F}-{EST_SAMPLES}samples", "estimators": EST_N,
                   "features": EST_F, "samples_per_step": EST_SAMPLES},
        "roofline": {"bound": "hbm", "kernel": "est_accumulate", "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5),
                     "traffic": None, "bytes_per_launch": acc_bytes, "copy_gbs": round(copy_gbs, 1)},
        "kernels": {"est_accumulate": {"launches": args.steps, "avg_ms": round(add_ms / args.steps, 4)},
                    "est_solve": {"launches": args.steps, "avg_ms": round(solve_ms / args.steps, 4)}},
    }
    E.free()
    if not args.no_cpu_baseline:
        # the oracle on a bounded sample (the estimators whose samples come
        # first), against a fresh set fed the batch once
        import oracle.estimator as oest
        F1 = ss.Estimators(EST_N, EST_F)
        F1.add(P, X, Y, stream=stream)
        coef, status = F1.solve(stream=stream)
        torch.cuda.synchronize()
        F1.free()
        n_pick = 2048
        s1 = int(ptr[n_pick])
        t0 = time.perf_counter()
        ref = oest.EstimatorSet(n_pick, EST_F)
        ref.add(ids[:s1], x[:s1], y[:s1])
        rc, rs = ref.solve()
        wall = time.perf_counter() - t0
        got_c, got_s = coef[:n_pick].cpu().numpy(), status[:n_pick].cpu().numpy()
        mism = int((got_s != rs).sum() + (~np.isclose(got_c, rc, rtol=1e-9, atol=1e-9)).any(axis=1).sum())
        result["cpu_baseline"] = {"value": round(s1 / wall, 1), "unit": "samples/s", "cores": 1, "kind": "oracle",
                                  "sample": f"the first {n_pick} estimators ({s1} samples), one thread, "
                                            f"{wall:.1f} s wall"}
        result["parity_sample"] = {"checked": n_pick, "mismatching_estimators": mism}
    print(json.dumps(result), flush=True)


def sched_run(S, g, synth, key, record=None, max_rounds=None, osch=None, deadline=None):
    """One scheduling run: rounds until every op is issued or done.  Rounds
    come at the stand-in executor's completion times: after a round that
    issues nothing, the next completion is fed back and the clock moves to it.
    With `record`, each round's (status, batch, partition, size of its
    snapshot graph) is appended (the size is read from the scheduler's state,
    outside what a caller needs).  `osch`: S is the oracle's scheduler.  Stops
    early at `max_rounds` or at the perf_counter `deadline`.  Returns (rounds,
    issued rounds)."""
    X = synth.Executor(g, key)
    rounds = issued_rounds = 0
    now = 0
    if record is not None:
        dst = np.repeat(np.arange(g.n_ops), np.diff(g.pred_ptr))  # consumer of each edge
    while (max_rounds is None or rounds < max_rounds) and (deadline is None or time.perf_counter() < deadline):
        st, batch, p = S.round(now)
        rounds += 1
        if record is not None:
            graph = 0
            if st in (0, 3):  # the snapshot's ops: issued, and done ones feeding an op not done
                state = S.state()[0] if osch is None else S.state
                done = state == 2
                open_ = np.bincount(g.pred_idx, weights=~done[dst], minlength=g.n_ops) > 0
                graph = int((state == 1).sum() + (done & open_).sum()) + (len(batch) if st == 3 else 0)
            record.append((st, tuple(batch), p, graph))
        if st == 0:
            issued_rounds += 1
            X.issue(batch, (S.state()[1] if osch is None else S.place)[batch], now)
            continue
        ev = X.next_completion()
        if ev is None:
            break
        now, v = ev
        S.complete(v, now)
    return rounds, issued_rounds


def sched_main(args):
    """The incremental loop of Alg. 1: one step is a whole scheduling run of the
    workload (every op issued), each round simulating all pre-defined
    partitions of its batch on the GPU; throughput in rounds per second."""
    import torch

    from paper_2608_15762_amd import ss, synth

    dev = torch.device("cuda:0")
    cid = args.workload
    cfg = synth.CONFIGS[cid]
    g = synth.build_gmg(cid)
    part = synth.partition_table(g, cid)
    prio = synth.request_priority(g)
    log(f"incremental loop on {cfg.name}: N={g.n_ops} partitions={len(part)} cap={args.batch_cap} "
        f"budget={args.budget}")
    copy_gbs = copy_bandwidth(torch, dev)
    reuse = args.prefix_reuse
    gpu_rec = []
    for i in range(args.warmup):
        S = ss.Scheduler(g, part, prio, args.budget, args.batch_cap, prefix_reuse=reuse)
        sched_run(S, g, synth, cid, record=gpu_rec if i == 0 else None)
        S.free()
        log(f"warmup run {i + 1}/{args.warmup} done")
    ss.kernel_timing(True)
    rounds = issued = 0
    t0 = time.perf_counter()
    for i in range(args.steps):
        S = ss.Scheduler(g, part, prio, args.budget, args.batch_cap, prefix_reuse=reuse)
        r, ir = sched_run(S, g, synth, cid)
        S.free()
        rounds += r
        issued += ir
        log(f"timed run {i + 1}/{args.steps} done: {r} rounds ({ir} issuing) in "
            f"{(time.perf_counter() - t0) / (i + 1) * 1e3:.0f} ms per run")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kernels = {}
    for k, name in ss.KERNEL_NAMES.items():
        n, ms = ss.kernel_time(k)
        kernels[name] = dict(launches=n, total_ms=round(ms, 3), avg_ms=round(ms / max(n, 1), 4))
    ss.kernel_timing(False)
    if not gpu_rec:  # no warmup: record one more run, untimed
        S = ss.Scheduler(g, part, prio, args.budget, args.batch_cap, prefix_reuse=reuse)
        sched_run(S, g, synth, cid, record=gpu_rec)
        S.free()
    # algorithmic bytes of the simulations: per candidate its placement row of
    # the round's snapshot graph and its outputs (makespan, violation, slack, sumfin)
    per_run, n_ops_sim = 0, 0
    dom = max((k for k in kernels if k != "select"), key=lambda k: kernels[k]["total_ms"])
    D, R = g.n_dev, g.n_req
    graphs = [n for st, batch, p, n in gpu_rec if st in (0, 3)]
    for n in graphs:
        per_run += len(part) * (n + 8 + 1 + 8 * R + 8)
        n_ops_sim += len(part) * n
    alg_bytes = per_run * args.steps
    achieved = alg_bytes / max(kernels[dom]["launches"], 1) / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    result = {
        "metric": "incremental scheduling rounds/sec (Alg. 1 loop, all partitions simulated per round, 1 GPU)",
        "value": round(issued / elapsed, 2), "unit": "rounds/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": f"{cfg.name}-incremental", "n_ops": g.n_ops, "partitions": len(part),
                   "batch_cap": args.batch_cap, "issue_budget": args.budget, "rounds_per_run": rounds // args.steps,
                   "issuing_rounds_per_run": issued // args.steps, "prefix_reuse": reuse,
                   "snapshot_ops_mean": round(float(np.mean(graphs)), 1) if graphs else 0,
                   "snapshot_ops_max": int(max(graphs)) if graphs else 0},
        "simulated_op_evals_per_s": round(n_ops_sim * args.steps / elapsed, 1),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 4), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 7), "traffic": None,
                     "bytes_per_launch": round(alg_bytes / max(kernels[dom]["launches"], 1)),
                     "copy_gbs": round(copy_gbs, 1)},
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        # the oracle loop on the same run, for as many rounds as fit in the CPU
        # time budget; its rounds must be the GPU's
        from oracle import sched as osch
        O = osch.Scheduler(g, part, prio, args.budget, args.batch_cap)
        rec = []
        t0 = time.perf_counter()
        sched_run(O, g, synth, cid, record=rec, osch=osch, deadline=t0 + args.cpu_seconds)
        n_issuing = sum(1 for x in rec if x[0] == 0)
        wall = time.perf_counter() - t0
        mism = sum(1 for a, b in zip(rec, gpu_rec) if a != b)
        result["cpu_baseline"] = {"value": round(n_issuing / wall, 3), "unit": "rounds/s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": f"the first {len(rec)} rounds ({n_issuing} issuing) of the same run, "
                                            f"one thread, {wall:.1f} s wall"}
        result["parity_sample"] = {"checked_rounds": len(rec), "mismatching_rounds": mism}
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.part == "estimator" and args.gpus == 1:
        return estimator_main(args)
    if args.part == "sched" and args.gpus == 1:
        return sched_main(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the candidate batch shards "
              "across GPUs by contiguous ranges, but this benchmark runs on one GPU only.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_15762_amd import ss, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cid = args.workload
    cfg = synth.CONFIGS[cid]
    g = synth.build_gmg(cid)
    B, N, D, R = cfg.n_cand, g.n_ops, g.n_dev, g.n_req
    if args.candidates > 0:
        B = min(B, args.candidates)
    log(f"workload {cfg.name}: N={N} E={g.n_edges} D={D} R={R} B={B}")
    copy_gbs = copy_bandwidth(torch, dev)
    log(f"device-to-device copy of {COPY_BYTES >> 20} MiB: {copy_gbs:.0f} GB/s")
    h = ss.Gmg(g)
    t0 = time.perf_counter()
    P = stage_placements(torch, synth, g, cid, B, dev, args.gen_chunk)
    log(f"staged {B * N / 1e9:.2f} GB of placements in HBM in {time.perf_counter() - t0:.1f} s")
    out = dict(makespan=torch.empty(B, dtype=torch.int64, device=dev),
               violation=torch.empty(B, dtype=torch.uint8, device=dev),
               peak=torch.empty((B, D), dtype=torch.int64, device=dev),
               slack=torch.empty((B, R), dtype=torch.int64, device=dev),
               sumfin=torch.empty(B, dtype=torch.int64, device=dev))
    best = torch.empty(2, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        ss.simulate_batch_into(h, P, out["makespan"], out["violation"], out["peak"], out["slack"], out["sumfin"],
                               stream=stream, dispatch=args.dispatch, links=args.links)
        ss.select_best(h, out["violation"], out["sumfin"], out=best, stream=stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    ss.kernel_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        torch.cuda.synchronize()
        log(f"timed step {i + 1}/{args.steps} done ({(time.perf_counter() - t0) / (i + 1) * 1e3:.1f} ms/step)")
    elapsed = time.perf_counter() - t0
    kernels = {}
    for k, name in ss.KERNEL_NAMES.items():
        n, ms = ss.kernel_time(k)
        kernels[name] = dict(launches=n, total_ms=round(ms, 3), avg_ms=round(ms / max(n, 1), 4))
    ss.kernel_timing(False)

    value = B * args.steps / elapsed
    bytes_per_cand = N + 8 + 8 * D + 1 + 8 * R + 8  # placements in; makespan, peak, violation, slack, sumfin out
    dom = max((k for k in kernels if k != "select"), key=lambda k: kernels[k]["total_ms"])
    launches_per_step = max(1, kernels[dom]["launches"] // args.steps)
    cand_per_launch = B / launches_per_step
    achieved = bytes_per_cand * cand_per_launch / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    traffic = measured_traffic().get(dom) if args.dispatch == "index" and args.links == "latency" else None
    if traffic is not None:
        traffic = round(traffic * cand_per_launch)
    # the integers the simulation computes its times in (the 32-bit kernels
    # when the loader proved every time of the workload fits)
    dtype = "u32" if ss.time_bits(h, args.dispatch, args.links) == 32 else "int64"
    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "candidates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "n_ops": N, "n_edges": g.n_edges, "n_dev": D, "n_req": R,
                   "candidates": B, "idle_slices_per_device": cfg.n_slices, "dispatch": args.dispatch,
                   "links": args.links},
        "op_evals_per_s": round(value * N, 1),
        "path_hbm_frac": round(value * bytes_per_cand / (HBM_PEAK_GBS * 1e9), 6),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6), "traffic": traffic,
                     "bytes_per_candidate": bytes_per_cand, "candidates_per_launch": cand_per_launch,
                     "copy_gbs": round(copy_gbs, 1)},
        "kernels": kernels,
    }
    torch.cuda.synchronize()
    bi, bk = best.cpu().tolist()
    result["best"] = {"index": bi, "sumfin": bk}
    if args.pipeline > 0:
        log(f"streaming the batch through the GPU in chunks of {args.pipeline}")
        rate, h2d = pipeline_rate(torch, ss, synth, g, cid, h, B, args.pipeline, out, best)
        bi2, bk2 = best.cpu().tolist()
        result["pipeline"] = {"chunk": args.pipeline, "value": round(rate, 1), "unit": "candidates/s",
                              "h2d_gbs": round(h2d, 1), "same_best": (bi2, bk2) == (bi, bk)}
    if not args.no_cpu_baseline:
        got = {k: v.cpu().numpy() for k, v in out.items()}
        log("running the oracle CPU baseline")
        cb, par = cpu_baseline(g, cid, B, args.cpu_seconds, got, args.dispatch, args.links,
                               split=ss.chunking(h, B, dispatch=args.dispatch))
        result["cpu_baseline"] = cb
        result["parity_sample"] = par
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
