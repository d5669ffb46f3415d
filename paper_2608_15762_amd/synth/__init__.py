"""Seeded synthetic inputs for the GMG what-if simulator.

This module builds Global Mapping Graph snapshots (Sec. 3.2) and batches of
candidate placements shaped like the paper's serving workloads.  It holds none
of the simulator's arithmetic (no ready times, no slice fitting, no transfer
costs, no memory accounting): only workload shapes, seeded draws and the
deadline/capacity parameters that define an input.  Both the oracle and the
HIP path consume what it produces, and it imports neither.

Workload recipe (stand-in for the paper's production traces and Llama-3 runs,
which are not available):

* Operators are Llama-style transformer layers, 10 ops per layer
  (rmsnorm, qkv, attn, o_proj, add, rmsnorm, gate_up, act, down, add) plus
  embed / lm_head, with two residual skip edges per layer (the layer-granular
  scheduling unit of Sec. 5.1).  Successive instances of one request are
  chained last op -> first op ("serving requests form dependency chains across
  graph instances", Sec. 3.4.2).
* Durations stand in for the linear operator estimator of Sec. 3.3.1: a
  roofline max(flops / 2.5e15, bytes / 8e12) seconds, rounded up to whole
  microseconds; output tensor sizes are the bf16 activation shapes.
* Idle slices follow the idle-slice statistics of the trace replay (Sec. 2,
  Fig. trace_replay): lognormal, median 2551.11 ms, sigma 1.0; busy windows are
  lognormal with median 2551.11 * 0.64 / 0.36 ms so that utilisation is 64% in
  expectation; each device starts at a random phase (busy with probability
  0.64, first window a uniform residual) so devices rarely align (Sec. 2).
* Every random number is SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) used
  as a counter-based generator: draw(key, n) = mix(key + (n + 1) * gamma).

Units: times are int64 microseconds, sizes int64 bytes.
"""
from __future__ import annotations

import copy
import ctypes
import heapq
import math
import os
import subprocess
import threading
from dataclasses import dataclass, field

import numpy as np

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
TIME_INF = (1 << 63) - 1
KiB, MiB, GiB = 1 << 10, 1 << 20, 1 << 30

# purposes (sub-stream ids under a config seed)
_P_OPS, _P_SLICES, _P_CAPS, _P_DEADLINES, _P_PLACEMENTS, _P_CALIB = 1, 2, 3, 4, 5, 6


def mix(z: int) -> int:
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def draw(key: int, n: int) -> int:
    """n-th SplitMix64 output under ``key`` (counter-based form)."""
    return mix((key + (n + 1) * GAMMA) & M64)


def mix_np(z: np.ndarray) -> np.ndarray:
    """mix over a uint64 array (multiplications wrap modulo 2^64, as in mix)."""
    z = np.asarray(z, np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def draw_np(key, n: np.ndarray) -> np.ndarray:
    """draw(key, n) for every n of an array (key an int or a uint64 array)."""
    with np.errstate(over="ignore"):
        return mix_np(np.asarray(key, np.uint64) + (np.asarray(n, np.uint64) + np.uint64(1)) * np.uint64(GAMMA))


def below(x: int, n: int) -> int:
    """floor(x * n / 2^64): maps a 64-bit draw to [0, n)."""
    return (int(x) * int(n)) >> 64


class Stream:
    """Sequential reader of one counter-based SplitMix64 stream."""

    def __init__(self, key: int):
        self.key = key & M64
        self.n = 0

    def next(self) -> int:
        x = draw(self.key, self.n)
        self.n += 1
        return x

    def uniform_int(self, lo: int, hi: int) -> int:
        lo, hi = int(lo), int(hi)
        return lo + below(self.next(), hi - lo + 1)

    def unit(self) -> float:
        """Uniform double in (0, 1]."""
        return ((self.next() >> 11) + 1) * (1.0 / (1 << 53))

    def normal(self) -> float:
        """Standard normal by Box-Muller (cosine branch)."""
        u1, u2 = self.unit(), self.unit()
        return math.sqrt(-2.0 * math.log(u1)) * math.cos(2.0 * math.pi * u2)

    def lognormal_us(self, median_us: float, sigma: float) -> int:
        return max(1, int(math.floor(median_us * math.exp(sigma * self.normal()) + 0.5)))


# --------------------------------------------------------------------------------------
# Operator shapes (bf16).  Decode: batch M=16 tokens at context L=2048.  Prefill: T=4096
# tokens, causal attention, lm_head on the last token only.
MODELS = {
    "8b": dict(H=4096, F=14336, nq=32, nkv=8, hd=128, layers=32, io=True),
    "70b": dict(H=8192, F=28672, nq=64, nkv=8, hd=128, layers=20, io=False),  # one 20-layer shard
    "1b": dict(H=2048, F=8192, nq=32, nkv=8, hd=64, layers=16, io=True),
}
VOCAB = 128256
DECODE_M, DECODE_CTX, PREFILL_T = 16, 2048, 4096
LAYER_KINDS = ("rmsnorm", "qkv", "attn", "o_proj", "add", "rmsnorm", "gate_up", "act", "down", "add")


def op_cost(model: str, phase: str, kind: str) -> tuple[int, int, int]:
    """(flops, bytes moved, output bytes) of one operator."""
    m = MODELS[model]
    H, F = m["H"], m["F"]
    Q, Hk = m["nq"] * m["hd"], m["nkv"] * m["hd"]
    M = DECODE_M if phase == "decode" else PREFILL_T
    if kind == "qkv":
        return 2 * M * H * (Q + 2 * Hk), 2 * H * (Q + 2 * Hk) + 2 * M * H + 2 * M * (Q + 2 * Hk), 2 * M * (Q + 2 * Hk)
    if kind == "attn":
        if phase == "decode":
            L = DECODE_CTX
            return 4 * M * L * Q, 4 * M * L * Hk + 2 * M * (Q + 2 * Hk) + 2 * M * Q, 2 * M * Q
        T = PREFILL_T
        return 2 * T * T * Q, 2 * T * (Q + 2 * Hk) + 2 * T * Q, 2 * T * Q
    if kind == "o_proj":
        return 2 * M * Q * H, 2 * Q * H + 2 * M * Q + 2 * M * H, 2 * M * H
    if kind == "gate_up":
        return 4 * M * H * F, 4 * H * F + 2 * M * H + 4 * M * F, 4 * M * F
    if kind == "act":
        return 3 * M * F, 6 * M * F, 2 * M * F
    if kind == "down":
        return 2 * M * F * H, 2 * F * H + 2 * M * F + 2 * M * H, 2 * M * H
    if kind == "rmsnorm":
        return 4 * M * H, 4 * M * H + 2 * H, 2 * M * H
    if kind == "add":
        return M * H, 6 * M * H, 2 * M * H
    if kind == "embed":
        return 0, 4 * M * H, 2 * M * H
    if kind == "lm_head":
        Mp = M if phase == "decode" else 1
        return 2 * Mp * H * VOCAB, 2 * H * VOCAB + 2 * Mp * H + 2 * Mp * VOCAB, 2 * Mp * VOCAB
    raise ValueError(kind)


def roofline_us(flops: int, moved: int) -> int:
    """max(ceil(flops / 2.5e15 s), ceil(bytes / 8e12 s)) in whole microseconds, >= 1."""
    t_compute = (2 * flops + 5_000_000_000 - 1) // 5_000_000_000
    t_memory = (moved + 8_000_000 - 1) // 8_000_000
    return max(1, t_compute, t_memory)


def request_graph(model: str, n_inst: int | None = None, n_ops: int | None = None):
    """Op kinds and edges of one request: instances of a model's graph chained
    last -> first, optionally truncated to ``n_ops`` operators.  Local op order
    is topological (every edge goes from a lower to a higher local index)."""
    m = MODELS[model]
    kinds: list[str] = []
    edges: list[tuple[int, int]] = []

    def add(kind):
        kinds.append(kind)
        return len(kinds) - 1

    prev_out = None
    inst = 0
    while True:
        if n_inst is not None and inst >= n_inst:
            break
        if n_ops is not None and len(kinds) >= n_ops:
            break
        if m["io"]:
            emb = add("embed")
            if prev_out is not None:
                edges.append((prev_out, emb))
            resid, chain = emb, emb
        else:
            resid, chain = prev_out, prev_out
        for _ in range(m["layers"]):
            n1 = add("rmsnorm")
            if chain is not None:
                edges.append((chain, n1))
            q = add("qkv"); edges.append((n1, q))
            a = add("attn"); edges.append((q, a))
            o = add("o_proj"); edges.append((a, o))
            a1 = add("add"); edges.append((o, a1))
            if resid is not None:
                edges.append((resid, a1))  # residual skip: layer input -> first add
            n2 = add("rmsnorm"); edges.append((a1, n2))
            g = add("gate_up"); edges.append((n2, g))
            ac = add("act"); edges.append((g, ac))
            dn = add("down"); edges.append((ac, dn))
            a2 = add("add"); edges.append((dn, a2))
            edges.append((a1, a2))  # residual skip: first add -> second add
            resid, chain = a2, a2
        if m["io"]:
            lm = add("lm_head"); edges.append((resid, lm))
            prev_out = lm
        else:
            prev_out = resid
        inst += 1
    if n_ops is not None and len(kinds) > n_ops:
        kinds = kinds[:n_ops]
        edges = [(u, v) for (u, v) in edges if v < n_ops]
    return kinds, edges


# --------------------------------------------------------------------------------------
@dataclass
class Config:
    cid: int
    name: str
    seed: int
    n_dev: int
    n_nodes: int
    n_slices: int
    n_cand: int
    tenants: list  # (model, phase, n_inst, n_ops) per request; model None = tiny random
    placement: dict  # recipe for the candidate generator
    cap_kind: str
    deadline_kind: str
    clip_slices: bool = False
    n_tiny_ops: int = 0


# Capacity of the tight-memory workload: the nearest-rank 70th percentile of
# max_d peak[d] over 4,096 uniform random placements of that workload (so that
# about 30% of random placements violate).  Written by
# tests/golden/calibrate_memory_cap.py, which runs only the oracle.
TIGHT_CAP_BYTES = 587_333_632

CONFIGS = {
    0: Config(0, "tiny-2dev-32op", 0, 2, 1, 4, 256, [(None, "decode", 1, None)],
              dict(mode_even=0, mode_odd=0, kmin=0, kmax=0, distinct=0), "tiny", "x1500", n_tiny_ops=32),
    1: Config(1, "llama8b-decode-8dev", 1, 8, 2, 16, 65536, [("8b", "decode", 1, None)],
              dict(mode_even=0, mode_odd=0, kmin=0, kmax=0, distinct=0), "hbm288", "x1500"),
    2: Config(2, "4tenant-32dev", 2, 32, 4, 64, 262144,
              [("8b", "decode", 2, None), ("8b", "prefill", 1, None), ("70b", "decode", 3, None), ("1b", "decode", 3, None)],
              dict(mode_even=1, mode_odd=1, kmin=0, kmax=16, distinct=0), "hbm288", "uniform1200_2000"),
    3: Config(3, "8tenant-10kop-64dev", 3, 64, 8, 64, 131072,
              [("8b", "prefill" if t % 4 == 3 else "decode", None, 1250) for t in range(8)],
              dict(mode_even=1, mode_odd=1, kmin=1, kmax=8, distinct=1), "tight", "uniform1200_2000"),
    4: Config(4, "16tenant-50kop-128dev", 4, 128, 16, 256, 1048576,
              [(("1b", "8b", "70b")[t % 3], "prefill" if t % 4 == 3 else "decode", None, 3125) for t in range(16)],
              dict(mode_even=0, mode_odd=1, kmin=1, kmax=16, distinct=1), "hbm288", "uniform1200_2000",
              clip_slices=True),
}


@dataclass
class Gmg:
    """A GMG snapshot in the array form both the oracle and the library take."""
    n_ops: int
    n_dev: int
    n_class: int
    n_link: int
    n_req: int
    pred_ptr: np.ndarray      # int32 [N+1]  CSR over predecessors
    pred_idx: np.ndarray      # int32 [E]    every entry < its op's index
    op_req: np.ndarray        # int32 [N]
    dur: np.ndarray           # int64 [N, C] microseconds, >= 1
    out_bytes: np.ndarray     # int64 [N]
    dev_class: np.ndarray     # int32 [D]
    link_class: np.ndarray    # uint8 [D, D]
    bw: np.ndarray            # int64 [K] bytes per microsecond
    lat: np.ndarray           # int64 [K] microseconds
    slice_ptr: np.ndarray     # int64 [D+1]
    slice_begin: np.ndarray   # int64 [S_total]
    slice_end: np.ndarray     # int64 [S_total]; the last slice of each device ends at TIME_INF
    cap: np.ndarray           # int64 [D] bytes
    release: np.ndarray       # int64 [R]
    deadline: np.ndarray      # int64 [R]
    kinds: list = field(default_factory=list)
    tenant_of: np.ndarray | None = None
    name: str = ""
    # a snapshot of a running schedule (optional): recorded completion time of
    # each done op (-1: not done), issue time of each op, the snapshot's time
    done_fin: np.ndarray | None = None   # int64 [N]
    issue_at: np.ndarray | None = None   # int64 [N]
    t_now: int = 0

    @property
    def n_edges(self) -> int:
        return int(self.pred_ptr[-1])

    def edges(self):
        for v in range(self.n_ops):
            for e in range(self.pred_ptr[v], self.pred_ptr[v + 1]):
                yield int(self.pred_idx[e]), v


def make_gmg(n_dev, kinds, edges, op_req, dur, out_bytes, slices, cap, release, deadline,
             link_class=None, bw=(50_000,), lat=(0,), dev_class=None, name="") -> Gmg:
    """Assemble a Gmg from plain Python lists (edges as (u, v) with u < v)."""
    N = len(dur)
    preds = [[] for _ in range(N)]
    for u, v in edges:
        preds[v].append(u)
    pred_ptr = np.zeros(N + 1, np.int32)
    for v in range(N):
        pred_ptr[v + 1] = pred_ptr[v] + len(preds[v])
    pred_idx = np.array([u for v in range(N) for u in sorted(preds[v])], np.int32)
    dur_arr = np.asarray(dur, np.int64).reshape(N, -1) if N else np.zeros((0, 1), np.int64)
    D = n_dev
    if link_class is None:
        link_class = np.zeros((D, D), np.uint8)
    if dev_class is None:
        dev_class = np.zeros(D, np.int32)
    sp = np.zeros(D + 1, np.int64)
    sb, se = [], []
    for d in range(D):
        for a, e in slices[d]:
            sb.append(a)
            se.append(e)
        sp[d + 1] = len(sb)
    return Gmg(N, D, dur_arr.shape[1] if N else 1, len(bw), len(release),
               pred_ptr, pred_idx, np.asarray(op_req, np.int32), dur_arr,
               np.asarray(out_bytes, np.int64), np.asarray(dev_class, np.int32),
               np.asarray(link_class, np.uint8), np.asarray(bw, np.int64), np.asarray(lat, np.int64),
               sp, np.asarray(sb, np.int64), np.asarray(se, np.int64), np.asarray(cap, np.int64),
               np.asarray(release, np.int64), np.asarray(deadline, np.int64), list(kinds), None, name)


# --------------------------------------------------------------------------------------
IDLE_MEDIAN_US = 2_551_110.0                  # p50 idle slice (trace replay, Sec. 2)
BUSY_MEDIAN_US = 2_551_110.0 * 0.64 / 0.36    # 64% utilisation in expectation
P_BUSY_FIRST = 0.64
CLIP_LO_US, CLIP_HI_US = 10_000, 20_000_000   # only slices in (10 ms, 20 s) were kept


def device_slices(key: int, n_slices: int, clip: bool) -> list[tuple[int, int]]:
    """``n_slices`` finite idle slices separated by busy windows, then an open tail."""
    st = Stream(key)

    def idle():
        x = st.lognormal_us(IDLE_MEDIAN_US, 1.0)
        return min(max(x, CLIP_LO_US), CLIP_HI_US) if clip else x

    def busy():
        x = st.lognormal_us(BUSY_MEDIAN_US, 1.0)
        return min(max(x, CLIP_LO_US), CLIP_HI_US) if clip else x

    t = 0
    first_busy = st.unit() <= P_BUSY_FIRST
    if first_busy:
        t += max(1, int(st.unit() * busy()))
    out = []
    for k in range(n_slices):
        length = idle()
        if k == 0 and not first_busy:
            length = max(1, int(st.unit() * length))
        out.append((t, t + length))
        t = t + length + busy()
    out.append((t, TIME_INF))
    return out


def _merge_requests(reqs):
    """Merge per-request graphs into one index order: by isolated ASAP start time
    (longest path of durations from the request's sources), then request id,
    then local index.  Because every duration is >= 1 this is topological."""
    keyed = []
    for r, (kinds, edges, durs, obytes) in enumerate(reqs):
        n = len(kinds)
        preds = [[] for _ in range(n)]
        for u, v in edges:
            preds[v].append(u)
        asap = [0] * n
        for v in range(n):
            for u in preds[v]:
                asap[v] = max(asap[v], asap[u] + durs[u])
        for v in range(n):
            keyed.append((asap[v], r, v))
    keyed.sort()
    gid = {}
    for i, (_, r, v) in enumerate(keyed):
        gid[(r, v)] = i
    N = len(keyed)
    kinds_all, op_req, dur, obytes = [None] * N, [0] * N, [0] * N, [0] * N
    edges_all = []
    for r, (kinds, edges, durs, ob) in enumerate(reqs):
        for v in range(len(kinds)):
            i = gid[(r, v)]
            kinds_all[i], op_req[i], dur[i], obytes[i] = kinds[v], r, durs[v], ob[v]
        for u, v in edges:
            edges_all.append((gid[(r, u)], gid[(r, v)]))
    return kinds_all, edges_all, op_req, dur, obytes


def build_gmg(cid: int) -> Gmg:
    cfg = CONFIGS[cid]
    seed = cfg.seed
    reqs = []
    if cfg.n_tiny_ops:
        # three Llama-style layers (30 ops) + embed + lm_head = 32 ops, 37 edges
        kinds, edges = request_graph("8b", n_inst=1)
        keep = 1 + 3 * 10
        kinds = kinds[:keep] + ["lm_head"]
        edges = [(u, v) for (u, v) in edges if v < keep] + [(keep - 1, keep)]
        st = Stream(draw(seed, _P_OPS))
        durs = [st.uniform_int(50, 2000) for _ in kinds]
        ob = [st.uniform_int(64 * KiB, 64 * MiB) for _ in kinds]
        reqs.append((kinds, edges, durs, ob))
    else:
        for model, phase, n_inst, n_ops in cfg.tenants:
            kinds, edges = request_graph(model, n_inst=n_inst, n_ops=n_ops)
            costs = [op_cost(model, phase, k) for k in kinds]
            durs = [roofline_us(f, m) for f, m, _ in costs]
            ob = [o for _, _, o in costs]
            reqs.append((kinds, edges, durs, ob))
    kinds, edges, op_req, dur, obytes = _merge_requests(reqs)
    D = cfg.n_dev
    dpn = D // cfg.n_nodes
    node = [d // dpn for d in range(D)]
    if cfg.n_nodes > 1:
        link = np.array([[0 if node[s] == node[t] else 1 for t in range(D)] for s in range(D)], np.uint8)
        bw, lat = (50_000, 12_500), (0, 0)
    else:
        link = np.zeros((D, D), np.uint8)
        bw, lat = (50_000,), (0,)
    skey = draw(seed, _P_SLICES)
    slices = [device_slices(draw(skey, d), cfg.n_slices, cfg.clip_slices) for d in range(D)]
    cst = Stream(draw(seed, _P_CAPS))
    if cfg.cap_kind == "tiny":
        cap = [4 * GiB - cst.uniform_int(1 * GiB, 3 * GiB) for _ in range(D)]
    elif cfg.cap_kind == "hbm288":
        cap = [288 * GiB - cst.uniform_int(150 * GiB, 250 * GiB) for _ in range(D)]
    elif cfg.cap_kind == "tight":
        cap = [TIGHT_CAP_BYTES if TIGHT_CAP_BYTES is not None else 288 * GiB] * D
    else:
        raise ValueError(cfg.cap_kind)
    R = len(reqs)
    iso = [0] * R
    for v, r in enumerate(op_req):
        iso[r] += dur[v]
    dst = Stream(draw(seed, _P_DEADLINES))
    release = [0] * R
    if cfg.deadline_kind == "x1500":
        permille = [1500] * R
    else:
        permille = [dst.uniform_int(1200, 2000) for _ in range(R)]
    deadline = [release[r] + (permille[r] * iso[r] + 999) // 1000 for r in range(R)]
    g = make_gmg(D, kinds, edges, op_req, dur, obytes, slices, cap, release, deadline,
                 link_class=link, bw=bw, lat=lat, name=cfg.name)
    g.tenant_of = np.asarray(op_req, np.int32)
    return g


def base_placement(g: Gmg, cid: int) -> np.ndarray:
    """Partition base placement (the pre-defined partitions of Sec. 3.4.2): request r
    runs on node r mod n_nodes; its operators, in index order, are cut into as many
    contiguous pipeline stages as the node has devices, balanced by cumulative
    duration, and stage s goes to the node's s-th device ordered by the start of its
    first idle slice (earliest available first, ties to the lower id)."""
    cfg = CONFIGS[cid]
    D = g.n_dev
    dpn = D // cfg.n_nodes
    first_idle = [int(g.slice_begin[g.slice_ptr[d]]) for d in range(D)]
    p = np.zeros(g.n_ops, np.uint8)
    for r in range(g.n_req):
        ops = np.nonzero(g.op_req == r)[0]
        node = r % cfg.n_nodes
        devs = sorted(range(node * dpn, (node + 1) * dpn), key=lambda d: (first_idle[d], d))
        w = g.dur[ops, 0]
        total = int(w.sum())
        before = 0
        for v, wv in zip(ops, w):
            stage = min(dpn - 1, (before * dpn) // max(total, 1))
            p[v] = devs[stage]
            before += int(wv)
    return p


def partition_table(g: Gmg, cid: int) -> np.ndarray:
    """Pre-defined partitions for the incremental loop (Sec. 3.4.2): for every node
    and every group size k in (devices per node, half of it, ..., 1), the node's
    devices (by id) split into groups of k; each group is one partition.  The
    mapping of a request's ops onto a partition is fixed: its ops, in index order,
    cut into k contiguous stages balanced by cumulative duration, stage s on the
    group's s-th device.  Returns part_dev [n_part][n_ops] (uint8)."""
    cfg = CONFIGS[cid]
    D = g.n_dev
    dpn = D // cfg.n_nodes
    sizes = []
    k = dpn
    while k >= 1:
        sizes.append(k)
        k //= 2
    groups = [list(range(n * dpn + j * k, n * dpn + (j + 1) * k))
              for n in range(cfg.n_nodes) for k in sizes for j in range(dpn // k)]
    out = np.zeros((len(groups), g.n_ops), np.uint8)
    for r in range(g.n_req):
        ops = np.nonzero(g.op_req == r)[0]
        w = g.dur[ops, 0]
        total = max(int(w.sum()), 1)
        before = np.concatenate([[0], np.cumsum(w)[:-1]]) if len(ops) else np.zeros(0, np.int64)
        for p, grp in enumerate(groups):
            stage = np.minimum(len(grp) - 1, (before * len(grp)) // total)
            out[p, ops] = np.asarray(grp, np.uint8)[stage]
    return out


def random_snapshot(g: Gmg, seed: int, done_p: float = 0.5, issue_span: int = 400, t_now: int | None = None,
                    issue: bool = True) -> Gmg:
    """A copy of g holding a random state of a running schedule: every op an
    issue time in [0, issue_span] (or none with issue=False); ops done with
    probability done_p when all their predecessors are done, finishing 1-60 us
    after the later of their issue and their predecessors' finishes; the
    snapshot's timestamp t_now (default: drawn up to the latest finish)."""
    st = Stream(draw(0x5A9 + seed, 2))
    N = g.n_ops
    iss = np.array([st.uniform_int(0, issue_span) for _ in range(N)], np.int64)
    done = np.full(N, -1, np.int64)
    for v in range(N):
        preds = g.pred_idx[g.pred_ptr[v]:g.pred_ptr[v + 1]]
        if st.unit() < done_p and all(done[u] >= 0 for u in preds):
            t = max([int(iss[v]) if issue else 0] + [int(done[u]) for u in preds])
            done[v] = t + st.uniform_int(1, 60)
    h = copy.deepcopy(g)
    h.done_fin = done
    h.issue_at = iss if issue else None
    h.t_now = int(st.uniform_int(0, int(max(done.max(), 0)) + 1)) if t_now is None else int(t_now)
    return h


class Executor:
    """Stand-in for the cluster that runs what the incremental loop issues
    (Sec. 3.5), reporting completions with their times.  An issued op runs
    once its predecessors have completed: it completes at the later of its
    issue time and its predecessors' completions, plus its duration estimate
    on its device's class scaled by a seeded factor in [0.75, 1.25] (at least
    1 us).  Completions come out in time order, ties to the lower op."""

    def __init__(self, g: Gmg, key: int):
        self.g = g
        self.key = key
        N = g.n_ops
        # plain lists: the loop runs once per completion
        pp = np.asarray(g.pred_ptr).tolist()
        pi = np.asarray(g.pred_idx).tolist()
        self.preds = [pi[pp[v]:pp[v + 1]] for v in range(N)]
        self.succ = [[] for _ in range(N)]
        for v in range(N):
            for u in self.preds[v]:
                self.succ[u].append(v)
        self.waiting = [len(p) for p in self.preds]  # predecessors not yet completed
        self.dur = np.asarray(g.dur).tolist()
        self.dev_class = np.asarray(g.dev_class).tolist()
        self.issue_t = [-1] * N
        self.dev = [0] * N
        self.done_t = [-1] * N
        self.events = []  # heap of (completion time, op)
        # op v's factor: the first unit() of Stream(draw(key, 0xE7EC + v)), for all ops at once
        x = draw_np(draw_np(key & M64, np.arange(N, dtype=np.uint64) + np.uint64(0xE7EC)), np.zeros(N, np.uint64))
        self.factor = (((x >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * (1.0 / (1 << 53))).tolist()

    def _start(self, v):
        t = self.issue_t[v]
        for u in self.preds[v]:
            t = max(t, self.done_t[u])
        w = self.dur[v][self.dev_class[self.dev[v]]]
        heapq.heappush(self.events, (t + max(1, int(round(w * (0.75 + 0.5 * self.factor[v])))), v))

    def issue(self, ops, devs, t: int):
        for v, d in zip(ops, devs):
            v = int(v)
            self.issue_t[v] = int(t)
            self.dev[v] = int(d)
            if self.waiting[v] == 0:
                self._start(v)

    def next_completion(self):
        """(time, op) of the next completion, or None when nothing runs."""
        if not self.events:
            return None
        t, v = heapq.heappop(self.events)
        self.done_t[v] = t
        for x in self.succ[v]:
            self.waiting[x] -= 1
            if self.waiting[x] == 0 and self.issue_t[x] >= 0:
                self._start(x)
        return t, v


def request_priority(g: Gmg) -> np.ndarray:
    """Per-request priority of the incremental loop: the deadline (earlier first)."""
    return np.asarray(g.deadline, np.int64).copy()


# --------------------------------------------------------------------------------------
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None
_lib_lock = threading.Lock()


def build_lib(force: bool = False) -> str:
    if force or not os.path.exists(_LIB_PATH):
        src = os.path.join(_HERE, "placements.c")
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", src, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _get_lib():
    global _lib
    with _lib_lock:
        if _lib is None:
            # SS_SYNTH_LIB: another build of the same source (the sanitizer run)
            lib = ctypes.CDLL(os.environ.get("SS_SYNTH_LIB") or build_lib())
            lib.synth_placements.restype = ctypes.c_int
            lib.synth_placements.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                             ctypes.c_int32]
            lib.synth_draw.restype = ctypes.c_uint64
            lib.synth_draw.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
            _lib = lib
    return _lib


def placements_from_recipe(root: int, n_ops: int, n_dev: int, recipe: dict, base, b0: int, nb: int,
                           out: np.ndarray | None = None, n_threads: int = 0) -> np.ndarray:
    lib = _get_lib()
    if out is None:
        out = np.empty((nb, n_ops), np.uint8)
    assert out.dtype == np.uint8 and out.flags.c_contiguous and out.shape == (nb, n_ops)
    if base is not None:
        base = np.ascontiguousarray(base, np.uint8)
        assert base.shape == (n_ops,)
    if n_threads <= 0:
        n_threads = min(16, os.cpu_count() or 1)
    rc = lib.synth_placements(root & M64, n_ops, n_dev, recipe["mode_even"], recipe["mode_odd"], recipe["kmin"],
                              recipe["kmax"], recipe["distinct"],
                              base.ctypes.data if base is not None else None, b0, nb, out.ctypes.data, n_threads)
    if rc != 0:
        raise ValueError("synth_placements rejected its arguments")
    return out


def placements(g: Gmg, cid: int, b0: int, nb: int, out=None, base=None, n_threads: int = 0) -> np.ndarray:
    """Candidates b0 .. b0+nb-1 of config ``cid`` as a row-major uint8 [nb, N] array."""
    cfg = CONFIGS[cid]
    rec = cfg.placement
    if base is None and (rec["mode_even"] == 1 or rec["mode_odd"] == 1):
        base = base_placement(g, cid)
    return placements_from_recipe(draw(cfg.seed, _P_PLACEMENTS), g.n_ops, g.n_dev, rec, base, b0, nb, out, n_threads)


def uniform_placements(g: Gmg, key: int, b0: int, nb: int, n_threads: int = 0) -> np.ndarray:
    rec = dict(mode_even=0, mode_odd=0, kmin=0, kmax=0, distinct=0)
    return placements_from_recipe(key, g.n_ops, g.n_dev, rec, None, b0, nb, None, n_threads)


def calibration_key(cid: int) -> int:
    return draw(CONFIGS[cid].seed, _P_CALIB)


# --------------------------------------------------------------------------------------
# Small random GMGs for fuzzing and hand cases.
def random_gmg(seed: int, n_ops: int, n_dev: int, n_req: int = 1, edge_p: float = 0.3, max_span: int = 6,
               n_slices: int = 3, n_class: int = 1, n_link: int = 1, max_dur: int = 40, max_bytes: int = 1000,
               zero_bytes_p: float = 0.1, slice_scale: int = 60, open_only: bool = False,
               cap_scale: int | None = None, lat_max: int = 3, bw_max: int = 50, rel_max: int = 0,
               cross_req_p: float = 0.1, max_outdeg: int | None = None) -> Gmg:
    """A small random GMG: a random DAG over ``n_ops`` ops (edges u -> v with
    v - max_span <= u < v), random slices, link classes, durations and sizes.
    ``max_outdeg`` drops edges that would give an op more successors (it
    changes no draw)."""
    st = Stream(draw(0xF022 + seed, 1))
    U = st.uniform_int
    op_req = [U(0, n_req - 1) for _ in range(n_ops)]
    edges = []
    outdeg = [0] * n_ops
    for v in range(n_ops):
        for u in range(max(0, v - max_span), v):
            if st.unit() < edge_p and (op_req[u] == op_req[v] or st.unit() < cross_req_p):
                if max_outdeg is None or outdeg[u] < max_outdeg:
                    edges.append((u, v))
                    outdeg[u] += 1
    dur = [[U(1, max_dur) for _ in range(n_class)] for _ in range(n_ops)]
    ob = [0 if st.unit() < zero_bytes_p else U(1, max_bytes) for _ in range(n_ops)]
    slices = []
    for d in range(n_dev):
        t = U(0, slice_scale // 2)
        sl = []
        if not open_only:
            for _ in range(U(0, n_slices)):
                a = t
                e = a + U(1, slice_scale)
                sl.append((a, e))
                t = e + U(0, slice_scale)
        sl.append((t if not open_only else 0, TIME_INF))
        slices.append(sl)
    dev_class = [U(0, n_class - 1) for _ in range(n_dev)]
    link = np.zeros((n_dev, n_dev), np.uint8)
    for s in range(n_dev):
        for t in range(n_dev):
            link[s, t] = U(0, n_link - 1) if s != t else 0
    bw = [U(1, bw_max) for _ in range(n_link)]
    lat = [U(0, lat_max) for _ in range(n_link)]
    total_b = sum(ob) + 1
    cs = cap_scale if cap_scale is not None else total_b
    cap = [U(0, cs) for _ in range(n_dev)]
    release = [U(0, rel_max) for _ in range(n_req)]
    deadline = [release[r] + U(0, 10 * max_dur * max(1, n_ops // max(1, n_req))) for r in range(n_req)]
    return make_gmg(n_dev, ["op"] * n_ops, edges, op_req, dur, ob, slices, cap, release, deadline,
                    link_class=link, bw=bw, lat=lat, dev_class=dev_class, name=f"random{seed}")
