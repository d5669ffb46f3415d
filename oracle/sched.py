"""Oracle for the incremental scheduling loop -- TEST INFRASTRUCTURE ONLY.

Written from the paper (SliceScheduler, arXiv 2608.15762), Sec. 3.4 and Alg. 1:
  - ops are unscheduled, issued or done;
  - the scheduled frontier holds the issued or done ops that have an
    unscheduled successor (their outputs stay on their accelerators as
    checkpoints); the unscheduled frontier holds the unscheduled ops whose
    predecessors are all issued or done (Sec. 3.4.1);
  - a round returns at once when the issued ops reach the budget or the
    unscheduled frontier is empty; otherwise it takes the highest-priority op
    of the unscheduled frontier, collects a small connected batch from it by
    following successors (capped), evaluates every pre-defined partition as a
    candidate placement of the batch by what-if simulation of the whole
    placed graph, discards infeasible candidates, keeps the one with the
    smallest simulated average completion time, writes it back and marks the
    batch issued (Alg. 1, Sec. 3.4.2).

Readings where the paper is silent (each is listed in the design notes):
  - priority: a smaller per-request priority value first (the workloads use
    the deadline), ties to the lower op index;
  - batch collection: starting from the chosen op, repeatedly add the
    lowest-index unscheduled successor of a batch op whose predecessors are
    all issued, done or already in the batch, until the cap or no such op;
  - the simulated graph of a round holds the scheduled (issued or done) ops
    in the order they were issued (the order of the device queues; a batch in
    index order), then the batch in index order: a topological order in which
    every candidate places the ops before the batch alike, and which later
    rounds only extend;
  - durations are the estimates: executor feedback marks an op done (it no
    longer counts against the budget); measured times refine the estimators
    (Sec. 3.3.1), not the simulated history;
  - candidate b is partition b; the score is the sum of finish times over the
    simulated graph (the ops before the batch are the same for every
    candidate, so the argmin is that of the batch's average completion);
    feasibility is memory only unless SLA is required; ties go to the lower
    partition index; with no feasible candidate nothing is issued.

The simulation itself is the C oracle (index-order dispatch).  Nothing here is
shared with the library.
"""
from __future__ import annotations

import numpy as np

import oracle

UNSCHEDULED, ISSUED, DONE = 0, 1, 2
ROUND_ISSUED, ROUND_BUDGET, ROUND_IDLE, ROUND_INFEASIBLE = 0, 1, 2, 3


class Scheduler:
    """The GMG of a whole run with per-op state; `part_dev[p][v]` is op v's
    device under partition p."""

    def __init__(self, g, part_dev, priority, budget: int, cap: int, require_sla: bool = False):
        self.g = g
        self.part = np.asarray(part_dev, np.uint8)
        assert self.part.ndim == 2 and self.part.shape[1] == g.n_ops
        self.priority = np.asarray(priority, np.int64)
        self.budget, self.cap, self.require_sla = int(budget), int(cap), bool(require_sla)
        N = g.n_ops
        self.state = np.full(N, UNSCHEDULED, np.uint8)
        self.place = np.zeros(N, np.uint8)
        self.issue_order = []  # scheduled ops in the order they were issued
        self.preds = [[int(g.pred_idx[e]) for e in range(g.pred_ptr[v], g.pred_ptr[v + 1])] for v in range(N)]
        self.succs = [[] for _ in range(N)]
        for v in range(N):
            for u in self.preds[v]:
                self.succs[u].append(v)

    # ---------------------------------------------------------------- frontiers (Sec. 3.4.1)
    def unscheduled_frontier(self):
        return [v for v in range(self.g.n_ops) if self.state[v] == UNSCHEDULED
                and all(self.state[u] != UNSCHEDULED for u in self.preds[v])]

    def scheduled_frontier(self):
        return [v for v in range(self.g.n_ops) if self.state[v] != UNSCHEDULED
                and any(self.state[x] == UNSCHEDULED for x in self.succs[v])]

    # ---------------------------------------------------------------- batch collection
    def collect(self, op):
        batch, inb = [op], {op}
        while len(batch) < self.cap:
            ok = [x for b in batch for x in self.succs[b]
                  if self.state[x] == UNSCHEDULED and x not in inb
                  and all(self.state[u] != UNSCHEDULED or u in inb for u in self.preds[x])]
            if not ok:
                break
            x = min(ok)
            batch.append(x)
            inb.add(x)
        return sorted(batch)

    # ---------------------------------------------------------------- the round's simulated graph
    def round_graph(self, batch):
        """(sub-GMG, op order): the scheduled ops in issue order, then the batch."""
        g = self.g
        order = self.issue_order + list(batch)
        new = {v: i for i, v in enumerate(order)}
        pred_ptr = [0]
        pred_idx = []
        for v in order:
            ps = sorted(new[u] for u in self.preds[v])
            pred_idx += ps
            pred_ptr.append(len(pred_idx))
        dur = np.array([g.dur[v] for v in order], np.int64).reshape(len(order), g.n_class)
        sub = type(g)(len(order), g.n_dev, g.n_class, g.n_link, g.n_req,
                      np.asarray(pred_ptr, np.int32), np.asarray(pred_idx, np.int32),
                      np.asarray([g.op_req[v] for v in order], np.int32), dur,
                      np.asarray([g.out_bytes[v] for v in order], np.int64), g.dev_class, g.link_class, g.bw, g.lat,
                      g.slice_ptr, g.slice_begin, g.slice_end, g.cap, g.release, g.deadline)
        return sub, order

    # ---------------------------------------------------------------- Alg. 1
    def round(self):
        """One round: (status, batch ops, chosen partition or -1)."""
        if int((self.state == ISSUED).sum()) >= self.budget:
            return ROUND_BUDGET, [], -1
        F = self.unscheduled_frontier()
        if not F:
            return ROUND_IDLE, [], -1
        op = min(F, key=lambda v: (int(self.priority[self.g.op_req[v]]), v))
        batch = self.collect(op)
        sub, order = self.round_graph(batch)
        n_pre = len(order) - len(batch)
        rows = np.empty((len(self.part), len(order)), np.uint8)
        rows[:, :n_pre] = self.place[order[:n_pre]]
        rows[:, n_pre:] = self.part[:, batch]
        res = oracle.simulate_batch(sub, rows, oracle.INDEX_ORDER)
        best, _ = oracle.select_best(res["violation"], res["sumfin"], res["slack"], self.require_sla)
        if best < 0:
            return ROUND_INFEASIBLE, batch, -1
        self.state[batch] = ISSUED
        self.place[batch] = self.part[best, batch]
        self.issue_order += list(batch)
        return ROUND_ISSUED, batch, int(best)

    def complete(self, v):
        """Feedback: issued op v is done."""
        assert self.state[v] == ISSUED
        self.state[v] = DONE
