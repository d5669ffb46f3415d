"""Oracle for the incremental scheduling loop -- TEST INFRASTRUCTURE ONLY.

Written from the paper (SliceScheduler, arXiv 2608.15762), Sec. 3.2, 3.3.2,
3.4 and Alg. 1:
  - ops are unscheduled, issued or done; the scheduling metadata of an op
    holds the time it was issued and the time it completed (Sec. 3.2);
  - the scheduled frontier holds the issued or done ops that have an
    unscheduled successor (their outputs stay on their accelerators as
    checkpoints); the unscheduled frontier holds the unscheduled ops whose
    predecessors are all issued or done (Sec. 3.4.1);
  - a round at time `now` returns at once when the issued ops reach the
    budget or the unscheduled frontier is empty; otherwise it takes the
    highest-priority op of the unscheduled frontier, collects a small
    connected batch from it by following successors (capped), evaluates
    every pre-defined partition as a candidate placement of the batch by a
    what-if simulation built from the snapshot (Sec. 3.3.2), discards
    infeasible candidates, keeps the one with the smallest simulated average
    completion time, writes it back and marks the batch issued at `now`
    (Alg. 1, Sec. 3.4.2);
  - executor feedback marks an issued op done at its completion time.

Readings where the paper is silent (each is listed in the design notes):
  - priority: a smaller per-request priority value first (the workloads use
    the deadline), ties to the lower op index;
  - batch collection: starting from the chosen op, repeatedly add the
    lowest-index unscheduled successor of a batch op whose predecessors are
    all issued, done or already in the batch, until the cap or no such op;
  - the simulated graph of a round (the snapshot) holds, in the order they
    were issued, the issued ops that are not done and the done ops whose
    output is still needed (a successor not done: a checkpoint, or the input
    of an op in flight), then the batch in index order.  Done ops keep their
    recorded completion; the issued ops and the batch are simulated with the
    estimates, each no earlier than its issue time (the batch's is `now`); a
    done op none of whose successors is still to run has no bearing on the
    future and is left out, so the graph holds the issue budget, the
    checkpoints and one batch, not the run's history;
  - memory is checked from `now` on (the simulation's peak over times at or
    after the snapshot's timestamp);
  - candidate b is partition b; the score is the sum of finish times over the
    simulated graph (the ops before the batch have the same schedule in every
    candidate: they precede the batch in every device queue and are issued
    no later); feasibility is memory only unless SLA is required; ties go to
    the lower partition index; with no feasible candidate nothing is issued;
  - rounds come at non-decreasing times; a completion is reported after the
    op's predecessors' completions and later than they and its issue.

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
        self.issue_t = np.full(N, -1, np.int64)
        self.done_t = np.full(N, -1, np.int64)
        self.now = 0
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

    # ---------------------------------------------------------------- the round's snapshot
    def kept(self, v):
        """In the snapshot: issued and not done, or done with a successor not done."""
        if self.state[v] == ISSUED:
            return True
        return self.state[v] == DONE and any(self.state[x] != DONE for x in self.succs[v])

    def round_graph(self, batch, now):
        """(sub-GMG with the running schedule's state, op order)."""
        g = self.g
        order = [v for v in self.issue_order if self.kept(v)] + list(batch)
        new = {v: i for i, v in enumerate(order)}
        pred_ptr, pred_idx = [0], []
        for v in order:
            ps = [new[u] for u in self.preds[v] if u in new]
            assert self.state[v] == DONE or len(ps) == len(self.preds[v])  # inputs of ops to run are all there
            pred_idx += sorted(ps)
            pred_ptr.append(len(pred_idx))
        dur = np.array([g.dur[v] for v in order], np.int64).reshape(len(order), g.n_class)
        sub = type(g)(len(order), g.n_dev, g.n_class, g.n_link, g.n_req,
                      np.asarray(pred_ptr, np.int32), np.asarray(pred_idx, np.int32),
                      np.asarray([g.op_req[v] for v in order], np.int32), dur,
                      np.asarray([g.out_bytes[v] for v in order], np.int64), g.dev_class, g.link_class, g.bw, g.lat,
                      g.slice_ptr, g.slice_begin, g.slice_end, g.cap, g.release, g.deadline)
        inb = set(batch)
        sub.done_fin = np.array([self.done_t[v] if self.state[v] == DONE else -1 for v in order], np.int64)
        sub.issue_at = np.array([now if v in inb else self.issue_t[v] for v in order], np.int64)
        sub.t_now = int(now)
        return sub, order

    # ---------------------------------------------------------------- Alg. 1
    def round(self, now: int):
        """One round at time `now`: (status, batch ops, chosen partition or -1)."""
        if now < self.now:
            raise ValueError("rounds come at non-decreasing times")
        self.now = int(now)
        if int((self.state == ISSUED).sum()) >= self.budget:
            return ROUND_BUDGET, [], -1
        F = self.unscheduled_frontier()
        if not F:
            return ROUND_IDLE, [], -1
        op = min(F, key=lambda v: (int(self.priority[self.g.op_req[v]]), v))
        batch = self.collect(op)
        sub, order = self.round_graph(batch, now)
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
        self.issue_t[batch] = now
        self.issue_order += list(batch)
        return ROUND_ISSUED, batch, int(best)

    def complete(self, v, t: int):
        """Feedback: issued op v completed at time t."""
        if self.state[v] != ISSUED:
            raise ValueError("op is not issued")
        if t <= self.issue_t[v] or any(self.state[u] != DONE or self.done_t[u] >= t for u in self.preds[v]):
            raise ValueError("a completion comes after the op's issue and its predecessors' completions")
        self.state[v] = DONE
        self.done_t[v] = int(t)
