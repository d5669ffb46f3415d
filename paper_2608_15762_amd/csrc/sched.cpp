// Incremental simulation-based scheduling (Alg. 1, Sec. 3.4) around the
// batched simulator: op states and the two scheduling frontiers of Sec. 3.4.1,
// batch collection, candidate partitions simulated in one ss_simulate_batch
// call on the GPU, selection by ss_select_best, write-back.
//
// Host-side state, per op: unscheduled / issued / done, the device chosen for
// it, its issue and completion times (the scheduling metadata of Sec. 3.2),
// the number of its predecessors still unscheduled (it is on the unscheduled
// frontier when that count is zero) and of its successors not done.  The
// frontier is kept ordered by (request priority, op), so the highest-priority
// op is its first element.
//
// A round at time `now` simulates the snapshot (Sec. 3.3.2): the issued ops
// that are not done and the done ops whose output still feeds an op to run,
// in the order they were issued, then the batch in index order, issued at
// `now`.  Done ops keep their recorded completion; the rest is simulated with
// the estimates, no op before its issue; memory is checked from `now` on.
// The ops before the batch precede it in every device queue and were issued
// no later, so they have one schedule in every candidate and the candidates'
// finish-time sums differ by the batch's alone.  A done op with no successor
// left to run is out of every later snapshot, so the graph is bounded by the
// issue budget, the checkpoints and one batch.
//
// Prefix reuse (SS_SCHED_PREFIX_REUSE): the chosen candidate's state after
// its round's graph is captured; while no completion arrives, the next
// round's graph is that graph followed by a new batch (the batch just issued
// joins the issued ops, the done ops still in play stay), so every candidate
// resumes after it.  Off by default: the candidates run in parallel lanes, so
// the capture's serial walk costs more than the walk each lane saves.
#include <algorithm>
#include <new>
#include <queue>
#include <set>
#include <vector>

#include "ss_internal.h"

struct ss_sched {
  int64_t N = 0, E = 0, D = 0, C = 0, K = 0, R = 0, P = 0;
  std::vector<int32_t> pred_ptr, pred_idx, op_req, dev_class, succ_ptr, succ_idx;
  std::vector<int64_t> dur, out_bytes, bw, lat, slice_ptr, slice_begin, slice_end, cap, release, deadline;
  std::vector<uint8_t> link_class;
  std::vector<uint8_t> part;  // [P][N]
  std::vector<int64_t> priority;
  int64_t budget = 0, batch_cap = 0;
  int flags = 0;
  int device = 0;
  std::vector<uint8_t> state, place;
  std::vector<int64_t> issue_t, done_t;  // -1 until issued / done
  int64_t now = 0;                       // time of the latest round
  // ops that can still be in a snapshot (issued, or done with a successor not
  // done), in the order they were issued; a done op leaves for good once its
  // last successor is done
  std::vector<int32_t> issue_order;
  std::vector<int32_t> open_succ;  // successors not done
  std::vector<int32_t> missing;  // unscheduled predecessors
  std::vector<uint8_t> rows;     // host candidate rows of the current round (kept: no new pages each round)
  std::set<std::pair<int64_t, int32_t>> frontier;
  int64_t n_issued = 0;
  // reused device buffers: candidate rows and per-candidate outputs
  void *dev_buf = nullptr;
  size_t dev_bytes = 0;
  // the chosen candidate's simulation state after the scheduled ops (the
  // prefix of the next round), and a second state to capture the next one in
  ss_state *prefix = nullptr, *next = nullptr;
  bool prefix_ok = false;  // no completion since prefix was captured
  bool reuse = false;      // prefix reuse enabled (SS_SCHED_PREFIX_REUSE)

};

namespace {

int sched_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

template <class T>
void copy_in(std::vector<T> &dst, const T *src, int64_t n) {
  dst.assign(src, src + n);
}

// Becomes issued: leaves the frontier, its successors lose a missing predecessor.
void mark_issued(ss_sched *s, int32_t v, uint8_t dev) {
  s->frontier.erase({s->priority[s->op_req[v]], v});
  s->state[v] = SS_OP_ISSUED;
  s->place[v] = dev;
  ++s->n_issued;
  for (int32_t q = s->succ_ptr[v]; q < s->succ_ptr[v + 1]; ++q) {
    const int32_t x = s->succ_idx[q];
    if (--s->missing[x] == 0 && s->state[x] == SS_OP_UNSCHEDULED) s->frontier.insert({s->priority[s->op_req[x]], x});
  }
}

// CollectConnectedGraph: from op, repeatedly the lowest-index unscheduled
// successor of a batch op whose predecessors are all scheduled or in the
// batch, up to the cap.
std::vector<int32_t> collect(const ss_sched *s, int32_t op) {
  std::vector<int32_t> batch{op};
  // per successor reached: its unscheduled predecessors not yet in the batch
  std::vector<int32_t> need((size_t)s->N, -1);
  std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> ready;
  auto add = [&](int32_t v) {
    for (int32_t q = s->succ_ptr[v]; q < s->succ_ptr[v + 1]; ++q) {
      const int32_t x = s->succ_idx[q];
      if (s->state[x] != SS_OP_UNSCHEDULED || x == op) continue;
      if (need[x] < 0) need[x] = s->missing[x];
      if (--need[x] == 0) ready.push(x);
    }
  };
  add(op);
  while ((int64_t)batch.size() < s->batch_cap && !ready.empty()) {
    const int32_t x = ready.top();
    ready.pop();
    batch.push_back(x);
    add(x);
  }
  std::sort(batch.begin(), batch.end());
  return batch;
}

}  // namespace

int ss_run_sched_create(const ss_sched_desc *d, ss_sched **out) {
  const ss_gmg_desc *g = d->gmg;
  // the loader's rules apply to the run's graph as a whole
  ss_gmg *probe = nullptr;
  int rc = ss_gmg_load(g, &probe);
  if (rc != SS_OK) return rc;
  ss_gmg_free(probe);
  ss_sched *s = new (std::nothrow) ss_sched();
  if (!s) return ss_set_error(SS_ERR_OOM, "ss_sched_create: host allocation failed");
  try {
    s->N = g->n_ops;
    s->E = g->n_edges;
    s->D = g->n_dev;
    s->C = g->n_class;
    s->K = g->n_link;
    s->R = g->n_req;
    s->P = d->n_part;
    copy_in(s->pred_ptr, g->pred_ptr, s->N + 1);
    copy_in(s->pred_idx, g->pred_idx, s->E);
    copy_in(s->op_req, g->op_req, s->N);
    copy_in(s->dev_class, g->dev_class, s->D);
    copy_in(s->dur, g->dur, s->N * s->C);
    copy_in(s->out_bytes, g->out_bytes, s->N);
    copy_in(s->bw, g->bw, s->K);
    copy_in(s->lat, g->lat, s->K);
    copy_in(s->slice_ptr, g->slice_ptr, s->D + 1);
    copy_in(s->slice_begin, g->slice_begin, g->slice_ptr[s->D]);
    copy_in(s->slice_end, g->slice_end, g->slice_ptr[s->D]);
    copy_in(s->cap, g->cap, s->D);
    copy_in(s->release, g->release, s->R);
    copy_in(s->deadline, g->deadline, s->R);
    copy_in(s->link_class, g->link_class, s->D * s->D);
    copy_in(s->part, d->part_dev, s->P * s->N);
    copy_in(s->priority, d->priority, s->R);
    s->budget = d->issue_budget;
    s->batch_cap = d->batch_cap;
    s->flags = d->flags;
    s->state.assign((size_t)s->N, SS_OP_UNSCHEDULED);
    s->place.assign((size_t)s->N, 0);
    s->issue_t.assign((size_t)s->N, -1);
    s->done_t.assign((size_t)s->N, -1);
    s->open_succ.assign((size_t)s->N, 0);
    s->reuse = (d->flags & SS_SCHED_PREFIX_REUSE) != 0;
    s->missing.assign((size_t)s->N, 0);
    s->succ_ptr.assign((size_t)s->N + 1, 0);
    s->succ_idx.assign((size_t)s->E, 0);
    for (int64_t v = 0; v < s->N; ++v) {
      s->missing[v] = s->pred_ptr[v + 1] - s->pred_ptr[v];
      for (int32_t e = s->pred_ptr[v]; e < s->pred_ptr[v + 1]; ++e) ++s->succ_ptr[s->pred_idx[e] + 1];
    }
    for (int64_t v = 0; v < s->N; ++v) s->open_succ[v] = s->succ_ptr[v + 1];
    for (int64_t v = 0; v < s->N; ++v) s->succ_ptr[v + 1] += s->succ_ptr[v];
    std::vector<int32_t> fill(s->succ_ptr.begin(), s->succ_ptr.end() - 1);
    for (int64_t v = 0; v < s->N; ++v)
      for (int32_t e = s->pred_ptr[v]; e < s->pred_ptr[v + 1]; ++e) s->succ_idx[fill[s->pred_idx[e]]++] = (int32_t)v;
    for (int64_t v = 0; v < s->N; ++v)
      if (s->missing[v] == 0) s->frontier.insert({s->priority[s->op_req[v]], (int32_t)v});
  } catch (const std::bad_alloc &) {
    delete s;
    return ss_set_error(SS_ERR_OOM, "ss_sched_create: host allocation failed");
  }
  if (hipGetDevice(&s->device) != hipSuccess) {
    delete s;
    return ss_set_error(SS_ERR_DEVICE, "hipGetDevice failed");
  }
  rc = ss_state_create(&s->prefix);
  if (rc == SS_OK) rc = ss_state_create(&s->next);
  if (rc != SS_OK) {
    ss_state_free(s->prefix);
    ss_state_free(s->next);
    delete s;
    return rc;
  }
  *out = s;
  return SS_OK;
}

void ss_run_sched_free(ss_sched *s) {
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(s->device);
  (void)hipDeviceSynchronize();
  if (s->dev_buf) {
    ss_pool_free(s->dev_buf, nullptr);
    (void)hipDeviceSynchronize();
  }
  (void)hipSetDevice(prev);
  ss_state_free(s->prefix);
  ss_state_free(s->next);
  delete s;
}

int ss_run_sched_round(ss_sched *s, int64_t now, int *status, int64_t *ops, int64_t *n_ops, int64_t *part,
                       hipStream_t stream) {
  *n_ops = 0;
  *part = -1;
  if (now < s->now) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_round: rounds come at non-decreasing times");
  s->now = now;
  if (s->n_issued >= s->budget) {
    *status = SS_ROUND_BUDGET;
    return SS_OK;
  }
  if (s->frontier.empty()) {
    *status = SS_ROUND_IDLE;
    return SS_OK;
  }
  const int32_t op = s->frontier.begin()->second;
  std::vector<int32_t> batch;
  std::vector<int32_t> order;
  try {
    batch = collect(s, op);
    // the snapshot's ops: done ops whose every successor is done leave for good
    size_t w = 0;
    for (const int32_t v : s->issue_order)
      if (s->state[v] == SS_OP_ISSUED || s->open_succ[v] > 0) s->issue_order[w++] = v;
    s->issue_order.resize(w);
    order = s->issue_order;
    order.insert(order.end(), batch.begin(), batch.end());
    s->issue_order.reserve(order.size());  // the write-back cannot fail half-way
  } catch (const std::bad_alloc &) {
    return ss_set_error(SS_ERR_OOM, "ss_sched_round: host allocation failed");
  }
  const int64_t Ns = (int64_t)order.size(), nb = (int64_t)batch.size(), npre = Ns - nb, P = s->P;

  // the round's graph: the snapshot's ops and the batch, renumbered; a done
  // op's predecessors outside the snapshot are dropped (it is not simulated)
  std::vector<int32_t> newid((size_t)s->N, -1), sp_ptr(1, 0), sp_idx, sreq((size_t)Ns);
  sp_idx.reserve(s->pred_idx.size());
  sp_ptr.reserve((size_t)Ns + 1);
  std::vector<int64_t> sdur((size_t)(Ns * s->C)), sbytes((size_t)Ns), sdone((size_t)Ns), sissue((size_t)Ns);
  for (int64_t i = 0; i < Ns; ++i) newid[order[i]] = (int32_t)i;
  for (int64_t i = 0; i < Ns; ++i) {
    const int32_t v = order[i];
    const size_t first = sp_idx.size();
    for (int32_t e = s->pred_ptr[v]; e < s->pred_ptr[v + 1]; ++e)
      if (newid[s->pred_idx[e]] >= 0) sp_idx.push_back(newid[s->pred_idx[e]]);
    std::sort(sp_idx.begin() + (std::ptrdiff_t)first, sp_idx.end());
    sp_ptr.push_back((int32_t)sp_idx.size());
    sreq[i] = s->op_req[v];
    for (int64_t c = 0; c < s->C; ++c) sdur[i * s->C + c] = s->dur[v * s->C + c];
    sbytes[i] = s->out_bytes[v];
    sdone[i] = s->state[v] == SS_OP_DONE ? s->done_t[v] : -1;
    sissue[i] = i < npre ? s->issue_t[v] : now;
  }
  ss_gmg_desc gd{};
  gd.n_ops = Ns;
  gd.n_edges = (int64_t)sp_idx.size();
  gd.n_dev = s->D;
  gd.n_class = s->C;
  gd.n_link = s->K;
  gd.n_req = s->R;
  gd.pred_ptr = sp_ptr.data();
  gd.pred_idx = sp_idx.data();
  gd.op_req = sreq.data();
  gd.dur = sdur.data();
  gd.out_bytes = sbytes.data();
  gd.dev_class = s->dev_class.data();
  gd.link_class = s->link_class.data();
  gd.bw = s->bw.data();
  gd.lat = s->lat.data();
  gd.slice_ptr = s->slice_ptr.data();
  gd.slice_begin = s->slice_begin.data();
  gd.slice_end = s->slice_end.data();
  gd.cap = s->cap.data();
  gd.release = s->release.data();
  gd.deadline = s->deadline.data();
  gd.done_fin = sdone.data();
  gd.issue_at = sissue.data();
  gd.t_now = now;

  // candidate b = partition b: the snapshot's ops where they are, the batch by the partition
  try {
    if (s->rows.size() < (size_t)(P * Ns)) s->rows.resize((size_t)(P * Ns));
  } catch (const std::bad_alloc &) {
    return ss_set_error(SS_ERR_OOM, "ss_sched_round: host allocation failed");
  }
  std::vector<uint8_t> &rows = s->rows;
  for (int64_t b = 0; b < P; ++b) {
    uint8_t *row = rows.data() + b * Ns;
    for (int64_t i = 0; i < npre; ++i) row[i] = s->place[order[i]];
    for (int64_t i = 0; i < nb; ++i) row[npre + i] = s->part[b * s->N + batch[i]];
  }

  ss_gmg *g = nullptr;
  int rc = ss_gmg_load(&gd, &g);
  if (rc != SS_OK) return rc;
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t sz_rows = align((size_t)(P * Ns) + 1), sz_ms = align((size_t)P * 8), sz_vi = align((size_t)P),
               sz_sl = align((size_t)(P * s->R) * 8 + 8), sz_best = align(16);
  const size_t need = sz_rows + 2 * sz_ms + sz_vi + sz_sl + sz_best;
  hipError_t err = hipSuccess;
  if (need > s->dev_bytes) {
    const size_t grow = std::max(need, 2 * s->dev_bytes);  // few reallocations as graphs vary
    if (s->dev_buf) {
      (void)hipStreamSynchronize(stream);
      ss_pool_free(s->dev_buf, stream);
      s->dev_buf = nullptr;
      s->dev_bytes = 0;
    }
    rc = ss_pool_alloc(s->device, grow, stream, &s->dev_buf);
    if (rc != SS_OK) {
      ss_gmg_free(g);
      return rc;
    }
    s->dev_bytes = grow;
  }
  unsigned char *p = static_cast<unsigned char *>(s->dev_buf);
  auto *d_rows = reinterpret_cast<uint8_t *>(p);
  auto *d_ms = reinterpret_cast<int64_t *>(p + sz_rows);
  auto *d_sum = reinterpret_cast<int64_t *>(p + sz_rows + sz_ms);
  auto *d_vi = reinterpret_cast<uint8_t *>(p + sz_rows + 2 * sz_ms);
  auto *d_sl = reinterpret_cast<int64_t *>(p + sz_rows + 2 * sz_ms + sz_vi);
  auto *d_best = reinterpret_cast<int64_t *>(p + sz_rows + 2 * sz_ms + sz_vi + sz_sl);
  int64_t best[2] = {-1, 0};
  err = hipMemcpyAsync(d_rows, rows.data(), (size_t)(P * Ns), hipMemcpyHostToDevice, stream);
  if (err == hipSuccess) {
    // every candidate resumes after the snapshot's ops when the state
    // captured at the last issuing round still describes them
    int64_t k = 0;
    (void)ss_state_info(s->prefix, &k);
    const ss_state *from = s->reuse && s->prefix_ok && k == npre ? s->prefix : nullptr;
    rc = ss_simulate_batch_resume(g, from, d_rows, P, d_ms, nullptr, d_vi, d_sl, d_sum, stream);
    if (rc == SS_OK)
      rc = ss_select_best(g, d_vi, d_sum, d_sl, P, s->flags & SS_SELECT_REQUIRE_SLA, d_best, stream);
    if (rc == SS_OK) err = hipMemcpyAsync(best, d_best, sizeof(best), hipMemcpyDeviceToHost, stream);
    if (rc == SS_OK && err == hipSuccess) err = hipStreamSynchronize(stream);
    if (rc == SS_OK && err == hipSuccess && best[0] >= 0 && s->reuse) {
      // the chosen candidate's schedule once more, captured for the next round
      rc = ss_state_capture(g, from, d_rows + best[0] * Ns, s->next, stream);
      if (rc == SS_OK) err = hipStreamSynchronize(stream);
      if (rc == SS_OK && err == hipSuccess) std::swap(s->prefix, s->next);
      s->prefix_ok = rc == SS_OK && err == hipSuccess;
    }
  }
  ss_gmg_free(g);
  if (rc != SS_OK) return rc;
  if (err != hipSuccess) return sched_fail(err, "ss_sched_round");

  for (int64_t i = 0; i < nb; ++i) ops[i] = batch[i];
  *n_ops = nb;
  if (best[0] < 0) {
    *status = SS_ROUND_INFEASIBLE;
    return SS_OK;
  }
  for (int64_t i = 0; i < nb; ++i) {
    mark_issued(s, batch[i], s->part[best[0] * s->N + batch[i]]);
    s->issue_t[batch[i]] = now;
  }
  s->issue_order.insert(s->issue_order.end(), batch.begin(), batch.end());
  *part = best[0];
  *status = SS_ROUND_ISSUED;
  return SS_OK;
}

int ss_run_sched_complete(ss_sched *s, int64_t op, int64_t t_done) {
  if (op < 0 || op >= s->N || s->state[op] != SS_OP_ISSUED)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_complete: op is not issued");
  if (t_done <= s->issue_t[op])
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_complete: completion not after the op's issue");
  if (t_done >= ((int64_t)1 << 62)) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_complete: time >= 2^62");
  for (int32_t e = s->pred_ptr[op]; e < s->pred_ptr[op + 1]; ++e) {
    const int32_t u = s->pred_idx[e];
    if (s->state[u] != SS_OP_DONE || s->done_t[u] >= t_done)
      return ss_set_error(SS_ERR_INVALID_ARG,
                          "ss_sched_complete: completion before a predecessor's completion");
  }
  s->state[op] = SS_OP_DONE;
  s->done_t[op] = t_done;
  --s->n_issued;
  for (int32_t e = s->pred_ptr[op]; e < s->pred_ptr[op + 1]; ++e) --s->open_succ[s->pred_idx[e]];
  s->prefix_ok = false;
  return SS_OK;
}

void ss_run_sched_state(const ss_sched *s, uint8_t *state, uint8_t *place, int64_t *issue_t, int64_t *done_t) {
  if (state) std::copy(s->state.begin(), s->state.end(), state);
  if (place) std::copy(s->place.begin(), s->place.end(), place);
  if (issue_t) std::copy(s->issue_t.begin(), s->issue_t.end(), issue_t);
  if (done_t) std::copy(s->done_t.begin(), s->done_t.end(), done_t);
}
