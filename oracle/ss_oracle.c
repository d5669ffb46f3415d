/*
 * Oracle for the GMG what-if simulator -- TEST INFRASTRUCTURE ONLY.
 *
 * Written from the paper (SliceScheduler, arXiv 2608.15762):
 *   - transfer estimator, Sec. 3.3.1: t = alpha * size + c per accelerator pair,
 *     taken in integer form as lat[k] + ceil(bytes / bw[k]) per link class k;
 *   - simulator construction, Sec. 3.3.2: an op is ready when its local
 *     predecessors have completed and the outputs of remote predecessors have
 *     arrived; a queue runs at most one op at a time; completion = start +
 *     operator estimate; ready and executing ops determine the tensors
 *     resident in HBM;
 *   - event-driven simulation and what-if, Sec. 3.3.3: advance every queue,
 *     score a placement from completion-time statistics;
 *   - selection, Sec. 3.4.2 and Alg. 1: discard placements that run out of
 *     memory, keep the one with the smallest average completion time.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - an op runs non-preemptively inside ONE idle slice of its device; after
 *     the last finite slice a device is free forever (open tail);
 *   - contract A serves each device's ops in index order (index order is the
 *     priority order of the GMG); the ready-time dispatch of Sec. 3.3.2 is
 *     the SSO_READY_ORDER variant;
 *   - a transfer is pure latency starting at the producer's finish, one per
 *     (tensor, destination device), shared by all consumers there; the
 *     SSO_LINK_PORTS variant arbitrates transfers over per-device ports
 *     instead, event by event (Sec. 3.5.2, see schedule_index_order_ports);
 *   - memory: an op's output occupies its device from the op's start until the
 *     later of its last local consumer's finish and its last outgoing
 *     transfer's arrival; a remote copy occupies the destination from the
 *     transfer's start (the producer's finish; the receive buffer exists
 *     before the data moves, Sec. 3.5.2) until its last consumer there
 *     finishes; outputs without consumers stay resident; intervals are
 *     half-open; a device violates when its peak exceeds its capacity;
 *   - a snapshot of a running schedule (Sec. 3.2 scheduling metadata: the
 *     issued and done timestamps; Sec. 3.3.2 builds the simulator from it):
 *     a done op is not simulated, it finished at its recorded time on its
 *     device; an op does not start before it was issued, and the transfer of
 *     an output to a device does not start before the first consumer there
 *     was issued (its Intent exists only from then on); the peak is that of
 *     the memory held at or after the snapshot's timestamp (every residency
 *     interval clipped to [t_now, inf)).
 *
 * Parity: pinned by closed forms, bounds, brute force and hand-worked cases in
 * the CPU test-suite (no printed worked example exists in the paper).
 */
#include "ss_oracle.h"

#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- estimators */

/* Transfer estimator X(u, s, t): zero on the same device, else
 * lat + ceil(out_bytes[u] / bw) of the (s, t) link class (Sec. 3.3.1). */
static int64_t transfer_time(const sso_gmg *g, int64_t u, int64_t s, int64_t t) {
  if (s == t) return 0;
  const int k = g->link_class[s * g->n_dev + t];
  const int64_t bytes = g->out_bytes[u];
  const int64_t bw = g->bw[k];
  return g->lat[k] + (bytes + bw - 1) / bw;
}

/* Operator estimator: duration of op v on device d (per device class). */
static int64_t op_duration(const sso_gmg *g, int64_t v, int64_t d) {
  return g->dur[v * g->n_class + g->dev_class[d]];
}

/* Earliest s >= t such that [s, s + w) lies inside one idle slice of device d.
 * Slices are sorted; the start max(t, a_k) does not decrease with k, so the
 * first slice that can hold the op gives the earliest start. */
static int64_t earliest_fit(const sso_gmg *g, int64_t d, int64_t t, int64_t w) {
  for (int64_t k = g->slice_ptr[d]; k < g->slice_ptr[d + 1]; ++k) {
    const int64_t a = g->slice_begin[k], e = g->slice_end[k];
    const int64_t s = t > a ? t : a;
    if (s + w <= e) return s;
  }
  return -1; /* not reached: the last slice of every device is open */
}

/* Ready time: the later of the request's release (and t0 = 0) and, over every
 * predecessor u, its finish plus the transfer of its output to v's device. */
static int64_t ready_time(const sso_gmg *g, const uint8_t *place, const int64_t *fin, int64_t v) {
  int64_t r = g->release[g->op_req[v]];
  if (r < 0) r = 0;
  for (int64_t e = g->pred_ptr[v]; e < g->pred_ptr[v + 1]; ++e) {
    const int64_t u = g->pred_idx[e];
    const int64_t arrive = fin[u] + transfer_time(g, u, place[u], place[v]);
    if (arrive > r) r = arrive;
  }
  return r;
}

/* ---------------------------------------------------------------- successors */

typedef struct {
  int64_t *ptr; /* [n_ops+1] */
  int64_t *idx; /* ascending within each op */
} succ_csr;

static int build_succ(const sso_gmg *g, succ_csr *s) {
  const int64_t N = g->n_ops, E = g->pred_ptr[N];
  s->ptr = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
  s->idx = (int64_t *)malloc(((size_t)E + 1) * sizeof(int64_t));
  int64_t *fill = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
  if (!s->ptr || !s->idx || !fill) {
    free(s->ptr); free(s->idx); free(fill);
    return -1;
  }
  for (int64_t e = 0; e < E; ++e) s->ptr[g->pred_idx[e] + 1]++;
  for (int64_t v = 0; v < N; ++v) s->ptr[v + 1] += s->ptr[v];
  /* visiting consumers v in increasing order keeps each list ascending */
  for (int64_t v = 0; v < N; ++v)
    for (int64_t e = g->pred_ptr[v]; e < g->pred_ptr[v + 1]; ++e) {
      const int64_t u = g->pred_idx[e];
      s->idx[s->ptr[u] + fill[u]++] = v;
    }
  free(fill);
  return 0;
}

static void free_succ(succ_csr *s) { free(s->ptr); free(s->idx); }

/* ---------------------------------------------------------------- snapshots */

static int64_t issue_time(const sso_gmg *g, int64_t v) { return g->issue_at ? g->issue_at[v] : 0; }

static int is_done(const sso_gmg *g, int64_t v) { return g->done_fin && g->done_fin[v] >= 0; }

/* Earliest start of the transfer of u's output to device e: the first issue
 * time among u's consumers on e (the Intent of the first one issued), never
 * before u finishes (the caller takes the later of the two). */
static int64_t transfer_floor(const sso_gmg *g, const succ_csr *sc, const uint8_t *place, int64_t u, int64_t e) {
  int64_t f = INT64_MAX;
  for (int64_t q = sc->ptr[u]; q < sc->ptr[u + 1]; ++q) {
    const int64_t x = sc->idx[q];
    if (place[x] == e && issue_time(g, x) < f) f = issue_time(g, x);
  }
  return f == INT64_MAX ? 0 : f;
}

/* Arrival on device e of u's output (u on another device): its transfer
 * starts once u has finished and the first consumer on e has been issued. */
static int64_t transfer_arrival(const sso_gmg *g, const succ_csr *sc, const uint8_t *place, const int64_t *fin,
                                int64_t u, int64_t e) {
  const int64_t floor_ = transfer_floor(g, sc, place, u, e);
  const int64_t start = fin[u] > floor_ ? fin[u] : floor_;
  return start + transfer_time(g, u, place[u], e);
}

/* ---------------------------------------------------------------- schedules */

/* Contract A: ops in index order; each starts at the earliest fit at or after
 * max(ready, the device's previous finish); one op at a time per device.  In
 * a snapshot a done op is not placed: it finished at its recorded time and
 * its device is free from then on; ready times also wait for the op's issue
 * and for transfers that start no earlier than their first consumer's issue. */
static void schedule_index_order(const sso_gmg *g, const uint8_t *place, const succ_csr *sc, int64_t *clock,
                                 int64_t *st, int64_t *fin) {
  for (int64_t d = 0; d < g->n_dev; ++d) clock[d] = 0;
  for (int64_t v = 0; v < g->n_ops; ++v) {
    const int64_t d = place[v];
    const int64_t w = op_duration(g, v, d);
    if (is_done(g, v)) {
      fin[v] = g->done_fin[v];
      st[v] = fin[v] - w;
      if (fin[v] > clock[d]) clock[d] = fin[v];
      continue;
    }
    int64_t ready = g->release[g->op_req[v]];
    if (ready < 0) ready = 0;
    if (issue_time(g, v) > ready) ready = issue_time(g, v);
    for (int64_t e = g->pred_ptr[v]; e < g->pred_ptr[v + 1]; ++e) {
      const int64_t u = g->pred_idx[e];
      const int64_t arrive = place[u] == d ? fin[u] : transfer_arrival(g, sc, place, fin, u, d);
      if (arrive > ready) ready = arrive;
    }
    const int64_t t = ready > clock[d] ? ready : clock[d];
    st[v] = earliest_fit(g, d, t, w);
    fin[v] = st[v] + w;
    clock[d] = fin[v];
  }
}

/* SSO_LINK_PORTS: transfers arbitrated over the devices' ports, as the
 * executor's arbitration does (Sec. 3.5.2), inside an event-driven simulation.
 *   - Compute queues are those of contract A: each device runs its ops in
 *     index order, one at a time, each at the earliest fit at or after
 *     max(ready, the device's previous finish).
 *   - The output of u is moved once to every other device that holds a
 *     consumer of u (one transfer per (tensor, destination device)).  Its
 *     Intent arrives when u finishes; the transfer is then pending.
 *   - The arbitration is triggered by every Intent arrival and every transfer
 *     completion.  At such an instant t the pending transfers are examined in
 *     order of request time, then producer index, then destination device,
 *     and each one whose source's send port and destination's receive port
 *     are both idle at t starts at t (so the started set shares no source and
 *     no destination); it holds both ports until it arrives, t + X.  Nothing
 *     is booked ahead of time.
 *   - A transfer whose estimate X is zero moves nothing: it completes at its
 *     request, takes no port and waits for none.
 *   - A consumer's remote input is there when its transfer arrives.
 * An op is placed as soon as every input's availability time is known and
 * the op ahead of it on its device is placed; its start depends on nothing
 * else, and it never precedes the instant at which it is placed, so placing
 * it then gives the same schedule as placing it at its ready time.
 * xs/xa receive the start and arrival of the transfer that serves each
 * successor entry (equal for every consumer of u on one device; unused for
 * local consumers).  order/n_order (nullable) receive the first successor
 * entry of each transfer in the order the transfers start.
 * Returns 0, or -1 on allocation failure. */
typedef struct { int64_t time, kind, id; } sim_event; /* kind 0: op finishes, 1: transfer arrives */

static int event_before(sim_event a, sim_event b) {
  if (a.time != b.time) return a.time < b.time;
  if (a.kind != b.kind) return a.kind < b.kind;
  return a.id < b.id;
}

static void event_push(sim_event *h, int64_t *n, sim_event x) {
  int64_t i = (*n)++;
  h[i] = x;
  while (i > 0) {
    const int64_t p = (i - 1) / 2;
    if (!event_before(h[i], h[p])) break;
    sim_event t = h[i]; h[i] = h[p]; h[p] = t;
    i = p;
  }
}

static sim_event event_pop(sim_event *h, int64_t *n) {
  sim_event top = h[0];
  h[0] = h[--(*n)];
  int64_t i = 0;
  for (;;) {
    const int64_t l = 2 * i + 1, r = l + 1;
    int64_t m = i;
    if (l < *n && event_before(h[l], h[m])) m = l;
    if (r < *n && event_before(h[r], h[m])) m = r;
    if (m == i) break;
    sim_event t = h[i]; h[i] = h[m]; h[m] = t;
    i = m;
  }
  return top;
}

/* First successor entry of u whose consumer runs on device e, or -1. */
static int64_t first_entry_to(const succ_csr *sc, const uint8_t *place, int64_t u, int64_t e) {
  for (int64_t q = sc->ptr[u]; q < sc->ptr[u + 1]; ++q)
    if (place[sc->idx[q]] == e) return q;
  return -1;
}

/* Start (or, with a zero estimate, complete) the transfer of u to e at t. */
static void set_transfer(const succ_csr *sc, const uint8_t *place, int64_t u, int64_t e, int64_t start,
                         int64_t arrive, int64_t *xs, int64_t *xa) {
  for (int64_t q = sc->ptr[u]; q < sc->ptr[u + 1]; ++q)
    if (place[sc->idx[q]] == e) {
      xs[q] = start;
      xa[q] = arrive;
    }
}

static int schedule_index_order_ports(const sso_gmg *g, const uint8_t *place, const succ_csr *sc, int64_t *clock,
                                      int64_t *st, int64_t *fin, int64_t *xs, int64_t *xa, int64_t *order,
                                      int64_t *n_order) {
  const int64_t N = g->n_ops, D = g->n_dev, E = sc->ptr[N];
  int64_t *dev_ptr = (int64_t *)calloc((size_t)D + 1, sizeof(int64_t));
  int64_t *dev_ops = (int64_t *)malloc(((size_t)N + 1) * sizeof(int64_t));
  int64_t *head = (int64_t *)malloc(((size_t)D + 1) * sizeof(int64_t));
  int64_t *send_until = (int64_t *)malloc(((size_t)D + 1) * sizeof(int64_t));
  int64_t *recv_until = (int64_t *)malloc(((size_t)D + 1) * sizeof(int64_t));
  char *dirty = (char *)calloc((size_t)D + 1, 1);
  /* pending transfers: producer, destination, request time (in arbitration order) */
  int64_t *pend_u = (int64_t *)malloc(((size_t)E + 1) * sizeof(int64_t));
  int64_t *pend_e = (int64_t *)malloc(((size_t)E + 1) * sizeof(int64_t));
  int64_t *fresh = (int64_t *)malloc(((size_t)D + 1) * sizeof(int64_t));
  sim_event *heap = (sim_event *)malloc(((size_t)N + E + 1) * sizeof(sim_event));
  int rc = -1;
  if (!dev_ptr || !dev_ops || !head || !send_until || !recv_until || !dirty || !pend_u || !pend_e || !fresh ||
      !heap)
    goto out;
  int64_t n_pend = 0, n_heap = 0, n_ord = 0;
  /* the compute queue of each device: its ops in index order */
  for (int64_t v = 0; v < N; ++v) dev_ptr[place[v] + 1]++;
  for (int64_t d = 0; d < D; ++d) dev_ptr[d + 1] += dev_ptr[d];
  for (int64_t d = 0; d < D; ++d) head[d] = dev_ptr[d];
  for (int64_t v = 0; v < N; ++v) dev_ops[head[place[v]]++] = v;
  for (int64_t d = 0; d < D; ++d) {
    head[d] = dev_ptr[d];
    clock[d] = send_until[d] = recv_until[d] = 0;
    dirty[d] = 1;
  }
  for (int64_t q = 0; q < E; ++q) xs[q] = xa[q] = -1;
  for (;;) {
    /* place every queue head whose inputs' availability is known */
    for (int64_t d = 0; d < D; ++d) {
      if (!dirty[d]) continue;
      dirty[d] = 0;
      for (; head[d] < dev_ptr[d + 1]; ++head[d]) {
        const int64_t v = dev_ops[head[d]];
        int64_t ready = g->release[g->op_req[v]];
        if (ready < 0) ready = 0;
        int known = 1;
        for (int64_t e = g->pred_ptr[v]; e < g->pred_ptr[v + 1] && known; ++e) {
          const int64_t u = g->pred_idx[e];
          int64_t avail;
          if (place[u] == d) {
            avail = fin[u]; /* earlier in this queue, hence placed */
          } else {
            avail = xa[first_entry_to(sc, place, u, d)];
            if (avail < 0) known = 0; /* its transfer has not started */
          }
          if (avail > ready) ready = avail;
        }
        if (!known) break;
        const int64_t w = op_duration(g, v, d);
        const int64_t t = ready > clock[d] ? ready : clock[d];
        st[v] = earliest_fit(g, d, t, w);
        fin[v] = st[v] + w;
        clock[d] = fin[v];
        event_push(heap, &n_heap, (sim_event){fin[v], 0, v});
      }
    }
    if (n_heap == 0) break;
    /* every event of the next instant t */
    const int64_t t = heap[0].time;
    while (n_heap > 0 && heap[0].time == t) {
      const sim_event ev = event_pop(heap, &n_heap);
      if (ev.kind != 0) continue; /* an arrival: its ports are idle from t on */
      const int64_t u = ev.id, du = place[u];
      /* Intents of u, one per remote destination device, by device id */
      int64_t nf = 0;
      for (int64_t q = sc->ptr[u]; q < sc->ptr[u + 1]; ++q) {
        const int64_t e = place[sc->idx[q]];
        if (e == du || first_entry_to(sc, place, u, e) != q) continue;
        int64_t i = nf++;
        while (i > 0 && fresh[i - 1] > e) { fresh[i] = fresh[i - 1]; --i; }
        fresh[i] = e;
      }
      for (int64_t i = 0; i < nf; ++i) {
        const int64_t e = fresh[i];
        if (transfer_time(g, u, du, e) == 0) { /* nothing moves */
          set_transfer(sc, place, u, e, t, t, xs, xa);
          if (order) order[n_ord] = first_entry_to(sc, place, u, e);
          ++n_ord;
          dirty[e] = 1;
        } else {
          pend_u[n_pend] = u;
          pend_e[n_pend] = e;
          ++n_pend;
        }
      }
    }
    /* arbitration at t: pending transfers in order, each started when both of
     * its ports are idle */
    int64_t kept = 0;
    for (int64_t i = 0; i < n_pend; ++i) {
      const int64_t u = pend_u[i], e = pend_e[i], s = place[u];
      if (send_until[s] <= t && recv_until[e] <= t) {
        const int64_t a = t + transfer_time(g, u, s, e);
        set_transfer(sc, place, u, e, t, a, xs, xa);
        send_until[s] = recv_until[e] = a;
        event_push(heap, &n_heap, (sim_event){a, 1, first_entry_to(sc, place, u, e)});
        if (order) order[n_ord] = first_entry_to(sc, place, u, e);
        ++n_ord;
        dirty[e] = 1;
      } else {
        pend_u[kept] = u;
        pend_e[kept] = e;
        ++kept;
      }
    }
    n_pend = kept;
  }
  if (n_order) *n_order = n_ord;
  rc = 0;
out:
  free(dev_ptr); free(dev_ops); free(head); free(send_until); free(recv_until); free(dirty);
  free(pend_u); free(pend_e); free(fresh); free(heap);
  return rc;
}

/* binary min-heap of (ready, op) pairs */
typedef struct { int64_t ready, op; } ready_item;

static int item_less(ready_item a, ready_item b) {
  return a.ready < b.ready || (a.ready == b.ready && a.op < b.op);
}

static void heap_push(ready_item *h, int64_t *n, ready_item x) {
  int64_t i = (*n)++;
  h[i] = x;
  while (i > 0) {
    const int64_t p = (i - 1) / 2;
    if (!item_less(h[i], h[p])) break;
    ready_item t = h[i]; h[i] = h[p]; h[p] = t;
    i = p;
  }
}

static ready_item heap_pop(ready_item *h, int64_t *n) {
  ready_item top = h[0];
  h[0] = h[--(*n)];
  int64_t i = 0;
  for (;;) {
    const int64_t l = 2 * i + 1, r = l + 1;
    int64_t m = i;
    if (l < *n && item_less(h[l], h[m])) m = l;
    if (r < *n && item_less(h[r], h[m])) m = r;
    if (m == i) break;
    ready_item t = h[i]; h[i] = h[m]; h[m] = t;
    i = m;
  }
  return top;
}

/* Ready-order variant: repeatedly dispatch the op with the earliest ready
 * time among those whose predecessors are all scheduled (ties to the lower
 * index), then place it on its device exactly as contract A does. */
static int schedule_ready_order(const sso_gmg *g, const uint8_t *place, const succ_csr *sc, int64_t *clock,
                                int64_t *st, int64_t *fin) {
  const int64_t N = g->n_ops;
  int64_t *missing = (int64_t *)malloc(((size_t)N + 1) * sizeof(int64_t));
  ready_item *heap = (ready_item *)malloc(((size_t)N + 1) * sizeof(ready_item));
  if (!missing || !heap) { free(missing); free(heap); return -1; }
  int64_t hn = 0;
  for (int64_t d = 0; d < g->n_dev; ++d) clock[d] = 0;
  for (int64_t v = 0; v < N; ++v) {
    missing[v] = g->pred_ptr[v + 1] - g->pred_ptr[v];
    if (missing[v] == 0) heap_push(heap, &hn, (ready_item){ready_time(g, place, fin, v), v});
  }
  while (hn > 0) {
    const ready_item it = heap_pop(heap, &hn);
    const int64_t v = it.op, d = place[v];
    const int64_t w = op_duration(g, v, d);
    const int64_t t = it.ready > clock[d] ? it.ready : clock[d];
    st[v] = earliest_fit(g, d, t, w);
    fin[v] = st[v] + w;
    clock[d] = fin[v];
    for (int64_t e = sc->ptr[v]; e < sc->ptr[v + 1]; ++e) {
      const int64_t x = sc->idx[e];
      if (--missing[x] == 0) heap_push(heap, &hn, (ready_item){ready_time(g, place, fin, x), x});
    }
  }
  free(missing);
  free(heap);
  return 0;
}

/* ---------------------------------------------------------------- memory */

typedef struct { int64_t dev, lo, hi, bytes; } interval;

/* The part of an interval at or after t0 (empty, [t0, t0), when it ended
 * before): memory is counted from the snapshot's timestamp on. */
static interval clip(interval iv, int64_t t0) {
  if (iv.lo < t0) iv.lo = t0;
  if (iv.hi < t0) iv.hi = t0;
  return iv;
}

/* Residency intervals of one scheduled candidate (see the memory reading in
 * the file header).  Returns the count, or -1 on allocation failure. */
static int64_t residency_intervals(const sso_gmg *g, const uint8_t *place, const succ_csr *sc, const int64_t *st,
                                   const int64_t *fin, const int64_t *xs, const int64_t *xa, interval **out) {
  const int64_t N = g->n_ops;
  int64_t cap = N + sc->ptr[N] + 1, n = 0;
  interval *iv = (interval *)malloc((size_t)cap * sizeof(interval));
  if (!iv) return -1;
  for (int64_t v = 0; v < N; ++v) {
    const int64_t d = place[v];
    const int64_t b = g->out_bytes[v];
    const int64_t s0 = sc->ptr[v], s1 = sc->ptr[v + 1];
    /* own output on d: from v's start until every local consumer has finished
     * and every outgoing transfer has arrived; kept forever without consumers */
    int64_t free_at = SSO_INF;
    if (s1 > s0) {
      free_at = fin[v];
      for (int64_t e = s0; e < s1; ++e) {
        const int64_t x = sc->idx[e], dx = place[x];
        const int64_t t = (dx == d) ? fin[x] : xa ? xa[e] : transfer_arrival(g, sc, place, fin, v, dx);
        if (t > free_at) free_at = t;
      }
    }
    iv[n++] = clip((interval){d, st[v], free_at, b}, g->t_now);
    /* one remote copy per destination device, from the transfer's start (v's
     * finish, not before the first consumer there was issued; with arbitrated
     * ports the admitted start) until the last consumer on that device
     * finishes */
    for (int64_t e = s0; e < s1; ++e) {
      const int64_t dx = place[sc->idx[e]];
      if (dx == d) continue;
      int seen = 0;
      for (int64_t e2 = s0; e2 < e; ++e2)
        if (place[sc->idx[e2]] == dx) seen = 1;
      if (seen) continue;
      int64_t last = 0;
      for (int64_t e2 = s0; e2 < s1; ++e2)
        if (place[sc->idx[e2]] == dx && fin[sc->idx[e2]] > last) last = fin[sc->idx[e2]];
      const int64_t floor_ = transfer_floor(g, sc, place, v, dx);
      iv[n++] = clip((interval){dx, xs ? xs[e] : fin[v] > floor_ ? fin[v] : floor_, last, b}, g->t_now);
    }
  }
  *out = iv;
  return n;
}

typedef struct { int64_t time; int64_t is_alloc; int64_t delta; } mem_event;

static int event_cmp(const void *pa, const void *pb) {
  const mem_event *a = (const mem_event *)pa, *b = (const mem_event *)pb;
  if (a->time != b->time) return a->time < b->time ? -1 : 1;
  /* at equal times frees come first: intervals are half-open */
  if (a->is_alloc != b->is_alloc) return a->is_alloc < b->is_alloc ? -1 : 1;
  return 0;
}

/* peak[d] = max over time of the bytes live on d; sweep over sorted endpoints */
static int peak_by_sweep(const sso_gmg *g, const interval *iv, int64_t n, int64_t *peak) {
  mem_event *ev = (mem_event *)malloc(((size_t)2 * n + 1) * sizeof(mem_event));
  if (!ev) return -1;
  for (int64_t d = 0; d < g->n_dev; ++d) {
    int64_t m = 0;
    for (int64_t i = 0; i < n; ++i) {
      if (iv[i].dev != d) continue;
      ev[m++] = (mem_event){iv[i].lo, 1, iv[i].bytes};
      if (iv[i].hi != SSO_INF) ev[m++] = (mem_event){iv[i].hi, 0, -iv[i].bytes};
    }
    qsort(ev, (size_t)m, sizeof(mem_event), event_cmp);
    int64_t live = 0, best = 0;
    for (int64_t i = 0; i < m; ++i) {
      live += ev[i].delta;
      if (live > best) best = live;
    }
    peak[d] = best;
  }
  free(ev);
  return 0;
}

/* peak[d] = max over allocation instants t of sum of bytes with lo <= t < hi */
static void peak_by_pairs(const sso_gmg *g, const interval *iv, int64_t n, int64_t *peak) {
  for (int64_t d = 0; d < g->n_dev; ++d) peak[d] = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t t = iv[i].lo;
    int64_t live = 0;
    for (int64_t j = 0; j < n; ++j)
      if (iv[j].dev == iv[i].dev && iv[j].lo <= t && t < iv[j].hi) live += iv[j].bytes;
    if (live > peak[iv[i].dev]) peak[iv[i].dev] = live;
  }
}

/* ---------------------------------------------------------------- what-if */

static int valid_placement(const sso_gmg *g, const uint8_t *place) {
  for (int64_t v = 0; v < g->n_ops; ++v)
    if (place[v] >= g->n_dev) return 0;
  return 1;
}

typedef struct {
  int64_t *st, *fin, *clock, *peak, *xs, *xa, *order;
} work_bufs;

static int simulate_with(const sso_gmg *g, const succ_csr *sc, const uint8_t *place, int dispatch,
                         const work_bufs *wb, int64_t *makespan, int64_t *peak, uint8_t *violation, int64_t *slack,
                         int64_t *sumfin) {
  int64_t *st = wb->st, *fin = wb->fin, *clock = wb->clock, *peak_buf = wb->peak;
  const int ports = dispatch == SSO_LINK_PORTS;
  const int64_t N = g->n_ops, D = g->n_dev, R = g->n_req;
  if (!valid_placement(g, place)) {
    /* a placement naming a device outside the set is not simulated */
    *makespan = INT64_MAX;
    *sumfin = INT64_MAX;
    *violation = 4;
    if (peak) for (int64_t d = 0; d < D; ++d) peak[d] = 0;
    if (slack) for (int64_t r = 0; r < R; ++r) slack[r] = INT64_MIN;
    return 0;
  }
  if ((g->done_fin || g->issue_at) && dispatch != SSO_INDEX_ORDER) return -3;
  if (dispatch == SSO_READY_ORDER) {
    if (schedule_ready_order(g, place, sc, clock, st, fin) != 0) return -1;
  } else if (ports) {
    if (schedule_index_order_ports(g, place, sc, clock, st, fin, wb->xs, wb->xa, 0, 0) != 0) return -1;
  } else {
    schedule_index_order(g, place, sc, clock, st, fin);
  }
  /* completion-time statistics (Sec. 3.3.3): makespan from t0 = 0, per-request
   * completion (its release when it has no ops) against its deadline, and the
   * sum of finish times (average completion time times N, Sec. 3.4.2) */
  int64_t ms = 0, sum = 0;
  for (int64_t v = 0; v < N; ++v) {
    if (fin[v] > ms) ms = fin[v];
    sum += fin[v];
  }
  *makespan = ms;
  *sumfin = sum;
  if (slack) {
    for (int64_t r = 0; r < R; ++r) slack[r] = g->release[r];
    for (int64_t v = 0; v < N; ++v)
      if (fin[v] > slack[g->op_req[v]]) slack[g->op_req[v]] = fin[v];
    for (int64_t r = 0; r < R; ++r) slack[r] = g->deadline[r] - slack[r];
  }
  interval *iv = 0;
  const int64_t n = residency_intervals(g, place, sc, st, fin, ports ? wb->xs : 0, ports ? wb->xa : 0, &iv);
  if (n < 0) return -1;
  const int rc = peak_by_sweep(g, iv, n, peak_buf);
  free(iv);
  if (rc != 0) return -1;
  uint8_t viol = 0;
  for (int64_t d = 0; d < D; ++d)
    if (peak_buf[d] > g->cap[d]) viol = 1;
  *violation = viol;
  if (peak) memcpy(peak, peak_buf, (size_t)D * sizeof(int64_t));
  return 0;
}

static int alloc_work(const sso_gmg *g, work_bufs *w) {
  const size_t N = (size_t)g->n_ops + 1, D = (size_t)g->n_dev + 1, E = (size_t)g->pred_ptr[g->n_ops] + 1;
  w->st = (int64_t *)malloc(N * sizeof(int64_t));
  w->fin = (int64_t *)malloc(N * sizeof(int64_t));
  w->clock = (int64_t *)malloc(D * sizeof(int64_t));
  w->peak = (int64_t *)malloc(D * sizeof(int64_t));
  w->order = (int64_t *)malloc(E * sizeof(int64_t));
  w->xs = (int64_t *)malloc(E * sizeof(int64_t));
  w->xa = (int64_t *)malloc(E * sizeof(int64_t));
  return (w->st && w->fin && w->clock && w->peak && w->order && w->xs && w->xa) ? 0 : -1;
}

static void free_work(work_bufs *w) {
  free(w->st); free(w->fin); free(w->clock); free(w->peak);
  free(w->order); free(w->xs); free(w->xa);
}

int sso_simulate_one(const sso_gmg *g, const uint8_t *place, int dispatch, int64_t *st, int64_t *fin,
                     int64_t *makespan, int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin) {
  succ_csr sc;
  work_bufs w;
  if (build_succ(g, &sc) != 0) return -1;
  if (alloc_work(g, &w) != 0) { free_succ(&sc); free_work(&w); return -1; }
  const int rc = simulate_with(g, &sc, place, dispatch, &w, makespan, peak, violation, slack, sumfin);
  if (rc == 0 && valid_placement(g, place)) {
    if (st) memcpy(st, w.st, (size_t)g->n_ops * sizeof(int64_t));
    if (fin) memcpy(fin, w.fin, (size_t)g->n_ops * sizeof(int64_t));
  }
  free_work(&w);
  free_succ(&sc);
  return rc;
}

int sso_simulate_batch(const sso_gmg *g, const uint8_t *places, int64_t B, int dispatch, int64_t *makespan,
                       int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin) {
  succ_csr sc;
  work_bufs w;
  if (build_succ(g, &sc) != 0) return -1;
  if (alloc_work(g, &w) != 0) { free_succ(&sc); free_work(&w); return -1; }
  int rc = 0;
  for (int64_t b = 0; b < B && rc == 0; ++b)
    rc = simulate_with(g, &sc, places + b * g->n_ops, dispatch, &w, &makespan[b], peak ? peak + b * g->n_dev : 0,
                       &violation[b], slack ? slack + b * g->n_req : 0, &sumfin[b]);
  free_work(&w);
  free_succ(&sc);
  return rc;
}

static int peak_common(const sso_gmg *g, const uint8_t *place, const int64_t *st, const int64_t *fin,
                       int64_t *peak, int pairwise) {
  succ_csr sc;
  if (build_succ(g, &sc) != 0) return -1;
  interval *iv = 0;
  const int64_t n = residency_intervals(g, place, &sc, st, fin, 0, 0, &iv);
  free_succ(&sc);
  if (n < 0) return -1;
  int rc = 0;
  if (pairwise)
    peak_by_pairs(g, iv, n, peak);
  else
    rc = peak_by_sweep(g, iv, n, peak);
  free(iv);
  return rc;
}

int sso_peak_sweep(const sso_gmg *g, const uint8_t *place, const int64_t *st, const int64_t *fin, int64_t *peak) {
  return peak_common(g, place, st, fin, peak, 0);
}

int sso_peak_pairwise(const sso_gmg *g, const uint8_t *place, const int64_t *st, const int64_t *fin,
                      int64_t *peak) {
  return peak_common(g, place, st, fin, peak, 1);
}

/* Alg. 1: record feasible candidates, return the best.  Feasible = no memory
 * violation and a valid placement; optionally also no missed deadline.  Best =
 * smallest key (sum of finish times = N x average completion time, or the
 * makespan), ties to the lower candidate index. */
void sso_select_best(int64_t B, int64_t n_req, const uint8_t *violation, const int64_t *key, const int64_t *slack,
                     int require_sla, int64_t *best_idx, int64_t *best_key) {
  int64_t bi = -1, bk = INT64_MAX;
  for (int64_t b = 0; b < B; ++b) {
    if (violation[b] != 0) continue;
    if (require_sla) {
      int ok = 1;
      for (int64_t r = 0; r < n_req; ++r)
        if (slack[b * n_req + r] < 0) ok = 0;
      if (!ok) continue;
    }
    if (bi < 0 || key[b] < bk) {
      bi = b;
      bk = key[b];
    }
  }
  *best_idx = bi;
  *best_key = bk;
}

int sso_port_transfers(const sso_gmg *g, const uint8_t *place, int64_t *op, int64_t *src, int64_t *dst,
                       int64_t *start, int64_t *arrive, int64_t *n) {
  *n = 0;
  if (!valid_placement(g, place)) return -2;
  succ_csr sc;
  work_bufs w;
  if (build_succ(g, &sc) != 0) return -1;
  int64_t *owner = (int64_t *)malloc(((size_t)sc.ptr[g->n_ops] + 1) * sizeof(int64_t));
  if (!owner || alloc_work(g, &w) != 0) {
    free(owner); free_succ(&sc); free_work(&w);
    return -1;
  }
  /* producer of every successor entry */
  for (int64_t v = 0; v < g->n_ops; ++v)
    for (int64_t q = sc.ptr[v]; q < sc.ptr[v + 1]; ++q) owner[q] = v;
  int64_t m = 0;
  int rc = schedule_index_order_ports(g, place, &sc, w.clock, w.st, w.fin, w.xs, w.xa, w.order, &m);
  for (int64_t i = 0; rc == 0 && i < m; ++i) { /* in the order the transfers started */
    const int64_t q = w.order[i], v = owner[q];
    op[i] = v;
    src[i] = place[v];
    dst[i] = place[sc.idx[q]];
    start[i] = w.xs[q];
    arrive[i] = w.xa[q];
  }
  if (rc == 0) *n = m;
  free(owner);
  free_work(&w);
  free_succ(&sc);
  return rc;
}
