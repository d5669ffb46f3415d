/*
 * Oracle for the GMG what-if simulator -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, sequential, deliberately unoptimised CPU implementation of what the
 * simulator computes, used by the tests, by the smoke check and by the
 * benchmark's CPU-baseline leg to judge the HIP implementation.  Nothing on the
 * product path links, loads or calls it.  It shares no code, header, table or
 * helper with the HIP library; the array layout of a GMG snapshot is the same
 * because both sides take the same generated input arrays.
 *
 * All quantities are int64: times in microseconds, sizes in bytes.
 */
#ifndef SS_ORACLE_H
#define SS_ORACLE_H
#include <stdint.h>

#define SSO_INF INT64_MAX

/* A GMG snapshot (Sec. 3.2): operator DAG (predecessor CSR, index order is a
 * topological order and the dispatch-priority order), per-(op, device class)
 * durations from the operator estimator, output tensor sizes, and the
 * accelerator set (device classes, pairwise link classes with linear transfer
 * estimators, idle slices, capacities), plus per-request release times and
 * deadlines. */
typedef struct {
  int64_t n_ops, n_dev, n_class, n_link, n_req;
  const int32_t *pred_ptr;   /* [n_ops+1] */
  const int32_t *pred_idx;   /* [n_edges], each < its op */
  const int32_t *op_req;     /* [n_ops] */
  const int64_t *dur;        /* [n_ops][n_class] */
  const int64_t *out_bytes;  /* [n_ops] */
  const int32_t *dev_class;  /* [n_dev] */
  const uint8_t *link_class; /* [n_dev][n_dev] */
  const int64_t *bw;         /* [n_link] bytes per microsecond */
  const int64_t *lat;        /* [n_link] microseconds */
  const int64_t *slice_ptr;  /* [n_dev+1] */
  const int64_t *slice_begin;/* idle slice starts */
  const int64_t *slice_end;  /* idle slice ends; last slice of a device ends at SSO_INF */
  const int64_t *cap;        /* [n_dev] */
  const int64_t *release;    /* [n_req] */
  const int64_t *deadline;   /* [n_req] */
  /* A snapshot of a running schedule (Sec. 3.2 scheduling metadata), both
   * optional (NULL: none), index-order dispatch only:
   *   done_fin[n_ops]  -1, or the recorded completion time of an op that is
   *                    done: it is not simulated, it finished then on its
   *                    device (free from then on); its output counts from
   *                    that time minus its estimate;
   *   issue_at[n_ops]  the time an op was issued: it does not start earlier,
   *                    and a transfer to it does not start before the first
   *                    of its destination's consumers was issued.
   * t_now is the snapshot's timestamp: peak memory is taken over times at or
   * after it (0 without a snapshot, where every residency starts at >= 0). */
  const int64_t *done_fin;
  const int64_t *issue_at;
  int64_t t_now;
} sso_gmg;

/* dispatch rules */
#define SSO_INDEX_ORDER 0  /* each device serves its ops in index (priority) order */
#define SSO_READY_ORDER 1  /* global earliest-ready-time-first dispatch */
#define SSO_LINK_PORTS 2   /* index order; transfers arbitrated event by event over per-device send and receive ports */

/* One candidate.  st/fin (length n_ops) and peak (n_dev), slack (n_req) may be
 * NULL.  Returns 0, -1 on allocation failure, -3 for a snapshot (done_fin or
 * issue_at) with another dispatch than SSO_INDEX_ORDER. */
int sso_simulate_one(const sso_gmg *g, const uint8_t *place, int dispatch, int64_t *st, int64_t *fin,
                     int64_t *makespan, int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin);

/* B candidates, placements row-major [B][n_ops]; outputs [B], [B][n_dev], [B], [B][n_req], [B]. */
int sso_simulate_batch(const sso_gmg *g, const uint8_t *places, int64_t B, int dispatch, int64_t *makespan,
                       int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin);

/* Per-device peak memory of a scheduled candidate, by a time sweep over the
 * interval endpoints, and by evaluating the live bytes at every allocation
 * instant directly (quadratic).  Both take the schedule (st, fin). */
int sso_peak_sweep(const sso_gmg *g, const uint8_t *place, const int64_t *st, const int64_t *fin, int64_t *peak);
int sso_peak_pairwise(const sso_gmg *g, const uint8_t *place, const int64_t *st, const int64_t *fin,
                      int64_t *peak);

/* The transfers of one candidate under SSO_LINK_PORTS, in the order they start:
 * producer op, source and destination device, start and arrival.  The arrays
 * hold at least n_edges entries; *n receives the count.  Returns 0, -1 on
 * allocation failure, -2 for a placement naming a device outside the set. */
int sso_port_transfers(const sso_gmg *g, const uint8_t *place, int64_t *op, int64_t *src, int64_t *dst,
                       int64_t *start, int64_t *arrive, int64_t *n);

/* Best feasible candidate: argmin over feasible b of (key[b], b); -1 if none. */
void sso_select_best(int64_t B, int64_t n_req, const uint8_t *violation, const int64_t *key,
                     const int64_t *slack, int require_sla, int64_t *best_idx, int64_t *best_key);

#endif
