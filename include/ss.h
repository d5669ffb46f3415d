/*
 * ss.h -- C ABI of the MI355X what-if simulator over the Global Mapping Graph.
 *
 * The method is SliceScheduler's global simulator (arXiv 2608.15762,
 * Sec. 3.3) driven by the parallel candidate loop of its incremental
 * scheduling algorithm (Alg. 1, Sec. 3.4): a GMG snapshot (Sec. 3.2) plus a
 * batch of candidate placements goes in; per candidate the simulated
 * makespan, per-device peak memory, a violation verdict and per-request SLA
 * slack come out, and the best feasible candidate is selected.
 *
 * Every entry point returns SS_OK (0) or a negative SS_ERR_* code and never
 * throws; ss_last_error() gives a message for the calling thread's last
 * failure.  All times are int64 microseconds and all sizes int64 bytes.
 */
#ifndef SS_H
#define SS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SS_OK 0
#define SS_ERR_INVALID_ARG (-1)  /* null pointer, negative count, unknown flag or layout */
#define SS_ERR_INVALID_GMG (-2)  /* the snapshot breaks a rule listed under ss_gmg_desc */
#define SS_ERR_OOM (-3)          /* host or device allocation failed */
#define SS_ERR_DEVICE (-4)       /* a HIP call or kernel launch failed */
#define SS_ERR_UNSUPPORTED (-5)  /* valid input beyond the library's limits (see ss_gmg_desc) */

#define SS_TIME_INF INT64_MAX    /* end of a device's last (open) idle slice */

#define SS_LAYOUT_ROW_MAJOR 0    /* placements[b * n_ops + v] = device of op v in candidate b */
#define SS_LAYOUT_OP_MAJOR 1     /* placements[v * B + b] = device of op v in candidate b */
#define SS_DISPATCH_READY 0x100  /* OR into layout: ready-time dispatch (see ss_simulate_batch) */
#define SS_LINK_PORTS 0x200      /* OR into layout: transfers arbitrated over device ports (see ss_simulate_batch) */

#define SS_VIOLATION_MEMORY 0x1  /* some device's peak memory exceeds its capacity */
#define SS_VIOLATION_INVALID 0x4 /* the placement names a device id >= n_dev; not simulated */

#define SS_SELECT_REQUIRE_SLA 0x1 /* feasible also requires every request's slack >= 0 */

typedef struct ss_gmg ss_gmg;

/*
 * A GMG snapshot (Sec. 3.2): the Shape DAG of the operators to place, their
 * estimator outputs, and the Accelerator Set with its pre-existing load.
 * All pointers are HOST pointers; ss_gmg_load copies what it needs, so the
 * caller may free them when it returns.
 *
 *   n_ops N        operators; index order is a topological order and is the
 *                  dispatch priority of every device queue (Sec. 3.3.2).
 *   pred_ptr[N+1], pred_idx[E]  predecessor CSR: the data dependencies of op v
 *                  are pred_idx[pred_ptr[v] .. pred_ptr[v+1]), strictly
 *                  increasing and each < v; pred_ptr[0] = 0.
 *   op_req[N]      request of each op, in [0, n_req).
 *   dur[N][n_class] operator estimator (Sec. 3.3.1): duration of op v on a
 *                  device of class c, >= 1.
 *   out_bytes[N]   size of op v's output tensor (Sec. 3.2 metadata), >= 0.
 *   dev_class[D]   class of each device, in [0, n_class).  1 <= D <= 255.
 *   link_class[D][D] link class of each ordered device pair (diagonal
 *                  ignored), in [0, n_link).
 *   bw[K], lat[K]  transfer estimator t = alpha*size + c per link class
 *                  (Sec. 3.3.1) in integer form lat + ceil(bytes / bw);
 *                  bw >= 1 byte/us, lat >= 0.
 *   slice_ptr[D+1], slice_begin[], slice_end[]  idle slices of device d are
 *                  [slice_begin[k], slice_end[k]) for k in
 *                  [slice_ptr[d], slice_ptr[d+1]): at least one, begin >= 0,
 *                  begin < end, end <= next begin, every end finite except the
 *                  last, which is SS_TIME_INF (the device is free from then on).
 *                  At most 65535 slices per device.
 *   cap[D]         memory available to the simulated tensors on each device.
 *   release[R], deadline[R]  per-request arrival (>= 0) and absolute SLA
 *                  deadline (|deadline| < 2^62).
 *
 * The state of a running schedule (Sec. 3.2 scheduling metadata: the issued
 * and done timestamps of the ops; Sec. 3.3.2 builds the simulator from it),
 * all optional (NULL / 0: a plan from an idle start):
 *   done_fin[N]    -1, or the recorded completion time (>= 0) of an op that
 *                  is done.  A done op is not simulated: it finished then on
 *                  the device its candidate names, which is free from then
 *                  on; its output counts from that time minus its estimate.
 *                  A done op's predecessors must be done and have finished
 *                  strictly earlier.
 *   issue_at[N]    the time (>= 0) each op was issued: it starts no earlier,
 *                  and the transfer of an output to a device starts no
 *                  earlier than the first issue time among its consumers on
 *                  that device (its Intent exists from then on).  A done op
 *                  must finish strictly after its issue time.
 *   t_now          the snapshot's timestamp (>= 0): peak memory is taken over
 *                  the times at or after it (every residency interval clipped
 *                  to [t_now, inf)).
 * A GMG with any of them simulates under index-order dispatch with latency-
 * only transfers (SS_DISPATCH_READY and SS_LINK_PORTS: SS_ERR_UNSUPPORTED).
 *
 * The loader also rejects snapshots whose time horizon could overflow:
 * H = T + sum_v max_c dur[v][c]
 *     + sum_v (outdeg(v) + 1) * max_k (lat[k] + ceil(out_bytes[v] / bw[k])),
 * with T the largest of the last-slice starts, releases, issue times, done
 * times and t_now, must stay below 2^62, N * H below 2^63, and
 * sum_v out_bytes[v] * (D + 1) below 2^63.
 */
typedef struct ss_gmg_desc {
  int64_t n_ops, n_edges, n_dev, n_class, n_link, n_req;
  const int32_t *pred_ptr;
  const int32_t *pred_idx;
  const int32_t *op_req;
  const int64_t *dur;
  const int64_t *out_bytes;
  const int32_t *dev_class;
  const uint8_t *link_class;
  const int64_t *bw;
  const int64_t *lat;
  const int64_t *slice_ptr;
  const int64_t *slice_begin;
  const int64_t *slice_end;
  const int64_t *cap;
  const int64_t *release;
  const int64_t *deadline;
  const int64_t *done_fin; /* nullable */
  const int64_t *issue_at; /* nullable */
  int64_t t_now;
} ss_gmg_desc;

/*
 * Validate a snapshot (rules above), precompute its transfer table and
 * successor lists, and stage it in the memory of the CURRENT HIP device
 * (once per GMG; Sec. 3.3.2 builds the simulator from the snapshot).
 * On success *out owns the staged copy until ss_gmg_free.  A loaded GMG is
 * read-only and may be used by concurrent calls on any streams of that device.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_INVALID_GMG, SS_ERR_OOM, SS_ERR_DEVICE.
 */
int ss_gmg_load(const ss_gmg_desc *desc, ss_gmg **out);

/* Release a GMG (synchronises the device first; its memory goes back to the
 * library's pool, see ss_release_cached_memory).  NULL is a no-op. */
void ss_gmg_free(ss_gmg *g);

/* Sizes of a loaded GMG; any output pointer may be NULL. */
int ss_gmg_info(const ss_gmg *g, int64_t *n_ops, int64_t *n_dev, int64_t *n_req);

/*
 * What-if simulation of B candidate placements at once (Sec. 3.3.3 and the
 * "in parallel" candidate loop of Alg. 1).  For each candidate b:
 *   - ops run in index order on their devices, one at a time, each starting
 *     at the earliest instant >= max(ready time, the device's previous
 *     finish) at which it fits entirely inside one idle slice; the ready time
 *     is the later of the request's release and, over the predecessors, their
 *     finish plus the transfer estimate when they ran on another device
 *     (Sec. 3.3.2); with a running schedule's state (see ss_gmg_desc) done
 *     ops keep their recorded finish, ops wait for their issue time and
 *     transfers for their destination's first issued consumer;
 *   - memory: an op's output occupies its device from the op's start until
 *     its last local consumer finishes and its last outgoing transfer has
 *     arrived (forever if it has no consumer); each (output, remote device)
 *     pair holds one copy there from the producer's finish until the last
 *     consumer on that device finishes; peak = the maximum over time of the
 *     bytes resident on a device (half-open intervals) (Sec. 3.3.2, 3.5.2).
 * Outputs (DEVICE pointers, caller-owned, row-major):
 *   out_makespan[B]      latest finish time (t0 = 0)              (required)
 *   out_peak_mem[B][D]   per-device peak bytes                    (nullable)
 *   out_violation[B]     SS_VIOLATION_* bits, 0 = feasible        (required)
 *   out_sla_slack[B][R]  deadline[r] - completion of request r (its release
 *                        when it has no ops); may be negative     (nullable)
 *   out_sumfin[B]        sum of finish times = N x the average completion
 *                        time that Sec. 3.4.2 minimises           (nullable)
 * With layout | SS_DISPATCH_READY the dispatch rule is the ready-time rule
 * of Sec. 3.3.2 instead of index order: of the ops whose predecessors have
 * all been dispatched, the one with the earliest ready time (ties to the lower
 * index) is dispatched next, at the earliest fit on its device at or after
 * max(ready time, that device's previous finish).  Memory follows the same
 * definitions with "last" meaning the consumer that finishes last.  Both
 * rules accept every GMG the loader accepts; the ready-time rule evaluates a
 * candidate with one wavefront instead of one lane, so it costs more per
 * candidate, and it needs scratch for N ready entries per candidate in flight.
 * A candidate naming a device >= n_dev is not simulated: violation =
 * SS_VIOLATION_INVALID, makespan = sumfin = INT64_MAX, peak = 0 and slack =
 * INT64_MIN.  This is a per-candidate result, not a call error.
 * With layout | SS_LINK_PORTS transfers contend for the devices' ports, after
 * the event-driven arbitration of Sec. 3.5.2: each device sends one tensor at
 * a time and receives one at a time.  The output of an op is moved once to
 * every other device holding a consumer; that transfer becomes pending when
 * the op finishes.  At every instant where an op finishes or a transfer
 * arrives, the pending transfers are examined in order of request time, then
 * producer index, then destination device, and each one whose send and
 * receive ports are both idle starts then and holds both until it arrives
 * (its estimate later); a zero estimate moves nothing and completes at once.
 * Compute queues stay index-ordered.  Consumers on the destination wait for
 * the arrival; the copy there is allocated at the transfer's start and the
 * producer's output is kept until its last transfer has arrived.  Index-order
 * dispatch only: with SS_DISPATCH_READY as well the call fails with
 * SS_ERR_UNSUPPORTED.  This variant simulates each candidate with one
 * wavefront, event by event, so it costs more per candidate than the
 * latency-only rule.
 * placements: DEVICE pointer, uint8, SS_LAYOUT_ROW_MAJOR [B][n_ops] or
 * SS_LAYOUT_OP_MAJOR [n_ops][B] (the layout the schedule pass reads: no
 * transpose of the batch before it), either one OR-ed with the flags above.
 * The call is asynchronous on hip_stream (NULL = the null stream); inputs must
 * stay valid and outputs are defined once that stream has been synchronised.
 * It takes stream-ordered scratch on hip_stream, for the duration of the
 * work, from the library's memory pool for g's device, which keeps that
 * memory for later calls (for a fixed workload, calls after the first
 * allocate no device memory; see ss_release_cached_memory).  With index-order
 * dispatch its scratch is at most the preferred workspace
 * (ss_simulate_workspace_size) and at most seven eighths of the memory the
 * call can get at its start (free device memory, the pool's unused memory and
 * idle blocks); smaller memory means smaller chunks.  When the pool runs
 * short anyway, the call waits for hip_stream's earlier work, returns its idle
 * memory to the driver and retries once, then halves its chunks.  A caller that
 * must own that memory passes it to ss_simulate_batch_ws instead (sized with
 * ss_simulate_workspace_size).  B = 0 is a no-op.  Results are bit-identical
 * to a sequential CPU evaluation of the same rules.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_OOM, SS_ERR_DEVICE, SS_ERR_UNSUPPORTED.
 */
int ss_simulate_batch(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout, int64_t *out_makespan,
                      int64_t *out_peak_mem, uint8_t *out_violation, int64_t *out_sla_slack, int64_t *out_sumfin,
                      void *hip_stream);

/*
 * Workspace of ss_simulate_batch_ws for a batch of B candidates with this
 * layout and these flags (the same what-if simulation, Sec. 3.3.3 and the
 * candidate loop of Alg. 1): *min_bytes is the smallest workspace with which
 * the call works (it then runs in chunks of a few candidates), *pref_bytes
 * the size at which it runs in the chunks it would choose itself; any size in
 * between works, larger chunks being faster.  Either pointer may be NULL (not
 * both).  B = 0 gives 0.  Launches nothing.  Errors: SS_ERR_INVALID_ARG,
 * SS_ERR_DEVICE, SS_ERR_UNSUPPORTED (as ss_simulate_batch would).
 */
int ss_simulate_workspace_size(const ss_gmg *g, int64_t B, int layout, int64_t *min_bytes, int64_t *pref_bytes);

/*
 * How ss_simulate_batch splits B candidates (the same simulation, Sec. 3.3.3,
 * and candidate loop of Alg. 1): *chunk candidates per schedule launch and
 * *sub per memory-pass launch inside a chunk (equal to *chunk where the
 * memory pass is not split), so that tests and benchmarks can check the
 * candidates at every boundary.  The sizes follow the memory the device has
 * free at the time of the query, as a call's would (a call that then runs
 * out of memory halves its chunks).  Launches nothing.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE, SS_ERR_UNSUPPORTED.
 */
int ss_simulate_chunking(const ss_gmg *g, int64_t B, int layout, int64_t *chunk, int64_t *sub);

/*
 * The width in bits of the integers a ss_simulate_batch call on g with these
 * flags computes its simulated times in (Sec. 3.3.2-3.3.3; the results are
 * the same either way): 32 when the loader proved that every time of the GMG
 * fits in 32 bits and the call takes the 32-bit kernels (index-order or
 * ready-time dispatch; byte sums are then 32-bit too when their bound allows
 * it, else 64-bit), 64 on the general path (a GMG beyond 32 bits, a running
 * schedule's state, SS_LINK_PORTS, or SS_PATH=generic in the environment).
 * Launches nothing.  Errors: SS_ERR_INVALID_ARG (g or bits NULL, an unknown
 * flag), SS_ERR_DEVICE, SS_ERR_UNSUPPORTED (as ss_simulate_batch would).
 */
int ss_simulate_time_bits(const ss_gmg *g, int layout, int *bits);

/*
 * ss_simulate_batch with a caller-owned workspace: the same arguments and
 * results, plus `workspace`, a DEVICE buffer of workspace_bytes (256-byte
 * aligned, at least ss_simulate_workspace_size's min_bytes) that the call
 * uses for all of its scratch: it allocates no device memory, creates no
 * events and runs every kernel on hip_stream.  The workspace belongs to the
 * call until hip_stream has completed it; two calls in flight at once need
 * two workspaces.  Errors: as ss_simulate_batch, and SS_ERR_INVALID_ARG for
 * a NULL, misaligned or too small workspace.
 */
int ss_simulate_batch_ws(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout, int64_t *out_makespan,
                         int64_t *out_peak_mem, uint8_t *out_violation, int64_t *out_sla_slack, int64_t *out_sumfin,
                         void *workspace, int64_t workspace_bytes, void *hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * ss_simulate_batch with the same arguments and results, whose scratch is a
 * fixed array of 128 MiB per GPU inside the library (held from the first call
 * on that GPU until the process ends).  It calls no hipMalloc or hipFree,
 * creates no events and runs every kernel on hip_stream; a batch is processed
 * in chunks that fit the array.  Every call on one GPU shares that array, so
 * calls that overlap on one GPU (other streams, other threads) race: order
 * them.  A batch whose smallest scratch (ss_simulate_workspace_size's
 * min_bytes) exceeds the array fails with SS_ERR_INVALID_ARG before anything
 * is launched.  Errors: as ss_simulate_batch, and SS_ERR_INVALID_ARG for such
 * a batch.
 */
int ss_simulate_batch_noalloc(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout,
                              int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                              int64_t *out_sla_slack, int64_t *out_sumfin, void *hip_stream);

/*
 * Prefix reuse for candidates that share their first ops (the ops before a
 * batch in Alg. 1's rounds, Sec. 3.4.2).  A state holds one simulated
 * candidate after the first k ops of a GMG: their finish times, every
 * device's clock and slice position, every request's completion so far, and
 * the running makespan and finish-time sum (device memory of the current
 * device, grown at capture).
 */
typedef struct ss_state ss_state;

/* An empty state (k = 0) on the current HIP device.  Errors: SS_ERR_INVALID_ARG,
 * SS_ERR_OOM, SS_ERR_DEVICE. */
int ss_state_create(ss_state **out);

/* Release a state (synchronises its device first).  NULL is a no-op. */
void ss_state_free(ss_state *st);

/* The number of ops the state holds (0 for an empty state or a failed capture). */
int ss_state_info(const ss_state *st, int64_t *n_ops);

/*
 * ss_simulate_batch (index-order dispatch, latency-only transfers, row-major
 * placements) resumed from `from`: the results are those of ss_simulate_batch
 * on the same arguments when `from` was captured from a simulation of a GMG
 * whose first k ops (and their predecessors, requests, durations, sizes) are
 * g's first k ops and whose placement of them is every candidate's (the
 * caller's contract, which with issue times also asks that ops k.. be issued
 * no earlier than ops ..k-1, as in the incremental loop, so that no later
 * consumer moves an earlier transfer; the library checks k <= n_ops and the
 * device and request counts).  Each candidate's schedule is walked from op k
 * only; the memory pass covers all ops.  from may be NULL or empty (a full simulation).
 * Placements of the first k ops are still checked against n_dev
 * (SS_VIOLATION_INVALID).  Asynchronous on hip_stream.  Errors:
 * SS_ERR_INVALID_ARG, SS_ERR_OOM, SS_ERR_DEVICE, SS_ERR_UNSUPPORTED.
 */
int ss_simulate_batch_resume(const ss_gmg *g, const ss_state *from, const uint8_t *placements, int64_t B,
                             int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                             int64_t *out_sla_slack, int64_t *out_sumfin, void *hip_stream);

/*
 * The schedule of one candidate (placement: DEVICE uint8 [n_ops]), resumed
 * from `from` as above, its state after all n_ops ops stored in capture
 * (capture != from; no memory pass, no outputs): the prefix for the next
 * call on a GMG that extends g with this placement of g's ops.  Asynchronous
 * on hip_stream (growing the state's buffer synchronises it first).  Errors:
 * SS_ERR_INVALID_ARG, SS_ERR_OOM, SS_ERR_DEVICE.
 */
int ss_state_capture(const ss_gmg *g, const ss_state *from, const uint8_t *placement, ss_state *capture,
                     void *hip_stream);

/*
 * Best-candidate selection of Alg. 1 / Sec. 3.4.2: discard infeasible
 * candidates (violation != 0, and with SS_SELECT_REQUIRE_SLA also any
 * negative slack), then take the smallest key, ties to the lowest index.
 * key is out_sumfin (the average-completion objective) or out_makespan.
 * violation[B], key[B], sla_slack[B][n_req] (needed only with
 * SS_SELECT_REQUIRE_SLA) are DEVICE pointers; out_best is a DEVICE int64[2]
 * receiving {index or -1, key or INT64_MAX}; it is also the reduction's only
 * scratch (the call allocates no device memory).  Asynchronous on hip_stream.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE.
 */
int ss_select_best(const ss_gmg *g, const uint8_t *violation, const int64_t *key, const int64_t *sla_slack,
                   int64_t B, int flags, int64_t *out_best, void *hip_stream);

/*
 * Kernel timing, for benchmarks.  While enabled (process-wide), every kernel
 * that ss_simulate_batch and ss_select_best launch is bracketed by a HIP
 * event pair recorded on the caller's stream.  ss_kernel_time waits for the
 * recorded events of one kernel kind, returns how many launches there were
 * and their summed duration in milliseconds, and forgets them.  Disabling
 * drops unread records.  Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE.
 */
#define SS_KERNEL_SCHEDULE 0     /* per-candidate list schedule (one lane per candidate) */
#define SS_KERNEL_MEMORY 1       /* per-device peak memory (one wave per candidate) */
#define SS_KERNEL_SELECT 2       /* best-candidate reduction (both passes) */
#define SS_KERNEL_INTERVALS 3    /* residency intervals into per-device buckets (fast path) */
#define SS_KERNEL_TRANSPOSE 4    /* layout changes between the passes (fast path) */
#define SS_KERNEL_ESTIMATOR 6    /* estimator accumulation, solves and predictions */
int ss_kernel_timing(int enable);
int ss_kernel_time(int kernel, int64_t *launches, double *total_ms);

/*
 * Online linear estimators (Sec. 3.3.1): the transfer estimator of an
 * accelerator pair, t = alpha * size + c, and the operator estimator of an
 * (accelerator type, template operator) pair, t = sum_j beta_j * phi_j(shape)
 * over shape-derived features (e.g. bmnk, bmk, bkn, bmn, 1 for a batched
 * matrix multiply), refined as the executor feeds back measured times.  An
 * estimator set holds n_est ordinary least-squares fits with n_feat (1..8)
 * features each.  Its state, on the HIP device current at creation, is every
 * fit's sufficient statistics in float64: sum x x^T, sum x y and the sample
 * count, accumulated over all samples added so far.  Calls on one set must be
 * ordered (one stream, or synchronised): concurrent calls race.
 */
#define SS_EST_MAX_FEAT 8
#define SS_EST_FITTED 0           /* coefficients solved */
#define SS_EST_UNDERDETERMINED 1  /* fewer samples than features; coefficients 0 */
#define SS_EST_SINGULAR 2         /* Gram matrix not positive definite (a Cholesky
                                     pivot <= 1e-12 x its diagonal entry); coefficients 0 */
typedef struct ss_est ss_est;

/* Create a set with zeroed statistics on the current device.  n_est >= 0,
 * 1 <= n_feat <= SS_EST_MAX_FEAT.  Errors: SS_ERR_INVALID_ARG, SS_ERR_OOM,
 * SS_ERR_DEVICE. */
int ss_est_create(int64_t n_est, int64_t n_feat, ss_est **out);

/* Release a set (synchronises its device first).  NULL is a no-op. */
void ss_est_free(ss_est *e);

/* Add n_samples feedback samples, grouped by estimator: the samples of
 * estimator i are rows [sample_ptr[i], sample_ptr[i+1]) of x[n_samples][n_feat]
 * (features) and y[n_samples] (measured times).  DEVICE pointers; sample_ptr
 * has n_est + 1 entries, non-decreasing from 0 to n_samples (ranges outside
 * [0, n_samples) are clamped to it, never read beyond it).  Asynchronous on
 * hip_stream; the sums of a set do not depend on how the device schedules the
 * work (a fixed reduction order).  Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE. */
int ss_est_add(ss_est *e, const int64_t *sample_ptr, int64_t n_samples, const double *x, const double *y,
               void *hip_stream);

/* Solve every fit: coef[n_est][n_feat] (DEVICE, float64) and status[n_est]
 * (DEVICE, SS_EST_*), from the normal equations by Cholesky factorisation.
 * Asynchronous on hip_stream.  Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE. */
int ss_est_solve(const ss_est *e, double *coef, int32_t *status, void *hip_stream);

/* Integer times for the simulator (durations of ss_gmg_desc.dur, or transfer
 * times): out_us[i] = max(1, ceil(x[i] . coef[est_of[i]])) for M queries.
 * DEVICE pointers: coef[n_est][n_feat], est_of[M], x[M][n_feat], out_us[M].
 * out_us[i] = 0 marks a query naming an estimator outside [0, n_est) or whose
 * prediction is not finite or reaches 2^62.  Asynchronous on hip_stream.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_DEVICE. */
int ss_est_predict(const double *coef, int64_t n_est, int64_t n_feat, const int32_t *est_of, const double *x,
                   int64_t M, int64_t *out_us, void *hip_stream);

/*
 * Incremental simulation-based scheduling (Alg. 1, Sec. 3.4).  A scheduler
 * holds the GMG of a whole run (every op that will be scheduled) with a state
 * per op (unscheduled, issued, done) and its scheduling metadata (Sec. 3.2:
 * the time it was issued, the time it completed), and keeps the two
 * frontiers of Sec. 3.4.1: the scheduled frontier (issued or done ops with an
 * unscheduled successor, whose outputs stay on their devices as checkpoints)
 * and the unscheduled frontier (unscheduled ops whose predecessors are all
 * issued or done).
 *
 * ss_sched_desc (HOST pointers, copied by ss_sched_create):
 *   gmg            the run's GMG; the loader's rules apply (ss_gmg_load); it
 *                  holds no running state (done_fin, issue_at NULL, t_now 0):
 *                  the scheduler keeps that.
 *   n_part, part_dev[n_part][n_ops]  the pre-defined partitions (Sec. 3.4.2):
 *                  partition p places op v on device part_dev[p][v] (< n_dev).
 *   priority[n_req] request priority, smaller first (for instance the
 *                  deadline); ties go to the lower op index.
 *   issue_budget   Alg. 1's budget on issued (not yet done) ops, >= 1.
 *   batch_cap      the batch cap of CollectConnectedGraph, >= 1.
 *   flags          SS_SELECT_REQUIRE_SLA (feasibility also requires every
 *                  request's slack >= 0) and SS_SCHED_PREFIX_REUSE (each
 *                  issuing round captures the chosen candidate's state, and
 *                  the next round resumes every candidate from it when no
 *                  completion came in between; same decisions, and slower
 *                  on the measured workloads: the candidates of a round run
 *                  in parallel lanes, so the capture's extra serial walk
 *                  costs more than the walk it saves), or 0.
 */
#define SS_SCHED_PREFIX_REUSE 0x2
#define SS_OP_UNSCHEDULED 0
#define SS_OP_ISSUED 1
#define SS_OP_DONE 2
#define SS_ROUND_ISSUED 0     /* a batch was placed and marked issued */
#define SS_ROUND_BUDGET 1     /* issued ops >= issue_budget: nothing done */
#define SS_ROUND_IDLE 2       /* the unscheduled frontier is empty (all ops scheduled) */
#define SS_ROUND_INFEASIBLE 3 /* no partition is feasible for the batch: nothing issued */

typedef struct ss_sched ss_sched;
typedef struct ss_sched_desc {
  const ss_gmg_desc *gmg;
  int64_t n_part;
  const uint8_t *part_dev;
  const int64_t *priority;
  int64_t issue_budget;
  int64_t batch_cap;
  int flags;
} ss_sched_desc;

/* Create a scheduler on the CURRENT HIP device; every op starts unscheduled.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_INVALID_GMG, SS_ERR_OOM, SS_ERR_DEVICE,
 * SS_ERR_UNSUPPORTED. */
int ss_sched_create(const ss_sched_desc *desc, ss_sched **out);

/* Release a scheduler (synchronises its device first).  NULL is a no-op. */
void ss_sched_free(ss_sched *s);

/*
 * One round of Alg. 1 at time `now` (>= the previous round's, < 2^62).
 * Returns at once (SS_ROUND_BUDGET, SS_ROUND_IDLE) when the issued ops reach
 * the budget or the unscheduled frontier is empty.  Otherwise: the
 * highest-priority op of the unscheduled frontier; its batch, collected by
 * repeatedly adding the lowest-index unscheduled successor of a batch op
 * whose predecessors are all issued, done or in the batch, up to batch_cap
 * ops; one candidate per partition, simulated together on the GPU
 * (ss_simulate_batch, index-order dispatch) over the snapshot (Sec. 3.3.2):
 * in the order they were issued (the device queues' order), the issued ops
 * that are not done and the done ops whose output still feeds an op to run,
 * then the batch in index order issued at `now`; done ops keep their
 * recorded completion, the others take their estimates and start no earlier
 * than their issue (see ss_gmg_desc), and memory is checked from `now` on;
 * the feasible candidate with the smallest sum of finish times (ties to the
 * lower partition) is written back and the batch marked issued at `now`.
 * out_ops (HOST, >= batch_cap entries) receives the batch in index order and
 * *out_n its size (also for SS_ROUND_INFEASIBLE, 0 otherwise); *out_part the
 * partition (-1 unless issued); *out_status an SS_ROUND_* value.  The call
 * runs its GPU work on hip_stream and synchronises it before returning.
 * Errors: SS_ERR_INVALID_ARG, SS_ERR_OOM, SS_ERR_DEVICE.
 */
int ss_sched_round(ss_sched *s, int64_t now, int *out_status, int64_t *out_ops, int64_t *out_n,
                   int64_t *out_part, void *hip_stream);

/* Executor feedback: issued op `op` completed at time t_done, which must be
 * later than its issue and than every predecessor's completion (each
 * predecessor reported first), and below 2^62.  It no longer counts against
 * the issue budget; its recorded completion enters the next snapshots while
 * an op to run still reads its output.  Errors: SS_ERR_INVALID_ARG. */
int ss_sched_complete(ss_sched *s, int64_t op, int64_t t_done);

/* Current state (SS_OP_*), device, issue time and completion time (-1 until
 * then) of every op, HOST arrays of n_ops entries; any may be NULL.  The
 * device of an unscheduled op is 0. */
int ss_sched_state(const ss_sched *s, uint8_t *state, uint8_t *place, int64_t *issue_t, int64_t *done_t);

/*
 * The library takes every device buffer (staged GMGs, scratch, scheduler and
 * state buffers) from one stream-ordered memory pool per device that keeps
 * freed memory for later calls: handing large buffers back to the driver and
 * allocating again soon after stalls for up to seconds.  A simulation call's
 * scratch is, in addition, kept as an idle block (at most four per device)
 * that a later call on any stream reuses after the block's last use, so that
 * calls whose sizes vary do not allocate each time.  An allocation that fails
 * for lack of memory first returns the idle blocks and the pool's unused
 * memory (after synchronising the calling stream) and is tried once more;
 * only then does the call fail with SS_ERR_OOM.  This call returns the idle
 * blocks and the pools' unused memory to the driver (synchronising each
 * device that has a pool first); buffers in use stay.  Errors: SS_ERR_DEVICE.
 */
int ss_release_cached_memory(void);

/* Message for the calling thread's most recent failed call ("" if none). */
const char *ss_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SS_H */
