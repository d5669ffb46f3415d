// C ABI entry points: argument checks, error reporting, dispatch to the
// kernel drivers.  The GMG loader lives in gmg_load.cpp.
#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include <climits>

#include "ss_internal.h"

struct SsTimingRec {
  int kernel;
  hipEvent_t start, stop;
};

namespace {
thread_local std::string g_last_error;
std::atomic<int> g_timing_on{0};
std::mutex g_timing_mu;
std::vector<SsTimingRec *> g_timing;

void drop_record(SsTimingRec *r) {
  (void)hipEventDestroy(r->start);
  (void)hipEventDestroy(r->stop);
  delete r;
}

int check_device(const ss_gmg *g) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return ss_set_error(SS_ERR_DEVICE, "hipGetDevice failed");
  if (cur != g->device)
    return ss_set_error(SS_ERR_INVALID_ARG, "the current HIP device is not the one the GMG was loaded on");
  return SS_OK;
}
}  // namespace

int ss_set_error(int code, const std::string &msg) {
  g_last_error = msg;
  return code;
}

void ss_clear_error() { g_last_error.clear(); }

extern "C" const char *ss_last_error(void) { return g_last_error.c_str(); }

namespace {
// Checks shared by the simulation entry points; fills the placement source
// and the dispatch flags.  SS_OK with B == 0 means there is nothing to do.
int check_simulate(const char *fn, const ss_gmg *g, const uint8_t *placements, int64_t B, int layout,
                   const int64_t *out_makespan, const uint8_t *out_violation, SsPlace *src, bool *ready,
                   bool *ports) {
  const std::string f(fn);
  if (!g) return ss_set_error(SS_ERR_INVALID_ARG, f + ": g is NULL");
  if (B < 0) return ss_set_error(SS_ERR_INVALID_ARG, f + ": B < 0");
  if ((layout & ~(SS_LAYOUT_OP_MAJOR | SS_DISPATCH_READY | SS_LINK_PORTS)) != 0)
    return ss_set_error(SS_ERR_INVALID_ARG, f + ": unknown layout");
  if ((layout & SS_LINK_PORTS) && (layout & SS_DISPATCH_READY))
    return ss_set_error(SS_ERR_UNSUPPORTED, f + ": SS_LINK_PORTS takes index-order dispatch only");
  src->p = placements;
  src->B = B;
  src->op_major = (layout & SS_LAYOUT_OP_MAJOR) != 0;
  *ready = (layout & SS_DISPATCH_READY) != 0;
  *ports = (layout & SS_LINK_PORTS) != 0;
  if (B == 0) return SS_OK;
  if (!out_makespan || !out_violation)
    return ss_set_error(SS_ERR_INVALID_ARG, f + ": out_makespan and out_violation are required");
  if (!placements && g->n_ops > 0) return ss_set_error(SS_ERR_INVALID_ARG, f + ": placements is NULL");
  return check_device(g);
}
}  // namespace

extern "C" int ss_simulate_batch(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout,
                                 int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                                 int64_t *out_sla_slack, int64_t *out_sumfin, void *hip_stream) {
  ss_clear_error();
  SsPlace src;
  bool ready = false, ports = false;
  const int rc = check_simulate("ss_simulate_batch", g, placements, B, layout, out_makespan, out_violation, &src,
                                &ready, &ports);
  if (rc != SS_OK || B == 0) return rc;
  SsWork W;
  return ss_run_simulate(g, src, out_makespan, out_peak_mem, out_violation, out_sla_slack, out_sumfin,
                         static_cast<hipStream_t>(hip_stream), ready, ports, W);
}

extern "C" int ss_simulate_workspace_size(const ss_gmg *g, int64_t B, int layout, int64_t *min_bytes,
                                          int64_t *pref_bytes) {
  ss_clear_error();
  if (min_bytes) *min_bytes = 0;
  if (pref_bytes) *pref_bytes = 0;
  if (!min_bytes && !pref_bytes) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_workspace_size: no output");
  SsPlace src;
  bool ready = false, ports = false;
  int64_t dummy_ms = 0;
  uint8_t dummy_vi = 0;
  const uint8_t dummy_p = 0;
  const int rc = check_simulate("ss_simulate_workspace_size", g, &dummy_p, B, layout, &dummy_ms, &dummy_vi, &src,
                                &ready, &ports);
  if (rc != SS_OK || B == 0) return rc;
  SsWork W;
  W.query = true;
  W.single = true;
  const int r2 = ss_run_simulate(g, src, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, ready, ports, W);
  if (r2 != SS_OK) return r2;
  if (min_bytes) *min_bytes = (int64_t)W.need_min;
  if (pref_bytes) *pref_bytes = (int64_t)W.need_pref;
  return SS_OK;
}

extern "C" int ss_simulate_chunking(const ss_gmg *g, int64_t B, int layout, int64_t *chunk, int64_t *sub) {
  ss_clear_error();
  if (!chunk || !sub) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_chunking: a NULL output");
  *chunk = *sub = 0;
  SsPlace src;
  bool ready = false, ports = false;
  int64_t dummy_ms = 0;
  uint8_t dummy_vi = 0;
  const uint8_t dummy_p = 0;
  const int rc = check_simulate("ss_simulate_chunking", g, &dummy_p, B, layout, &dummy_ms, &dummy_vi, &src, &ready,
                                &ports);
  if (rc != SS_OK || B == 0) return rc;
  SsWork W;
  W.query = true;
  const int r2 = ss_run_simulate(g, src, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, ready, ports, W);
  if (r2 != SS_OK) return r2;
  *chunk = W.chunk;
  *sub = W.sub;
  return SS_OK;
}

extern "C" int ss_simulate_time_bits(const ss_gmg *g, int layout, int *bits) {
  ss_clear_error();
  if (!bits) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_time_bits: bits is NULL");
  *bits = 0;
  SsPlace src;
  bool ready = false, ports = false;
  const int rc = check_simulate("ss_simulate_time_bits", g, nullptr, 0, layout, nullptr, nullptr, &src, &ready, &ports);
  if (rc != SS_OK) return rc;
  const int rd = check_device(g);
  if (rd != SS_OK) return rd;
  return ss_simulate_time_bits_of(g, ready, ports, bits);
}

extern "C" int ss_simulate_batch_ws(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout,
                                    int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                                    int64_t *out_sla_slack, int64_t *out_sumfin, void *workspace,
                                    int64_t workspace_bytes, void *hip_stream) {
  ss_clear_error();
  SsPlace src;
  bool ready = false, ports = false;
  const int rc = check_simulate("ss_simulate_batch_ws", g, placements, B, layout, out_makespan, out_violation, &src,
                                &ready, &ports);
  if (rc != SS_OK || B == 0) return rc;
  if (!workspace || workspace_bytes <= 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_ws: workspace is NULL or empty");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_ws: workspace is not 256-byte aligned");
  SsWork W;
  W.ptr = workspace;
  W.bytes = (size_t)workspace_bytes;
  W.single = true;
  return ss_run_simulate(g, src, out_makespan, out_peak_mem, out_violation, out_sla_slack, out_sumfin,
                         static_cast<hipStream_t>(hip_stream), ready, ports, W);
}

extern "C" int ss_est_create(int64_t n_est, int64_t n_feat, ss_est **out) {
  ss_clear_error();
  if (!out) return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_create: out is NULL");
  *out = nullptr;
  if (n_est < 0 || n_feat < 1 || n_feat > SS_EST_MAX_FEAT)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_create: n_est < 0 or n_feat outside 1..8");
  if (n_est > INT32_MAX || n_est > (int64_t(1) << 40) / (n_feat * n_feat + n_feat + 1))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_create: n_est too large");
  return ss_run_est_create(n_est, n_feat, out);
}

extern "C" void ss_est_free(ss_est *e) {
  if (e) ss_run_est_free(e);
}

namespace {
int check_est_device(const ss_est *e) {
  int dev = 0, cur = 0;
  ss_run_est_info(e, nullptr, nullptr, &dev);
  if (hipGetDevice(&cur) != hipSuccess) return ss_set_error(SS_ERR_DEVICE, "hipGetDevice failed");
  if (cur != dev) return ss_set_error(SS_ERR_INVALID_ARG, "the current HIP device is not the estimator set's");
  return SS_OK;
}
}  // namespace

extern "C" int ss_est_add(ss_est *e, const int64_t *sample_ptr, int64_t n_samples, const double *x, const double *y,
                          void *hip_stream) {
  ss_clear_error();
  if (!e) return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_add: e is NULL");
  int64_t n_est = 0;
  ss_run_est_info(e, &n_est, nullptr, nullptr);
  if (n_samples < 0 || !sample_ptr || (n_samples > 0 && (!x || !y)))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_add: n_samples < 0 or a NULL array");
  const int rc = check_est_device(e);
  if (rc != SS_OK) return rc;
  return ss_run_est_add(e, sample_ptr, n_samples, x, y, static_cast<hipStream_t>(hip_stream));
}

extern "C" int ss_est_solve(const ss_est *e, double *coef, int32_t *status, void *hip_stream) {
  ss_clear_error();
  if (!e || !coef || !status) return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_solve: a NULL argument");
  const int rc = check_est_device(e);
  if (rc != SS_OK) return rc;
  return ss_run_est_solve(e, coef, status, static_cast<hipStream_t>(hip_stream));
}

extern "C" int ss_est_predict(const double *coef, int64_t n_est, int64_t n_feat, const int32_t *est_of,
                              const double *x, int64_t M, int64_t *out_us, void *hip_stream) {
  ss_clear_error();
  if (n_est < 0 || n_feat < 1 || n_feat > SS_EST_MAX_FEAT || M < 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_predict: bad n_est, n_feat or M");
  if (M > 0 && (!coef || !est_of || !x || !out_us))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_est_predict: a NULL array");
  return ss_run_est_predict(coef, n_est, n_feat, est_of, x, M, out_us, static_cast<hipStream_t>(hip_stream));
}

extern "C" int ss_select_best(const ss_gmg *g, const uint8_t *violation, const int64_t *key,
                              const int64_t *sla_slack, int64_t B, int flags, int64_t *out_best, void *hip_stream) {
  ss_clear_error();
  if (!g || !out_best) return ss_set_error(SS_ERR_INVALID_ARG, "ss_select_best: g and out_best are required");
  if (B < 0 || (flags & ~SS_SELECT_REQUIRE_SLA))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_select_best: B < 0 or unknown flag");
  const int require_sla = (flags & SS_SELECT_REQUIRE_SLA) && g->n_req > 0;
  if (B > 0 && (!violation || !key || (require_sla && !sla_slack)))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_select_best: violation, key (and slack with REQUIRE_SLA) required");
  const int rc = check_device(g);
  if (rc != SS_OK) return rc;
  return ss_run_select(g, violation, key, sla_slack, B, require_sla, out_best, static_cast<hipStream_t>(hip_stream));
}

SsTimingRec *ss_timing_start(int kernel, hipStream_t stream) {
  if (!g_timing_on.load()) return nullptr;
  auto *r = new SsTimingRec{kernel, nullptr, nullptr};
  if (hipEventCreate(&r->start) != hipSuccess || hipEventCreate(&r->stop) != hipSuccess ||
      hipEventRecord(r->start, stream) != hipSuccess) {
    drop_record(r);
    return nullptr;
  }
  return r;
}

void ss_timing_stop(SsTimingRec *r, hipStream_t stream) {
  if (!r) return;
  if (hipEventRecord(r->stop, stream) != hipSuccess) {
    drop_record(r);
    return;
  }
  std::lock_guard<std::mutex> lk(g_timing_mu);
  g_timing.push_back(r);
}

extern "C" int ss_kernel_timing(int enable) {
  ss_clear_error();
  g_timing_on.store(enable ? 1 : 0);
  if (!enable) {
    std::lock_guard<std::mutex> lk(g_timing_mu);
    for (auto *r : g_timing) drop_record(r);
    g_timing.clear();
  }
  return SS_OK;
}

extern "C" int ss_kernel_time(int kernel, int64_t *launches, double *total_ms) {
  ss_clear_error();
  if (!launches || !total_ms || kernel < SS_KERNEL_SCHEDULE || kernel > SS_KERNEL_ESTIMATOR)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_kernel_time: bad kernel id or NULL output");
  std::lock_guard<std::mutex> lk(g_timing_mu);
  int64_t n = 0;
  double ms = 0.0;
  int rc = SS_OK;
  std::vector<SsTimingRec *> keep;
  for (auto *r : g_timing) {
    if (r->kernel != kernel) {
      keep.push_back(r);
      continue;
    }
    float t = 0.f;
    if (hipEventSynchronize(r->stop) != hipSuccess || hipEventElapsedTime(&t, r->start, r->stop) != hipSuccess)
      rc = ss_set_error(SS_ERR_DEVICE, "ss_kernel_time: reading a timing event failed");
    ms += t;
    ++n;
    drop_record(r);
  }
  g_timing.swap(keep);
  *launches = n;
  *total_ms = ms;
  return rc;
}

extern "C" int ss_sched_create(const ss_sched_desc *d, ss_sched **out) {
  ss_clear_error();
  if (!out) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: out is NULL");
  *out = nullptr;
  if (!d || !d->gmg) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: desc or desc->gmg is NULL");
  if (d->n_part < 1 || d->n_part > INT32_MAX || !d->part_dev)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: n_part < 1 or part_dev is NULL");
  if (d->gmg->n_req > 0 && !d->priority) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: priority is NULL");
  if (d->issue_budget < 1 || d->batch_cap < 1)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: issue_budget and batch_cap must be >= 1");
  if (d->flags & ~(SS_SELECT_REQUIRE_SLA | SS_SCHED_PREFIX_REUSE))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: unknown flags");
  if (d->gmg->done_fin || d->gmg->issue_at || d->gmg->t_now != 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: the run's GMG holds no running state (the scheduler "
                                            "keeps it)");
  const int64_t N = d->gmg->n_ops, D = d->gmg->n_dev;
  if (N < 0 || D < 1) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: bad GMG sizes");
  if (d->n_part > (int64_t(1) << 40) / std::max<int64_t>(N, 1))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: n_part * n_ops too large");
  for (int64_t i = 0; i < d->n_part * N; ++i)
    if (d->part_dev[i] >= D) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_create: part_dev names a device >= n_dev");
  return ss_run_sched_create(d, out);
}

extern "C" void ss_sched_free(ss_sched *s) {
  if (s) ss_run_sched_free(s);
}

extern "C" int ss_sched_round(ss_sched *s, int64_t now, int *out_status, int64_t *out_ops, int64_t *out_n,
                              int64_t *out_part, void *hip_stream) {
  ss_clear_error();
  if (!s || !out_status || !out_ops || !out_n || !out_part)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_round: NULL argument");
  if (now < 0 || now >= ((int64_t)1 << 62)) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_round: now out of range");
  return ss_run_sched_round(s, now, out_status, out_ops, out_n, out_part, static_cast<hipStream_t>(hip_stream));
}

extern "C" int ss_sched_complete(ss_sched *s, int64_t op, int64_t t_done) {
  ss_clear_error();
  if (!s) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_complete: s is NULL");
  return ss_run_sched_complete(s, op, t_done);
}

extern "C" int ss_sched_state(const ss_sched *s, uint8_t *state, uint8_t *place, int64_t *issue_t, int64_t *done_t) {
  ss_clear_error();
  if (!s) return ss_set_error(SS_ERR_INVALID_ARG, "ss_sched_state: s is NULL");
  ss_run_sched_state(s, state, place, issue_t, done_t);
  return SS_OK;
}

extern "C" int ss_state_create(ss_state **out) {
  ss_clear_error();
  if (!out) return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_create: out is NULL");
  *out = nullptr;
  ss_state *st = new (std::nothrow) ss_state();
  if (!st) return ss_set_error(SS_ERR_OOM, "ss_state_create: host allocation failed");
  if (hipGetDevice(&st->device) != hipSuccess) {
    delete st;
    return ss_set_error(SS_ERR_DEVICE, "hipGetDevice failed");
  }
  *out = st;
  return SS_OK;
}

extern "C" void ss_state_free(ss_state *st) {
  if (!st) return;
  if (st->mem) {
    int prev = 0;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(st->device);
    (void)hipDeviceSynchronize();
    ss_pool_free(st->mem, nullptr);
    (void)hipDeviceSynchronize();
    (void)hipSetDevice(prev);
  }
  delete st;
}

extern "C" int ss_state_info(const ss_state *st, int64_t *n_ops) {
  ss_clear_error();
  if (!st) return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_info: st is NULL");
  if (n_ops) *n_ops = st->k;
  return SS_OK;
}

namespace {
bool state_fits(const ss_state *from, const ss_gmg *g) {
  return !from || from->k == 0 ||
         (from->k <= g->n_ops && from->d == g->n_dev && from->r == g->n_req && from->device == g->device);
}
}  // namespace

extern "C" int ss_simulate_batch_resume(const ss_gmg *g, const ss_state *from, const uint8_t *placements, int64_t B,
                                        int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                                        int64_t *out_sla_slack, int64_t *out_sumfin, void *hip_stream) {
  ss_clear_error();
  if (!g) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_resume: g is NULL");
  if (B < 0) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_resume: B < 0");
  if (!state_fits(from, g))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_resume: the state does not fit this GMG");
  if (B == 0) return SS_OK;
  if (!out_makespan || !out_violation)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_resume: out_makespan and out_violation are required");
  if (!placements && g->n_ops > 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_resume: placements is NULL");
  const int rc = check_device(g);
  if (rc != SS_OK) return rc;
  return ss_run_simulate_resume(g, from, placements, B, out_makespan, out_peak_mem, out_violation, out_sla_slack,
                                out_sumfin, static_cast<hipStream_t>(hip_stream));
}

extern "C" int ss_state_capture(const ss_gmg *g, const ss_state *from, const uint8_t *placement, ss_state *capture,
                                void *hip_stream) {
  ss_clear_error();
  if (!g || !capture) return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_capture: g or capture is NULL");
  if (!state_fits(from, g)) return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_capture: the state does not fit this GMG");
  if (capture == from || capture->device != g->device)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_capture: capture must be its own state on g's device");
  if (!placement && g->n_ops > 0) return ss_set_error(SS_ERR_INVALID_ARG, "ss_state_capture: placement is NULL");
  const int rc = check_device(g);
  if (rc != SS_OK) return rc;
  return ss_run_state_capture(g, from, placement, capture, static_cast<hipStream_t>(hip_stream));
}
