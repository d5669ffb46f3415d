// Internal declarations of the simulator library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "ss.h"

// Device-resident GMG, passed by value to every kernel.  Times and sizes are
// int64; indices int32 (the loader enforces N, E < 2^31).
struct GmgView {
  int32_t n_ops, n_dev, n_class, n_link, n_req;
  const int32_t *pred_ptr, *pred_idx;  // predecessor CSR
  const int32_t *succ_ptr, *succ_idx;  // successor CSR, ascending within an op
  const int32_t *succ_pe;              // [E] position of each successor entry's edge in the predecessor CSR
  const int32_t *op_req, *dev_class, *slice_ptr;
  const int64_t *dur;        // [N][n_class]
  const int64_t *out_bytes;  // [N]
  const int64_t *xfer;       // [N][n_link]: lat[k] + ceil(out_bytes[v] / bw[k])
  const int64_t *slice_begin, *slice_end;
  const int64_t *cap, *release, *deadline;
  const uint8_t *link_class;  // [D][D]
  // a running schedule's state (null / 0 without one): recorded finish of
  // done ops (-1: not done), issue times, the snapshot's timestamp
  const int64_t *done_fin, *issue_at;
  int64_t t_now;
  // 32-bit copies of every time quantity, present when the loader proved the
  // whole time horizon (all starts, finishes, frees and finite slice bounds)
  // stays below 2^32 - 1, there are at most 65535 ops, 65535 edges and 65535
  // slices per device, and every output size fits in 32 bits; the open slice end becomes 0xFFFFFFFF.  The 32-bit slice
  // arrays hold one spare entry past the last slice.
  int32_t time32;
  const uint32_t *dur32, *xfer32, *slice_begin32, *slice_end32, *release32;
  // Per-op fields of the 32-bit path, field-major [kOpMetaFields][meta_stride]
  // so a wave reads the fields of 64 consecutive ops with one coalesced load
  // per field (meta_stride = N rounded up to 64 plus one spare block, >= 128).
  const uint32_t *op_meta;
  int32_t meta_stride;
  // link classes as bits (two classes at most): bit b of word [a][b >> 5] is
  // link_class[a][b]; link_words = ceil(n_dev / 32).  Null with more classes.
  const uint32_t *link_bits;
  int32_t link_words;
  // when the link classes follow device groups (two classes at most: one for
  // every pair in the same group, the other across groups): group id per
  // device and the class of a same-group pair; null otherwise
  const uint8_t *link_grp;
  int32_t link_same;
  // with such groups: s when device a's group is a >> s (contiguous groups of
  // 2^s devices), else -1
  int32_t link_shift;
  const uint32_t *bytes32;  // out_bytes as u32
  // the peak pass's byte sums: sizes divided by 2^peak_shift (their common
  // power of two) sum below 2^32 over every output and one copy per consumer
  // edge (peak_narrow), so 32-bit sums are exact
  int32_t peak_shift, peak_narrow;
  // first two successors of each op as u16 (0xFFFF: none), when no op has more
  const uint32_t *succ2;
  // with succ2 and fewer than 65,535 edges: the predecessor-edge index of each
  // of those two successor entries, same packing
  const uint32_t *succ2_pe;
  // time -> slice lookup per device, for buckets of 2^lut_shift us: entry
  // [d][b] concerns the first slice k of d ending at or after b << lut_shift;
  // lut_w holds {begin, end} of slices k and k+1, lut_k the device-local k
  const uint32_t *lut_k;
  const uint4 *lut_w;
  int32_t lut_nb, lut_shift;
  // ready-time dispatch: the n_src ops without predecessors sorted by
  // (release of their request, index); src_keys holds them as release << 16 |
  // op on the 32-bit path
  const int32_t *src_ops;
  const uint64_t *src_keys;
  int32_t n_src;
};

// Fields of op_meta for op v.  Predecessors beyond the first four and link
// class counts above two are read from the CSR and xfer32 tables instead.
enum OpMetaField {
  kMetaDur = 0,   // dur32[v] when there is one device class, else 0
  kMetaReq = 1,   // request id | predecessor count << 16 (count saturates at 0xFFFF)
  kMetaRel = 2,   // release32 of the op's request
  kMetaP01 = 3,   // predecessors 0 and 1 as u16 (0xFFFF: none)
  kMetaP23 = 4,   // predecessors 2 and 3
  kMetaX = 5,     // 8 fields: transfer time of predecessor i over link class k at kMetaX + 2 i + k
  kMetaE0 = 13,   // pred_ptr[v]
  kOpMetaFields = 14
};

struct ss_gmg {
  int device = 0;
  int64_t n_ops = 0, n_edges = 0, n_dev = 0, n_class = 0, n_link = 0, n_req = 0;
  int64_t max_slices = 0;  // largest slice count of any device
  int64_t horizon = 0;     // loader's upper bound on every simulated time
  int64_t max_indeg = 0;   // largest predecessor count of any op
  int64_t max_outdeg = 0;  // largest successor count of any op
  bool snapshot = false;   // done_fin, issue_at or t_now given (general index-order path only)
  void *dev_mem = nullptr;
  // second stream of the memory passes (the peak evaluation of one sub-chunk
  // overlaps the interval pass of the next): the device's (ss_device_aux)
  hipStream_t aux = nullptr;
  // the device's scratch pool (ss_device_pool), also holding dev_mem
  hipMemPool_t pool = nullptr;
  GmgView view{};
};

// The process-wide stream-ordered pool of a device: every device buffer of
// the library comes from it, and freed memory stays in it (release threshold:
// never) until ss_release_cached_memory.  Handing large buffers back to the
// driver and allocating again soon after stalls for up to seconds.  Returns
// nullptr (with the error recorded) when the pool cannot be made.
hipMemPool_t ss_device_pool(int device);
// Requests to the pool are rounded up to the next size of the form
// 2^k x {1, 1.25, 1.5, 1.75}: calls whose scratch grows a little each time (the
// incremental loop's rounds, whose graph gains a batch per round) reuse the
// pool's blocks instead of taking new memory from the driver every call.
inline size_t ss_pool_round(size_t x) {
  if (x <= 4096) return 4096;
  int k = 63 - __builtin_clzll((unsigned long long)x);  // 2^k <= x < 2^(k+1)
  const size_t base = size_t(1) << k, q = base >> 2;
  return base + ((x - base + q - 1) / q) * q;
}
// A block from `pool` on `stream`, its size rounded by ss_pool_round.  On
// running out of memory the device's idle scratch blocks and the pool's unused
// memory are given back (once the stream's earlier work has completed) and the
// allocation is retried once.
hipError_t ss_pool_malloc(void **p, size_t bytes, hipMemPool_t pool, hipStream_t stream);

// Per-call scratch.  Repeated calls whose sizes vary (the rounds of the
// incremental loop grow their graph op by op) would otherwise allocate from
// the pool at almost every call, and the runtime's pool stalls for up to
// seconds on such churn.  ss_scratch_get takes the smallest idle block of the
// device that holds `bytes` (the calling stream first waits for the block's
// last use), else a new block from the pool with a quarter of headroom;
// ss_scratch_put returns it as idle, marked by an event on `stream`, and
// frees the device's smallest idle block to the pool when more than four are
// idle.  Idle blocks stay until ss_release_cached_memory or an allocation
// that runs out of memory.
struct SsScratch {
  void *p = nullptr;
  size_t bytes = 0;
};
hipError_t ss_scratch_get(int device, hipMemPool_t pool, size_t bytes, hipStream_t stream, SsScratch *s);
// A scratch budget for one call: `cap`, or `eighths` eighths of the memory
// the call could get (the device's free memory, the pool's reserved but
// unused memory and the device's idle scratch blocks) when that is less.
// Taken at each call, so a budget cut by memory that others held grows back
// once they release it.
int64_t ss_scratch_budget(int device, hipMemPool_t pool, int64_t cap, int eighths = 6);
hipError_t ss_scratch_put(int device, SsScratch *s, hipStream_t stream);
// A buffer from the device's pool, ready for use on any stream when it returns
// (allocated on `stream`, which is synchronised), and its release.
int ss_pool_alloc(int device, size_t bytes, hipStream_t stream, void **out);
void ss_pool_free(void *p, hipStream_t stream);
// The process-wide second stream of a device (default priority, non-blocking),
// made once: creating and destroying streams as objects come and go remaps the
// few hardware queues and stalled host calls for up to a second.  nullptr
// (with the error recorded) when it cannot be made.
hipStream_t ss_device_aux(int device);

// A captured simulation state (ss_simulate_batch_resume): one candidate after
// its first k ops of a GMG with d devices and r requests.  One device
// allocation: fin[cap_n] | clk[cap_d] | comp[cap_r] | scal[2] | cur[cap_d].
struct ss_state {
  int device = 0;
  int64_t k = 0, d = 0, r = 0;
  int64_t cap_n = 0, cap_d = 0, cap_r = 0;
  void *mem = nullptr;
  int64_t *fin = nullptr, *clk = nullptr, *comp = nullptr, *scal = nullptr;
  int32_t *cur = nullptr;
};

// Record an error message for ss_last_error() and return the code.
int ss_set_error(int code, const std::string &msg);
void ss_clear_error();

// Optional per-kernel event timing (abi.cpp): returns a started record or
// nullptr when timing is off; ss_timing_stop closes it on the same stream.
struct SsTimingRec;
SsTimingRec *ss_timing_start(int kernel, hipStream_t stream);
void ss_timing_stop(SsTimingRec *rec, hipStream_t stream);

// Incremental scheduling loop (sched.cpp).  Arguments are already checked.
int ss_run_sched_create(const ss_sched_desc *d, ss_sched **out);
void ss_run_sched_free(ss_sched *s);
int ss_run_sched_round(ss_sched *s, int64_t now, int *status, int64_t *ops, int64_t *n_ops, int64_t *part,
                       hipStream_t stream);
int ss_run_sched_complete(ss_sched *s, int64_t op, int64_t t_done);
void ss_run_sched_state(const ss_sched *s, uint8_t *state, uint8_t *place, int64_t *issue_t, int64_t *done_t);

// Where a simulation call takes its scratch (device memory beyond its inputs
// and outputs) from: the device's pool (ptr null), or a caller's workspace of
// `bytes`, which the call then splits into chunks that fit and never
// allocates beyond.  single: every kernel on the caller's stream (no second
// stream, no events; one set of interval records).  query: the call only
// reports need_min (the smallest workspace that works) and need_pref (what
// the pool path takes for this batch) and launches nothing.
struct SsWork {
  void *ptr = nullptr;
  size_t bytes = 0;
  bool single = false;
  bool query = false;
  size_t need_min = 0, need_pref = 0;
  int64_t chunk = 0, sub = 0;  // query: candidates per chunk and per memory-pass sub-chunk of the pool path
};
// Placements of a call: row-major [B][n_ops], or op-major [n_ops][B].
struct SsPlace {
  const uint8_t *p = nullptr;
  int64_t B = 0;
  bool op_major = false;
};

// Kernel drivers (simulate.hip / select.hip).  Arguments are already checked.
// The width of the integers (32 or 64) the simulation of a call with these
// flags computes its times in.
int ss_simulate_time_bits_of(const ss_gmg *g, bool ready_dispatch, bool link_ports, int *bits);
int ss_run_simulate(const ss_gmg *g, SsPlace P, int64_t *makespan, int64_t *peak, uint8_t *violation,
                    int64_t *slack, int64_t *sumfin, hipStream_t stream, bool ready_dispatch, bool link_ports,
                    SsWork &W);
// Resumption from a captured state (general schedule kernel; the 32-bit
// memory passes when the GMG has a 32-bit horizon); from may be null or empty.
int ss_run_simulate_resume(const ss_gmg *g, const ss_state *from, const uint8_t *placements, int64_t B,
                           int64_t *makespan, int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin,
                           hipStream_t stream);
// The schedule of one candidate (resumed from `from`), its state stored in capture.
int ss_run_state_capture(const ss_gmg *g, const ss_state *from, const uint8_t *placement, ss_state *capture,
                         hipStream_t stream);
// Memory passes of the 32-bit path over int64 finish rows (sim_fast.hip).  With
// arr64 (transfers over device ports) the arrivals per predecessor edge,
// [edge][arr_stride] int64 from the first candidate of P: copies start at
// their transfer's start and own outputs are kept until their last arrival.
int ss_run_memory_fast(const ss_gmg *g, const uint8_t *P, const int64_t *fin64, int64_t B, int64_t *peak,
                       uint8_t *violation, hipStream_t stream, const int64_t *arr64 = nullptr,
                       int64_t arr_stride = 0);
// Fast path (sim_fast.hip): 32-bit times, N <= 65535.
size_t ss_fast_schedule_lds(const ss_gmg *g);
int ss_run_simulate_fast(const ss_gmg *g, SsPlace P, int64_t *makespan, int64_t *peak, uint8_t *violation,
                         int64_t *slack, int64_t *sumfin, hipStream_t stream, SsWork &W);
// Ready-time dispatch on the fast path (sim_fast.hip).
size_t ss_ready_schedule_lds(const ss_gmg *g);
int ss_run_simulate_ready(const ss_gmg *g, SsPlace P, int64_t *makespan, int64_t *peak, uint8_t *violation,
                          int64_t *slack, int64_t *sumfin, hipStream_t stream, SsWork &W);
// Candidate rows [nb][n_ops] of candidates [b0, b0 + nb) from op-major
// placements [n_ops][B] (sim_fast.hip).
hipError_t ss_rows_from_op_major(const uint8_t *P, int64_t n_ops, int64_t B, int64_t b0, int64_t nb, uint8_t *rows,
                                 hipStream_t stream);
// Estimators (estimator.hip).  Arguments are already checked.
int ss_run_est_create(int64_t n_est, int64_t n_feat, ss_est **out);
void ss_run_est_free(ss_est *e);
int ss_run_est_info(const ss_est *e, int64_t *n_est, int64_t *n_feat, int *device);
int ss_run_est_add(const ss_est *e, const int64_t *ptr, int64_t n_samples, const double *x, const double *y,
                   hipStream_t stream);
int ss_run_est_solve(const ss_est *e, double *coef, int32_t *status, hipStream_t stream);
int ss_run_est_predict(const double *coef, int64_t n_est, int64_t n_feat, const int32_t *est_of, const double *x,
                       int64_t M, int64_t *out, hipStream_t stream);
int ss_run_select(const ss_gmg *g, const uint8_t *violation, const int64_t *key, const int64_t *slack, int64_t B,
                  int require_sla, int64_t *out_best, hipStream_t stream);
