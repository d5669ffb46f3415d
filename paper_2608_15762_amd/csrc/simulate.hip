// Batched what-if simulation kernels for gfx950 (one HIP source, no other targets).
//
// schedule_kernel: one lane per candidate.  The lane walks the ops in index
//   order (the dispatch priority of every device queue) and computes each op's
//   ready time, its earliest fit into an idle slice of its device after the
//   device's previous finish, and its finish time (Sec. 3.3.2-3.3.3).  The
//   per-candidate device clocks and slice cursors live in LDS laid out
//   [device][lane], so the 64 lanes of a wave hit 64 distinct banks whatever
//   device each one touches.  Op-indexed GMG data is the same for every lane
//   (all lanes are at the same op), so it is read with wave-uniform loads.
//   Finish times go to a per-chunk scratch row for the memory pass.  With a
//   running schedule's state in the GMG (Sec. 3.2, 3.3.2) a done op keeps its
//   recorded finish and frees its device from then on, an op waits for its
//   issue time, and a transfer for the first issue among its destination's
//   consumers (xfer_floor).
//
// port_event_schedule: transfer arbitration (SS_LINK_PORTS, Sec. 3.5.2)
//   event by event, one wave per candidate (see below).
//
// ready_schedule_general: the ready-time dispatch rule, one wave per
//   candidate (the ready set is searched by the whole wave at every step).
//
// memory_kernel: one wave per candidate.  It groups the candidate's ops by
//   device, then for each device builds the endpoints of the residency
//   intervals resident there (own outputs and remote copies, Sec. 3.3.2),
//   sorts them in LDS by (time, free-before-allocate) with a bitonic network
//   and takes the maximum prefix sum of the byte deltas: the device's peak.
//   A device with more endpoints than fit in LDS uses the same code on a
//   per-workgroup global buffer.
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cstring>

#include "ss_internal.h"

namespace {

constexpr int kWave = 64;
constexpr int kMemCap = 2048;                     // endpoints of one device sorted in LDS
constexpr int64_t kFinBudget = int64_t(16) << 30; // bytes of finish-time scratch per chunk
constexpr int kMemBlocksPerCU = 4;

__device__ __forceinline__ int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }

// Running schedule (GMG issue times given): the transfer of u's output to
// device e starts no earlier than the first issue time among u's consumers
// placed on e, the moment its Intent exists.  0 when none is there.
__device__ int64_t xfer_floor(const GmgView &G, const uint8_t *prow, int u, int e) {
  int64_t f = INT64_MAX;
  const int q1 = G.succ_ptr[u + 1];
  for (int q = G.succ_ptr[u]; q < q1; ++q) {
    const int x = G.succ_idx[q];
    if (prow[x] == e && G.issue_at[x] < f) f = G.issue_at[x];
  }
  return f == INT64_MAX ? 0 : f;
}

// ------------------------------------------------------------------ schedule
// Resumption from a captured state (ss_simulate_batch_resume): every
// candidate places its first k0 ops as the captured run did, so a lane starts
// at op k0 with the captured device clocks, slice cursors, request
// completions, makespan and finish-time sum; the finish times of ops < k0 are
// already in its row (fill_prefix).  With cap_* set (one candidate) the lane
// stores its state after its last op.
struct Resume {
  int32_t k0 = 0;
  const int64_t *clk = nullptr, *comp = nullptr, *scal = nullptr;  // [D], [R], {makespan, sum}
  const int32_t *cur = nullptr;                                    // [D]
  const uint32_t *bad = nullptr;  // [nb]: nonzero when the candidate's first k0 ops name a device >= D
  int64_t *cap_clk = nullptr, *cap_scal = nullptr;
  int32_t *cap_cur = nullptr;
};

__global__ __launch_bounds__(256) void zero_u32(uint32_t *__restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0;
}

// Flags the candidates whose first k0 placements name a device >= D (rows
// read with consecutive threads on consecutive bytes).
__global__ __launch_bounds__(256) void prefix_check(const uint8_t *__restrict__ P, int64_t nb, int64_t N, int64_t k0,
                                                    int D, uint32_t *__restrict__ bad) {
  const int64_t total = nb * k0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t c = i / k0, v = i - c * k0;
    if (P[c * N + v] >= D) atomicOr(&bad[c], 1u);
  }
}

// Copies the captured finish times of ops [0, k0) into every candidate's row.
__global__ __launch_bounds__(256) void fill_prefix(int64_t *__restrict__ fin, int64_t nb, int64_t N, int64_t k0,
                                                   const int64_t *__restrict__ pre) {
  const int64_t total = nb * k0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t c = i / k0, v = i - c * k0;
    fin[c * N + v] = pre[v];
  }
}

__global__ __launch_bounds__(kWave) void schedule_kernel(const GmgView G, const uint8_t *__restrict__ P,
                                                         int64_t nb, int64_t *__restrict__ fin,
                                                         int64_t *__restrict__ comp, const Resume RS,
                                                         int64_t *__restrict__ makespan,
                                                         int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
                                                         uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class, K = G.n_link;
  const int lane = threadIdx.x;
  int64_t *clk = reinterpret_cast<int64_t *>(lds_raw);                        // [D][64]
  uint16_t *cur = reinterpret_cast<uint16_t *>(lds_raw + (size_t)D * kWave * 8);  // [D][64]
  const int64_t c = (int64_t)blockIdx.x * kWave + lane;
  if (c >= nb) return;
  const uint8_t *prow = P + c * N;
  int64_t *frow = fin + c * N;
  const bool from = RS.clk != nullptr;
  for (int d = 0; d < D; ++d) {
    clk[d * kWave + lane] = from ? RS.clk[d] : 0;
    cur[d * kWave + lane] = from ? (uint16_t)RS.cur[d] : 0;
  }
  for (int r = 0; r < R; ++r) comp[(int64_t)r * nb + c] = from ? RS.comp[r] : G.release[r];

  bool invalid = false;
  int64_t ms = from ? RS.scal[0] : 0, sum = from ? RS.scal[1] : 0;
  if (RS.bad) invalid = RS.bad[c] != 0;  // the prefix is not walked, but must name devices
  for (int v = RS.k0; v < N; ++v) {
    int d = prow[v];
    if (d >= D) {  // not a device of the set: finish the walk on device 0, report sentinels
      invalid = true;
      d = 0;
    }
    const int r = G.op_req[v];
    const int slot = d * kWave + lane;
    const int64_t done = G.done_fin ? G.done_fin[v] : -1;
    int64_t f;
    if (done >= 0) {
      // done (running schedule): it finished at its recorded time; the
      // device is free from then on
      f = done;
      clk[slot] = imax(clk[slot], f);
    } else {
      const int64_t w = G.dur[(int64_t)v * C + G.dev_class[d]];
      // ready: release (and issue time), and every predecessor's finish plus
      // its transfer (started no earlier than the transfer's Intent)
      int64_t ready = G.release[r];
      if (G.issue_at) ready = imax(ready, G.issue_at[v]);
      const int e1 = G.pred_ptr[v + 1];
      for (int e = G.pred_ptr[v]; e < e1; ++e) {
        const int u = G.pred_idx[e];
        int64_t t = frow[u];
        int du = prow[u];
        if (du >= D) du = 0;
        if (du != d) {
          if (G.issue_at) t = imax(t, xfer_floor(G, prow, u, d));
          t += G.xfer[(int64_t)u * K + G.link_class[du * D + d]];
        }
        ready = imax(ready, t);
      }
      // one op at a time: not before the device's previous finish; then the
      // first idle slice that holds [s, s + w) (the cursor only moves forward)
      const int64_t t = imax(ready, clk[slot]);
      const int sbase = G.slice_ptr[d];
      int k = cur[slot];
      int64_t s;
      for (;;) {
        const int64_t a = G.slice_begin[sbase + k], e = G.slice_end[sbase + k];
        s = imax(t, a);
        if (s + w <= e) break;
        ++k;
      }
      cur[slot] = (uint16_t)k;
      f = s + w;
      clk[slot] = f;
    }
    frow[v] = f;
    ms = imax(ms, f);
    sum += f;
    int64_t *cr = comp + (int64_t)r * nb + c;
    *cr = imax(*cr, f);
  }
  if (RS.cap_clk) {  // one candidate: its state after its last op
    for (int d = 0; d < D; ++d) {
      RS.cap_clk[d] = clk[d * kWave + lane];
      RS.cap_cur[d] = cur[d * kWave + lane];
    }
    RS.cap_scal[0] = ms;
    RS.cap_scal[1] = sum;
  }
  if (invalid) {
    makespan[c] = INT64_MAX;
    if (sumfin) sumfin[c] = INT64_MAX;
    if (slack)
      for (int r = 0; r < R; ++r) slack[c * R + r] = INT64_MIN;
    violation[c] = SS_VIOLATION_INVALID;
  } else {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = sum;
    if (slack)
      for (int r = 0; r < R; ++r) slack[c * R + r] = G.deadline[r] - comp[(int64_t)r * nb + c];
    violation[c] = 0;
  }
}

// ------------------------------------------------------------------ ready-time dispatch
// The dispatch rule of Sec. 3.3.2 on the general path: among the ops whose
// predecessors have all been scheduled, the one with the earliest ready time
// (ties to the lower index) runs next, at the earliest fit on its device at or
// after max(ready time, the device's previous finish).  One wave per
// candidate.  Ready ops are (ready, op) pairs held kGenSlots per lane, and
// beyond that in the candidate's spill list (at most N entries: ready ops form
// an antichain), scanned while non-empty; sources come from the presorted
// src_ops list.  A device's clock never decreases, so its slice cursor (LDS)
// only moves forward.  The wave writes finish times (candidate rows, as
// schedule_kernel does) and the per-candidate outputs; request completions
// live in comp rows [candidate][R].
constexpr int kGenSlots = 4;

__device__ __forceinline__ bool pair_less(int64_t r1, int o1, int64_t r2, int o2) {
  return r1 < r2 || (r1 == r2 && o1 < o2);
}

__device__ __forceinline__ void wave_min_pair(int64_t &r, int &o) {
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    const int64_t r2 = __shfl_xor(r, off, kWave);
    const int o2 = __shfl_xor(o, off, kWave);
    if (pair_less(r2, o2, r, o)) {
      r = r2;
      o = o2;
    }
  }
}

__global__ __launch_bounds__(kWave) void ready_schedule_general(
    const GmgView G, const uint8_t *__restrict__ P, int64_t *__restrict__ fin, int32_t *__restrict__ missing,
    int64_t *__restrict__ spill_r, int32_t *__restrict__ spill_o, int64_t *__restrict__ comp,
    int64_t *__restrict__ makespan, int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
    uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class, K = G.n_link;
  const int lane = threadIdx.x;
  int64_t *clk = reinterpret_cast<int64_t *>(lds_raw);                     // [D]
  int32_t *cur = reinterpret_cast<int32_t *>(lds_raw + (size_t)D * 8);   // [D] slice cursor
  const int64_t c = blockIdx.x;
  const uint8_t *prow = P + c * N;
  int64_t *frow = fin + c * N;
  int32_t *mrow = missing + c * N;
  int64_t *srr = spill_r + c * N;
  int32_t *sro = spill_o + c * N;
  int64_t *crow = comp + c * R;
  bool bad = false;
  for (int v = lane; v < N; v += kWave) bad |= prow[v] >= (uint8_t)D;
  if (__any(bad)) {
    if (lane == 0) {
      makespan[c] = INT64_MAX;
      if (sumfin) sumfin[c] = INT64_MAX;
      violation[c] = SS_VIOLATION_INVALID;
    }
    if (slack)
      for (int r = lane; r < R; r += kWave) slack[c * R + r] = INT64_MIN;
    return;
  }
  for (int d = lane; d < D; d += kWave) {
    clk[d] = 0;
    cur[d] = 0;
  }
  for (int r = lane; r < R; r += kWave) crow[r] = G.release[r];
  for (int v = lane; v < N; v += kWave) mrow[v] = G.pred_ptr[v + 1] - G.pred_ptr[v];
  __syncthreads();  // LDS state and this wave's rows before the loop reads them

  constexpr int64_t kNoR = INT64_MAX;
  constexpr int kNoO = INT32_MAX;
  int64_t sr[kGenSlots];
  int so[kGenSlots];
#pragma unroll
  for (int k = 0; k < kGenSlots; ++k) {
    sr[k] = kNoR;
    so[k] = kNoO;
  }
  int sp = 0, ns = 0;  // next source, spill length (wave-uniform)
  int64_t ms = 0, sum = 0;
  for (int step = 0; step < N; ++step) {
    int64_t mr = sr[0];
    int mo = so[0];
#pragma unroll
    for (int k = 1; k < kGenSlots; ++k)
      if (pair_less(sr[k], so[k], mr, mo)) {
        mr = sr[k];
        mo = so[k];
      }
    int64_t wr = mr;
    int wo = mo;
    wave_min_pair(wr, wo);
    int64_t xr = kNoR;
    int xo = kNoO, xi = 0;
    if (ns > 0) {  // smallest spilled pair and its position
      int li = 0;
      for (int i = lane; i < ns; i += kWave) {
        const int64_t r = srr[i];
        const int o = sro[i];
        if (pair_less(r, o, xr, xo)) {
          xr = r;
          xo = o;
          li = i;
        }
      }
      const int64_t lr = xr;
      const int lo = xo;
      wave_min_pair(xr, xo);
      xi = __shfl(li, __ffsll((unsigned long long)__ballot(lr == xr && lo == xo)) - 1, kWave);
    }
    int64_t qr = kNoR;
    int qo = kNoO;
    if (sp < G.n_src) {
      qo = G.src_ops[sp];
      qr = G.release[G.op_req[qo]];
    }
    int v;
    int64_t ready;
    if (pair_less(qr, qo, wr, wo) && pair_less(qr, qo, xr, xo)) {
      v = qo;
      ready = qr;
      ++sp;
    } else if (pair_less(xr, xo, wr, wo)) {
      v = xo;
      ready = xr;
      --ns;
      if (lane == 0) {  // the last entry fills the hole
        srr[xi] = srr[ns];
        sro[xi] = sro[ns];
      }
    } else {
      v = wo;
      ready = wr;
      const int owner = __ffsll((unsigned long long)__ballot(mr == wr && mo == wo)) - 1;
      if (lane == owner) {
        bool done = false;
#pragma unroll
        for (int k = 0; k < kGenSlots; ++k)
          if (!done && so[k] == wo) {
            sr[k] = kNoR;
            so[k] = kNoO;
            done = true;
          }
      }
    }
    const int d = prow[v];
    const int64_t w = G.dur[(int64_t)v * C + G.dev_class[d]];
    const int64_t t = imax(ready, clk[d]);
    const int sbase = G.slice_ptr[d];
    int k = cur[d];
    int64_t s;
    for (;;) {
      const int64_t a = G.slice_begin[sbase + k], e = G.slice_end[sbase + k];
      s = imax(t, a);
      if (s + w <= e) break;
      ++k;
    }
    const int64_t f = s + w;
    const int r = G.op_req[v];
    const int64_t cr = crow[r];
    __syncthreads();  // every lane has read the LDS state and the rows
    if (lane == 0) {
      cur[d] = k;
      clk[d] = f;
      frow[v] = f;
      crow[r] = imax(cr, f);
    }
    __syncthreads();
    ms = imax(ms, f);
    sum += f;
    // successors whose last missing predecessor this was become ready
    const int q1 = G.succ_ptr[v + 1];
    for (int q = G.succ_ptr[v]; q < q1; ++q) {
      const int x = G.succ_idx[q];
      const int left = mrow[x] - 1;
      __syncthreads();
      if (lane == 0) mrow[x] = left;
      __syncthreads();
      if (left == 0) {
        const int dx = prow[x];
        int64_t rx = G.release[G.op_req[x]];
        const int e1 = G.pred_ptr[x + 1];
        for (int e = G.pred_ptr[x]; e < e1; ++e) {
          const int u = G.pred_idx[e];
          const int du = prow[u];
          int64_t tu = u == v ? f : frow[u];
          if (du != dx) tu += G.xfer[(int64_t)u * K + G.link_class[du * D + dx]];
          rx = imax(rx, tu);
        }
        bool placed = false;
#pragma unroll
        for (int kk = 0; kk < kGenSlots; ++kk) {
          if (!placed) {
            const unsigned long long free_lanes = __ballot(so[kk] == kNoO);
            if (free_lanes) {
              if (lane == __ffsll(free_lanes) - 1) {
                sr[kk] = rx;
                so[kk] = x;
              }
              placed = true;
            }
          }
        }
        if (!placed) {
          if (lane == 0) {
            srr[ns] = rx;
            sro[ns] = x;
          }
          ++ns;
          __syncthreads();
        }
      }
    }
  }
  if (lane == 0) {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = sum;
    violation[c] = 0;
  }
  __syncthreads();
  if (slack)
    for (int r = lane; r < R; r += kWave) slack[c * R + r] = G.deadline[r] - crow[r];
}

// ------------------------------------------------------------------ transfer ports, event by event
// The arbitration of Sec. 3.5.2 inside an event-driven simulation (one wave
// per candidate):
//   - compute queues are those of contract A: a device runs its ops in index
//     order, one at a time, each at the earliest fit at or after
//     max(ready, the device's previous finish);
//   - the output of u is moved once to every other device that holds a
//     consumer of u; its transfer becomes pending when u finishes;
//   - at every instant where an op finishes or a transfer arrives, the
//     pending transfers are examined in order of request time, producer index
//     and destination device, and each one whose source's send port and
//     destination's receive port are both idle starts then and holds both
//     until it arrives (a zero estimate moves nothing and completes at once);
//   - an op is placed as soon as every input's availability is known and
//     the op ahead of it on its device is placed (its start depends on
//     nothing else, and it never lies before the current instant).
// Per device in LDS: its queue (a range of the candidate's op list, ops of
// the device in index order), the queue head and the first placed op not yet
// finished (ops of a device finish in queue order), the clock and slice
// cursor, both port clocks, the arrival of the transfer now entering it, and
// the earliest unprocessed finish.  The next instant is a wave minimum over
// the devices.  Pending transfers (producer << 8 | destination) are a list
// in global scratch kept in examination order: appended at each instant in
// producer then destination order, scanned 64 at a time, compacted.
// Arrivals go to arr ([predecessor edge][candidate], every edge from u into
// the destination), which the memory pass reads: copies allocated at their
// transfer's start, own outputs kept until their last arrival.
constexpr int64_t kNever = INT64_MAX;

struct PortLds {
  int32_t *qbeg, *head, *done, *cur;
  int64_t *clk, *send_until, *recv_until, *arr_evt, *next_fin, *comp;
  uint8_t *dirty, *seen;
};

size_t port_schedule_lds(int D, int R) {
  return (size_t)(D + 1) * 4 + (size_t)D * 3 * 4 + (size_t)D * 5 * 8 + (size_t)R * 8 + (size_t)D * 2 + 64;
}

__device__ __forceinline__ PortLds port_lds(unsigned char *raw, int D, int R) {
  PortLds L;
  int64_t *p64 = reinterpret_cast<int64_t *>(raw);
  L.clk = p64;
  L.send_until = p64 + D;
  L.recv_until = p64 + 2 * D;
  L.arr_evt = p64 + 3 * D;
  L.next_fin = p64 + 4 * D;
  L.comp = p64 + 5 * D;
  int32_t *p32 = reinterpret_cast<int32_t *>(L.comp + R);
  L.qbeg = p32;
  L.head = p32 + D + 1;
  L.done = p32 + 2 * D + 1;
  L.cur = p32 + 3 * D + 1;
  L.dirty = reinterpret_cast<uint8_t *>(p32 + 4 * D + 1);
  L.seen = L.dirty + D;
  return L;
}

// Sets the arrival of u's transfer to device e on every edge from u into e.
__device__ __forceinline__ void port_set_arrivals(const GmgView &G, const uint8_t *prow, int u, int e, int64_t a,
                                                  int64_t *arr, int64_t nb, int64_t c, int q_begin, int q_step) {
  const int q1 = G.succ_ptr[u + 1];
  for (int q = G.succ_ptr[u] + q_begin; q < q1; q += q_step)
    if (prow[G.succ_idx[q]] == e) arr[(int64_t)G.succ_pe[q] * nb + c] = a;
}

__global__ __launch_bounds__(kWave) void port_event_schedule(const GmgView G, const uint8_t *__restrict__ P,
                                                             int64_t nb, int64_t *__restrict__ fin,
                                                             int64_t *__restrict__ arr, int32_t *__restrict__ lists,
                                                             int64_t *__restrict__ pend_all, int64_t pend_cap,
                                                             int64_t *__restrict__ makespan,
                                                             int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
                                                             uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class, K = G.n_link;
  const int E = G.pred_ptr[N];
  const int lane = threadIdx.x;
  const int64_t c = blockIdx.x;
  const uint8_t *prow = P + c * N;
  int64_t *frow = fin + c * N;
  int32_t *list = lists + c * N;
  int64_t *pend = pend_all + c * pend_cap;
  PortLds L = port_lds(lds_raw, D, R);

  // a candidate naming a device outside the set is not simulated
  bool bad = false;
  for (int v = lane; v < N; v += kWave) bad = bad || prow[v] >= D;
  if (__ballot(bad)) {
    if (lane == 0) {
      makespan[c] = INT64_MAX;
      if (sumfin) sumfin[c] = INT64_MAX;
      violation[c] = SS_VIOLATION_INVALID;
    }
    if (slack)
      for (int r = lane; r < R; r += kWave) slack[c * R + r] = INT64_MIN;
    return;
  }
  // every device's queue: its ops in index order
  for (int d = lane; d < D; d += kWave) L.head[d] = 0;
  __syncthreads();
  for (int v = lane; v < N; v += kWave) atomicAdd(&L.head[prow[v]], 1);
  __syncthreads();
  if (lane == 0) {
    int s = 0;
    for (int d = 0; d < D; ++d) {
      const int n = L.head[d];
      L.qbeg[d] = s;
      L.done[d] = s;  // fill position while the lists are written
      s += n;
    }
    L.qbeg[D] = s;
  }
  __syncthreads();
  for (int v0 = 0; v0 < N; v0 += kWave) {
    const int v = v0 + lane;
    const int d = v < N ? prow[v] : -1;
    // lanes of this chunk on the same device, lower lanes first
    uint64_t peers = (uint64_t)__ballot(v < N);
    for (int b = 0; b < 8; ++b) {
      const uint64_t m = (uint64_t)__ballot(v < N && ((d >> b) & 1));
      peers &= (v < N && ((d >> b) & 1)) ? m : ~m;
    }
    const int below = __popcll(peers & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
    const int base = v < N ? L.done[d] : 0;
    __syncthreads();
    if (v < N) {
      list[base + below] = v;
      if (below == 0) L.done[d] = base + __popcll(peers);
    }
    __syncthreads();
  }
  for (int d = lane; d < D; d += kWave) {
    L.head[d] = L.done[d] = L.qbeg[d];
    L.cur[d] = 0;
    L.clk[d] = L.send_until[d] = L.recv_until[d] = 0;
    L.arr_evt[d] = L.next_fin[d] = kNever;
    L.dirty[d] = 1;
    L.seen[d] = 0;
  }
  for (int r = lane; r < R; r += kWave) L.comp[r] = G.release[r];
  for (int e = lane; e < E; e += kWave) arr[(int64_t)e * nb + c] = -1;  // not started yet
  __syncthreads();

  int64_t ms = 0, sum = 0;
  int64_t npend = 0;
  bool stuck = false;
  // every instant consumes at least one finish or arrival, so N + E + 1
  // instants are enough; the bound only guarantees that the wave exits
  for (int64_t step = 0;; ++step) {
    if (step > (int64_t)N + E + 1) {
      stuck = true;
      break;
    }
    // place every queue head whose inputs' availability is known
    for (int d = lane; d < D; d += kWave) {
      if (!L.dirty[d]) continue;
      L.dirty[d] = 0;
      const int qend = L.qbeg[d + 1];
      int h = L.head[d];
      for (; h < qend; ++h) {
        const int v = list[h];
        int64_t ready = G.release[G.op_req[v]];
        bool known = true;
        for (int pe = G.pred_ptr[v]; pe < G.pred_ptr[v + 1]; ++pe) {
          const int u = G.pred_idx[pe];
          int64_t a;
          if (prow[u] == d) {
            a = frow[u];  // earlier in this queue, hence placed
          } else {
            a = arr[(int64_t)pe * nb + c];
            if (a < 0) {
              known = false;
              break;
            }
          }
          ready = imax(ready, a);
        }
        if (!known) break;
        const int64_t w = G.dur[(int64_t)v * C + G.dev_class[d]];
        const int64_t t = imax(ready, L.clk[d]);
        const int sb = G.slice_ptr[d];
        int k = L.cur[d];
        int64_t s;
        for (;;) {
          s = imax(t, G.slice_begin[sb + k]);
          if (s + w <= G.slice_end[sb + k]) break;
          ++k;
        }
        L.cur[d] = k;
        const int64_t f = s + w;
        frow[v] = f;
        L.clk[d] = f;
        if (L.done[d] == h) L.next_fin[d] = f;  // the first placed op not yet finished
        ms = imax(ms, f);
        sum += f;
        atomicMax(reinterpret_cast<unsigned long long *>(&L.comp[G.op_req[v]]), (unsigned long long)f);
      }
      L.head[d] = h;
    }
    __syncthreads();
    // the next instant: a finish or an arrival
    int64_t t = kNever;
    for (int d = lane; d < D; d += kWave) t = min(t, min(L.next_fin[d], L.arr_evt[d]));
    for (int o = kWave / 2; o >= 1; o >>= 1) t = min(t, (int64_t)__shfl_xor(t, o, kWave));
    if (t == kNever) break;
    // arrivals at t: the ports they held are idle from t on
    for (int d = lane; d < D; d += kWave)
      if (L.arr_evt[d] == t) L.arr_evt[d] = kNever;
    // finishes at t, in producer index order: their Intents, by destination
    for (;;) {
      int u = INT_MAX;
      for (int d = lane; d < D; d += kWave)
        if (L.next_fin[d] == t) u = min(u, list[L.done[d]]);
      for (int o = kWave / 2; o >= 1; o >>= 1) u = min(u, __shfl_xor(u, o, kWave));
      if (u == INT_MAX) break;
      const int du = prow[u];
      __syncthreads();
      if (lane == 0) {
        const int nd = ++L.done[du];
        L.next_fin[du] = nd < L.head[du] ? frow[list[nd]] : kNever;
      }
      for (int q = G.succ_ptr[u] + lane; q < G.succ_ptr[u + 1]; q += kWave) {
        const int e = prow[G.succ_idx[q]];
        if (e != du) L.seen[e] = 1;
      }
      __syncthreads();
      for (int d0 = 0; d0 < D; d0 += kWave) {
        const int d = d0 + lane;
        const bool mark = d < D && L.seen[d];
        uint64_t m = (uint64_t)__ballot(mark);
        if (mark) L.seen[d] = 0;
        while (m) {  // destinations in increasing device order
          const int e = d0 + __ffsll((unsigned long long)m) - 1;
          m &= m - 1;
          const int64_t x = G.xfer[(int64_t)u * K + G.link_class[du * D + e]];
          if (x == 0) {  // nothing moves: complete at its request
            port_set_arrivals(G, prow, u, e, t, arr, nb, c, lane, kWave);
            if (lane == 0) L.dirty[e] = 1;
          } else {
            if (lane == 0) pend[npend] = (int64_t)u << 8 | e;
            ++npend;
          }
        }
      }
      __syncthreads();
    }
    // arbitration at t: pending transfers in order, each started when both of
    // its ports are idle; the rest kept in order
    int64_t kept = 0;
    for (int64_t b0 = 0; b0 < npend; b0 += kWave) {
      const int64_t i = b0 + lane;
      const bool valid = i < npend;
      const int64_t ent = valid ? pend[i] : 0;
      const int u = (int)(ent >> 8), e = (int)(ent & 255), s = valid ? prow[u] : 0;
      const int64_t x = valid ? G.xfer[(int64_t)u * K + G.link_class[s * D + e]] : 0;
      bool started = false;
      __syncthreads();
      for (;;) {
        const bool elig = valid && !started && L.send_until[s] <= t && L.recv_until[e] <= t;
        const uint64_t m = (uint64_t)__ballot(elig);
        if (!m) break;
        const int first = __ffsll((unsigned long long)m) - 1;
        if (lane == first) {
          const int64_t a = t + x;
          L.send_until[s] = a;
          L.recv_until[e] = a;
          L.arr_evt[e] = a;
          L.dirty[e] = 1;
          port_set_arrivals(G, prow, u, e, a, arr, nb, c, 0, 1);
          started = true;
        }
        __syncthreads();
      }
      const bool keep = valid && !started;
      const uint64_t km = (uint64_t)__ballot(keep);
      const int pos = __popcll(km & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
      __syncthreads();
      if (keep) pend[kept + pos] = ent;
      kept += __popcll(km);
    }
    npend = kept;
    __syncthreads();
  }
  // completion-time statistics (Sec. 3.3.3); every queue has run out (a
  // queue left with ops would be a defect: its makespan reads -1)
  for (int d = lane; d < D; d += kWave) stuck = stuck || L.head[d] < L.qbeg[d + 1];
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    ms = imax(ms, (int64_t)__shfl_xor(ms, o, kWave));
    sum += (int64_t)__shfl_xor(sum, o, kWave);
  }
  if (__ballot(stuck)) ms = -1;
  if (lane == 0) {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = sum;
    violation[c] = 0;
  }
  if (slack)
    for (int r = lane; r < R; r += kWave) slack[c * R + r] = G.deadline[r] - L.comp[r];
}

// ------------------------------------------------------------------ memory
// Interval endpoints contributed by op y placed on device e: its own output
// (allocated at its start, freed when its last local consumer has finished and
// its last outgoing transfer has arrived; never for an op without consumers)
// and, for every remote predecessor whose last consumer on e is y, that
// predecessor's copy on e (allocated at the predecessor's finish, freed at y's
// finish).  Key = 2 * time + (1 for an allocation), so frees sort first at
// equal times (half-open intervals).  Zero-byte tensors contribute nothing.
// kReady: the copy's last consumer on e is the one that finishes last (index
// order and finish order agree under index-order dispatch).  kPorts: arrivals
// come from the port reservations (arr, [edge][candidate]); a copy is
// allocated at its transfer's start = arrival - estimate.
// A running schedule's state in the GMG (index order, latency transfers):
// transfers start no earlier than xfer_floor; with done ops, whose recorded
// finishes need not follow index order, the last consumer is the one with the
// latest (finish, index); every time is clipped to t_now, from which on the
// peak is taken (t_now = 0 otherwise, where no time is negative).
template <bool kWrite, bool kReady, bool kPorts, class KP, class VP>
__device__ int op_events(const GmgView &G, const uint8_t *prow, const int64_t *frow, int y, int e, KP keys,
                         VP vals, int w, const int64_t *arr, int64_t nb, int64_t c) {
  const int C = G.n_class, K = G.n_link, D = G.n_dev;
  const int64_t T0 = G.t_now;
  int n = 0;
  const int64_t fy = frow[y];
  const int64_t by = G.out_bytes[y];
  if (by > 0) {
    if (kWrite) {
      keys[w] = 2 * imax(fy - G.dur[(int64_t)y * C + G.dev_class[e]], T0) + 1;
      vals[w] = by;
    }
    ++n;
    const int x0 = G.succ_ptr[y], x1 = G.succ_ptr[y + 1];
    if (x1 > x0) {
      if (kWrite) {
        int64_t F = fy;
        for (int q = x0; q < x1; ++q) {
          const int x = G.succ_idx[q];
          const int dx = prow[x];
          int64_t t;
          if (dx == e) {
            t = frow[x];
          } else if (kPorts) {
            t = arr[(int64_t)G.succ_pe[q] * nb + c];
          } else {
            t = G.issue_at ? imax(fy, xfer_floor(G, prow, y, dx)) : fy;
            t += G.xfer[(int64_t)y * K + G.link_class[e * D + dx]];
          }
          F = imax(F, t);
        }
        keys[w + n] = 2 * imax(F, T0);
        vals[w + n] = -by;
      }
      ++n;
    }
  }
  const int p1 = G.pred_ptr[y + 1];
  for (int q = G.pred_ptr[y]; q < p1; ++q) {
    const int u = G.pred_idx[q];
    if (prow[u] == e) continue;
    const int64_t bu = G.out_bytes[u];
    if (bu == 0) continue;
    bool last = true;  // no consumer of u on e after y?
    const int s0 = G.succ_ptr[u];
    if (!kReady && !kPorts && G.done_fin) {
      for (int s = s0; s < G.succ_ptr[u + 1]; ++s) {
        const int x = G.succ_idx[s];
        if (x != y && prow[x] == e && (frow[x] > fy || (frow[x] == fy && x > y))) {
          last = false;
          break;
        }
      }
    } else if (kReady) {  // one op at a time on e: finishes there are distinct
      for (int s = s0; s < G.succ_ptr[u + 1]; ++s) {
        const int x = G.succ_idx[s];
        if (prow[x] == e && frow[x] > fy) {
          last = false;
          break;
        }
      }
    } else {
      for (int s = G.succ_ptr[u + 1] - 1; s >= s0; --s) {
        const int x = G.succ_idx[s];
        if (x <= y) break;
        if (prow[x] == e) {
          last = false;
          break;
        }
      }
    }
    if (!last) continue;
    if (kWrite) {
      int64_t t0;
      if (kPorts)
        t0 = arr[(int64_t)q * nb + c] - G.xfer[(int64_t)u * K + G.link_class[prow[u] * D + e]];
      else
        t0 = G.issue_at ? imax(frow[u], xfer_floor(G, prow, u, e)) : frow[u];
      keys[w + n] = 2 * imax(t0, T0) + 1;
      vals[w + n] = bu;
      keys[w + n + 1] = 2 * imax(fy, T0);
      vals[w + n + 1] = -bu;
    }
    n += 2;
  }
  return n;
}

template <class KP, class VP>
__device__ __forceinline__ void compare_swap(KP keys, VP vals, int i, int l) {
  const int64_t ki = keys[i], kl = keys[l];
  if (kl < ki) {
    const int64_t vi = vals[i], vl = vals[l];
    keys[i] = kl;
    keys[l] = ki;
    vals[i] = vl;
    vals[l] = vi;
  }
}

// Ascending bitonic sort of n (key, value) pairs by one wave.  Every
// comparator puts the smaller key at the lower index, so the virtual padding
// up to the next power of two (keys = +inf) never moves and pairs that reach
// into it are skipped.
template <class KP, class VP>
__device__ void sort_pairs(KP keys, VP vals, int n, int lane) {
  if (n < 2) return;
  int lg = 0;
  while ((1 << lg) < n) ++lg;
  const int half_total = 1 << (lg - 1);
  for (int kb = 1; kb <= lg; ++kb) {
    const int k = 1 << kb, hmask = (k >> 1) - 1;
    for (int q = lane; q < half_total; q += kWave) {
      const int base = (q >> (kb - 1)) << kb, off = q & hmask;
      const int l = base + k - 1 - off;
      if (l < n) compare_swap(keys, vals, base + off, l);
    }
    __syncthreads();
    for (int jb = kb - 2; jb >= 0; --jb) {
      const int j = 1 << jb;
      for (int q = lane; q < half_total; q += kWave) {
        const int i = ((q >> jb) << (jb + 1)) + (q & (j - 1));
        if (i + j < n) compare_swap(keys, vals, i, i + j);
      }
      __syncthreads();
    }
  }
}

// Maximum over prefixes of the sorted deltas (= peak live bytes, >= 0).
template <class VP>
__device__ int64_t max_prefix_sum(VP vals, int n, int lane) {
  int64_t carry = 0, best = 0;
  for (int base = 0; base < n; base += kWave) {
    const int i = base + lane;
    int64_t s = i < n ? vals[i] : 0;
    for (int o = 1; o < kWave; o <<= 1) {
      const int64_t y = __shfl_up(s, o, kWave);
      if (lane >= o) s += y;
    }
    s += carry;
    int64_t m = i < n ? s : INT64_MIN;
    for (int o = kWave / 2; o >= 1; o >>= 1) m = imax(m, __shfl_xor(m, o, kWave));
    best = imax(best, m);
    carry = __shfl(s, kWave - 1, kWave);
  }
  return best;
}

__device__ __forceinline__ int wave_exclusive_scan(int x, int lane, int *total) {
  int s = x;
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(s, o, kWave);
    if (lane >= o) s += y;
  }
  *total = __shfl(s, kWave - 1, kWave);
  return s - x;
}

template <bool kReady, bool kPorts>
__global__ __launch_bounds__(kWave) void memory_kernel(const GmgView G, const uint8_t *__restrict__ P, int64_t nb,
                                                       const int64_t *__restrict__ fin,
                                                       const int64_t *__restrict__ arr, int32_t *__restrict__ bydev_all,
                                                       int64_t *__restrict__ gkeys_all,
                                                       int64_t *__restrict__ gvals_all, int64_t slot_cap,
                                                       int64_t *__restrict__ peak, uint8_t *__restrict__ violation) {
  __shared__ int64_t skeys[kMemCap];
  __shared__ int64_t svals[kMemCap];
  __shared__ int32_t start[257];
  __shared__ int32_t fillp[256];
  const int D = G.n_dev, N = G.n_ops;
  const int lane = threadIdx.x;
  int32_t *bydev = bydev_all + (int64_t)blockIdx.x * N;
  int64_t *gkeys = gkeys_all + (int64_t)blockIdx.x * slot_cap;
  int64_t *gvals = gvals_all + (int64_t)blockIdx.x * slot_cap;
  for (int64_t c = blockIdx.x; c < nb; c += gridDim.x) {
    const uint8_t *prow = P + c * N;
    const int64_t *frow = fin + c * N;
    if (violation[c] & SS_VIOLATION_INVALID) {
      if (peak)
        for (int d = lane; d < D; d += kWave) peak[c * D + d] = 0;
      continue;
    }
    // group the ops by device (order inside a device is irrelevant: the
    // endpoints are sorted afterwards)
    for (int d = lane; d <= D; d += kWave) start[d] = 0;
    __syncthreads();
    for (int v = lane; v < N; v += kWave) atomicAdd(&start[prow[v]], 1);
    __syncthreads();
    if (lane == 0) {
      int s = 0;
      for (int d = 0; d < D; ++d) {
        const int t = start[d];
        start[d] = s;
        fillp[d] = s;
        s += t;
      }
      start[D] = s;
    }
    __syncthreads();
    for (int v = lane; v < N; v += kWave) bydev[atomicAdd(&fillp[prow[v]], 1)] = v;
    __syncthreads();

    uint8_t viol = 0;
    for (int e = 0; e < D; ++e) {
      const int lo = start[e], hi = start[e + 1];
      int64_t pk = 0;
      if (hi > lo) {
        int mine = 0;
        for (int q = lo + lane; q < hi; q += kWave)
          mine += op_events<false, kReady, kPorts>(G, prow, frow, bydev[q], e, (int64_t *)nullptr, (int64_t *)nullptr,
                                                   0, arr, nb, c);
        int total;
        int w = wave_exclusive_scan(mine, lane, &total);
        if (total <= kMemCap) {
          for (int q = lo + lane; q < hi; q += kWave)
            w += op_events<true, kReady, kPorts>(G, prow, frow, bydev[q], e, skeys, svals, w, arr, nb, c);
          __syncthreads();
          sort_pairs(skeys, svals, total, lane);
          pk = max_prefix_sum(svals, total, lane);
        } else {
          for (int q = lo + lane; q < hi; q += kWave)
            w += op_events<true, kReady, kPorts>(G, prow, frow, bydev[q], e, gkeys, gvals, w, arr, nb, c);
          __syncthreads();
          sort_pairs(gkeys, gvals, total, lane);
          pk = max_prefix_sum(gvals, total, lane);
        }
        __syncthreads();
      }
      if (peak && lane == 0) peak[c * D + e] = pk;
      if (pk > G.cap[e]) viol = SS_VIOLATION_MEMORY;
    }
    if (lane == 0) violation[c] = viol;
    __syncthreads();
  }
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

}  // namespace

// General path: int64 times, any size the loader accepts; either dispatch rule.
// from: resume every candidate after the state's ops; capture (B == 1): store
// the candidate's state after its last op and skip the memory pass; mem_fast:
// the 32-bit memory passes instead of memory_kernel.
static int run_simulate_generic(const ss_gmg *g, SsPlace src, int64_t *makespan, int64_t *peak, uint8_t *violation,
                                int64_t *slack, int64_t *sumfin, hipStream_t stream, bool ready, bool ports,
                                SsWork &W, const ss_state *from = nullptr, ss_state *capture = nullptr,
                                bool mem_fast = false) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev, R = g->n_req, B = src.B;
  const int64_t slot_cap = 2 * (N + E) + 2;
  if (slot_cap >= INT32_MAX) return ss_set_error(SS_ERR_UNSUPPORTED, "n_ops + n_edges too large for the memory pass");
  if (ready && ports) return ss_set_error(SS_ERR_UNSUPPORTED, "transfer ports take index-order dispatch only");
  const void *sched_fn = ready   ? reinterpret_cast<const void *>(&ready_schedule_general)
                         : ports ? reinterpret_cast<const void *>(&port_event_schedule)
                                 : reinterpret_cast<const void *>(&schedule_kernel);
  const size_t sched_lds = ready   ? (size_t)D * (sizeof(int64_t) + sizeof(int32_t))
                           : ports ? port_schedule_lds((int)D, (int)R)
                                   : (size_t)D * kWave * (sizeof(int64_t) + sizeof(uint16_t));
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  size_t lds_max = 0;
  {
    int v = 0;
    err = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, g->device);
    if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
    lds_max = (size_t)v;
  }
  if (sched_lds > lds_max) return ss_set_error(SS_ERR_UNSUPPORTED, "device state of the schedule pass exceeds LDS");
  if ((W.ptr || W.query) && (from || capture || mem_fast))
    return ss_set_error(SS_ERR_UNSUPPORTED, "a caller's workspace serves full simulations only");

  // per candidate: finish times and request completions; with ready-time
  // dispatch also missing-predecessor counts and the spill list; with
  // transfer ports also an arrival per edge, the op list by device and the
  // pending transfers; with op-major input the chunk's placement rows
  const int64_t per_cand = N * 8 + R * 8 + (ready ? N * (4 + 8 + 4) : 0) + (ports ? E * 8 + N * 4 + E * 8 : 0) +
                           (src.op_major ? N : 0);
  const bool resumed = from && from->k > 0;
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  struct Plan {
    int64_t chunk, nslots;
    size_t sz_fin, sz_comp, sz_miss, sz_spr, sz_spo, sz_bydev, sz_ev, sz_port, sz_arr, sz_bad, sz_rows, total;
  };
  auto plan_of = [&](int64_t chunk) {
    Plan q{};
    q.chunk = chunk = std::min<int64_t>(std::max<int64_t>(1, chunk), B);
    q.nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kMemBlocksPerCU, chunk));
    q.sz_fin = align((size_t)chunk * N * 8 + 8);
    q.sz_comp = align((size_t)chunk * R * 8 + 8);
    q.sz_miss = ready ? align((size_t)chunk * N * 4 + 4) : 0;
    q.sz_spr = ready ? align((size_t)chunk * N * 8 + 8) : 0;
    q.sz_spo = ready ? align((size_t)chunk * N * 4 + 4) : 0;
    q.sz_bydev = align((size_t)q.nslots * N * 4 + 4);
    q.sz_ev = align((size_t)q.nslots * slot_cap * 8);
    q.sz_port = ports ? align((size_t)chunk * N * 4 + 4) + align((size_t)chunk * (E + 1) * 8) : 0;
    q.sz_arr = ports ? align((size_t)E * chunk * 8 + 8) : 0;
    q.sz_bad = resumed ? align((size_t)chunk * 4) : 0;
    q.sz_rows = src.op_major ? align((size_t)chunk * N + 1) : 0;
    q.total = q.sz_fin + q.sz_comp + q.sz_miss + q.sz_spr + q.sz_spo + q.sz_bydev + 2 * q.sz_ev + q.sz_port +
              q.sz_arr + q.sz_bad + q.sz_rows;
    return q;
  };
  // chunks of whole waves within the finish-time budget
  int64_t pref_chunk = kFinBudget / std::max<int64_t>(1, per_cand);
  pref_chunk = std::max<int64_t>(kWave, pref_chunk / kWave * kWave);
  const Plan pmin = plan_of(1);
  if (W.query) {
    W.need_min = pmin.total;
    W.need_pref = plan_of(pref_chunk).total;
    W.chunk = W.sub = plan_of(pref_chunk).chunk;
    return SS_OK;
  }
  err = hipFuncSetAttribute(sched_fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sched_lds);
  if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");
  Plan pl = plan_of(pref_chunk);
  SsScratch scr;
  void *scratch = nullptr;
  if (W.ptr) {  // the caller's workspace: the largest chunk that fits
    if (pmin.total > W.bytes)
      return ss_set_error(SS_ERR_INVALID_ARG, "workspace of " + std::to_string(W.bytes) +
                                                   " bytes is smaller than this call's minimum of " +
                                                   std::to_string(pmin.total));
    int64_t lo = 1, hi = pl.chunk;  // plan_of(lo) fits
    while (lo < hi) {
      const int64_t mid = lo + (hi - lo + 1) / 2;
      if (plan_of(mid).total <= W.bytes) lo = mid;
      else hi = mid - 1;
    }
    pl = plan_of(lo >= kWave ? lo / kWave * kWave : lo);
    scratch = W.ptr;
  } else {
    err = ss_scratch_get(g->device, g->pool, pl.total, stream, &scr);
    if (err != hipSuccess) return hip_fail(err, "allocating the simulation scratch");
    scratch = scr.p;
  }
  const int64_t chunk = pl.chunk, nslots = pl.nslots;
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *fin = reinterpret_cast<int64_t *>(take(pl.sz_fin));
  auto *comp = reinterpret_cast<int64_t *>(take(pl.sz_comp));
  auto *miss = reinterpret_cast<int32_t *>(take(pl.sz_miss));
  auto *spr = reinterpret_cast<int64_t *>(take(pl.sz_spr));
  auto *spo = reinterpret_cast<int32_t *>(take(pl.sz_spo));
  auto *bydev = reinterpret_cast<int32_t *>(take(pl.sz_bydev));
  auto *gkeys = reinterpret_cast<int64_t *>(take(pl.sz_ev));
  auto *gvals = reinterpret_cast<int64_t *>(take(pl.sz_ev));
  auto *port = ports ? reinterpret_cast<int64_t *>(take(pl.sz_port)) : nullptr;
  auto *arr = ports ? reinterpret_cast<int64_t *>(take(pl.sz_arr)) : nullptr;
  auto *bad = resumed ? reinterpret_cast<uint32_t *>(take(pl.sz_bad)) : nullptr;
  auto *rows = src.op_major ? reinterpret_cast<uint8_t *>(take(pl.sz_rows)) : nullptr;
  Resume RS;
  if (resumed) {
    RS.k0 = (int32_t)from->k;
    RS.clk = from->clk;
    RS.cur = from->cur;
    RS.comp = from->comp;
    RS.scal = from->scal;
  }
  if (capture) {
    RS.cap_clk = capture->clk;
    RS.cap_cur = capture->cur;
    RS.cap_scal = capture->scal;
  }

  int rc = SS_OK;
  for (int64_t b0 = 0; b0 < B && rc == SS_OK; b0 += chunk) {
    const int64_t nb = std::min(chunk, B - b0);
    const uint8_t *Pc = src.p + b0 * N;
    if (src.op_major) {
      err = ss_rows_from_op_major(src.p, N, B, b0, nb, rows, stream);
      if (err != hipSuccess) {
        rc = hip_fail(err, "transpose launch");
        break;
      }
      Pc = rows;
    }
    SsTimingRec *t_sched = ss_timing_start(SS_KERNEL_SCHEDULE, stream);
    if (ready)
      hipLaunchKernelGGL(ready_schedule_general, dim3((unsigned)nb), dim3(kWave), sched_lds, stream, G, Pc, fin, miss,
                         spr, spo, comp, makespan + b0, sumfin ? sumfin + b0 : nullptr,
                         slack ? slack + b0 * R : nullptr, violation + b0);
    else {
      if (RS.k0 > 0) {
        const unsigned grid = (unsigned)std::min<int64_t>((nb * RS.k0 + 255) / 256, 4096);
        hipLaunchKernelGGL(fill_prefix, dim3(grid), dim3(256), 0, stream, fin, nb, N, (int64_t)RS.k0,
                           static_cast<const int64_t *>(from->fin));
        hipLaunchKernelGGL(zero_u32, dim3((unsigned)std::min<int64_t>((nb + 255) / 256, 1024)), dim3(256), 0, stream,
                           bad, nb);
        hipLaunchKernelGGL(prefix_check, dim3(grid), dim3(256), 0, stream, Pc, nb, N, (int64_t)RS.k0, (int)D, bad);
        RS.bad = bad;
      }
      if (ports) {  // event by event, one wave per candidate
        auto *lists = reinterpret_cast<int32_t *>(port);
        auto *pend = reinterpret_cast<int64_t *>(reinterpret_cast<unsigned char *>(port) +
                                                  align((size_t)chunk * N * 4 + 4));
        hipLaunchKernelGGL(port_event_schedule, dim3((unsigned)nb), dim3(kWave), sched_lds, stream, G, Pc, nb, fin,
                           arr, lists, pend, E + 1, makespan + b0, sumfin ? sumfin + b0 : nullptr,
                           slack ? slack + b0 * R : nullptr, violation + b0);
      } else {
        hipLaunchKernelGGL(schedule_kernel, dim3((unsigned)((nb + kWave - 1) / kWave)), dim3(kWave),
                           sched_lds, stream, G, Pc, nb, fin, comp, RS, makespan + b0,
                           sumfin ? sumfin + b0 : nullptr, slack ? slack + b0 * R : nullptr, violation + b0);
      }
      if (capture) {  // one candidate: its finish times and request completions
        err = hipMemcpyAsync(capture->fin, fin, (size_t)N * 8, hipMemcpyDeviceToDevice, stream);
        if (err == hipSuccess)
          err = hipMemcpyAsync(capture->comp, comp, (size_t)R * 8, hipMemcpyDeviceToDevice, stream);
        if (err != hipSuccess) {
          rc = hip_fail(err, "capturing the simulation state");
          break;
        }
      }
    }
    err = hipGetLastError();
    ss_timing_stop(t_sched, stream);
    if (err != hipSuccess) {
      rc = hip_fail(err, "schedule launch");
      break;
    }
    if (capture) continue;  // the state is all a capture needs
    if (mem_fast) {  // with ports the arrivals, [edge][nb] for this chunk, go along
      rc = ss_run_memory_fast(g, Pc, fin, nb, peak ? peak + b0 * D : nullptr, violation + b0, stream,
                              ports ? static_cast<const int64_t *>(arr) : nullptr, nb);
      continue;
    }
    const int64_t grid = std::min<int64_t>(nb, nslots);
    SsTimingRec *t_mem = ss_timing_start(SS_KERNEL_MEMORY, stream);
    auto *mem_fn = ready ? &memory_kernel<true, false> : ports ? &memory_kernel<false, true> : &memory_kernel<false, false>;
    hipLaunchKernelGGL(mem_fn, dim3((unsigned)grid), dim3(kWave), 0, stream, G, Pc, nb,
                       static_cast<const int64_t *>(fin), static_cast<const int64_t *>(arr), bydev, gkeys, gvals,
                       slot_cap, peak ? peak + b0 * D : nullptr, violation + b0);
    err = hipGetLastError();
    ss_timing_stop(t_mem, stream);
    if (err != hipSuccess) rc = hip_fail(err, "memory_kernel launch");
  }
  if (!W.ptr) {
    err = ss_scratch_put(g->device, &scr, stream);
    if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "releasing the scratch");
  }
  return rc;
}

// Path choice: the 32-bit fast path when the loader enabled it and its LDS
// state fits; SS_PATH=generic or SS_PATH=fast in the environment forces one
// (fast is still refused when the GMG does not qualify).  A GMG holding a
// running schedule's state never qualifies: the loader keeps it off the 32-bit
// tables, so it takes schedule_kernel and memory_kernel.
// The kernels a call takes: the general int64 ones (generic), and with
// transfer ports whether the memory pass is the 32-bit one.
static int simulate_route(const ss_gmg *g, bool ready_dispatch, bool link_ports, bool *generic,
                          bool *ports_mem_fast) {
  if (g->snapshot && (ready_dispatch || link_ports))
    return ss_set_error(SS_ERR_UNSUPPORTED,
                        "a running schedule's state (done_fin, issue_at, t_now) takes index-order dispatch and "
                        "latency-only transfers");
  int lds_max = 0;
  hipError_t err = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  const bool fast_ok = g->view.time32 && (ready_dispatch ? ss_ready_schedule_lds(g) : ss_fast_schedule_lds(g)) <=
                                             (size_t)lds_max;
  const char *path = std::getenv("SS_PATH");
  if (path && std::strcmp(path, "fast") == 0 && (!fast_ok || link_ports))
    return ss_set_error(SS_ERR_UNSUPPORTED, "SS_PATH=fast but this GMG or dispatch needs the general path");
  // transfer ports: the event-driven schedule of the general path, whose
  // memory pass is the 32-bit one when the GMG fits the branch-free interval
  // writer (SS_PATH=generic: the general kernels throughout)
  const bool force_generic = path && std::strcmp(path, "generic") == 0;
  *generic = !fast_ok || link_ports || force_generic;
  *ports_mem_fast = link_ports && !force_generic && g->view.time32 && g->n_ops > 0 && g->n_class == 1 &&
                    g->n_link <= 2 && g->max_outdeg <= 2 && g->view.succ2_pe;
  return SS_OK;
}

int ss_simulate_time_bits_of(const ss_gmg *g, bool ready_dispatch, bool link_ports, int *bits) {
  bool generic = false, ports_mem_fast = false;
  const int rc = simulate_route(g, ready_dispatch, link_ports, &generic, &ports_mem_fast);
  if (rc == SS_OK) *bits = generic ? 64 : 32;
  return rc;
}

int ss_run_simulate(const ss_gmg *g, SsPlace P, int64_t *makespan, int64_t *peak, uint8_t *violation,
                    int64_t *slack, int64_t *sumfin, hipStream_t stream, bool ready_dispatch, bool link_ports,
                    SsWork &W) {
  bool generic = false, ports_mem_fast = false;
  const int route = simulate_route(g, ready_dispatch, link_ports, &generic, &ports_mem_fast);
  if (route != SS_OK) return route;
  if (generic)
    return run_simulate_generic(g, P, makespan, peak, violation, slack, sumfin, stream, ready_dispatch, link_ports, W,
                                nullptr, nullptr, ports_mem_fast && !W.ptr && !W.query);
  if (ready_dispatch) return ss_run_simulate_ready(g, P, makespan, peak, violation, slack, sumfin, stream, W);
  return ss_run_simulate_fast(g, P, makespan, peak, violation, slack, sumfin, stream, W);
}

// The state's buffer grows to hold a capture of g (synchronising the stream
// before the old buffer is released).
static int state_reserve(ss_state *st, const ss_gmg *g, hipStream_t stream) {
  const int64_t n = g->n_ops, d = g->n_dev, r = g->n_req;
  if (st->mem && n <= st->cap_n && d <= st->cap_d && r <= st->cap_r) return SS_OK;
  const int64_t cn = std::max<int64_t>(n, 2 * st->cap_n), cd = std::max<int64_t>(d, st->cap_d),
                cr = std::max<int64_t>(r, st->cap_r);
  const size_t bytes = (size_t)(cn + cd + cr + 2) * 8 + (size_t)cd * 4 + 16;
  if (st->mem) {
    const hipError_t err = hipStreamSynchronize(stream);
    if (err != hipSuccess) return hip_fail(err, "releasing a state buffer");
    ss_pool_free(st->mem, stream);
    st->mem = nullptr;
  }
  const int rc = ss_pool_alloc(g->device, bytes, stream, &st->mem);
  if (rc != SS_OK) {
    st->mem = nullptr;
    st->cap_n = st->cap_d = st->cap_r = 0;
    st->k = 0;
    return rc;
  }
  auto *p = static_cast<int64_t *>(st->mem);
  st->fin = p;
  st->clk = p + cn;
  st->comp = st->clk + cd;
  st->scal = st->comp + cr;
  st->cur = reinterpret_cast<int32_t *>(st->scal + 2);
  st->cap_n = cn;
  st->cap_d = cd;
  st->cap_r = cr;
  st->k = 0;
  return SS_OK;
}

int ss_run_simulate_resume(const ss_gmg *g, const ss_state *from, const uint8_t *P, int64_t B, int64_t *makespan,
                           int64_t *peak, uint8_t *violation, int64_t *slack, int64_t *sumfin, hipStream_t stream) {
  SsWork W;
  SsPlace src;
  src.p = P;
  src.B = B;
  return run_simulate_generic(g, src, makespan, peak, violation, slack, sumfin, stream, false, false, W, from, nullptr,
                              g->view.time32 && g->n_ops > 0);
}

int ss_run_state_capture(const ss_gmg *g, const ss_state *from, const uint8_t *placement, ss_state *capture,
                         hipStream_t stream) {
  int rc = state_reserve(capture, g, stream);
  if (rc != SS_OK) return rc;
  // the schedule kernel's per-candidate outputs, unused here
  void *outs = nullptr;
  hipError_t err = ss_pool_malloc(&outs, 256 + (size_t)g->n_req * 8 + 8, g->pool, stream);
  if (err != hipSuccess) return hip_fail(err, "allocating capture outputs");
  auto *o = static_cast<int64_t *>(outs);
  SsWork W;
  SsPlace src;
  src.p = placement;
  src.B = 1;
  rc = run_simulate_generic(g, src, o, nullptr, reinterpret_cast<uint8_t *>(o + 2), o + 4, o + 1, stream, false,
                            false, W, from, capture);
  err = hipFreeAsync(outs, stream);
  if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "hipFreeAsync");
  capture->k = rc == SS_OK ? g->n_ops : 0;
  capture->d = g->n_dev;
  capture->r = g->n_req;
  return rc;
}
