// Fast path of the batched what-if simulation (gfx950), used when the loader
// proved that every simulated time fits in 32 bits and N <= 65535.
//
// fast_schedule: one lane per candidate, ops in index order (Sec. 3.3.2-3.3.3).
//   Per (device, lane) LDS state, laid out [device][lane] so the 64 lanes of a
//   wave fall in distinct banks whatever device each one touches:
//     clk  u32  effective clock = max(device's last finish, current slice start)
//     cur  u16  current idle slice (relative index)
//     cnt  u16  ops placed on the device so far
//   An op first tries the current slice (one load of its end); only when it
//   does not fit does the lane walk forward through later slices.  Each op's
//   finish time and its rank among the ops of its device are written to the
//   candidate's scratch row; the per-device op counts at the end.
//
// fast_memory: one wave per candidate.
//   1. A pass over the ops in index order (lanes = consecutive ops, so the
//      candidate's rows are read with coalesced loads) writes every residency
//      interval into a per-device bucket: an op's own output at the slot given
//      by its rank (so a device's own intervals are in index order, hence in
//      start-time order), and one copy per (output, remote device).
//   2. Per device, only the copy allocations are sorted (LDS bitonic); they
//      are merged with the already sorted own allocations by binary-search
//      ranks, every free is scattered by binary search onto the first
//      allocation at or after it (frees precede allocations at equal times),
//      and peak = max over allocation instants of (bytes allocated so far -
//      bytes freed so far).  No full sort of all endpoints is needed.
#include <climits>

#include "ss_internal.h"

namespace {

constexpr int kWave = 64;
constexpr int kCap = 1024;            // allocations of one device evaluated in LDS
constexpr uint32_t kInf32 = 0xFFFFFFFFu;
constexpr int64_t kScratchBudget = int64_t(16) << 30;
constexpr int kMemBlocksPerCU = 4;

__device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ int64_t imax64(int64_t a, int64_t b) { return a > b ? a : b; }

// ------------------------------------------------------------------ schedule
__global__ __launch_bounds__(kWave) void fast_schedule(const GmgView G, const uint8_t *__restrict__ P, int64_t nb,
                                                       uint32_t *__restrict__ fin, uint16_t *__restrict__ rank,
                                                       uint16_t *__restrict__ dcnt, int64_t *__restrict__ makespan,
                                                       int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
                                                       uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class, K = G.n_link;
  const int lane = threadIdx.x;
  uint32_t *clk = reinterpret_cast<uint32_t *>(lds_raw);                               // [D][64]
  uint32_t *comp = clk + (size_t)D * kWave;                                            // [R][64]
  uint16_t *cur = reinterpret_cast<uint16_t *>(comp + (size_t)R * kWave);              // [D][64]
  uint16_t *cnt = cur + (size_t)D * kWave;                                             // [D][64]
  const int64_t c = (int64_t)blockIdx.x * kWave + lane;
  if (c >= nb) return;
  const uint8_t *prow = P + c * N;
  uint32_t *frow = fin + c * N;
  uint16_t *rrow = rank + c * N;
  for (int d = 0; d < D; ++d) {
    clk[d * kWave + lane] = G.slice_begin32[G.slice_ptr[d]];
    cur[d * kWave + lane] = 0;
    cnt[d * kWave + lane] = 0;
  }
  for (int r = 0; r < R; ++r) comp[r * kWave + lane] = G.release32[r];

  bool invalid = false;
  uint32_t ms = 0;
  uint64_t sum = 0;
  for (int v = 0; v < N; ++v) {
    int d = prow[v];
    if (d >= D) {
      invalid = true;
      d = 0;
    }
    const uint32_t w = G.dur32[v * C + G.dev_class[d]];
    const int r = G.op_req[v];
    uint32_t ready = G.release32[r];
    const int e1 = G.pred_ptr[v + 1];
    for (int e = G.pred_ptr[v]; e < e1; ++e) {
      const int u = G.pred_idx[e];
      uint32_t t = frow[u];
      int du = prow[u];
      if (du >= D) du = 0;
      if (du != d) t += G.xfer32[u * K + G.link_class[du * D + d]];
      ready = umax32(ready, t);
    }
    const int slot = d * kWave + lane;
    const int sbase = G.slice_ptr[d];
    int k = cur[slot];
    uint32_t s = umax32(ready, clk[slot]);  // clk already includes the current slice's start
    if (s + w > G.slice_end32[sbase + k]) {
      // does not fit in the current slice: first later slice that holds it
      // (every later slice starts after the device's last finish)
      for (;;) {
        ++k;
        const uint32_t a = G.slice_begin32[sbase + k];
        const uint32_t t = umax32(ready, a);
        if (t + w <= G.slice_end32[sbase + k]) {
          s = t;
          break;
        }
      }
      cur[slot] = (uint16_t)k;
    }
    const uint32_t f = s + w;
    clk[slot] = f;
    const uint16_t rk = cnt[slot];
    cnt[slot] = rk + 1;
    frow[v] = f;
    rrow[v] = rk;
    ms = umax32(ms, f);
    sum += f;
    uint32_t *cr = comp + r * kWave + lane;
    *cr = umax32(*cr, f);
  }
  uint16_t *crow = dcnt + c * D;
  for (int d = 0; d < D; ++d) crow[d] = cnt[d * kWave + lane];
  if (invalid) {
    makespan[c] = INT64_MAX;
    if (sumfin) sumfin[c] = INT64_MAX;
    if (slack)
      for (int r = 0; r < R; ++r) slack[c * R + r] = INT64_MIN;
    violation[c] = SS_VIOLATION_INVALID;
  } else {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = (int64_t)sum;
    if (slack)
      for (int r = 0; r < R; ++r) slack[c * R + r] = G.deadline[r] - (int64_t)comp[r * kWave + lane];
    violation[c] = 0;
  }
}

// ------------------------------------------------------------------ memory
struct Records {  // SoA interval records: [lo, hi) with bytes
  uint32_t *lo, *hi;
  int64_t *b;
};

// Intervals of op v (own output, and one copy per remote destination device).
// kWrite = false only counts the copies per destination (atomics on ccnt).
template <bool kWrite>
__device__ void op_intervals(const GmgView &G, const uint8_t *prow, const uint32_t *frow, const uint16_t *rrow, int v,
                             const int *own_off, int *cfill, Records own, Records cp) {
  const int D = G.n_dev, K = G.n_link, C = G.n_class;
  const int d = prow[v];
  const int64_t b = G.out_bytes[v];
  const int x0 = G.succ_ptr[v], x1 = G.succ_ptr[v + 1];
  if (kWrite) {
    const uint32_t f = frow[v];
    uint32_t F = kInf32;  // kept forever without consumers
    if (x1 > x0) {
      F = f;
      for (int q = x0; q < x1; ++q) {
        const int x = G.succ_idx[q];
        const int dx = prow[x];
        const uint32_t t = (dx == d) ? frow[x] : f + G.xfer32[v * K + G.link_class[d * D + dx]];
        F = umax32(F, t);
      }
    }
    const int pos = own_off[d] + rrow[v];
    own.lo[pos] = f - G.dur32[v * C + G.dev_class[d]];
    own.hi[pos] = F;
    own.b[pos] = b;
  }
  if (b == 0) return;
  for (int q = x0; q < x1; ++q) {
    const int e = prow[G.succ_idx[q]];
    if (e == d) continue;
    bool first = true;
    for (int q2 = x0; q2 < q; ++q2)
      if (prow[G.succ_idx[q2]] == e) first = false;
    if (!first) continue;
    const int pos = atomicAdd(&cfill[e], 1);
    if (kWrite) {
      uint32_t g = 0;
      for (int q2 = q; q2 < x1; ++q2) {
        const int x = G.succ_idx[q2];
        if (prow[x] == e) g = umax32(g, frow[x]);
      }
      cp.lo[pos] = frow[v];
      cp.hi[pos] = g;
      cp.b[pos] = b;
    }
  }
}

__device__ __forceinline__ int lower_bound_u32(const uint32_t *a, int n, uint32_t x) {  // first i with a[i] >= x
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < x)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

__device__ __forceinline__ int upper_bound_u32(const uint32_t *a, int n, uint32_t x) {  // first i with a[i] > x
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] <= x)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// ascending bitonic sort of n (u32 key, i64 payload) pairs by one wave
template <class KP, class VP>
__device__ void sort_u32_pairs(KP keys, VP vals, int n, int lane) {
  if (n < 2) return;
  int lg = 0;
  while ((1 << lg) < n) ++lg;
  const int half_total = 1 << (lg - 1);
  for (int kb = 1; kb <= lg; ++kb) {
    const int k = 1 << kb, hmask = (k >> 1) - 1;
    for (int q = lane; q < half_total; q += kWave) {
      const int base = (q >> (kb - 1)) << kb, off = q & hmask;
      const int i = base + off, l = base + k - 1 - off;
      if (l < n) {
        const uint32_t ki = keys[i], kl = keys[l];
        if (kl < ki) {
          const int64_t vi = vals[i];
          keys[i] = kl;
          keys[l] = ki;
          vals[i] = vals[l];
          vals[l] = vi;
        }
      }
    }
    __syncthreads();
    for (int jb = kb - 2; jb >= 0; --jb) {
      const int j = 1 << jb;
      for (int q = lane; q < half_total; q += kWave) {
        const int i = ((q >> jb) << (jb + 1)) + (q & (j - 1)), l = i + j;
        if (l < n) {
          const uint32_t ki = keys[i], kl = keys[l];
          if (kl < ki) {
            const int64_t vi = vals[i];
            keys[i] = kl;
            keys[l] = ki;
            vals[i] = vals[l];
            vals[l] = vi;
          }
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int64_t wave_incl_scan64(int64_t x, int lane) {
  for (int o = 1; o < kWave; o <<= 1) {
    const int64_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

// Peak of one device from its own records (start-sorted) and copy records.
// Work arrays (LDS or a global slot buffer): sk/sb (own then copy allocations),
// mk/mb (merged allocations, then allocated-so-far), fd (bytes freed).
template <class UP, class IP, class FP>
__device__ int64_t device_peak(const Records own, int o0, int n1, const Records cp, int c0, int n4, UP sk, IP sb,
                               UP mk, IP mb, FP fd, int lane) {
  const int na = n1 + n4;
  for (int i = lane; i < n1; i += kWave) {
    sk[i] = own.lo[o0 + i];
    sb[i] = own.b[o0 + i];
  }
  for (int j = lane; j < n4; j += kWave) {
    sk[n1 + j] = cp.lo[c0 + j];
    sb[n1 + j] = cp.b[c0 + j];
  }
  __syncthreads();
  sort_u32_pairs(sk + n1, sb + n1, n4, lane);
  // merge the two sorted runs by ranks (own before copy at equal keys)
  for (int i = lane; i < n1; i += kWave) {
    const int pos = i + lower_bound_u32(sk + n1, n4, sk[i]);
    mk[pos] = sk[i];
    mb[pos] = sb[i];
  }
  for (int j = lane; j < n4; j += kWave) {
    const int pos = j + upper_bound_u32(sk, n1, sk[n1 + j]);
    mk[pos] = sk[n1 + j];
    mb[pos] = sb[n1 + j];
  }
  for (int i = lane; i < na; i += kWave) fd[i] = 0;
  __syncthreads();
  // bytes allocated up to and including each allocation
  int64_t carry = 0;
  for (int base = 0; base < na; base += kWave) {
    const int i = base + lane;
    int64_t x = i < na ? mb[i] : 0;
    x = wave_incl_scan64(x, lane) + carry;
    if (i < na) mb[i] = x;
    carry = __shfl(x, kWave - 1, kWave);
  }
  // each free lands on the first allocation at or after its time
  for (int i = lane; i < n1; i += kWave) {
    const uint32_t h = own.hi[o0 + i];
    if (h == kInf32) continue;
    const int pos = lower_bound_u32(mk, na, h);
    if (pos < na) atomicAdd(reinterpret_cast<unsigned long long *>(&fd[pos]), (unsigned long long)own.b[o0 + i]);
  }
  for (int j = lane; j < n4; j += kWave) {
    const int pos = lower_bound_u32(mk, na, cp.hi[c0 + j]);
    if (pos < na) atomicAdd(reinterpret_cast<unsigned long long *>(&fd[pos]), (unsigned long long)cp.b[c0 + j]);
  }
  __syncthreads();
  int64_t freed = 0, best = 0;
  for (int base = 0; base < na; base += kWave) {
    const int i = base + lane;
    int64_t x = i < na ? (int64_t)fd[i] : 0;
    x = wave_incl_scan64(x, lane) + freed;
    int64_t live = i < na ? mb[i] - x : 0;
    for (int o = kWave / 2; o >= 1; o >>= 1) live = imax64(live, __shfl_xor(live, o, kWave));
    best = imax64(best, live);
    freed = __shfl(x, kWave - 1, kWave);
  }
  __syncthreads();
  return best;
}

__global__ __launch_bounds__(kWave) void fast_memory(const GmgView G, const uint8_t *__restrict__ P, int64_t nb,
                                                     const uint32_t *__restrict__ fin,
                                                     const uint16_t *__restrict__ rank,
                                                     const uint16_t *__restrict__ dcnt, Records own_all,
                                                     Records cp_all, uint32_t *__restrict__ wk_all,
                                                     int64_t *__restrict__ wb_all, int64_t slot_cap,
                                                     int64_t *__restrict__ peak, uint8_t *__restrict__ violation) {
  __shared__ uint32_t s_sk[kCap], s_mk[kCap];
  __shared__ int64_t s_sb[kCap], s_mb[kCap];
  __shared__ uint64_t s_fd[kCap];
  __shared__ int own_off[257], cp_off[257], cfill[256];
  const int D = G.n_dev, N = G.n_ops, E = G.pred_ptr[N];
  const int lane = threadIdx.x;
  const Records own{own_all.lo + (int64_t)blockIdx.x * N, own_all.hi + (int64_t)blockIdx.x * N,
                    own_all.b + (int64_t)blockIdx.x * N};
  const Records cp{cp_all.lo + (int64_t)blockIdx.x * E, cp_all.hi + (int64_t)blockIdx.x * E,
                   cp_all.b + (int64_t)blockIdx.x * E};
  uint32_t *g_sk = wk_all + (int64_t)blockIdx.x * 2 * slot_cap;
  uint32_t *g_mk = g_sk + slot_cap;
  int64_t *g_sb = wb_all + (int64_t)blockIdx.x * 3 * slot_cap;
  int64_t *g_mb = g_sb + slot_cap;
  uint64_t *g_fd = reinterpret_cast<uint64_t *>(g_mb + slot_cap);

  for (int64_t c = blockIdx.x; c < nb; c += gridDim.x) {
    if (violation[c] & SS_VIOLATION_INVALID) {
      if (peak)
        for (int d = lane; d < D; d += kWave) peak[c * D + d] = 0;
      continue;
    }
    const uint8_t *prow = P + c * N;
    const uint32_t *frow = fin + c * N;
    const uint16_t *rrow = rank + c * N;
    // own buckets from the per-device op counts; copy buckets counted here
    if (lane == 0) {
      int s = 0;
      for (int d = 0; d < D; ++d) {
        own_off[d] = s;
        s += dcnt[c * D + d];
      }
      own_off[D] = s;
    }
    for (int d = lane; d < D; d += kWave) cfill[d] = 0;
    __syncthreads();
    for (int v = lane; v < N; v += kWave) op_intervals<false>(G, prow, frow, rrow, v, own_off, cfill, own, cp);
    __syncthreads();
    if (lane == 0) {
      int s = 0;
      for (int d = 0; d < D; ++d) {
        cp_off[d] = s;
        s += cfill[d];
        cfill[d] = cp_off[d];
      }
      cp_off[D] = s;
    }
    __syncthreads();
    for (int v = lane; v < N; v += kWave) op_intervals<true>(G, prow, frow, rrow, v, own_off, cfill, own, cp);
    __syncthreads();

    uint8_t viol = 0;
    for (int e = 0; e < D; ++e) {
      const int o0 = own_off[e], n1 = own_off[e + 1] - o0;
      const int c0 = cp_off[e], n4 = cp_off[e + 1] - c0;
      int64_t pk = 0;
      if (n1 + n4 > 0) {
        if (n1 + n4 <= kCap)
          pk = device_peak(own, o0, n1, cp, c0, n4, s_sk, s_sb, s_mk, s_mb, s_fd, lane);
        else
          pk = device_peak(own, o0, n1, cp, c0, n4, g_sk, g_sb, g_mk, g_mb, g_fd, lane);
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

size_t ss_fast_schedule_lds(const ss_gmg *g) {
  return (size_t)g->n_dev * kWave * (4 + 2 + 2) + (size_t)g->n_req * kWave * 4;
}

int ss_run_simulate_fast(const ss_gmg *g, const uint8_t *P, int64_t B, int64_t *makespan, int64_t *peak,
                         uint8_t *violation, int64_t *slack, int64_t *sumfin, hipStream_t stream) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev, R = g->n_req;
  const size_t sched_lds = ss_fast_schedule_lds(g);
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  err = hipFuncSetAttribute(reinterpret_cast<const void *>(&fast_schedule), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)sched_lds);
  if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");

  const int64_t per_cand = N * (4 + 2) + D * 2;
  int64_t chunk = kScratchBudget / std::max<int64_t>(1, per_cand);
  chunk = std::max<int64_t>(kWave, chunk / kWave * kWave);
  chunk = std::min<int64_t>(chunk, B);
  const int64_t nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kMemBlocksPerCU, chunk));
  const int64_t slot_cap = N + E + 1;  // most allocations one device can hold

  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t sz_fin = align((size_t)chunk * N * 4 + 4);
  const size_t sz_rank = align((size_t)chunk * N * 2 + 2);
  const size_t sz_cnt = align((size_t)chunk * D * 2 + 2);
  const size_t n_own = (size_t)nslots * N + 1, n_cp = (size_t)nslots * E + 1;
  const size_t sz_own = align(n_own * 4) * 2 + align(n_own * 8);
  const size_t sz_cp = align(n_cp * 4) * 2 + align(n_cp * 8);
  const size_t sz_wk = align((size_t)nslots * 2 * slot_cap * 4);
  const size_t sz_wb = align((size_t)nslots * 3 * slot_cap * 8);
  void *scratch = nullptr;
  err = hipMallocAsync(&scratch, sz_fin + sz_rank + sz_cnt + sz_own + sz_cp + sz_wk + sz_wb, stream);
  if (err != hipSuccess) return hip_fail(err, "hipMallocAsync of simulation scratch");
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *fin = reinterpret_cast<uint32_t *>(take(sz_fin));
  auto *rank = reinterpret_cast<uint16_t *>(take(sz_rank));
  auto *dcnt = reinterpret_cast<uint16_t *>(take(sz_cnt));
  Records own{reinterpret_cast<uint32_t *>(take(align(n_own * 4))), reinterpret_cast<uint32_t *>(take(align(n_own * 4))),
              reinterpret_cast<int64_t *>(take(align(n_own * 8)))};
  Records cp{reinterpret_cast<uint32_t *>(take(align(n_cp * 4))), reinterpret_cast<uint32_t *>(take(align(n_cp * 4))),
             reinterpret_cast<int64_t *>(take(align(n_cp * 8)))};
  auto *wk = reinterpret_cast<uint32_t *>(take(sz_wk));
  auto *wb = reinterpret_cast<int64_t *>(take(sz_wb));

  int rc = SS_OK;
  for (int64_t b0 = 0; b0 < B && rc == SS_OK; b0 += chunk) {
    const int64_t nb = std::min(chunk, B - b0);
    const uint8_t *Pc = P + b0 * N;
    SsTimingRec *t_sched = ss_timing_start(SS_KERNEL_SCHEDULE, stream);
    hipLaunchKernelGGL(fast_schedule, dim3((unsigned)((nb + kWave - 1) / kWave)), dim3(kWave), sched_lds, stream, G,
                       Pc, nb, fin, rank, dcnt, makespan + b0, sumfin ? sumfin + b0 : nullptr,
                       slack ? slack + b0 * R : nullptr, violation + b0);
    err = hipGetLastError();
    ss_timing_stop(t_sched, stream);
    if (err != hipSuccess) {
      rc = hip_fail(err, "fast_schedule launch");
      break;
    }
    const int64_t grid = std::min<int64_t>(nb, nslots);
    SsTimingRec *t_mem = ss_timing_start(SS_KERNEL_MEMORY, stream);
    hipLaunchKernelGGL(fast_memory, dim3((unsigned)grid), dim3(kWave), 0, stream, G, Pc, nb,
                       static_cast<const uint32_t *>(fin), static_cast<const uint16_t *>(rank),
                       static_cast<const uint16_t *>(dcnt), own, cp, wk, wb, slot_cap,
                       peak ? peak + b0 * D : nullptr, violation + b0);
    err = hipGetLastError();
    ss_timing_stop(t_mem, stream);
    if (err != hipSuccess) rc = hip_fail(err, "fast_memory launch");
  }
  err = hipFreeAsync(scratch, stream);
  if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "hipFreeAsync");
  return rc;
}
