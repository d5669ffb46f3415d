// Fast path of the batched what-if simulation (gfx950), used when the loader
// proved that every simulated time fits in 32 bits and N <= 65535.
//
// Per chunk of candidates:
//   fast_schedule one lane per candidate, ops in index order (Sec. 3.3.2-3.3.3).
//                 Per (device, lane) LDS state laid out [device][lane], so a
//                 wave's 64 lanes fall in distinct banks whatever device each
//                 touches: effective clock u32 (= max(last finish, current
//                 slice start)) and slice cursor u16.  An op first tries the
//                 current slice; only when it does not fit does the lane walk
//                 forward through later slices.  While op v is placed, the
//                 next op's device, predecessor values and slice end are
//                 already being fetched.  The lane reads its placement row in
//                 16-op blocks; finish times are written op-major.
//   transpose     finish times back to candidate rows
// then per sub-chunk of candidates:
//   fast_intervals one wave per candidate, lanes = consecutive ops (coalesced
//                 row reads), almost no LDS so many waves hide the gathers.
//                 A 64-key sort across the wave groups each chunk of ops by
//                 device, giving every op its rank among the ops of its device
//                 (and per-device counts and in-degree sums) without
//                 same-address atomics.  Writes every residency interval
//                 (Sec. 3.3.2) into a per-device bucket: own outputs at their
//                 rank (so a device's own intervals are start-sorted), one copy
//                 per (output, remote device) in a region bounded by the
//                 device's summed in-degree.
//   fast_peaks    one wave per candidate.  Per device: sort only the copy
//                 allocations (LDS bitonic), merge them with the sorted own
//                 allocations by binary-search ranks, scatter every free onto
//                 the first allocation at or after it (frees precede
//                 allocations at equal times), and take the maximum of
//                 allocated-so-far minus freed-so-far over the allocations.
#include <climits>

#include "ss_internal.h"

namespace {

constexpr int kWave = 64;
constexpr int kCap = 1024;            // allocations of one device evaluated in LDS
constexpr uint32_t kInf32 = 0xFFFFFFFFu;
constexpr int64_t kScratchBudget = int64_t(32) << 30;  // schedule scratch per chunk
constexpr int64_t kRecordBudget = int64_t(12) << 30;   // interval records per sub-chunk
constexpr int kPeakBlocksPerCU = 4;
constexpr int kMaxPre = 4;            // predecessors fetched one op ahead

__device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ int64_t imax64(int64_t a, int64_t b) { return a > b ? a : b; }

// ------------------------------------------------------------------ transpose
// 64 x 64 tiles through LDS: both the read and the write are coalesced.
template <class T>
__global__ __launch_bounds__(256) void transpose_tiles(const T *__restrict__ in, int64_t rows, int64_t cols,
                                                       T *__restrict__ out) {
  __shared__ T tile[64][65];
  const int64_t c0 = (int64_t)blockIdx.x * 64, r0 = (int64_t)blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = in[r * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) out[c * rows + r] = tile[tx][i];
  }
}

// ------------------------------------------------------------------ schedule
__device__ __forceinline__ uint32_t xfer_of(const GmgView &G, int u, int du, int d) {
  const int K = G.n_link;
  if (K == 1) return G.xfer32[u];
  const int k = G.link_class[du * G.n_dev + d];
  if (K == 2) {  // both entries are wave-uniform loads
    const uint32_t x0 = G.xfer32[2 * u], x1 = G.xfer32[2 * u + 1];
    return k ? x1 : x0;
  }
  return G.xfer32[u * K + k];
}

// The lane streams its candidate's placement row (row-major, as the caller
// passes it) in 16-op blocks, one block ahead; finish times are op-major
// ([op][candidate]) so every per-op finish-time load or store of a wave is one
// contiguous 64-element segment.
template <bool kVec16>
__global__ __launch_bounds__(kWave) void fast_schedule(const GmgView G, const uint8_t *__restrict__ P, int64_t nb,
                                                       uint32_t *__restrict__ finT, int64_t *__restrict__ makespan,
                                                       int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
                                                       uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class;
  const int lane = threadIdx.x;
  uint32_t *clk = reinterpret_cast<uint32_t *>(lds_raw);                  // [D][64]
  uint32_t *comp = clk + (size_t)D * kWave;                               // [R][64]
  int32_t *sbase = reinterpret_cast<int32_t *>(comp + (size_t)R * kWave);  // [D+1] slice ranges of the devices
  int32_t *dcls = sbase + D + 1;                                          // [D] device class
  uint16_t *cur = reinterpret_cast<uint16_t *>(dcls + D);                 // [D][64]
  for (int d = lane; d <= D; d += kWave) {
    sbase[d] = G.slice_ptr[d];
    if (d < D) dcls[d] = G.dev_class[d];
  }
  __syncthreads();
  const int64_t c = (int64_t)blockIdx.x * kWave + lane;
  if (c >= nb) return;
  const uint8_t *prow = P + c * N;
  for (int d = 0; d < D; ++d) {
    clk[d * kWave + lane] = G.slice_begin32[sbase[d]];
    cur[d * kWave + lane] = 0;
  }
  for (int r = 0; r < R; ++r) comp[r * kWave + lane] = G.release32[r];

  // placement stream
  uint4 blk = make_uint4(0, 0, 0, 0), nxt = make_uint4(0, 0, 0, 0);
  if (kVec16) {
    if (N > 0) blk = *reinterpret_cast<const uint4 *>(prow);
    if (N > 16) nxt = *reinterpret_cast<const uint4 *>(prow + 16);
  }
  auto dev_of = [&](int v) -> int {  // device of op v (v in the current block)
    const int q = (v >> 2) & 3;
    const uint32_t w = q == 0 ? blk.x : q == 1 ? blk.y : q == 2 ? blk.z : blk.w;
    return (int)((w >> (8 * (v & 3))) & 0xFFu);
  };

  bool invalid = false;
  uint32_t ms = 0;
  uint64_t sum = 0;
  int d = 0;
  uint32_t E = 0;  // end of the current slice of op v's device
  if (N > 0) {
    d = kVec16 ? dev_of(0) : prow[0];
    if (d >= D) {
      invalid = true;
      d = 0;
    }
    E = G.slice_end32[sbase[d]];
  }
  uint32_t pf[kMaxPre];  // finish and device of op v's first predecessors (fetched during op v-1)
  int pd[kMaxPre];
#pragma unroll
  for (int i = 0; i < kMaxPre; ++i) {
    pf[i] = 0;
    pd[i] = 0;
  }
  uint32_t f_prev = 0;
  int d_prev = 0;
  for (int v = 0; v < N; ++v) {
    int dn_raw = 0;
    if (!kVec16 && v + 1 < N) dn_raw = prow[v + 1];  // in flight while op v is placed
    const uint32_t w = (C == 1) ? G.dur32[v] : G.dur32[v * C + dcls[d]];
    const int r = G.op_req[v];
    // ready: release, and every predecessor's finish plus its transfer
    uint32_t ready = G.release32[r];
    const int e0 = G.pred_ptr[v], e1 = G.pred_ptr[v + 1];
#pragma unroll
    for (int i = 0; i < kMaxPre; ++i) {
      if (e0 + i < e1) {
        const int u = G.pred_idx[e0 + i];
        const bool last = (u == v - 1);
        uint32_t t = last ? f_prev : pf[i];
        const int du = last ? d_prev : pd[i];
        if (du != d) t += xfer_of(G, u, du, d);
        ready = umax32(ready, t);
      }
    }
    for (int e = e0 + kMaxPre; e < e1; ++e) {  // more predecessors than were fetched ahead
      const int u = G.pred_idx[e];
      uint32_t t;
      int du;
      if (u == v - 1) {
        t = f_prev;
        du = d_prev;
      } else {
        t = finT[(int64_t)u * nb + c];
        du = prow[u];
        if (du >= D) du = 0;
      }
      if (du != d) t += xfer_of(G, u, du, d);
      ready = umax32(ready, t);
    }
    // one op at a time, in the current idle slice if it fits there, else in the
    // first later slice that holds it (later slices start after the device's
    // last finish, so only the ready time and the slice start matter there)
    const int slot = d * kWave + lane;
    uint32_t s = umax32(ready, clk[slot]);
    if (s + w > E) {
      const int sb = sbase[d];
      int k = cur[slot];
      for (;;) {
        ++k;
        const uint32_t t = umax32(ready, G.slice_begin32[sb + k]);
        if (t + w <= G.slice_end32[sb + k]) {
          s = t;
          break;
        }
      }
      cur[slot] = (uint16_t)k;
    }
    const uint32_t f = s + w;
    clk[slot] = f;
    finT[(int64_t)v * nb + c] = f;
    ms = umax32(ms, f);
    sum += f;
    uint32_t *cr = comp + r * kWave + lane;
    *cr = umax32(*cr, f);
    f_prev = f;
    d_prev = d;
    if (v + 1 < N) {  // fetch what op v+1 needs while this wave moves on
      const int q0 = G.pred_ptr[v + 1], q1 = G.pred_ptr[v + 2];
#pragma unroll
      for (int i = 0; i < kMaxPre; ++i) {
        if (q0 + i < q1) {
          const int u = G.pred_idx[q0 + i];
          if (u != v) {
            pf[i] = finT[(int64_t)u * nb + c];
            const int du = prow[u];
            pd[i] = du >= D ? 0 : du;
          }
        }
      }
      if (kVec16) {
        if (((v + 1) & 15) == 0) {  // next block becomes current; fetch the one after
          blk = nxt;
          if (v + 17 < N) nxt = *reinterpret_cast<const uint4 *>(prow + v + 17);
        }
        dn_raw = dev_of(v + 1);
      }
      d = dn_raw;
      if (d >= D) {
        invalid = true;
        d = 0;
      }
      E = G.slice_end32[sbase[d] + cur[d * kWave + lane]];
    }
  }
  if (invalid) {
    makespan[c] = INT64_MAX;
    if (sumfin) sumfin[c] = INT64_MAX;
    if (slack)
      for (int rr = 0; rr < R; ++rr) slack[c * R + rr] = INT64_MIN;
    violation[c] = SS_VIOLATION_INVALID;
  } else {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = (int64_t)sum;
    if (slack)
      for (int rr = 0; rr < R; ++rr) slack[c * R + rr] = G.deadline[rr] - (int64_t)comp[rr * kWave + lane];
    violation[c] = 0;
  }
}

// ------------------------------------------------------------------ memory
// An interval record: {allocation time, free time (kInf32 = never), bytes}.
using Rec = uint3;

// Intervals of op v: its own output at slot own_pos of its device's bucket,
// and one copy per remote destination device (slot taken with an LDS atomic).
__device__ void op_intervals(const GmgView &G, const uint8_t *prow, const uint32_t *frow, int v, int own_pos,
                             int *cfill, Rec *own, Rec *cp) {
  const int C = G.n_class;
  const int d = prow[v];
  const uint32_t b = (uint32_t)G.out_bytes[v];
  const int x0 = G.succ_ptr[v], x1 = G.succ_ptr[v + 1];
  const uint32_t f = frow[v];
  uint32_t F = kInf32;  // kept forever without consumers
  if (x1 > x0) {
    F = f;
    for (int q = x0; q < x1; ++q) {
      const int x = G.succ_idx[q];
      const int dx = prow[x];
      F = umax32(F, (dx == d) ? frow[x] : f + xfer_of(G, v, d, dx));
    }
  }
  own[own_pos] = Rec{f - G.dur32[v * C + G.dev_class[d]], F, b};
  if (b == 0) return;
  for (int q = x0; q < x1; ++q) {
    const int e = prow[G.succ_idx[q]];
    if (e == d) continue;
    bool first = true;
    for (int q2 = x0; q2 < q; ++q2)
      if (prow[G.succ_idx[q2]] == e) first = false;
    if (!first) continue;
    uint32_t g = 0;  // the copy lives until its last consumer on e finishes
    for (int q2 = q; q2 < x1; ++q2) {
      const int x = G.succ_idx[q2];
      if (prow[x] == e) g = umax32(g, frow[x]);
    }
    cp[atomicAdd(&cfill[e], 1)] = Rec{f, g, b};
  }
}

// Ascending sort of the 64 lanes' keys: bitonic network over lane shuffles.
__device__ __forceinline__ uint32_t wave_sort64(uint32_t key, int lane) {
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint32_t other = __shfl_xor(key, j, kWave);
      const bool asc = (lane & k) == 0, low = (lane & j) == 0;
      key = (asc == low) ? min(key, other) : max(key, other);
    }
  }
  return key;
}

// Groups a chunk of 64 ops by device.  For the op of this lane (device d,
// active = it exists): rank = how many ops of the chunk with lower index are
// on the same device.  Lanes that end a device's group in sorted order get
// that device (grp_dev, else -1), the group size and the group's sum of val.
__device__ __forceinline__ void chunk_groups(int d, bool active, int val, int lane, int &rank, int &grp_dev,
                                             int &grp_cnt, int &grp_sum) {
  const uint32_t key = ((active ? (uint32_t)d : 0x3FFu) << 6) | (uint32_t)lane;
  const uint32_t sk = wave_sort64(key, lane);
  const int sd = (int)(sk >> 6), src = (int)(sk & 63u);
  const int sval = __shfl(val, src, kWave);
  const int prev = __shfl_up(sd, 1, kWave), next = __shfl_down(sd, 1, kWave);
  int start = (lane == 0 || prev != sd) ? lane : 0;
  int sum = sval;
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(start, o, kWave);
    if (lane >= o) start = max(start, y);
  }
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(sum, o, kWave);
    if (lane - o >= start) sum += y;
  }
  const bool tail = lane == kWave - 1 || next != sd;
  grp_dev = (tail && sd != 0x3FF) ? sd : -1;
  grp_cnt = lane - start + 1;
  grp_sum = sum;
  rank = __builtin_amdgcn_ds_permute(src << 2, lane - start);
}

// Per-candidate bucket geometry written by fast_intervals, read by fast_peaks.
__device__ __forceinline__ int meta_stride(int D) { return 3 * (D + 1); }

__global__ __launch_bounds__(kWave) void fast_intervals(const GmgView G, const uint8_t *__restrict__ P,
                                                        const uint32_t *__restrict__ fin, int64_t j0,
                                                        Rec *__restrict__ own_all, Rec *__restrict__ cp_all,
                                                        int32_t *__restrict__ meta,
                                                        const uint8_t *__restrict__ violation) {
  __shared__ int own_off[257], cp_off[257], cfill[256], ocnt[256], base[256];
  const int D = G.n_dev, N = G.n_ops, E = G.pred_ptr[G.n_ops];
  const int lane = threadIdx.x;
  const int64_t j = blockIdx.x, c = j0 + j;
  if (violation[c] & SS_VIOLATION_INVALID) return;
  const uint8_t *prow = P + c * N;
  const uint32_t *frow = fin + c * N;
  Rec *own = own_all + j * N;
  Rec *cp = cp_all + j * E;
  for (int d = lane; d < D; d += kWave) {
    cfill[d] = 0;
    ocnt[d] = 0;
    base[d] = 0;
  }
  __syncthreads();
  // ops per device, and summed in-degree (copies landing on a device <= it)
  for (int v0 = 0; v0 < N; v0 += kWave) {
    const int v = v0 + lane;
    const bool act = v < N;
    const int d = act ? prow[v] : 0;
    const int indeg = act ? G.pred_ptr[v + 1] - G.pred_ptr[v] : 0;
    int rank, gd, gcnt, gsum;
    chunk_groups(d, act, indeg, lane, rank, gd, gcnt, gsum);
    if (gd >= 0) {
      ocnt[gd] += gcnt;
      cfill[gd] += gsum;
    }
    __syncthreads();
  }
  if (lane == 0) {
    int so = 0, sc = 0;
    for (int d = 0; d < D; ++d) {
      own_off[d] = so;
      so += ocnt[d];
      cp_off[d] = sc;
      sc += cfill[d];
      cfill[d] = cp_off[d];
    }
    own_off[D] = so;
    cp_off[D] = sc;
  }
  __syncthreads();
  for (int v0 = 0; v0 < N; v0 += kWave) {
    const int v = v0 + lane;
    const bool act = v < N;
    const int d = act ? prow[v] : 0;
    int rank, gd, gcnt, gsum;
    chunk_groups(d, act, 0, lane, rank, gd, gcnt, gsum);
    const int pos = act ? own_off[d] + base[d] + rank : 0;
    __syncthreads();
    if (gd >= 0) base[gd] += gcnt;
    if (act) op_intervals(G, prow, frow, v, pos, cfill, own, cp);
    __syncthreads();
  }
  int32_t *m = meta + j * meta_stride(D);
  for (int d = lane; d <= D; d += kWave) {
    m[d] = own_off[d];
    m[D + 1 + d] = cp_off[d];
    m[2 * (D + 1) + d] = d < D ? cfill[d] - cp_off[d] : 0;
  }
}

// Up to 4 searches per lane in lockstep (independent LDS loads in flight):
// r[j] = first index i in a[0, n) with a[i] >= x[j] (kUpper: a[i] > x[j]).
template <bool kUpper, class UP>
__device__ __forceinline__ void search4(UP a, int n, const uint32_t (&x)[4], int (&r)[4]) {
  int b[4] = {0, 0, 0, 0};
  if (n == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = 0;
    return;
  }
  int len = n;
  while (len > 1) {
    const int half = len >> 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t v = a[b[j] + half];
      if (kUpper ? (v <= x[j]) : (v < x[j])) b[j] += half;
    }
    len -= half;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t v = a[b[j]];
    r[j] = b[j] + ((kUpper ? (v <= x[j]) : (v < x[j])) ? 1 : 0);
  }
}

// ascending bitonic sort of n (u32 key, u64 payload) pairs by one wave
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
          const uint64_t vi = vals[i];
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
            const uint64_t vi = vals[i];
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

__device__ __forceinline__ int wave_incl_scan32(int x, int lane) {
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

constexpr int kSmallGap = 16;  // copies between two own allocations sorted by one lane

// In-place inclusive prefix sum of a[0, n): each lane scans its own contiguous
// run, one wave scan combines the runs.  Callers fence before and after.
template <class CP>
__device__ void prefix_inplace(CP a, int n, int lane) {
  const int m = (n + kWave - 1) / kWave, lo = lane * m, hi = min(n, lo + m);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  int run = wave_incl_scan32(s, lane) - s;
  for (int i = lo; i < hi; ++i) {
    run += a[i];
    a[i] = run;
  }
}

// max(0, max_i sum_{k <= i} (alloc[k] - freed[k])): the peak live bytes, the
// maximum being taken at allocation instants (each position is one).
template <class IP, class FP>
__device__ int64_t max_live(IP alloc, FP freed, int n, int lane) {
  const int m = (n + kWave - 1) / kWave, lo = lane * m, hi = min(n, lo + m);
  int64_t s = 0;
  for (int i = lo; i < hi; ++i) s += alloc[i] - (int64_t)freed[i];
  int64_t run = wave_incl_scan64(s, lane) - s, best = 0;
  for (int i = lo; i < hi; ++i) {
    run += alloc[i] - (int64_t)freed[i];
    best = imax64(best, run);
  }
  for (int o = kWave / 2; o >= 1; o >>= 1) best = imax64(best, __shfl_xor(best, o, kWave));
  return best;
}

// Peak of one device from its own records (start-sorted) and copy records.
// Work arrays (LDS, or a global slot buffer when too large):
//   sk/sp  allocation times and {free time, bytes} of own (first n1) then copy records
//   sq     per copy: (gap << 16 | slot), kept in fd's storage until fd is needed;
//          gap counts / prefix in gc (n1 + 2 ints)
//   mk/mb  merged allocation times and bytes; fd bytes freed just before each
template <class UP, class PP, class IP, class FP, class CP>
__device__ int64_t device_peak(const Rec *own, int o0, int n1, const Rec *cp, int c0, int n4, UP sk, PP sp, CP gc,
                               UP mk, IP mb, FP fd, int lane) {
  constexpr int kB = 8;
  uint32_t *sq = reinterpret_cast<uint32_t *>(fd);
  const int na = n1 + n4;
  for (int base = lane; base < na; base += kB * kWave) {  // all loads of a batch in flight together
    Rec r[kB];
#pragma unroll
    for (int j = 0; j < kB; ++j) {
      const int i = base + j * kWave;
      if (i < na) r[j] = i < n1 ? own[o0 + i] : cp[c0 + i - n1];
    }
#pragma unroll
    for (int j = 0; j < kB; ++j) {
      const int i = base + j * kWave;
      if (i < na) {
        sk[i] = r[j].x;
        sp[i] = ((uint64_t)r[j].y << 32) | r[j].z;
      }
    }
  }
  for (int i = lane; i <= n1 + 1; i += kWave) gc[i] = 0;
  __syncthreads();
  // each copy falls in the gap after the last own allocation at or before it
  int big = 0;  // largest slot this lane saw
  for (int base = lane; base < n4; base += 4 * kWave) {
    uint32_t x[4];
    int r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = base + j * kWave < n4 ? sk[n1 + base + j * kWave] : 0;
    search4<true>(sk, n1, x, r);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + j * kWave;
      if (i < n4) {
        const int slot = atomicAdd(&gc[r[j] + 1], 1);
        sq[i] = ((uint32_t)r[j] << 16) | (uint32_t)slot;
        big = max(big, slot + 1);
      }
    }
  }
  for (int o = kWave / 2; o >= 1; o >>= 1) big = max(big, __shfl_xor(big, o, kWave));
  __syncthreads();
  const bool small_gaps = big <= kSmallGap;
  if (small_gaps) {
    // gc[g + 1] = copies in gap g  ->  gc[g] = copies in gaps before g
    prefix_inplace(gc, n1 + 2, lane);
    __syncthreads();
    // own allocation i follows gaps 0..i ; a copy in gap g follows own 0..g-1
    for (int i = lane; i < n1; i += kWave) {
      const int pos = i + gc[i + 1];
      mk[pos] = sk[i];
      mb[pos] = (int64_t)(sp[i] & 0xFFFFFFFFu);
    }
    for (int i = lane; i < n4; i += kWave) {
      const int g = (int)(sq[i] >> 16), slot = (int)(sq[i] & 0xFFFFu);
      const int pos = g + gc[g] + slot;
      mk[pos] = sk[n1 + i];
      mb[pos] = (int64_t)(sp[n1 + i] & 0xFFFFFFFFu);
    }
    __syncthreads();
    // order the copies inside each gap (at most kSmallGap of them)
    for (int g = lane; g <= n1; g += kWave) {
      const int s0 = g + gc[g], cnt = gc[g + 1] - gc[g];
      for (int a = 1; a < cnt; ++a) {
        const uint32_t key = mk[s0 + a];
        const int64_t val = mb[s0 + a];
        int z = a - 1;
        while (z >= 0 && mk[s0 + z] > key) {
          mk[s0 + z + 1] = mk[s0 + z];
          mb[s0 + z + 1] = mb[s0 + z];
          --z;
        }
        mk[s0 + z + 1] = key;
        mb[s0 + z + 1] = val;
      }
    }
  } else {
    // large gaps: sort the copies, then merge the two runs by ranks
    sort_u32_pairs(sk + n1, sp + n1, n4, lane);
    for (int base = lane; base < n1; base += 4 * kWave) {
      uint32_t x[4];
      int r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = base + j * kWave < n1 ? sk[base + j * kWave] : 0;
      search4<false>(sk + n1, n4, x, r);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = base + j * kWave;
        if (i < n1) {
          mk[i + r[j]] = x[j];
          mb[i + r[j]] = (int64_t)(sp[i] & 0xFFFFFFFFu);
        }
      }
    }
    for (int base = lane; base < n4; base += 4 * kWave) {
      uint32_t x[4];
      int r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = base + j * kWave < n4 ? sk[n1 + base + j * kWave] : 0;
      search4<true>(sk, n1, x, r);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = base + j * kWave;
        if (i < n4) {
          mk[i + r[j]] = x[j];
          mb[i + r[j]] = (int64_t)(sp[n1 + i] & 0xFFFFFFFFu);
        }
      }
    }
  }
  __syncthreads();
  for (int i = lane; i < na; i += kWave) fd[i] = 0;
  __syncthreads();
  // each free lands on the first allocation at or after its time
  for (int base = lane; base < na; base += 4 * kWave) {
    uint32_t x[4];
    int r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = base + j * kWave < na ? (uint32_t)(sp[base + j * kWave] >> 32) : kInf32;
    search4<false>(mk, na, x, r);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = base + j * kWave;
      if (i < na && x[j] != kInf32 && r[j] < na)
        atomicAdd(reinterpret_cast<unsigned long long *>(&fd[r[j]]),
                  (unsigned long long)(sp[i] & 0xFFFFFFFFu));
    }
  }
  __syncthreads();
  const int64_t best = max_live(mb, fd, na, lane);
  __syncthreads();
  return best;
}

__global__ __launch_bounds__(kWave) void fast_peaks(const GmgView G, int64_t j0, int64_t nj,
                                                    const Rec *__restrict__ own_all, const Rec *__restrict__ cp_all,
                                                    const int32_t *__restrict__ meta, uint32_t *__restrict__ wk_all,
                                                    uint64_t *__restrict__ wb_all, int32_t *__restrict__ wc_all,
                                                    int64_t slot_cap, int64_t *__restrict__ peak,
                                                    uint8_t *__restrict__ violation) {
  __shared__ uint32_t s_sk[kCap], s_mk[kCap];
  __shared__ uint64_t s_sp[kCap], s_fd[kCap];
  __shared__ int64_t s_mb[kCap];
  __shared__ int s_gc[kCap + 2];
  const int D = G.n_dev, N = G.n_ops, E = G.pred_ptr[G.n_ops];
  const int lane = threadIdx.x;
  uint32_t *g_sk = wk_all + (int64_t)blockIdx.x * 2 * slot_cap;
  uint32_t *g_mk = g_sk + slot_cap;
  uint64_t *g_sp = wb_all + (int64_t)blockIdx.x * 3 * slot_cap;
  int64_t *g_mb = reinterpret_cast<int64_t *>(g_sp + slot_cap);
  uint64_t *g_fd = g_sp + 2 * slot_cap;
  int32_t *g_gc = wc_all + (int64_t)blockIdx.x * (slot_cap + 2);
  for (int64_t j = blockIdx.x; j < nj; j += gridDim.x) {
    const int64_t c = j0 + j;
    if (violation[c] & SS_VIOLATION_INVALID) {
      if (peak)
        for (int d = lane; d < D; d += kWave) peak[c * D + d] = 0;
      continue;
    }
    const Rec *own = own_all + j * N;
    const Rec *cp = cp_all + j * E;
    const int32_t *m = meta + j * meta_stride(D);
    uint8_t viol = 0;
    for (int e = 0; e < D; ++e) {
      const int o0 = m[e], n1 = m[e + 1] - o0;
      const int c0 = m[D + 1 + e], n4 = m[2 * (D + 1) + e];
      int64_t pk = 0;
      if (n1 + n4 > 0) {
        if (n1 + n4 <= kCap && n1 + 2 <= kCap + 2)
          pk = device_peak(own, o0, n1, cp, c0, n4, s_sk, s_sp, s_gc, s_mk, s_mb, s_fd, lane);
        else
          pk = device_peak(own, o0, n1, cp, c0, n4, g_sk, g_sp, g_gc, g_mk, g_mb, g_fd, lane);
      }
      if (peak && lane == 0) peak[c * D + e] = pk;
      if (pk > G.cap[e]) viol = SS_VIOLATION_MEMORY;
    }
    if (lane == 0) violation[c] = viol;
  }
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

}  // namespace

size_t ss_fast_schedule_lds(const ss_gmg *g) {
  return (size_t)g->n_dev * kWave * (4 + 2) + (size_t)g->n_req * kWave * 4 + (size_t)(g->n_dev + 1) * 8;
}

int ss_run_simulate_fast(const ss_gmg *g, const uint8_t *P, int64_t B, int64_t *makespan, int64_t *peak,
                         uint8_t *violation, int64_t *slack, int64_t *sumfin, hipStream_t stream) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev, R = g->n_req;
  const size_t sched_lds = ss_fast_schedule_lds(g);
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  // 16-byte placement blocks need every row (and so the batch) 16-byte aligned
  const bool vec16 = N % 16 == 0 && (reinterpret_cast<uintptr_t>(P) & 15) == 0;
  err = hipFuncSetAttribute(vec16 ? reinterpret_cast<const void *>(&fast_schedule<true>)
                                  : reinterpret_cast<const void *>(&fast_schedule<false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)sched_lds);
  if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");

  // chunk: op-major and row-major finish times
  const int64_t per_cand = N * (4 + 4);
  int64_t chunk = kScratchBudget / std::max<int64_t>(1, per_cand);
  chunk = std::max<int64_t>(kWave, chunk / kWave * kWave);
  chunk = std::min<int64_t>(chunk, int64_t(65535) * 64);  // transpose grids index 64-candidate tiles in y
  chunk = std::min<int64_t>(chunk, B);
  // sub-chunk: interval records of each candidate (own N, copies <= E)
  const int64_t rec_per_cand = (N + E) * (int64_t)sizeof(uint3) + 3 * (D + 1) * 4;
  int64_t sub = std::max<int64_t>(1, kRecordBudget / std::max<int64_t>(1, rec_per_cand));
  sub = std::min<int64_t>(sub, chunk);
  const int64_t nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kPeakBlocksPerCU, sub));
  const int64_t slot_cap = N + E + 1;  // most allocations one device can hold

  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t sz_fin = align((size_t)chunk * N * 4 + 4);
  const size_t sz_own = align(((size_t)sub * N + 1) * sizeof(uint3));
  const size_t sz_cp = align(((size_t)sub * E + 1) * sizeof(uint3));
  const size_t sz_meta = align((size_t)sub * 3 * (D + 1) * 4);
  const size_t sz_wk = align((size_t)nslots * 2 * slot_cap * 4);
  const size_t sz_wb = align((size_t)nslots * 3 * slot_cap * 8);
  const size_t sz_wc = align((size_t)nslots * (slot_cap + 2) * 4);
  void *scratch = nullptr;
  err = hipMallocAsync(&scratch,
                       2 * sz_fin + sz_own + sz_cp + sz_meta + sz_wk + sz_wb + sz_wc,
                       stream);
  if (err != hipSuccess) return hip_fail(err, "hipMallocAsync of simulation scratch");
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *finT = reinterpret_cast<uint32_t *>(take(sz_fin));
  auto *fin = reinterpret_cast<uint32_t *>(take(sz_fin));
  auto *own = reinterpret_cast<Rec *>(take(sz_own));
  auto *cp = reinterpret_cast<Rec *>(take(sz_cp));
  auto *meta = reinterpret_cast<int32_t *>(take(sz_meta));
  auto *wk = reinterpret_cast<uint32_t *>(take(sz_wk));
  auto *wb = reinterpret_cast<uint64_t *>(take(sz_wb));
  auto *wc = reinterpret_cast<int32_t *>(take(sz_wc));

  int rc = SS_OK;
  auto check = [&](const char *what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess && rc == SS_OK) rc = hip_fail(e, what);
    return rc == SS_OK;
  };
  for (int64_t b0 = 0; b0 < B && rc == SS_OK; b0 += chunk) {
    const int64_t nb = std::min(chunk, B - b0);
    const uint8_t *Pc = P + b0 * N;
    SsTimingRec *ts = ss_timing_start(SS_KERNEL_SCHEDULE, stream);
    const dim3 sgrid((unsigned)((nb + kWave - 1) / kWave));
    if (vec16)
      hipLaunchKernelGGL(fast_schedule<true>, sgrid, dim3(kWave), sched_lds, stream, G, Pc, nb, finT, makespan + b0,
                         sumfin ? sumfin + b0 : nullptr, slack ? slack + b0 * R : nullptr, violation + b0);
    else
      hipLaunchKernelGGL(fast_schedule<false>, sgrid, dim3(kWave), sched_lds, stream, G, Pc, nb, finT, makespan + b0,
                         sumfin ? sumfin + b0 : nullptr, slack ? slack + b0 * R : nullptr, violation + b0);
    ss_timing_stop(ts, stream);
    if (!check("fast_schedule launch")) break;
    SsTimingRec *tt = nullptr;
    tt = ss_timing_start(SS_KERNEL_TRANSPOSE, stream);
    if (N > 0) {  // op-major -> candidates' rows for the memory passes
      const dim3 tg((unsigned)((nb + 63) / 64), (unsigned)((N + 63) / 64));
      hipLaunchKernelGGL(transpose_tiles<uint32_t>, tg, dim3(256), 0, stream, static_cast<const uint32_t *>(finT),
                         (int64_t)N, nb, fin);
    }
    ss_timing_stop(tt, stream);
    if (!check("transpose launch")) break;
    for (int64_t j0 = 0; j0 < nb && rc == SS_OK; j0 += sub) {
      const int64_t nj = std::min(sub, nb - j0);
      SsTimingRec *ti = ss_timing_start(SS_KERNEL_INTERVALS, stream);
      hipLaunchKernelGGL(fast_intervals, dim3((unsigned)nj), dim3(kWave), 0, stream, G, Pc,
                         static_cast<const uint32_t *>(fin), j0, own, cp, meta,
                         static_cast<const uint8_t *>(violation + b0));
      ss_timing_stop(ti, stream);
      if (!check("fast_intervals launch")) break;
      SsTimingRec *tm = ss_timing_start(SS_KERNEL_MEMORY, stream);
      hipLaunchKernelGGL(fast_peaks, dim3((unsigned)std::min<int64_t>(nj, nslots)), dim3(kWave), 0, stream, G, j0, nj,
                         static_cast<const Rec *>(own), static_cast<const Rec *>(cp),
                         static_cast<const int32_t *>(meta), wk, wb, wc, slot_cap, peak ? peak + b0 * D : nullptr,
                         violation + b0);
      ss_timing_stop(tm, stream);
      if (!check("fast_peaks launch")) break;
    }
  }
  err = hipFreeAsync(scratch, stream);
  if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "hipFreeAsync");
  return rc;
}
