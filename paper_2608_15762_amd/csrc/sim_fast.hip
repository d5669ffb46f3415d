// Fast path of the batched what-if simulation (gfx950), used when the loader
// proved that every simulated time fits in 32 bits and N <= 65535.
//
// Index-order dispatch, per chunk of candidates:
//   transpose     candidates' placement rows -> op-major [op][candidate]
//   fast_schedule one lane per candidate, ops in index order (Sec. 3.3.2-3.3.3).
//                 Per (device, lane) LDS state laid out [device][lane], so a
//                 wave's 64 lanes fall in distinct banks whatever device each
//                 touches: the device clock (last finish) only.  The idle
//                 slice that holds an op comes from a per-device time ->
//                 slice lookup taken two ops ahead at a lower bound of the
//                 op's finish.  The next ops' devices, predecessor values,
//                 link classes and lookups are already in flight (a
//                 software pipeline).  Finish times are written op-major
//                 (the schedule's own reads) and, eight ops at a time from
//                 registers, into each candidate's row for the memory passes.
//   transpose     finish times to candidate rows instead when N % 4 != 0
//                 (rows not 16-byte aligned)
// then per sub-chunk of candidates:
//   fast_intervals one wave per candidate, lanes = consecutive ops (coalesced
//                 row reads).  Pass A ranks every op among the ops of its
//                 device (lanes sharing a device from a 64-bit lane mask per
//                 device in LDS) into a rank table and counts per device.
//                 Pass B writes every residency interval (Sec. 3.3.2) into a
//                 per-device bucket: own outputs at their rank (so a device's
//                 own intervals are start-sorted), one copy per (output,
//                 remote device) in a region bounded by the device's summed
//                 in-degree, each event tagged with where it falls among the
//                 device's own starts (exact, or a small window around a
//                 known rank).  For graphs of out-degree <= 2 pass B is
//                 branch free and software-pipelined over chunks, and stages
//                 both kinds of record in LDS to write them in 32-byte pairs.
//   fast_peaks    persistent waves that take candidates from a ticket
//                 counter; per candidate, devices in turn, each device's
//                 records in registers (the next device's loaded meanwhile):
//                 per-gap sums of allocations and frees between consecutive
//                 own starts give the exact live bytes at every own start;
//                 only gaps holding copies and frees whose bound exceeds the
//                 best so far are swept event by event.
// The peak pass of a sub-chunk runs on a second stream beside the interval
// pass of the next ones (three record sets, so an interval pass rarely waits
// for the peak pass that still reads its set).  The schedule of
// the next chunk waits for the last peak pass: its launch is exactly one round
// of resident waves, and waves placed late behind another kernel's would add
// a second round.
// Ready-time dispatch (the rule of Sec. 3.3.2), per chunk:
//   ready_schedule one wave per candidate, the ready set in registers (a
//                 spill list beyond), finish times in candidate rows and each
//                 op's rank in dispatch order; then fast_intervals with those
//                 ranks and fast_peaks as above.
#include <atomic>
#include <climits>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "ss_internal.h"

namespace {

constexpr int kWave = 64;
constexpr uint32_t kInf32 = 0xFFFFFFFFu;
constexpr int64_t kScratchBudget = int64_t(32) << 30;  // schedule scratch per chunk
// index-order 32-bit path: the chunk buffers of its preferred layout (larger
// chunks mean fewer pipeline fills and drains of the memory passes); the
// whole layout, record sets included, is then fitted to the memory the call
// can get (ss_scratch_budget) and halved while it does not fit
constexpr int64_t kFastScratchBudget = int64_t(96) << 30;
constexpr int64_t kRecordBudget = int64_t(32) << 30;   // sizes the sub-chunks (record bytes of about two sets)
constexpr int kPeakBlocksPerCU = 8;  // fast_peaks: 2 waves per SIMD (198 or 224 registers)

__device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ int64_t imax64(int64_t a, int64_t b) { return a > b ? a : b; }

// Orders the LDS accesses of a one-wave workgroup at this point.  A wave's LDS
// operations complete in issue order, so only the compiler must keep accesses
// on their side; unlike __syncthreads there is no wait for outstanding global
// memory operations.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Zero fill (used for counters that kernels take work tickets from).
__global__ __launch_bounds__(256) void fill_zero_u32(uint32_t *__restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0;
}

// ------------------------------------------------------------------ transpose
// 64 x 64 tiles through LDS: both the read and the write are coalesced.
// in: rows x cols with row pitch `pitch` elements; out: cols x rows, dense.
template <class T>
__global__ __launch_bounds__(256) void transpose_tiles(const T *__restrict__ in, int64_t rows, int64_t cols,
                                                       int64_t pitch, T *__restrict__ out) {
  __shared__ T tile[64][65];
  const int64_t c0 = (int64_t)blockIdx.x * 64, r0 = (int64_t)blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = in[r * pitch + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) out[c * rows + r] = tile[tx][i];
  }
}

// 32-bit matrices whose row and column counts and pitch are multiples of 4
// (16-byte aligned buffers): a workgroup takes a strip of 64 columns and walks
// kStripTiles tiles of 64 rows down it, each tile read and written as 16-byte
// vectors through LDS (a wave moves four 256-byte row segments per access).
// The next tile's loads are in flight while the current one is written out,
// and the output segments of consecutive tiles, which share the lines where a
// row's segments meet, are written by the same workgroup.
constexpr int kStripTiles = 16;
__global__ __launch_bounds__(256) void transpose_u32_strips(const uint32_t *__restrict__ in, int64_t rows,
                                                            int64_t cols, int64_t pitch, uint32_t *__restrict__ out) {
  __shared__ uint32_t tile[64][65];
  const int64_t c0 = (int64_t)blockIdx.x * 64, rb = (int64_t)blockIdx.y * (64 * kStripTiles);
  const int t = threadIdx.x, sub = t & 15, grp = t >> 4;
  // read side: rows grp + 16j of the tile, columns 4 sub .. 4 sub + 3;
  // write side: columns grp + 16j of the tile (output rows), rows 4 sub .. 4 sub + 3
  const bool col_in = c0 + 4 * sub < cols;
  auto load = [&](int64_t r0, uint4 (&v)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t r = r0 + grp + 16 * j;
      v[j] = (col_in && r < rows) ? *reinterpret_cast<const uint4 *>(in + r * pitch + c0 + 4 * sub)
                                  : uint4{0u, 0u, 0u, 0u};
    }
  };
  const int64_t left = (rows - rb + 63) / 64;  // >= 1: the grid covers the rows
  const int ntile = left < kStripTiles ? (int)left : kStripTiles;
  uint4 v[4];
  load(rb, v);
  for (int k = 0; k < ntile; ++k) {
    const int64_t r0 = rb + (int64_t)k * 64;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t *row = tile[grp + 16 * j] + 4 * sub;
      row[0] = v[j].x;
      row[1] = v[j].y;
      row[2] = v[j].z;
      row[3] = v[j].w;
    }
    __syncthreads();
    if (k + 1 < ntile) load(r0 + 64, v);
    const int64_t r = r0 + 4 * sub;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int oc = grp + 16 * j;
      if (c0 + oc < cols && r < rows)
        *reinterpret_cast<uint4 *>(out + (c0 + oc) * rows + r) =
            uint4{tile[4 * sub][oc], tile[4 * sub + 1][oc], tile[4 * sub + 2][oc], tile[4 * sub + 3][oc]};
    }
    __syncthreads();
  }
}

// Byte matrices whose sizes and input pitch are multiples of 4 (and 4-byte
// aligned input): 128 x 128 tiles moved as 4-byte words on both sides. A word
// read holds 4 columns of one row; a word written packs 4 rows of one column,
// gathered byte by byte from LDS (row pitch 33 words).  Workgroups go to the
// 8 XCDs round-robin by launch order, each XCD with its own L2; tiles are
// renumbered so that each XCD takes consecutive tiles of a row band, whose
// row segments share the 128-byte lines they straddle (the row pitch need
// not be a multiple of 128), and a line is fetched once instead of twice.
__global__ __launch_bounds__(256) void transpose_u8_words(const uint8_t *__restrict__ in, int64_t rows, int64_t cols,
                                                          int64_t pitch, uint8_t *__restrict__ out) {
  __shared__ uint32_t tile[128 * 33];
  const uint32_t gx = gridDim.x, total = gx * gridDim.y, L = blockIdx.y * gx + blockIdx.x;
  const uint32_t xcd = L % 8u, per = total / 8u, extra = total % 8u;
  const uint32_t Lr = xcd * per + min(xcd, extra) + L / 8u;  // a bijection of [0, total)
  const int64_t c0 = (int64_t)(Lr % gx) * 128, r0 = (int64_t)(Lr / gx) * 128;
  const int w = threadIdx.x & 31, i0 = threadIdx.x >> 5;
  const bool col_in = c0 + 4 * w < cols;
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int i = i0 + 8 * p;
    if (col_in && r0 + i < rows)
      tile[i * 33 + w] = *reinterpret_cast<const uint32_t *>(in + (r0 + i) * pitch + c0 + 4 * w);
  }
  __syncthreads();
  const uint8_t *t8 = reinterpret_cast<const uint8_t *>(tile);
  const int q = w;  // rows 4q..4q+3 of the tile
  const bool row_in = r0 + 4 * q < rows;
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int c = i0 + 8 * p;
    if (row_in && c0 + c < cols) {
      const uint32_t v = (uint32_t)t8[(4 * q) * 132 + c] | (uint32_t)t8[(4 * q + 1) * 132 + c] << 8 |
                         (uint32_t)t8[(4 * q + 2) * 132 + c] << 16 | (uint32_t)t8[(4 * q + 3) * 132 + c] << 24;
      *reinterpret_cast<uint32_t *>(out + (c0 + c) * rows + r0 + 4 * q) = v;
    }
  }
}

// ------------------------------------------------------------------ schedule
// link class of a transfer from device a to device b (at most two classes)
__device__ __forceinline__ uint32_t link_bit(const GmgView &G, uint32_t a, uint32_t b) {
  return (G.link_bits[a * G.link_words + (b >> 5)] >> (b & 31)) & 1u;
}

__device__ __forceinline__ uint32_t xfer_of(const GmgView &G, int u, int du, int d) {
  const int K = G.n_link;
  if (K == 1) return G.xfer32[u];
  if (K == 2) {  // both entries are wave-uniform loads
    const uint32_t k = link_bit(G, (uint32_t)du, (uint32_t)d);
    const uint32_t x0 = G.xfer32[2 * u], x1 = G.xfer32[2 * u + 1];
    return k ? x1 : x0;
  }
  return G.xfer32[u * K + G.link_class[du * G.n_dev + d]];
}

// Software pipeline of the schedule, for target op T (one lane per candidate):
//   T-4  load the op's device from the op-major placements, and the finish
//        time and device of its first kPipePre predecessors when they are op
//        T-5 or older (op-major finish times written earlier by this lane;
//        two steps pass before they are used, which covers the latency of
//        rows far back that have left the cache);
//   T-2  resolve each predecessor: ops T-4, T-3 and T-2 from a three-deep
//        register history (op T-1's device is already loaded), the rest from
//        the T-4 loads, kept for step T; gather the link class of each predecessor
//        transfer, the op's duration on its device, and the device's current
//        slice end plus the next slice's bounds;
//   T    ready time (only a predecessor T-1 still comes from the history),
//        placement, stores.
// Uniform per-op fields come from op_meta through a 64-op window that
// advances by 32 ops (lane j holds op w0+j), broadcast with one readlane
// each.  Row offsets are 32 x 32-bit products (a chunk holds fewer than 2^32
// candidates).  Stage state is indexed by
// T mod 4, static in the four-way unrolled loop.  Loads are unconditional
// (indices clamped, unused values discarded by selects) so the loop body has
// no branch around a memory operation and the compiler can keep the loads of
// later stages in flight while op T waits only for its own.
constexpr int kPipePre = 2;  // predecessors handled by the pipeline; more go through the CSR
constexpr int kRowOps = 8;   // finish times a lane gathers in registers before it writes them to its own row
constexpr int kWindowStep = 32;  // ops per advance of the op-field window

struct SchedPipe {
  uint32_t dq[4];                // device of the target op (raw byte)
  uint32_t pf[4][kPipePre];      // predecessor finish times (raw loads)
  uint32_t pd[4][kPipePre];      // predecessor devices (raw loads)
  uint32_t lc[4][kPipePre];      // link class between predecessor and target device
  uint32_t xf[4][kPipePre];      // with device groups: transfer time to the target device
  uint32_t wq[4];                // duration on the target device
  uint32_t le[4];                // time -> slice lookup entry at a lower bound of the op's finish
  uint4 lw[4];                   // its {begin, end} of slices lk and lk+1
};
// kLink: 0 = link classes from device groups (LDS), 1 = bit table (two
// classes), 2 = byte table (more classes), 3 = device groups of 2^s
// consecutive devices (group = device >> s).  With groups (0, 3) stage T-2
// computes each predecessor's transfer time itself.
template <int kLink, bool kOverflow, bool kOneClass>
__global__ __launch_bounds__(kWave) void fast_schedule(const GmgView G, const uint8_t *__restrict__ PT, int64_t ppitch,
                                                       int64_t nb,
                                                       uint32_t *__restrict__ finT, int64_t *__restrict__ makespan,
                                                       int64_t *__restrict__ sumfin, int64_t *__restrict__ slack,
                                                       uint8_t *__restrict__ violation, uint32_t *__restrict__ finR) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = kOneClass ? 1 : G.n_class, K = G.n_link;
  const int lane = threadIdx.x;
  uint32_t *clk = reinterpret_cast<uint32_t *>(lds_raw);                  // [D][64]
  uint32_t *comp = clk + (size_t)D * kWave;                               // [R][64]
  int32_t *sbase = reinterpret_cast<int32_t *>(comp + (size_t)R * kWave);  // [D+1] slice ranges of the devices
  int32_t *dcls = sbase + D + 1;                                          // [D] device class
  uint8_t *lgrp = reinterpret_cast<uint8_t *>(dcls + D);                  // [D] link group (kLink 0)
  for (int d = lane; d <= D; d += kWave) {
    sbase[d] = G.slice_ptr[d];
    if (d < D) dcls[d] = G.dev_class[d];
    if (kLink == 0 && d < D) lgrp[d] = G.link_grp[d];
  }
  const uint32_t lsame = (uint32_t)G.link_same, lshift = (uint32_t)max(G.link_shift, 0);
  constexpr bool kGroups = kLink == 0 || kLink == 3;
  __syncthreads();
  // Every lane runs (readlane needs the field blocks loaded in all lanes); a
  // lane past the batch end shadows the last candidate, computing and storing
  // exactly what that candidate's lane stores.
  const int64_t c_raw = (int64_t)blockIdx.x * kWave + lane;
  const bool live = c_raw < nb;
  const int64_t c = live ? c_raw : nb - 1;
  for (int d = 0; d < D; ++d) clk[d * kWave + lane] = G.slice_begin32[sbase[d]];
  for (int r = 0; r < R; ++r) comp[r * kWave + lane] = G.release32[r];
  if (N == 0) {
    if (live) {
      makespan[c] = 0;
      if (sumfin) sumfin[c] = 0;
      if (slack)
        for (int rr = 0; rr < R; ++rr) slack[c * R + rr] = G.deadline[rr] - (int64_t)G.release32[rr];
      violation[c] = 0;
    }
    return;
  }

  const int ms_ = G.meta_stride;
  // Fields of ops [w0, w0 + 64) in mA (lane j: op w0 + j), of [w0 + 32,
  // w0 + 96) in mB.  The window advances by 32 ops, so every op a step reads
  // (T .. T+3) lies in mA and a field costs one readlane.
  uint32_t mA[kOpMetaFields], mB[kOpMetaFields];
#pragma unroll
  for (int f = 0; f < kOpMetaFields; ++f) {
    mA[f] = G.op_meta[(int64_t)f * ms_ + lane];
    mB[f] = G.op_meta[(int64_t)f * ms_ + kWindowStep + lane];
  }
  int w0 = 0;
  auto meta = [&](int f, int t) -> uint32_t { return (uint32_t)__builtin_amdgcn_readlane((int)mA[f], t - w0); };
  auto pred_of = [](uint32_t p01, int i) -> uint32_t { return i ? (p01 >> 16) : (p01 & 0xFFFFu); };

  bool invalid = false;
  // A loaded value is left untouched until the stage that consumes it, so the
  // wait for it lands there and not right after the load.
  auto clampD = [&](uint32_t x) -> uint32_t { return x >= (uint32_t)D ? 0u : x; };
  const uint64_t nbu = (uint64_t)(uint32_t)nb;  // a chunk holds fewer than 2^32 candidates
  const uint8_t *const PTc = PT + c;
  uint32_t *const finTc = finT + c;
  uint32_t *const finRc = finR ? finR + (uint64_t)(uint32_t)c * (uint32_t)N : nullptr;
  const uint64_t ppu = (uint64_t)ppitch;  // placement rows: the caller's op-major pitch, or the chunk's
  auto row = [&](int t) -> uint64_t { return (uint64_t)(uint32_t)t * nbu; };
  auto prow = [&](int t) -> uint64_t { return (uint64_t)(uint32_t)t * ppu; };
  auto load_dev = [&](int t) -> uint32_t { return PTc[prow(t)]; };
  SchedPipe S;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    S.dq[q] = load_dev(q < N ? q : N - 1);
    S.wq[q] = S.le[q] = 0;
    S.lw[q] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < kPipePre; ++i) S.pf[q][i] = S.pd[q][i] = S.lc[q][i] = 0;
  }

  // with finR: the lane's finish times of ops 8k .. 8k+7 (op T in slot T mod 8)
  uint32_t rb[kRowOps];
#pragma unroll
  for (int k = 0; k < kRowOps; ++k) rb[k] = 0;
  // Results of the last three ops: h1 = op T (after its step), h2 and h3 before it.
  uint32_t h1f = 0, h1d = 0, h2f = 0, h2d = 0, h3f = 0, h3d = 0;

  // Stage T-2 for target op t = T+2, after op T.
  auto stage2 = [&](auto qq, int T) {
    constexpr int q1 = (decltype(qq)::value + 1) & 3, q2 = (decltype(qq)::value + 2) & 3;
    const int t = min(T + 2, N - 1);  // past the end: computed and never used
    const uint32_t dt = clampD(S.dq[q2]);
    const uint32_t p01 = meta(kMetaP01, t), np = meta(kMetaReq, t) >> 16;
    // lower bound of op t's finish: its release, the predecessors finished by
    // now (op t-1 is not) with the cheaper link class, the device clock now
    uint32_t lb = meta(kMetaRel, t);
    const uint32_t gdt = kLink == 0 ? (uint32_t)lgrp[dt] : kLink == 3 ? dt >> lshift : 0u;
#pragma unroll
    for (int i = 0; i < kPipePre; ++i) {
      const int u = (int)pred_of(p01, i);
      const uint32_t du = u == T + 1 ? clampD(S.dq[q1])
                          : u == T   ? h1d
                          : u == T - 1 ? h2d
                          : u == T - 2 ? h3d
                                       : clampD(S.pd[q2][i]);
      uint32_t lc;
      if (kLink == 0) lc = (uint32_t)lgrp[du] == gdt ? lsame : 1u - lsame;
      else if (kLink == 3) lc = du >> lshift == gdt ? lsame : 1u - lsame;
      else if (kLink == 1) lc = link_bit(G, du, dt);  // zero with one class
      else lc = G.link_class[du * D + dt];
      S.lc[q2][i] = lc;
      const uint32_t fu = u == T ? h1f : u == T - 1 ? h2f : u == T - 2 ? h3f : S.pf[q2][i];
      // resolved for the step (a predecessor T+1 takes its finish from the
      // step's history; its device is already final)
      S.pd[q2][i] = du;
      S.pf[q2][i] = fu;
      // transfer time in the bound: exact with device groups, else the
      // cheapest class (the fields hold classes 0 and 1), else none
      const uint32_t x0 = meta(kMetaX + 2 * i, t), x1 = meta(kMetaX + 2 * i + 1, t);
      const uint32_t xm = kGroups ? (lc ? x1 : x0) : kLink == 1 ? min(x0, x1) : 0u;
      const uint32_t xe = du != dt ? xm : 0u;
      if (kGroups) S.xf[q2][i] = xe;  // exact
      lb = ((uint32_t)i < np && u != T + 1) ? umax32(lb, fu + xe) : lb;
    }
    S.wq[q2] = kOneClass ? meta(kMetaDur, t) : G.dur32[(int64_t)t * C + dcls[dt]];
    lb = umax32(lb, clk[(int)dt * kWave + lane]) + (kOneClass ? meta(kMetaDur, t) : 0u);
    const uint32_t e = dt * (uint32_t)G.lut_nb + (uint32_t)min((int)(lb >> G.lut_shift), G.lut_nb - 1);
    S.le[q2] = e;
    S.lw[q2] = G.lut_w[e];
  };
  // Stage T-4 for target op t = T+4: predecessors u <= T-1 (the others are
  // forwarded from the register history when op t runs).
  auto stage3 = [&](auto qq, int T) {
    constexpr int q3 = decltype(qq)::value;
    const int t = min(T + 4, N - 1);
    const uint32_t p01 = meta(kMetaP01, t);
#pragma unroll
    for (int i = 0; i < kPipePre; ++i) {
      const int u = (int)pred_of(p01, i);
      const int us = u < T ? u : 0;  // rows not yet written (or absent) read row 0, never used
      S.pf[q3][i] = finTc[row(us)];
      S.pd[q3][i] = PTc[prow(us)];
    }
  };

  uint32_t ms = 0;
  uint64_t sum = 0;
  stage2(std::integral_constant<int, 2>(), -2);
  stage2(std::integral_constant<int, 3>(), -1);
  stage3(std::integral_constant<int, 2>(), -2);  // ops 2 and 3: every predecessor comes from the history
  stage3(std::integral_constant<int, 3>(), -1);

  auto step = [&](auto qq, int T) {
    constexpr int q0 = decltype(qq)::value;
    const uint32_t draw = S.dq[q0];
    invalid |= draw >= (uint32_t)D;
    const uint32_t d = clampD(draw);
    const int slot = (int)d * kWave + lane;
    uint32_t s = clk[slot];
    const uint32_t rq = meta(kMetaReq, T), np = rq >> 16;
    const int r = (int)(rq & 0xFFFFu);
    const uint32_t w = S.wq[q0];
    uint32_t ready = meta(kMetaRel, T);
    const uint32_t p01 = meta(kMetaP01, T);
#pragma unroll
    for (int i = 0; i < kPipePre; ++i) {
      const int u = (int)pred_of(p01, i);
      const uint32_t tt = u == T - 1 ? h1f : S.pf[q0][i];
      const uint32_t du = S.pd[q0][i];
      uint32_t x;
      if (kGroups) {
        x = S.xf[q0][i];  // zero on the same device
      } else if (kLink == 2) {
        x = G.xfer32[(int64_t)(u < T ? u : 0) * K + S.lc[q0][i]];
      } else {
        const uint32_t x0 = meta(kMetaX + 2 * i, T), x1 = meta(kMetaX + 2 * i + 1, T);
        x = S.lc[q0][i] ? x1 : x0;
      }
      const uint32_t a = tt + (kGroups || du != d ? x : 0u);
      ready = (uint32_t)i < np ? umax32(ready, a) : ready;
    }
    if (kOverflow && np > (uint32_t)kPipePre) {  // predecessors past the pipelined ones
      const int e0 = (int)meta(kMetaE0, T);
      for (int e = e0 + kPipePre; e < e0 + (int)np; ++e) {
        const int u = G.pred_idx[e];
        uint32_t tt, du;
        if (u == T - 1) {
          tt = h1f;
          du = h1d;
        } else {
          tt = finTc[row(u)];
          du = PTc[prow(u)];
          if (du >= (uint32_t)D) du = 0;
        }
        if (du != d) tt += xfer_of(G, u, (int)du, (int)d);
        ready = umax32(ready, tt);
      }
    }
    // One op at a time, in the first idle slice that holds it from its ready
    // time and the device clock on.  Slices before lk end before the lookup
    // bucket starts, hence before any finish the op can have; slices that
    // end before the clock cannot hold it either (durations are >= 1), so
    // the answer is the first of lk, lk+1, ... that fits, almost always one
    // of the two whose bounds are already in registers.
    s = umax32(s, ready);
    {
      const uint4 lw = S.lw[q0];
      const uint32_t t0 = umax32(s, lw.x), t1 = umax32(s, lw.z);
      if (t0 + w <= lw.y) {
        s = t0;
      } else if (t1 + w <= lw.w) {
        s = t1;
      } else {
        const int sb = sbase[d];
        for (int k = (int)G.lut_k[S.le[q0]] + 2;; ++k) {
          const uint32_t t = umax32(s, G.slice_begin32[sb + k]);
          if (t + w <= G.slice_end32[sb + k]) {
            s = t;
            break;
          }
        }
      }
    }
    const uint32_t f = s + w;
    clk[slot] = f;
    finTc[row(T)] = f;
    if (finRc) {  // the candidate's own row, kRowOps finish times at a time
      // T mod 4 is q0 (steps come four to a block that starts at a multiple
      // of 4), so the slot is q0 or q0 + 4 by the wave-uniform bit T & 4
      const bool hi = (T & 4) != 0;
      rb[q0] = hi ? rb[q0] : f;
      rb[q0 + 4] = hi ? f : rb[q0 + 4];
      if (q0 == 3 && hi) {
        uint4 *dst = reinterpret_cast<uint4 *>(finRc + (T - (kRowOps - 1)));
        dst[0] = make_uint4(rb[0], rb[1], rb[2], rb[3]);
        dst[1] = make_uint4(rb[4], rb[5], rb[6], rb[7]);
      }
    }
    atomicMax(&comp[r * kWave + lane], f);
    ms = umax32(ms, f);
    sum += f;
    h3f = h2f;
    h3d = h2d;
    h2f = h1f;
    h2d = h1d;
    h1f = f;
    h1d = d;
    stage2(qq, T);
    stage3(qq, T);
    S.dq[q0] = load_dev(min(T + 4, N - 1));
  };

  const int n_main = N / kWindowStep * kWindowStep;
  for (; w0 < n_main; w0 += kWindowStep) {
    if (w0 > 0) {
#pragma unroll
      for (int f = 0; f < kOpMetaFields; ++f) {
        mA[f] = mB[f];
        mB[f] = G.op_meta[(int64_t)f * ms_ + min(w0 + kWindowStep + lane, ms_ - 1)];
      }
    }
    for (int T = w0; T < w0 + kWindowStep; T += 4) {
      step(std::integral_constant<int, 0>(), T);
      step(std::integral_constant<int, 1>(), T + 1);
      step(std::integral_constant<int, 2>(), T + 2);
      step(std::integral_constant<int, 3>(), T + 3);
    }
  }
  if (n_main < N) {  // last partial block
    if (n_main > 0) {
#pragma unroll
      for (int f = 0; f < kOpMetaFields; ++f) mA[f] = mB[f];
    }
    w0 = n_main;
    for (int T = n_main; T < N; T += 4) {
      step(std::integral_constant<int, 0>(), T);
      if (T + 1 < N) step(std::integral_constant<int, 1>(), T + 1);
      if (T + 2 < N) step(std::integral_constant<int, 2>(), T + 2);
      if (T + 3 < N) step(std::integral_constant<int, 3>(), T + 3);
    }
  }
  if (finRc) {  // the last N mod kRowOps finish times
#pragma unroll
    for (int k = 0; k < kRowOps; ++k)
      if (k < (N & (kRowOps - 1))) finRc[(N & ~(kRowOps - 1)) + k] = rb[k];
  }
  if (!live) return;
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

// ------------------------------------------------------------------ ready-time dispatch
// The dispatch rule of Sec. 3.3.2: among the ops whose predecessors have all
// been scheduled, the one with the earliest ready time runs next (ties to the
// lower index), at the earliest fit on its device at or after max(ready time,
// the device's previous finish).  One wave per candidate.  Ready ops are keys
// ready << 16 | op (unique, so the order is total).  They live in the lanes'
// registers (kReadySlots per lane); when those are full they go to the
// candidate's spill list in global memory (at most N entries: ready ops form
// an antichain), which is scanned while non-empty.  Sources (no predecessors)
// come from a presorted list instead.  The next op is the smallest key of the
// three.  The wave writes the finish times (candidate rows), each op's rank
// among its device's ops in dispatch order (the order the memory pass needs),
// and the per-candidate outputs.
constexpr int kReadySlots = 4;

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
  for (int o = kWave / 2; o >= 1; o >>= 1) {
    const uint64_t y = __shfl_xor(x, o, kWave);
    x = y < x ? y : x;
  }
  return x;
}

__global__ __launch_bounds__(kWave) void ready_schedule(const GmgView G, const uint8_t *__restrict__ P,
                                                        uint32_t *__restrict__ fin, uint16_t *__restrict__ rank,
                                                        uint16_t *__restrict__ missing, uint64_t *__restrict__ spill,
                                                        int64_t *__restrict__ makespan, int64_t *__restrict__ sumfin,
                                                        int64_t *__restrict__ slack, uint8_t *__restrict__ violation,
                                                        const uint32_t *__restrict__ only) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class;
  const int lane = threadIdx.x;
  if (only && only[blockIdx.x] == 0) return;  // candidates the lane kernel has already placed
  uint32_t *clk = reinterpret_cast<uint32_t *>(lds_raw);  // [D]
  uint32_t *comp = clk + D;                               // [R]
  uint32_t *cnt = comp + R;                               // [D] ops dispatched per device
  int32_t *sbase = reinterpret_cast<int32_t *>(cnt + D);  // [D+1]
  int32_t *dcls = sbase + D + 1;                          // [D]
  const int64_t c = blockIdx.x;
  const uint8_t *prow = P + c * N;
  uint32_t *frow = fin + c * N;
  uint16_t *rrow = rank + c * N;
  uint16_t *mrow = missing + c * N;
  uint64_t *srow = spill + c * N;
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
  for (int d = lane; d <= D; d += kWave) {
    sbase[d] = G.slice_ptr[d];
    if (d < D) {
      dcls[d] = G.dev_class[d];
      cnt[d] = 0;
    }
  }
  for (int r = lane; r < R; r += kWave) comp[r] = G.release32[r];
  const uint32_t *indeg = G.op_meta + (int64_t)kMetaReq * G.meta_stride;  // predecessor count << 16
  for (int v = lane; v < N; v += kWave) mrow[v] = (uint16_t)(indeg[v] >> 16);
  wave_lds_fence();
  for (int d = lane; d < D; d += kWave) clk[d] = G.slice_begin32[sbase[d]];
  __syncthreads();  // LDS state and the missing-predecessor row before the loop reads them

  constexpr uint64_t kNone = ~0ull;
  uint64_t slot[kReadySlots];
#pragma unroll
  for (int k = 0; k < kReadySlots; ++k) slot[k] = kNone;
  int sp = 0, ns = 0;  // next source, spill length (wave-uniform)
  uint32_t ms = 0;
  uint64_t sum = 0;
  for (int step = 0; step < N; ++step) {
    uint64_t my = slot[0];
#pragma unroll
    for (int k = 1; k < kReadySlots; ++k) my = slot[k] < my ? slot[k] : my;
    const uint64_t wm = wave_min_u64(my);
    uint64_t sm = kNone;
    int si = 0;
    if (ns > 0) {  // smallest spilled key and its position
      uint64_t lm = kNone;
      int li = 0;
      for (int i = lane; i < ns; i += kWave) {
        const uint64_t k = srow[i];
        li = k < lm ? i : li;
        lm = k < lm ? k : lm;
      }
      sm = wave_min_u64(lm);
      if (sm != kNone) si = __shfl(li, __ffsll((unsigned long long)__ballot(lm == sm)) - 1, kWave);
    }
    const uint64_t sk = sp < G.n_src ? G.src_keys[sp] : kNone;
    uint64_t key;
    if (sk < wm && sk < sm) {
      key = sk;
      ++sp;
    } else if (sm < wm) {
      key = sm;
      --ns;
      if (lane == 0) srow[si] = srow[ns];  // the last entry fills the hole
    } else {
      key = wm;
      const int owner = __ffsll((unsigned long long)__ballot(my == wm)) - 1;
      if (lane == owner) {
        bool done = false;
#pragma unroll
        for (int k = 0; k < kReadySlots; ++k)
          if (!done && slot[k] == wm) {
            slot[k] = kNone;
            done = true;
          }
      }
    }
    const int v = (int)(key & 0xFFFFu);
    const uint32_t ready = (uint32_t)(key >> 16);
    const int d = prow[v];
    const uint32_t w = G.dur32[(int64_t)v * C + dcls[d]];
    uint32_t s = umax32(ready, clk[d]);
    {  // the first idle slice that holds [s', s' + w) with s' >= s; slices
       // before the table's entry end before s + w
      const uint32_t e = (uint32_t)d * (uint32_t)G.lut_nb + (uint32_t)min((int)((s + w) >> G.lut_shift), G.lut_nb - 1);
      const uint4 lw = G.lut_w[e];
      const uint32_t t0 = umax32(s, lw.x), t1 = umax32(s, lw.z);
      if (t0 + w <= lw.y) {
        s = t0;
      } else if (t1 + w <= lw.w) {
        s = t1;
      } else {
        const int sb = sbase[d];
        for (int k = (int)G.lut_k[e] + 2;; ++k) {
          const uint32_t t = umax32(s, G.slice_begin32[sb + k]);
          if (t + w <= G.slice_end32[sb + k]) {
            s = t;
            break;
          }
        }
      }
    }
    const uint32_t f = s + w;
    const int r = G.op_req[v];
    const uint32_t rk = cnt[d];
    wave_lds_fence();
    if (lane == 0) {
      clk[d] = f;
      cnt[d] = rk + 1;
      comp[r] = umax32(comp[r], f);
      frow[v] = f;
      rrow[v] = (uint16_t)rk;
    }
    __threadfence_block();  // the wave reads these back in later steps
    ms = umax32(ms, f);
    sum += f;
    // successors whose last missing predecessor this was become ready
    for (int q = G.succ_ptr[v]; q < G.succ_ptr[v + 1]; ++q) {
      const int x = G.succ_idx[q];
      const int left = (int)mrow[x] - 1;
      if (lane == 0) mrow[x] = (uint16_t)left;
      __threadfence_block();
      if (left == 0) {
        const int dx = prow[x];
        uint32_t rx = G.release32[G.op_req[x]];
        for (int e = G.pred_ptr[x]; e < G.pred_ptr[x + 1]; ++e) {
          const int u = G.pred_idx[e];
          const int du = prow[u];
          uint32_t t = u == v ? f : frow[u];
          if (du != dx) t += xfer_of(G, u, du, dx);
          rx = umax32(rx, t);
        }
        const uint64_t nk = (uint64_t)rx << 16 | (uint64_t)x;
        bool placed = false;
#pragma unroll
        for (int k = 0; k < kReadySlots; ++k) {
          if (!placed) {
            const unsigned long long free_lanes = __ballot(slot[k] == kNone);
            if (free_lanes) {
              if (lane == __ffsll(free_lanes) - 1) slot[k] = nk;
              placed = true;
            }
          }
        }
        if (!placed) {
          if (lane == 0) srow[ns] = nk;
          ++ns;
          __threadfence_block();
        }
      }
    }
  }
  if (lane == 0) {
    makespan[c] = ms;
    if (sumfin) sumfin[c] = (int64_t)sum;
    violation[c] = 0;
  }
  if (slack)
    for (int rr = lane; rr < R; rr += kWave) slack[c * R + rr] = G.deadline[rr] - (int64_t)comp[rr];
}

size_t ready_schedule_lds(int D, int R) { return (size_t)(3 * D + R + 1 + D) * 4; }

// The same rule with one lane per candidate (64 candidates per wave): the
// ready set is a lane's own, kLaneSlots keys in registers; device clocks and
// request completions in LDS [device or request][lane]; ranks per device in
// global scratch [device][candidate]; finish times and ranks in the
// candidate rows the memory pass reads.  An op is ready when none of its
// predecessors' finish times is still unset (the rows start cleared), so no
// per-op counters are kept.  A candidate whose ready set outgrows the slots
// is flagged (ovf) and handed to ready_schedule, which redoes it whole; a
// placement naming a device >= D is walked on device 0 and reported invalid.
constexpr int kLaneSlots = 32;
constexpr uint32_t kFinUnset = 0xFFFFFFFFu;  // above every finish (the horizon is below 2^32 - 1)

// kPacked (0, 2 or 4): with at most two successors per op (succ2) and at most
// kPacked predecessors, an op's successors and their predecessors, requests
// and releases come from the packed per-op fields, all loaded unconditionally
// (indices clamped, results discarded when unused) so that a step waits for
// three levels of dependent loads; 0 walks the CSR lists.
template <int kPacked>
__global__ __launch_bounds__(kWave) void ready_lanes(const GmgView G, const uint8_t *__restrict__ P, int64_t nb,
                                                     uint32_t *__restrict__ fin, uint16_t *__restrict__ rank,
                                                     uint16_t *__restrict__ cnt, uint32_t *__restrict__ ovf,
                                                     int64_t *__restrict__ makespan, int64_t *__restrict__ sumfin,
                                                     int64_t *__restrict__ slack, uint8_t *__restrict__ violation) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const int D = G.n_dev, N = G.n_ops, R = G.n_req, C = G.n_class;
  uint32_t *clk = reinterpret_cast<uint32_t *>(lds_raw);  // [D][64]
  uint32_t *comp = clk + (size_t)D * kWave;                // [R][64]
  const int lane = threadIdx.x;
  const int64_t c0 = (int64_t)blockIdx.x * kWave, c = c0 + lane;
  const int rows = (int)min<int64_t>(kWave, nb - c0);
  for (int r = 0; r < rows; ++r) {  // the wave clears its candidates' finish rows, coalesced
    uint32_t *fr = fin + (c0 + r) * N;
    for (int v = lane; v < N; v += kWave) fr[v] = kFinUnset;
  }
  for (int d = 0; d < D; ++d) clk[d * kWave + lane] = 0;
  for (int r = 0; r < R; ++r) comp[r * kWave + lane] = G.release32[r];
  const bool act = c < nb;
  if (act)
    for (int d = 0; d < D; ++d) cnt[(int64_t)d * nb + c] = 0;
  __syncthreads();  // every row cleared before a lane reads its own
  if (!act) return;
  const uint8_t *prow = P + c * N;
  uint32_t *frow = fin + c * N;
  uint16_t *rrow = rank + c * N;
  const int64_t ms_ = G.meta_stride;
  const uint32_t *m_req = G.op_meta + kMetaReq * ms_, *m_rel = G.op_meta + kMetaRel * ms_,
                 *m_p01 = G.op_meta + kMetaP01 * ms_, *m_p23 = G.op_meta + kMetaP23 * ms_;
  constexpr uint64_t kNone = ~0ull;
  uint64_t slot[kLaneSlots];
#pragma unroll
  for (int k = 0; k < kLaneSlots; ++k) slot[k] = kNone;
  int sp = 0;
  uint64_t sk = G.n_src > 0 ? G.src_keys[0] : kNone;  // the next source's key, loaded a step ahead
  bool bad = false, over = false;
  uint32_t ms = 0;
  uint64_t sum = 0;
  // a ready key for successor x of v (finish f) when none of x's
  // predecessors is unset, else kNone
  auto ready_key = [&](int x, int v, uint32_t f, int dx, uint32_t rel, int np, const int *pu) -> uint64_t {
    uint32_t rx = rel;
    bool ok = true;
#pragma unroll
    for (int i = 0; i < (kPacked ? kPacked : 1); ++i) {
      const bool use = i < np;
      const int u = use ? pu[i] : v;  // loads from a valid op either way
      uint32_t t = u == v ? f : frow[u];
      int du = prow[u];
      if (du >= D) du = 0;
      if (du != dx) t += xfer_of(G, u, du, dx);
      ok &= !use || frow[u] != kFinUnset || u == v;
      if (use) rx = umax32(rx, t);
    }
    return ok ? ((uint64_t)rx << 16 | (uint64_t)x) : kNone;
  };
  auto insert = [&](uint64_t nk) {
    bool placed = false;
#pragma unroll
    for (int k = 0; k < kLaneSlots; ++k)
      if (!placed && slot[k] == kNone) {
        slot[k] = nk;
        placed = true;
      }
    over |= !placed;
  };
  for (int step = 0; step < N && !over; ++step) {
    uint64_t my = slot[0];
#pragma unroll
    for (int k = 1; k < kLaneSlots; ++k) my = slot[k] < my ? slot[k] : my;
    uint64_t key;
    if (sk < my) {
      key = sk;
      ++sp;
      sk = sp < G.n_src ? G.src_keys[sp] : kNone;
    } else {
      key = my;
      bool done = false;
#pragma unroll
      for (int k = 0; k < kLaneSlots; ++k)
        if (!done && slot[k] == my) {
          slot[k] = kNone;
          done = true;
        }
    }
    if (key == kNone) {  // nothing ready before every op ran: only after a lost key
      over = true;
      break;
    }
    const int v = (int)(key & 0xFFFFu);
    const uint32_t ready = (uint32_t)(key >> 16);
    // the successors' fields, requested before the placement needs them
    uint32_t s2 = 0, xs[2] = {0, 0}, xreq[2], xrel[2], xp01[2], xp23[2];
    int xd[2];
    if (kPacked) {
      s2 = G.succ2[v];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint32_t x = (s2 >> (16 * i)) & 0xFFFFu;
        xs[i] = x == 0xFFFFu ? 0u : x;
        xreq[i] = m_req[xs[i]];
        xrel[i] = m_rel[xs[i]];
        xp01[i] = m_p01[xs[i]];
        xp23[i] = kPacked > 2 ? m_p23[xs[i]] : 0xFFFFFFFFu;
        xd[i] = prow[xs[i]];
      }
    }
    int d = prow[v];
    if (d >= D) {
      bad = true;
      d = 0;
    }
    const uint32_t w = C == 1 ? G.dur32[v] : G.dur32[(int64_t)v * C + G.dev_class[d]];
    uint32_t s = umax32(ready, clk[d * kWave + lane]);
    {  // the first idle slice that holds [s', s' + w) with s' >= s
      const uint32_t e = (uint32_t)d * (uint32_t)G.lut_nb + (uint32_t)min((int)((s + w) >> G.lut_shift), G.lut_nb - 1);
      const uint4 lw = G.lut_w[e];
      const uint32_t t0 = umax32(s, lw.x), t1 = umax32(s, lw.z);
      if (t0 + w <= lw.y) {
        s = t0;
      } else if (t1 + w <= lw.w) {
        s = t1;
      } else {
        const int sb = G.slice_ptr[d];
        for (int k = (int)G.lut_k[e] + 2;; ++k) {
          const uint32_t t = umax32(s, G.slice_begin32[sb + k]);
          if (t + w <= G.slice_end32[sb + k]) {
            s = t;
            break;
          }
        }
      }
    }
    const uint32_t f = s + w;
    clk[d * kWave + lane] = f;
    uint16_t *cd = cnt + (int64_t)d * nb + c;
    const uint16_t rk = *cd;
    *cd = (uint16_t)(rk + 1);
    rrow[v] = rk;
    frow[v] = f;
    uint32_t *cr = comp + (m_req[v] & 0xFFFFu) * kWave + lane;
    *cr = umax32(*cr, f);
    ms = umax32(ms, f);
    sum += f;
    // successors whose last unset predecessor this was become ready
    if (kPacked) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        if (((s2 >> (16 * i)) & 0xFFFFu) != 0xFFFFu) {
          int dx = xd[i];
          if (dx >= D) dx = 0;
          const int pu[4] = {(int)(xp01[i] & 0xFFFFu), (int)(xp01[i] >> 16), (int)(xp23[i] & 0xFFFFu),
                             (int)(xp23[i] >> 16)};
          const uint64_t nk = ready_key((int)xs[i], v, f, dx, xrel[i], (int)(xreq[i] >> 16), pu);
          if (nk != kNone) insert(nk);
        }
      }
    } else {
      const int q1 = G.succ_ptr[v + 1];
      for (int q = G.succ_ptr[v]; q < q1; ++q) {
        const int x = G.succ_idx[q];
        int dx = prow[x];
        if (dx >= D) dx = 0;
        uint32_t rx = G.release32[G.op_req[x]];
        bool ok = true;
        const int e1 = G.pred_ptr[x + 1];
        for (int e = G.pred_ptr[x]; e < e1; ++e) {
          const int u = G.pred_idx[e];
          uint32_t t = u == v ? f : frow[u];
          if (t == kFinUnset) {
            ok = false;
            break;
          }
          int du = prow[u];
          if (du >= D) du = 0;
          if (du != dx) t += xfer_of(G, u, du, dx);
          rx = umax32(rx, t);
        }
        if (ok) insert((uint64_t)rx << 16 | (uint64_t)x);
      }
    }
  }
  ovf[c] = over ? 1u : 0u;
  if (over) return;  // ready_schedule writes this candidate's outputs
  if (bad) {
    makespan[c] = INT64_MAX;
    if (sumfin) sumfin[c] = INT64_MAX;
    if (slack)
      for (int r = 0; r < R; ++r) slack[c * R + r] = INT64_MIN;
    violation[c] = SS_VIOLATION_INVALID;
    return;
  }
  makespan[c] = ms;
  if (sumfin) sumfin[c] = (int64_t)sum;
  violation[c] = 0;
  if (slack)
    for (int r = 0; r < R; ++r) slack[c * R + r] = G.deadline[r] - (int64_t)comp[r * kWave + lane];
}

// ------------------------------------------------------------------ memory
// Residency intervals (Sec. 3.3.2) are written by fast_intervals into
// per-device buckets and evaluated by fast_peaks.
//   own record  {start, free time (kInf32: never), bytes, free locator}
//   copy record {allocation time, free time, bytes, alloc window << 16 | free gap}
// A device's own starts S[0..m) (its ops in index order) are sorted, and
// every event is placed by how many own starts precede it, its gap:
//   allocation of a copy at time c:  #{k : S[k] <= c}
//   free at time h:                  #{k : S[k] <  h}
// (frees precede allocations at equal times: intervals are half-open).  The
// writer knows each gap exactly or nearly: a free at the finish of a local
// op of rank k has gap k + 1 (durations are at least 1); a copy is allocated
// shortly before its first consumer of rank k starts, so its gap lies in
// [k-3, k+1]; a transfer-bound free of an op of rank k lies in [k+1, k+5].
// A locator holds the exact gap, or (kLocWindow) the start L of a window
// [L, L+4] that is checked and, if the gap lies outside, replaced by a
// binary search.
using Rec = uint4;
constexpr uint32_t kLocWindow = 0x80000000u;

// Records per candidate: own N plus a spare at index N, copies at most E plus
// a spare at E, each region rounded to whole blocks of kBlockRecs records so
// that every candidate's regions start on a block.
constexpr int kBlockShift = 2, kBlockRecs = 1 << kBlockShift;  // 64-byte lines
__host__ __device__ __forceinline__ int64_t own_stride(int64_t N) {
  return (N + 1 + kBlockRecs - 1) & ~int64_t(kBlockRecs - 1);
}
__host__ __device__ __forceinline__ int64_t cp_stride(int64_t E) {
  return (E + 1 + kBlockRecs - 1) & ~int64_t(kBlockRecs - 1);
}

__device__ __forceinline__ uint32_t loc_window(int L) { return kLocWindow | (uint32_t)max(L, 0); }

// Intervals of op v (device d, rank rv among the ops of d): its own output at
// slot own_pos of d's bucket, one copy per remote destination device (slot
// taken with an LDS atomic).
__device__ void op_intervals(const GmgView &G, const uint8_t *prow, const uint32_t *frow, const uint16_t *rk, int v,
                             int d, int rv, int own_pos, int *cfill, Rec *own, Rec *cp) {
  const int C = G.n_class;
  const uint32_t b = G.bytes32[v];
  const int x0 = G.succ_ptr[v], x1 = G.succ_ptr[v + 1];
  const uint32_t f = frow[v];
  uint32_t F = kInf32, loc = 0;  // kept forever without consumers
  if (x1 > x0) {
    // the local consumer that finishes last (with index-order dispatch: the last one)
    uint32_t L = f, A = 0;
    int rl = rv;
    for (int q = x0; q < x1; ++q) {
      const int x = G.succ_idx[q];
      const int dx = prow[x];
      if (dx == d) {
        if (frow[x] > L) {
          L = frow[x];
          rl = rk[x];
        }
      } else {
        A = umax32(A, f + xfer_of(G, v, d, dx));
      }
    }
    if (A > L) {
      F = A;
      loc = loc_window(rv + 1);
    } else {
      F = L;
      loc = (uint32_t)(rl + 1);
    }
  }
  own[own_pos] = Rec{f - (C == 1 ? G.dur32[v] : G.dur32[v * C + G.dev_class[d]]), F, b, loc};
  if (b == 0) return;
  for (int q = x0; q < x1; ++q) {
    const int xf = G.succ_idx[q];
    const int e = prow[xf];
    if (e == d) continue;
    bool first = true;
    for (int q2 = x0; q2 < q; ++q2)
      if (prow[G.succ_idx[q2]] == e) first = false;
    if (!first) continue;
    // the copy is allocated before the consumer on e that starts first (lowest
    // rank) and lives until the consumer on e that finishes last
    int y = xf, ra = rk[xf];
    for (int q2 = q + 1; q2 < x1; ++q2) {
      const int x = G.succ_idx[q2];
      if (prow[x] == e) {
        if (frow[x] > frow[y]) y = x;
        ra = min(ra, (int)rk[x]);
      }
    }
    const int ry = rk[y];
    cp[atomicAdd(&cfill[e], 1)] = Rec{f, frow[y], b, (uint32_t)max(ra - 3, 0) << 16 | (uint32_t)(ry + 1)};
  }
}

// Per-candidate bucket geometry written by fast_intervals, read by fast_peaks.
__device__ __forceinline__ int meta_stride(int D) { return 3 * (D + 1); }

// One wave per candidate.  Pass A ranks every op among the ops of its device
// (rank table rk) and counts ops and in-degrees per device (copies landing on
// a device are at most its summed in-degree); pass B writes the records.
// Each candidate's own and copy regions hold one spare record past the end
// (index N, resp. E) that absorbs the stores of lanes with nothing to write.
//
// kFast (one device class, at most two link classes, at most two successors
// per op): pass B is branch free, reads each op's successors from succ2, and
// software-pipelines the chunks of 64 ops: while chunk i is evaluated, the
// op fields of chunk i+1 are in flight, and its successors' fields are
// requested as soon as those arrive.
struct IvOp {  // fields of the lane's op
  uint32_t d, rv, f, b, w, s2, x0, x1, pe;
};
struct IvSucc {  // device, finish and rank of the first two successors (with ports: their inputs' arrivals)
  uint32_t dx0, dx1, fx0, fx1, rx0, rx1, ax0, ax1;
};

// Store staging of the own records.  A block of a bucket holds the records
// of positions 2L, 2L+1.  A device's own records of one chunk have
// consecutive positions [first, last], and with index ranks no later chunk
// writes below them, so block L of a bucket [start, end) is complete once
// position min(2L+1, end-1) has been produced.  A record's role:
//   open   its block began in an earlier chunk: staged in LDS; the record
//          that completes the block (close) queues it for a cooperative write
//   direct its block lies inside this chunk's run and is complete: stored
//   tail   its block begins in this chunk and is not complete: staged
// Copies (kStageCp) are staged the same way, a block per destination device,
// when the pass runs alone; beside the peak pass on a second stream they are
// stored directly, since there the LDS of their blocks costs more occupancy
// than the whole blocks save.
constexpr int kRoleNone = 0, kRoleDirect = 1, kRoleOpen = 2, kRoleClose = 6, kRoleTail = 8;

template <int kShift>
__device__ __forceinline__ int line_role(int p, int first, int last, int end) {
  constexpr int kRecs = 1 << kShift;
  const int L = p >> kShift, Lo = first >> kShift, Ll = last >> kShift;
  if (L == Lo) {
    const int closer = min((Lo << kShift) + kRecs - 1, end - 1);
    return (closer <= last && p == closer) ? kRoleClose : kRoleOpen;
  }
  const bool done = (L << kShift) + kRecs - 1 <= last || (last == end - 1 && L == Ll);
  return done ? kRoleDirect : kRoleTail;
}

// Staged blocks: records in 32-byte pairs (a smaller stage leaves more waves
// per CU, which this kernel needs).
constexpr int kOwnShift = 1, kOwnRecs = 1 << kOwnShift;
constexpr int kCpShift = 1, kCpRecs = 1 << kCpShift;

// kGivenRanks: the rank table already holds every op's rank on its device
// (dispatch order), pass A only counts.  kShiftLinks (with kFast): link
// classes follow contiguous device groups of 2^s devices, so a transfer's
// class comes from the two device ids instead of the bit table.  kPorts (with
// kFast, index ranks): transfers were arbitrated over device ports, and arr
// holds every candidate's arrival per predecessor edge (rows of E, like fin):
// an own output is kept until its last remote arrival, a copy is allocated at
// its transfer's start (arrival minus estimate).
template <bool kFast, bool kGivenRanks, bool kShiftLinks, bool kPorts, bool kStageCp>
__global__ __launch_bounds__(kWave) void fast_intervals(const GmgView G, const uint8_t *__restrict__ P,
                                                        const uint32_t *__restrict__ fin, int64_t j0,
                                                        Rec *__restrict__ own_all, Rec *__restrict__ cp_all,
                                                        int32_t *__restrict__ meta, uint16_t *__restrict__ rank_all,
                                                        const uint8_t *__restrict__ violation,
                                                        const uint32_t *__restrict__ arr) {
  // LDS (dynamic, sized by the device count): bucket offsets and fill
  // pointers; with staged stores (kFast with index ranks) also the open block
  // of every device's own bucket (and copy bucket) and the queues of complete
  // blocks
  constexpr bool kStage = kFast && !kGivenRanks;
  constexpr bool kCpSt = kStage && kStageCp;
  extern __shared__ __align__(16) unsigned char iv_lds[];
  const int Dv = G.n_dev;
  Rec *obuf = reinterpret_cast<Rec *>(iv_lds);                           // [D][kOwnRecs]
  Rec *cbuf = obuf + (kStage ? kOwnRecs * Dv : 0);                       // [D][kCpRecs]
  int *own_off = reinterpret_cast<int *>(cbuf + (kCpSt ? kCpRecs * Dv : 0));  // [D+1]
  int *cp_off = own_off + Dv + 1;                                          // [D+1]
  int *cfill = cp_off + Dv + 1;                                            // [D] next copy slot
  int *base = cfill + Dv;  // [D] ops counted so far; with staging then the next own position
  int *nocopy = base + Dv;                                                 // [64]
  uint32_t *fq = reinterpret_cast<uint32_t *>(nocopy + kWave);  // [64] own blocks to write
  uint32_t *fc = fq + kWave;                                    // [128] copy blocks to write
  int &fqn = *reinterpret_cast<int *>(fc + (kCpSt ? 2 * kWave : 0));
  int &fcn = *(&fqn + 1);
  // pass A's masks of the lanes on each device: on the own-record stage (not
  // used before pass B), else past the end
  uint64_t *dmask = kStage ? reinterpret_cast<uint64_t *>(obuf)
                           : reinterpret_cast<uint64_t *>((reinterpret_cast<uintptr_t>(&fcn + 1) + 7) & ~uintptr_t(7));
  const int D = G.n_dev, N = G.n_ops, E = G.pred_ptr[G.n_ops], K = G.n_link;
  const int lane = threadIdx.x;
  const int64_t j = blockIdx.x, c = j0 + j;
  if (violation[c] & SS_VIOLATION_INVALID) return;
  const uint8_t *prow = P + c * N;
  const uint32_t *frow = fin + c * N;
  const uint32_t *arow = kPorts ? arr + c * E : nullptr;
  uint16_t *rk = rank_all + j * N;
  Rec *own = own_all + j * own_stride(N);
  Rec *cp = cp_all + j * cp_stride(E);
  const uint32_t *indeg_f = G.op_meta + (int64_t)kMetaReq * G.meta_stride;  // predecessor count << 16
  for (int d = lane; d < D; d += kWave) {
    cfill[d] = 0;
    base[d] = 0;
    dmask[d] = 0;
  }
  wave_lds_fence();
  {
    int vn = min(lane, N - 1);
    uint32_t dn = N > 0 ? prow[vn] : 0, in = N > 0 ? indeg_f[vn] : 0;
    for (int v0 = 0; v0 < N; v0 += kWave) {
      const int v = v0 + lane;
      const bool act = v < N;
      const int d = (int)dn, indeg = act ? (int)(in >> 16) : 0;
      vn = min(v0 + kWave + lane, N - 1);  // next chunk, in flight meanwhile
      dn = prow[vn];
      in = indeg_f[vn];
      if (!kGivenRanks) {  // rank = ops of d so far + lower lanes of this chunk on d
        // the lanes on d: each lane sets its bit in d's mask, reads the mask
        // back once every lane has, and clears it once every lane has read
        // (a wave's LDS operations complete in order)
        if (act) atomicOr(reinterpret_cast<unsigned long long *>(&dmask[d]), 1ull << lane);
        wave_lds_fence();
        const uint64_t peers = act ? dmask[d] : 0ull;
        wave_lds_fence();
        if (act) {
          dmask[d] = 0;
          rk[v] = (uint16_t)(base[d] + __builtin_amdgcn_mbcnt_hi((uint32_t)(peers >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u)));
        }
      }
      if (act) {  // counts: the order of these adds does not matter
        atomicAdd(&base[d], 1);
        atomicAdd(&cfill[d], indeg);
      }
    }
  }
  if (lane == 0) {
    int so = 0, sc = 0;
    for (int d = 0; d < D; ++d) {
      own_off[d] = so;
      so += base[d];
      cp_off[d] = sc;
      sc += cfill[d];
      cfill[d] = cp_off[d];
    }
    own_off[D] = so;
    cp_off[D] = sc;
  }
  if (kStage) {
    for (int d = lane; d < D; d += kWave) base[d] = own_off[d];
    if (lane == 0) fqn = fcn = 0;
  }
  __syncthreads();  // also orders the rank-table stores before the loads below
  if (!kFast) {
    for (int v0 = 0; v0 < N; v0 += kWave) {
      const int v = v0 + lane;
      if (v < N) {
        const int d = prow[v], rv = rk[v];
        op_intervals(G, prow, frow, rk, v, d, rv, own_off[d] + rv, cfill, own, cp);
      }
    }
  } else if (N > 0) {
    auto load_op = [&](int v) -> IvOp {
      IvOp a;
      a.d = prow[v];
      a.rv = rk[v];
      a.f = frow[v];
      a.b = G.bytes32[v];
      a.w = G.dur32[v];
      a.s2 = G.succ2[v];
      a.x0 = G.xfer32[v * K];
      a.x1 = G.xfer32[v * K + K - 1];
      a.pe = kPorts ? G.succ2_pe[v] : 0u;
      return a;
    };
    auto load_succ = [&](const IvOp &a, int v) -> IvSucc {
      const uint32_t x0 = a.s2 & 0xFFFFu, x1 = a.s2 >> 16;
      const int y0 = x0 == 0xFFFFu ? v : (int)x0, y1 = x1 == 0xFFFFu ? v : (int)x1;
      uint32_t ax0 = 0, ax1 = 0;
      if (kPorts) {  // an absent successor reads edge 0 (E >= 1 when there is one), never used
        const uint32_t e0 = a.pe & 0xFFFFu, e1 = a.pe >> 16;
        ax0 = arow[e0 == 0xFFFFu ? 0u : e0];
        ax1 = arow[e1 == 0xFFFFu ? 0u : e1];
      }
      return IvSucc{prow[y0], prow[y1], frow[y0], frow[y1], rk[y0], rk[y1], ax0, ax1};
    };
    nocopy[lane] = 0;
    int vq = min(lane, N - 1);
    IvOp a = load_op(vq);
    IvSucc sc = load_succ(a, vq);
    for (int v0 = 0; v0 < N; v0 += kWave) {
      const bool act = v0 + lane < N;
      const int vn = min(v0 + kWave + lane, N - 1);
      const IvOp an = load_op(vn);  // next chunk
      const uint32_t d = a.d, x0 = a.s2 & 0xFFFFu, x1 = a.s2 >> 16;
      const bool has0 = x0 != 0xFFFFu, has1 = x1 != 0xFFFFu;
      const bool loc0 = has0 && sc.dx0 == d, loc1 = has1 && sc.dx1 == d;
      auto link_of = [&](uint32_t u, uint32_t w) -> uint32_t {
        if (!kShiftLinks) return link_bit(G, u, w);
        const uint32_t s = (uint32_t)G.link_shift, same = (uint32_t)G.link_same;
        return (u >> s) == (w >> s) ? same : 1u - same;
      };
      const uint32_t X0 = link_of(d, sc.dx0) ? a.x1 : a.x0;  // transfer to each successor's device
      const uint32_t X1 = link_of(d, sc.dx1) ? a.x1 : a.x0;
      // own output: until the local consumer that finishes last
      uint32_t L = a.f, rl = a.rv, A = 0;
      rl = (loc0 && sc.fx0 > L) ? sc.rx0 : rl;
      L = (loc0 && sc.fx0 > L) ? sc.fx0 : L;
      rl = (loc1 && sc.fx1 > L) ? sc.rx1 : rl;
      L = (loc1 && sc.fx1 > L) ? sc.fx1 : L;
      // arrival of each remote transfer (two successors on one remote device
      // share the first one's transfer)
      const uint32_t T0 = kPorts ? sc.ax0 : a.f + X0, T1 = kPorts ? sc.ax1 : a.f + X1;
      A = (has0 && !loc0) ? umax32(A, T0) : A;
      A = (has1 && !loc1) ? umax32(A, T1) : A;
      const bool arrive = A > L;
      const uint32_t F = !has0 ? kInf32 : arrive ? A : L;
      const uint32_t loc = !has0 ? 0u : arrive ? loc_window((int)a.rv + 1) : rl + 1;
      const Rec ro = Rec{a.f - a.w, F, a.b, loc};
      const int po = own_off[d] + (int)a.rv;
      // copies: one per remote successor device
      const bool same = has1 && sc.dx1 == sc.dx0;
      const bool c0 = act && has0 && !loc0 && a.b != 0;
      const bool c1 = act && has1 && !loc1 && !same && a.b != 0;
      int *const f0 = c0 ? &cfill[sc.dx0] : &nocopy[lane], *const f1 = c1 ? &cfill[sc.dx1] : &nocopy[lane];
      int qo = 0, q0 = 0, q1 = 0;
      if (kStage) {  // first position of each destination's run in this chunk
        if (kCpSt) {
          q0 = *f0;
          q1 = *f1;
        }
        qo = base[d];  // d is valid in every lane (inactive lanes repeat the last op)
        atomicAdd(&base[d], act ? 1 : 0);
      }
      const int s0 = atomicAdd(f0, c0 ? 1 : 0);
      const int s1 = atomicAdd(f1, c1 ? 1 : 0);
      // both successors on one remote device: allocated before the one that
      // starts first, freed after the one that finishes last
      const bool late1 = same && sc.fx1 > sc.fx0;
      const uint32_t ry0 = late1 ? sc.rx1 : sc.rx0, hi0 = late1 ? sc.fx1 : sc.fx0;
      const uint32_t ra0 = same ? min(sc.rx0, sc.rx1) : sc.rx0;
      const uint32_t st0 = kPorts ? T0 - X0 : a.f, st1 = kPorts ? T1 - X1 : a.f;  // transfer starts
      const Rec r0 = Rec{st0, hi0, a.b, (uint32_t)max((int)ra0 - 3, 0) << 16 | (ry0 + 1)};
      const Rec r1 = Rec{st1, sc.fx1, a.b, (uint32_t)max((int)sc.rx1 - 3, 0) << 16 | (sc.rx1 + 1)};
      const uint32_t dx0 = sc.dx0, dx1 = sc.dx1;
      sc = load_succ(an, vn);  // the next chunk's successors, in flight during the stores
      if (!kStage) {
        own[act ? po : N] = ro;
        cp[c0 ? s0 : E] = r0;
        cp[c1 ? s1 : E] = r1;
      } else {
        if (!kCpSt) {
          if (c0) cp[s0] = r0;
          if (c1) cp[s1] = r1;
        }
        wave_lds_fence();
        // each destination's positions in this chunk form one run [first, last]
        const int eo = base[d] - 1, bo = own_off[d + 1];
        const int ko = act ? line_role<kOwnShift>(po, qo, eo, bo) : kRoleNone;
        int k0 = kRoleNone, k1 = kRoleNone;
        if (kCpSt) {
          const int e0 = *f0 - 1, e1 = *f1 - 1;
          k0 = c0 ? line_role<kCpShift>(s0, q0, e0, INT_MAX) : kRoleNone;
          k1 = c1 ? line_role<kCpShift>(s1, q1, e1, INT_MAX) : kRoleNone;
        }
        // blocks complete inside this chunk: stored directly
        if (ko == kRoleDirect) own[po] = ro;
        if (k0 == kRoleDirect) cp[s0] = r0;
        if (k1 == kRoleDirect) cp[s1] = r1;
        // the block open since earlier chunks: staged, and queued once complete
        if (ko & kRoleOpen) obuf[d * kOwnRecs + (po & (kOwnRecs - 1))] = ro;
        if (k0 & kRoleOpen) cbuf[dx0 * kCpRecs + (s0 & (kCpRecs - 1))] = r0;
        if (k1 & kRoleOpen) cbuf[dx1 * kCpRecs + (s1 & (kCpRecs - 1))] = r1;
        if (ko == kRoleClose) fq[atomicAdd(&fqn, 1)] = d << 20 | (uint32_t)(po >> kOwnShift);
        if (k0 == kRoleClose) fc[atomicAdd(&fcn, 1)] = dx0 << 20 | (uint32_t)(s0 >> kCpShift);
        if (k1 == kRoleClose) fc[atomicAdd(&fcn, 1)] = dx1 << 20 | (uint32_t)(s1 >> kCpShift);
        wave_lds_fence();
        // write the queued blocks, adjacent lanes to adjacent records
        const int nq = fqn;
        for (int qb = 0; qb < nq; qb += kWave / kOwnRecs) {
          const int qi = qb + (lane >> kOwnShift), part = lane & (kOwnRecs - 1);
          if (qi < nq) {  // bounds and record read together; a slot outside the bucket goes to the spare
            const uint32_t ent = fq[qi];
            const int dv = (int)(ent >> 20), pos = (int)(ent & 0xFFFFFu) * kOwnRecs + part;
            const int lo = own_off[dv], hi = own_off[dv + 1];
            const Rec r = obuf[dv * kOwnRecs + part];
            own[((pos >= lo) & (pos < hi)) ? pos : N] = r;
          }
        }
        if (kCpSt) {
          const int nc = fcn;
          for (int qb = 0; qb < nc; qb += kWave / kCpRecs) {
            const int qi = qb + (lane >> kCpShift), part = lane & (kCpRecs - 1);
            if (qi < nc) {
              const uint32_t ent = fc[qi];
              const int dv = (int)(ent >> 20), pos = (int)(ent & 0xFFFFFu) * kCpRecs + part;
              const int lo = cp_off[dv];
              const Rec r = cbuf[dv * kCpRecs + part];
              cp[pos >= lo ? pos : E] = r;
            }
          }
        }
        wave_lds_fence();
        // a block begun in this chunk but not complete: staged for later chunks
        if (ko == kRoleTail) obuf[d * kOwnRecs + (po & (kOwnRecs - 1))] = ro;
        if (k0 == kRoleTail) cbuf[dx0 * kCpRecs + (s0 & (kCpRecs - 1))] = r0;
        if (k1 == kRoleTail) cbuf[dx1 * kCpRecs + (s1 & (kCpRecs - 1))] = r1;
        if (lane == 0) fqn = fcn = 0;
      }
      a = an;
    }
    if (kCpSt) {  // copy blocks still open (a bucket ends short of its reserve)
      wave_lds_fence();
      for (int e = lane; e < D; e += kWave) {
        const int end = cfill[e], lo = max(end & ~(kCpRecs - 1), cp_off[e]);
        for (int pos = lo; pos < end; ++pos) cp[pos] = cbuf[e * kCpRecs + (pos & (kCpRecs - 1))];
      }
    }
  }
  wave_lds_fence();
  int32_t *m = meta + j * meta_stride(D);
  for (int d = lane; d <= D; d += kWave) {
    m[d] = own_off[d];
    m[D + 1 + d] = cp_off[d];
    m[2 * (D + 1) + d] = d < D ? cfill[d] - cp_off[d] : 0;
  }
}

// Gap of x among the sorted S[0, m): #{k : S[k] <= x} (kLe) or S[k] < x.
// gap_win decides it from six independent probes when the answer lies in
// [L, L+4] (ok), gap_search covers the rest.
template <bool kLe, class UP>
__device__ __forceinline__ int gap_win(UP S, int m, uint32_t x, int L, bool &ok) {
  if (m == 0) {
    ok = true;
    return 0;
  }
  L = min(L, m);
  auto hit = [&](uint32_t sv) { return kLe ? sv <= x : sv < x; };
  const uint32_t sm1 = S[max(L - 1, 0)];
  uint32_t sv[5];
#pragma unroll
  for (int q = 0; q < 5; ++q) sv[q] = S[min(L + q, m - 1)];
  ok = (L == 0 || hit(sm1)) && (L + 4 >= m || !hit(sv[4]));
  int g = L;
#pragma unroll
  for (int q = 0; q < 4; ++q) g += (L + q < m && hit(sv[q])) ? 1 : 0;
  return g;
}

template <bool kLe, class UP>
__device__ int gap_search(UP S, int m, uint32_t x) {
  int lo = 0, n = m;
  while (n > 0) {
    const int half = n >> 1;
    if (kLe ? S[lo + half] <= x : S[lo + half] < x) {
      lo += half + 1;
      n -= half + 1;
    } else {
      n = half;
    }
  }
  return lo;
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

// max(0, max_i sum_{k <= i} delta[k]): the peak live bytes, the maximum being
// taken at allocation instants (each position is one).
template <class DP>
__device__ int64_t max_live(DP delta, int n, int lane) {
  const int m = (n + kWave - 1) / kWave, lo = lane * m, hi = min(n, lo + m);
  int64_t s = 0;
  for (int i = lo; i < hi; ++i) s += delta[i];
  int64_t run = wave_incl_scan64(s, lane) - s, best = 0;
  for (int i = lo; i < hi; ++i) {
    run += delta[i];
    best = imax64(best, run);
  }
  for (int o = kWave / 2; o >= 1; o >>= 1) best = imax64(best, __shfl_xor(best, o, kWave));
  return best;
}

// Peak of one device: m own records (start-sorted) and nc copy records.
// Allocations are merged in time order as
//   [copies of gap 0] own 0 [copies of gap 1] own 1 ... own m-1 [copies of gap m]
// so own k sits at k + CG[k+1] and the copy of in-gap rank r of gap g at
// g + CG[g] + r, where CG[g] counts the copies in gaps before g; a free of gap
// g lands before the first allocation at or after it: g + CG[g] + the copies
// of gap g allocated before it.  Work arrays (the workgroup's global slot
// memory):
//   ak  own starts S[0, m), then the copy times grouped by gap
//   ag  gap counts / CG[0, m+2), then per copy (gap << 16 | slot in gap)
//   dl  by merged position: bytes allocated there minus bytes freed just before
template <class UP, class IP, class DP>
__device__ int64_t device_peak(const Rec *own, int m, const Rec *cp, int nc, UP ak, IP ag, DP dl, int lane) {
  constexpr int kB = 8;
  const int na = m + nc;
  UP bt = ak + m;                                           // grouped copy times
  uint32_t *qg = reinterpret_cast<uint32_t *>(ag + m + 2);  // per copy: gap << 16 | slot
  for (int base = lane; base < m; base += kB * kWave) {      // a batch of loads in flight together
    uint32_t r[kB];
#pragma unroll
    for (int q = 0; q < kB; ++q)
      if (base + q * kWave < m) r[q] = own[base + q * kWave].x;
#pragma unroll
    for (int q = 0; q < kB; ++q)
      if (base + q * kWave < m) ak[base + q * kWave] = r[q];
  }
  for (int i = lane; i < na; i += kWave) dl[i] = 0;
  for (int i = lane; i < m + 2; i += kWave) ag[i] = 0;
  wave_lds_fence();
  // gap of every copy allocation, and its slot inside the gap: the window
  // probes of four rows are in flight together, searches only where needed
  for (int base = lane; base < nc; base += 4 * kWave) {
    uint32_t x[4], L[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const Rec r = cp[min(base + q * kWave, nc - 1)];
      x[q] = r.x;
      L[q] = r.w >> 16;
    }
    int g[4];
    bool ok[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) g[q] = gap_win<true>(ak, m, x[q], (int)L[q], ok[q]);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = base + q * kWave;
      if (i < nc) {
        if (!ok[q]) g[q] = gap_search<true>(ak, m, x[q]);
        const int slot = atomicAdd(&ag[g[q] + 1], 1);
        qg[i] = (uint32_t)g[q] << 16 | (uint32_t)slot;
      }
    }
  }
  wave_lds_fence();
  prefix_inplace(ag, m + 2, lane);  // ag[g] = CG[g]
  wave_lds_fence();
  for (int i = lane; i < nc; i += kWave) bt[ag[qg[i] >> 16] + (qg[i] & 0xFFFFu)] = cp[i].x;
  for (int k = lane; k < m; k += kWave) dl[k + ag[k + 1]] = own[k].z;
  wave_lds_fence();
  // copy allocations: rank inside the gap by (time, slot)
  for (int i = lane; i < nc; i += kWave) {
    const Rec r = cp[i];
    const int g = (int)(qg[i] >> 16), s0 = ag[g], s1 = ag[g + 1], me = s0 + (int)(qg[i] & 0xFFFFu);
    int rank = 0;
    for (int z = s0; z < s1; ++z) {
      const uint32_t t = bt[z];
      rank += (t < r.x || (t == r.x && z < me)) ? 1 : 0;
    }
    dl[g + s0 + rank] = r.z;
  }
  wave_lds_fence();
  // frees: gap (exact or by window), then the copies of that gap allocated before
  auto place_free = [&](int g, uint32_t h, uint32_t bytes) {
    const int s0 = ag[g], s1 = ag[g + 1];
    int pos = g + s0;
    for (int z = s0; z < s1; ++z) pos += bt[z] < h ? 1 : 0;
    if (pos < na) atomicAdd(reinterpret_cast<unsigned long long *>(&dl[pos]), (unsigned long long)(-(int64_t)bytes));
  };
  // (gaps are clamped to [0, m] so that no record content can widen a loop)
  for (int i = lane; i < nc; i += kWave) {
    const Rec r = cp[i];
    place_free(min((int)(r.w & 0xFFFFu), m), r.y, r.z);
  }
  for (int k = lane; k < m; k += kWave) {
    const Rec r = own[k];
    if (r.y != kInf32) {
      int g = min((int)r.w, m);
      if (r.w & kLocWindow) {
        bool ok;
        g = gap_win<false>(ak, m, r.y, (int)(r.w & 0xFFFFu), ok);
        if (!ok) g = gap_search<false>(ak, m, r.y);
      }
      place_free(g, r.y, r.z);
    }
  }
  wave_lds_fence();
  const int64_t best = max_live(dl, na, lane);
  wave_lds_fence();
  return best;
}

// Aggregate evaluation of one device (own starts S[0, m) sorted, nc copies).
// With the merged order [gap 0] own 0 [gap 1] own 1 ... own m-1 [gap m] (a
// gap's events: its copy allocations and the frees that land before the next
// own allocation), let L[g] be the live bytes after all events of gap g:
//   L[g] = sum_{g' <= g} (copies_g' - frees_g') + sum_{k < g} own_k,
// so the live bytes at own allocation k are L[k] + own_k, exact from per-gap
// sums alone.  Inside gap g the live bytes at a copy allocation are at most
// U[g] = L[g] + frees_g (every copy counted, no free), and equal to it when
// the gap holds no free.  Only a "hard" gap, holding copies and frees with
// U[g] above the best exact value so far, needs its events in time order;
// those few events are collected and swept exactly.
constexpr int kAggCap = 512;   // own allocations per device for the aggregate method in LDS
constexpr int kAggCopies = 1024;
constexpr int kHardCap = 128;  // events of hard gaps per device

// Per-gap byte sums: int64 in general; u32 when the loader proved that every
// byte that can be live on one device at once sums below 2^32 once all sizes
// are divided by their common power of two (GmgView::peak_narrow): the sums
// are then exact modulo 2^32 and every value compared lies in [0, 2^32).
template <class Acc>
struct AggLds {
  uint32_t S[kAggCap];        // own starts
  Acc dg[kAggCap + 1];        // per gap: copies allocated (+ own_{g-1}), then L[g]
  Acc fg[kAggCap + 1];        // per gap: freed bytes, then the live bytes at the gap's start
  uint32_t cg[kAggCopies];    // per copy: allocation gap << 16 | free gap
  uint8_t hard[kAggCap + 1];
  uint32_t ht[kHardCap], hb[kHardCap], hx[kHardCap];  // collected events: time, bytes, gap << 1 | is_alloc
  int hn;
};

// A device's share of one candidate's records.
struct DevSpan {
  const Rec *own, *cp;
  int m, nc;
};

constexpr int kOwnPer = kAggCap / kWave;    // own records per lane held in registers
constexpr int kCpPer = kAggCopies / kWave;  // copy records per lane
constexpr int kCpPre = 8;                   // copy rows loaded ahead; the rest when needed

__device__ __forceinline__ bool agg_fits(const DevSpan &s) { return s.m < kAggCap && s.nc <= kAggCopies; }

// Record k of a device sits in register k / 64 of lane k % 64.  The loads are
// unconditional (a load under a branch is waited for at the join): rows past
// the end repeat the last record, or the region's spare record when the
// device has none, and are never used.
__device__ __forceinline__ void load_own(Rec (&ro)[kOwnPer], const DevSpan &s, int lane) {
#pragma unroll
  for (int q = 0; q < kOwnPer; ++q) ro[q] = s.own[min(q * kWave + lane, max(s.m - 1, 0))];
}

__device__ __forceinline__ void load_cp(Rec (&rc)[kCpPre], const DevSpan &s, int lane) {
#pragma unroll
  for (int q = 0; q < kCpPre; ++q) rc[q] = s.cp[min(q * kWave + lane, max(s.nc - 1, 0))];
}

__device__ __forceinline__ void lds_add(uint32_t *p, uint32_t v) { atomicAdd(p, v); }
__device__ __forceinline__ void lds_add(int64_t *p, int64_t v) {
  atomicAdd(reinterpret_cast<unsigned long long *>(p), (unsigned long long)v);
}
__device__ __forceinline__ uint32_t wave_max_acc(uint32_t x) {
  for (int o = kWave / 2; o >= 1; o >>= 1) x = umax32(x, (uint32_t)__shfl_xor((int)x, o, kWave));
  return x;
}
__device__ __forceinline__ int64_t wave_max_acc(int64_t x) {
  for (int o = kWave / 2; o >= 1; o >>= 1) x = imax64(x, __shfl_xor(x, o, kWave));
  return x;
}
__device__ __forceinline__ uint32_t wave_scan_acc(uint32_t x, int lane) {  // modulo 2^32
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}
__device__ __forceinline__ int64_t wave_scan_acc(int64_t x, int lane) { return wave_incl_scan64(x, lane); }

// Peak of one device whose records the caller loaded into ro and rc (it fits
// the LDS arrays: agg_fits).  Once a record array has been used for the last
// time it is refilled with the records of the next device (nxt, when pf), so
// those loads overlap the rest of this device's work; the own sizes (and
// the gaps of the own frees) stay in registers past that.  Sizes are divided
// by 2^sh (kNarrow).  Returns -1 if the hard events overflow (the caller then
// uses device_peak).
template <bool kNarrow>
__device__ int64_t device_peak_agg(const DevSpan &cur, Rec (&ro)[kOwnPer], Rec (&rc)[kCpPre], const DevSpan &nxt,
                                   bool pf, AggLds<typename std::conditional<kNarrow, uint32_t, int64_t>::type> &A,
                                   int lane, int sh) {
  using Acc = typename std::conditional<kNarrow, uint32_t, int64_t>::type;
  const int m = cur.m, nc = cur.nc;
  auto size_of = [&](uint32_t z) -> uint32_t { return kNarrow ? z >> sh : z; };
  // own k: start, and its allocation as the opening value of gap k + 1
  uint32_t obr[kOwnPer];  // size of own k = q * 64 + lane
#pragma unroll
  for (int q = 0; q < kOwnPer; ++q) {
    const int k = q * kWave + lane;
    obr[q] = size_of(ro[q].z);
    if (k < m) {
      A.S[k] = ro[q].x;
      A.dg[k + 1] = (Acc)obr[q];
    }
    if (k <= m) {
      A.fg[k] = 0;
      A.hard[k] = 0;
    }
  }
  if (lane == 0) {
    A.dg[0] = 0;
    A.hn = 0;
  }
  wave_lds_fence();
  // copies: allocation gap (window probes, four rows at a time), free gap exact
#pragma unroll
  for (int q0 = 0; q0 < kCpPer; q0 += 4) {
    if (q0 * kWave < nc) {
      Rec r4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        r4[q] = q0 + q < kCpPre ? rc[(q0 + q) % kCpPre] : cur.cp[min((q0 + q) * kWave + lane, nc - 1)];
      int g[4];
      bool ok[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) g[q] = gap_win<true>(A.S, m, r4[q].x, (int)(r4[q].w >> 16), ok[q]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = (q0 + q) * kWave + lane;
        if (i < nc) {
          const Rec r = r4[q];
          if (!ok[q]) g[q] = gap_search<true>(A.S, m, r.x);
          const int gf = min((int)(r.w & 0xFFFFu), m);
          A.cg[i] = (uint32_t)g[q] << 16 | (uint32_t)gf;
          lds_add(&A.dg[g[q]], (Acc)size_of(r.z));
          lds_add(&A.fg[gf], (Acc)size_of(r.z));
        }
      }
    }
  }
  if (pf) load_cp(rc, nxt, lane);
  // own frees: exact gap or window probes; the gap is kept (0xFFFF: never freed)
  uint32_t ogr[kOwnPer / 2];  // u16 pairs: free gap of own q * 64 + lane in half q & 1 of word q / 2
#pragma unroll
  for (int q = 0; q < kOwnPer / 2; ++q) ogr[q] = 0xFFFFFFFFu;
#pragma unroll
  for (int q0 = 0; q0 < kOwnPer; q0 += 4) {
    if (q0 * kWave < m) {
      int g[4];
      bool ok[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ok[q] = true;
        g[q] = min((int)ro[q0 + q].w, m);
        if (ro[q0 + q].w & kLocWindow)
          g[q] = gap_win<false>(A.S, m, ro[q0 + q].y, (int)(ro[q0 + q].w & 0xFFFFu), ok[q]);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = (q0 + q) * kWave + lane;
        if (k < m) {
          const Rec r = ro[q0 + q];
          if (r.y != kInf32) {
            if (!ok[q]) g[q] = gap_search<false>(A.S, m, r.y);
            const int half = 16 * ((q0 + q) & 1);
            ogr[(q0 + q) >> 1] = (ogr[(q0 + q) >> 1] & ~(0xFFFFu << half)) | (uint32_t)g[q] << half;
            lds_add(&A.fg[g[q]], (Acc)obr[q0 + q]);
          }
        }
      }
    }
  }
  if (pf) load_own(ro, nxt, lane);
  wave_lds_fence();
  // L[g] = prefix of dg - fg.  Every loop below runs a fixed number of rows
  // (m < kAggCap, nc <= kAggCopies) with clamped, unconditional LDS loads, so
  // that each row's loads overlap.
  {
    const int n = m + 1, per = (n + kWave - 1) / kWave, lo = lane * per;
    Acc v[kOwnPer];
    Acc sacc = 0;
#pragma unroll
    for (int t = 0; t < kOwnPer; ++t) {
      const int g = min(lo + t, n - 1);
      v[t] = A.dg[g] - A.fg[g];
      if (t >= per || lo + t >= n) v[t] = 0;
      sacc += v[t];
    }
    Acc run = wave_scan_acc(sacc, lane) - sacc;
#pragma unroll
    for (int t = 0; t < kOwnPer; ++t) {
      run += v[t];
      if (t < per && lo + t < n) A.dg[lo + t] = run;
    }
  }
  wave_lds_fence();
  // P0 at own allocations, exact values of copy-only gaps; the live bytes at
  // each gap's start (after own g - 1) replace its frees in fg
  Acc best = 0;
  Acc bound[kOwnPer];  // per gap of this lane: L + frees when the gap holds copies and frees, else 0
#pragma unroll
  for (int q = 0; q < kOwnPer; ++q) {
    const int g = q * kWave + lane, gc = min(g, m), gp = max(gc - 1, 0);
    // size of own g - 1: the previous lane's, or lane 63's of the row before
    const uint32_t up = (uint32_t)__shfl_up((int)obr[q], 1, kWave);
    const uint32_t wrap = q > 0 ? (uint32_t)__shfl((int)obr[q > 0 ? q - 1 : 0], kWave - 1, kWave) : 0u;
    const uint32_t ob_prev = lane > 0 ? up : wrap;
    const Acc L = A.dg[gc], F = A.fg[gc];
    const Acc prev = gc > 0 ? A.dg[gp] + (Acc)ob_prev : (Acc)0;
    const Acc copies = L - prev + F;
    bound[q] = 0;
    if (g <= m) {
      if (g < m) best = best > L + (Acc)obr[q] ? best : L + (Acc)obr[q];
      if (copies > 0 && F == 0) best = best > L ? best : L;  // copies only: all of them precede own g
      if (copies > 0 && F > 0) bound[q] = L + F;
      A.fg[g] = prev;
    }
  }
  best = wave_max_acc(best);
  bool any = false;
#pragma unroll
  for (int q = 0; q < kOwnPer; ++q) {
    if (bound[q] > best) {
      A.hard[q * kWave + lane] = 1;
      any = true;
    }
  }
  auto widen = [&](Acc x) -> int64_t { return kNarrow ? (int64_t)x << sh : (int64_t)x; };
  if (!__any(any)) return widen(best);
  wave_lds_fence();
  // collect the events of the hard gaps
  auto push = [&](uint32_t t, uint32_t b, uint32_t x) {
    const int at = atomicAdd(&A.hn, 1);
    if (at < kHardCap) {
      A.ht[at] = t;
      A.hb[at] = b;
      A.hx[at] = x;
    }
  };
#pragma unroll
  for (int q0 = 0; q0 < kCpPer; q0 += 4) {
    if (q0 * kWave < nc) {
      uint32_t gg[4];
      bool ha[4], hf[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) gg[q] = A.cg[min((q0 + q) * kWave + lane, nc - 1)];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ha[q] = A.hard[gg[q] >> 16];
        hf[q] = A.hard[gg[q] & 0xFFFFu];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = (q0 + q) * kWave + lane;
        if (i < nc && (ha[q] || hf[q])) {
          const Rec r = cur.cp[i];
          if (ha[q]) push(r.x, size_of(r.z), (gg[q] >> 16) << 1 | 1u);
          if (hf[q]) push(r.y, size_of(r.z), (gg[q] & 0xFFFFu) << 1);
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kOwnPer; ++q) {
    const int k = q * kWave + lane;
    const uint32_t gf = (ogr[q >> 1] >> (16 * (q & 1))) & 0xFFFFu;
    if (k < m && gf != 0xFFFFu && A.hard[gf]) push(cur.own[k].y, obr[q], gf << 1);
  }
  wave_lds_fence();
  const int hn = A.hn;
  if (hn > kHardCap) return -1;
  // live bytes at each collected copy allocation: the gap's start value plus
  // its copies up to it (ties by position) minus its frees at or before it
  for (int e = lane; e < hn; e += kWave) {
    const uint32_t x = A.hx[e];
    if (!(x & 1u)) continue;
    const int g = (int)(x >> 1);
    const uint32_t t = A.ht[e];
    Acc live = A.fg[g];
    for (int z = 0; z < hn; ++z) {
      const uint32_t xz = A.hx[z];
      if ((int)(xz >> 1) != g) continue;
      const uint32_t tz = A.ht[z];
      if (xz & 1u) {
        if (tz < t || (tz == t && z <= e)) live += (Acc)A.hb[z];
      } else if (tz <= t) {
        live -= (Acc)A.hb[z];
      }
    }
    best = best > live ? best : live;
  }
  return widen(wave_max_acc(best));
}

// Blocks take candidates from a ticket counter (zero at launch) rather than
// in a fixed stride: a block that starts late, or shares its CU with another
// kernel's waves, takes fewer candidates instead of holding up the launch.
template <bool kNarrow>
__global__ __launch_bounds__(kWave) void fast_peaks(const GmgView G, int64_t j0, int64_t nj,
                                                    const Rec *__restrict__ own_all, const Rec *__restrict__ cp_all,
                                                    const int32_t *__restrict__ meta, uint32_t *__restrict__ wk_all,
                                                    int64_t *__restrict__ wb_all, int64_t slot_cap,
                                                    uint32_t *__restrict__ ticket, int64_t *__restrict__ peak,
                                                    uint8_t *__restrict__ violation) {
  __shared__ AggLds<typename std::conditional<kNarrow, uint32_t, int64_t>::type> s_agg;
  const int D = G.n_dev, N = G.n_ops, E = G.pred_ptr[G.n_ops];
  const int lane = threadIdx.x;
  uint32_t *g_ak = wk_all + (int64_t)blockIdx.x * 2 * (slot_cap + 2);
  int32_t *g_ag = reinterpret_cast<int32_t *>(g_ak + slot_cap + 2);
  int64_t *g_dl = wb_all + (int64_t)blockIdx.x * slot_cap;
  // the next candidate's ticket is fetched while the current one runs
  uint32_t tk = lane == 0 ? atomicAdd(ticket, 1u) : 0u;
  for (int64_t j = (uint32_t)__shfl((int)tk, 0, kWave); j < nj; j = (uint32_t)__shfl((int)tk, 0, kWave)) {
    tk = lane == 0 ? atomicAdd(ticket, 1u) : 0u;
    const int64_t c = j0 + j;
    if (violation[c] & SS_VIOLATION_INVALID) {
      if (peak)
        for (int d = lane; d < D; d += kWave) peak[c * D + d] = 0;
      continue;
    }
    const Rec *own = own_all + j * own_stride(N);
    const Rec *cp = cp_all + j * cp_stride(E);
    const int32_t *mt = meta + j * meta_stride(D);
    auto span = [&](int e) {
      const int o0 = mt[e];
      return DevSpan{own + o0, cp + mt[D + 1 + e], mt[e + 1] - o0, mt[2 * (D + 1) + e]};
    };
    uint8_t viol = 0;
    // each device's records are loaded while the previous device is evaluated
    Rec ro[kOwnPer], rc[kCpPre];
    DevSpan cur = span(0);
    if (agg_fits(cur)) {
      load_own(ro, cur, lane);
      load_cp(rc, cur, lane);
    }
    for (int e = 0; e < D; ++e) {
      const DevSpan nxt = e + 1 < D ? span(e + 1) : cur;
      const bool pf = e + 1 < D && agg_fits(nxt);
      int64_t pk = 0;
      if (cur.m + cur.nc > 0 && agg_fits(cur)) {
        pk = device_peak_agg<kNarrow>(cur, ro, rc, nxt, pf, s_agg, lane, G.peak_shift);
      } else if (pf) {
        load_own(ro, nxt, lane);
        load_cp(rc, nxt, lane);
      }
      if (pk < 0 || (cur.m + cur.nc > 0 && !agg_fits(cur)))
        pk = device_peak(cur.own, cur.m, cur.cp, cur.nc, g_ak, g_ag, g_dl, lane);
      if (peak && lane == 0) peak[c * D + e] = pk;
      if (pk > G.cap[e]) viol = SS_VIOLATION_MEMORY;
      cur = nxt;
    }
    if (lane == 0) violation[c] = viol;
  }
}

template <int kLink>
const void *schedule_fn(bool overflow, bool one_class) {
  if (overflow)
    return one_class ? reinterpret_cast<const void *>(&fast_schedule<kLink, true, true>)
                     : reinterpret_cast<const void *>(&fast_schedule<kLink, true, false>);
  return one_class ? reinterpret_cast<const void *>(&fast_schedule<kLink, false, true>)
                   : reinterpret_cast<const void *>(&fast_schedule<kLink, false, false>);
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

// Sub-chunk scratch of the memory passes.  The records (own, cp, meta) come in
// kRecSets sets used in turn: the interval pass of sub-chunk i runs on the
// caller's stream while peak passes of earlier sub-chunks run on the GMG's
// second stream; events order each peak pass after its interval pass, and the
// reuse of a set after the peak pass that read it.
constexpr int kRecSets = 3;
struct MemPass {
  Rec *own[kRecSets], *cp[kRecSets];
  int32_t *meta[kRecSets];
  uint16_t *rank;  // given ranks: candidate rows of the whole chunk; else sub rows
  uint32_t *wk;
  int64_t *wb;
  uint32_t *ticket;  // one zeroed counter per peak launch of the call
  int64_t n_ticket;
  int64_t sub, nslots, slot_cap;
  bool iv_fast;
  bool single;  // every pass on the caller's stream, one record set, no events
  int sets;     // record sets in use: kRecSets, or 1 when single
  hipStream_t aux;
  hipEvent_t iv_done[kRecSets], pk_done[kRecSets];
  int64_t it;  // sub-chunks issued so far in this call
};

int mem_pass_events(MemPass &M) {
  for (int k = 0; k < kRecSets; ++k) {
    M.iv_done[k] = M.pk_done[k] = nullptr;
  }
  M.it = 0;
  if (M.single) return SS_OK;
  for (int k = 0; k < kRecSets; ++k) {
    hipError_t err = hipEventCreateWithFlags(&M.iv_done[k], hipEventDisableTiming);
    if (err == hipSuccess) err = hipEventCreateWithFlags(&M.pk_done[k], hipEventDisableTiming);
    if (err != hipSuccess) return hip_fail(err, "hipEventCreateWithFlags");
  }
  M.it = 0;
  return SS_OK;
}

// Joins the second stream back into the caller's and releases the events
// (always, also after an error, before the scratch is freed).
int mem_pass_join(MemPass &M, hipStream_t stream) {
  if (M.single) return SS_OK;
  hipError_t err = hipSuccess;
  hipEvent_t done = nullptr;
  err = hipEventCreateWithFlags(&done, hipEventDisableTiming);
  if (err == hipSuccess) err = hipEventRecord(done, M.aux);
  if (err == hipSuccess) err = hipStreamWaitEvent(stream, done, 0);
  if (done) (void)hipEventDestroy(done);
  for (int k = 0; k < kRecSets; ++k) {
    if (M.iv_done[k]) (void)hipEventDestroy(M.iv_done[k]);
    if (M.pk_done[k]) (void)hipEventDestroy(M.pk_done[k]);
  }
  if (err != hipSuccess) {
    (void)hipStreamSynchronize(M.aux);  // the scratch must outlive the second stream's work
    return hip_fail(err, "joining the memory-pass stream");
  }
  return SS_OK;
}

// Dynamic LDS of fast_intervals: per-device offsets and fill pointers, and
// with staged stores the open blocks of every device's buckets.
size_t intervals_lds(int D, bool stage, bool stage_cp) {
  return (stage ? (size_t)D * kOwnRecs * sizeof(Rec) : 0) + (stage_cp ? (size_t)D * kCpRecs * sizeof(Rec) : 0) +
         (size_t)(4 * D + 2 + 2 * kWave + (stage_cp ? 2 * kWave : 0) + 2) * sizeof(int) +
         (stage ? 0 : (size_t)D * 8 + 8);  // lane masks per device (on the own-record stage when staged)
}

// Residency intervals, then peaks, for the nb candidates of one chunk (their
// placements Pc and finish-time rows fin), sub candidates at a time.
// arr (rows of arrivals per predecessor edge, transfers arbitrated over
// ports) is null in the latency model; with it, the branch-free writer with
// index ranks is required.
int memory_passes(const ss_gmg *g, MemPass &M, const uint8_t *Pc, const uint32_t *fin, int64_t nb,
                  bool given_ranks, int64_t *peak, uint8_t *violation, hipStream_t stream,
                  const uint32_t *arr = nullptr) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops;
  for (int64_t j0 = 0; j0 < nb; j0 += M.sub, ++M.it) {
    const int64_t nj = std::min(M.sub, nb - j0);
    const int set = (int)(M.it % M.sets);
    hipError_t err = hipSuccess;
    if (!M.single && M.it >= M.sets) err = hipStreamWaitEvent(stream, M.pk_done[set], 0);  // its buffers are free again
    if (err != hipSuccess) return hip_fail(err, "hipStreamWaitEvent");
    uint16_t *rank = given_ranks ? M.rank + j0 * N : M.rank;
    if (arr && (!M.iv_fast || given_ranks))
      return ss_set_error(SS_ERR_UNSUPPORTED, "port arrivals need the branch-free interval writer");
    const bool shift = G.link_shift >= 0;
    // copy records staged when this pass runs alone (one stream)
    const bool scp = M.single;
    auto staged = [&](auto shift_c, auto ports_c) -> const void * {
      constexpr bool kS = decltype(shift_c)::value, kP = decltype(ports_c)::value;
      return scp ? reinterpret_cast<const void *>(&fast_intervals<true, false, kS, kP, true>)
                 : reinterpret_cast<const void *>(&fast_intervals<true, false, kS, kP, false>);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    const void *fn =
        arr ? (shift ? staged(T_(), T_()) : staged(F_(), T_()))
        : M.iv_fast
            ? (given_ranks ? (shift ? reinterpret_cast<const void *>(&fast_intervals<true, true, true, false, false>)
                                    : reinterpret_cast<const void *>(&fast_intervals<true, true, false, false, false>))
                           : (shift ? staged(T_(), F_()) : staged(F_(), F_())))
            : (given_ranks ? reinterpret_cast<const void *>(&fast_intervals<false, true, false, false, false>)
                           : reinterpret_cast<const void *>(&fast_intervals<false, false, false, false, false>));
    const uint8_t *vi = violation;
    Rec *own = M.own[set], *cp = M.cp[set];
    int32_t *meta = M.meta[set];
    void *args[] = {const_cast<GmgView *>(&G), const_cast<uint8_t **>(&Pc), const_cast<uint32_t **>(&fin),
                    &j0, &own, &cp, &meta, &rank, &vi, const_cast<uint32_t **>(&arr)};
    // the branch-free writer with index ranks stages its stores
    const size_t lds = intervals_lds((int)g->n_dev, M.iv_fast && !given_ranks, M.iv_fast && !given_ranks && scp);
    err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");
    SsTimingRec *ti = ss_timing_start(SS_KERNEL_INTERVALS, stream);
    err = hipLaunchKernel(fn, dim3((unsigned)nj), dim3(kWave), args, lds, stream);
    ss_timing_stop(ti, stream);
    if (err == hipSuccess) err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(err, "fast_intervals launch");
    hipStream_t ps = M.single ? stream : M.aux;  // the peak pass's stream
    if (!M.single) {
      err = hipEventRecord(M.iv_done[set], stream);
      if (err == hipSuccess) err = hipStreamWaitEvent(M.aux, M.iv_done[set], 0);
      if (err != hipSuccess) return hip_fail(err, "ordering the peak pass");
    }
    if (M.it >= M.n_ticket) return ss_set_error(SS_ERR_DEVICE, "memory passes: more peak launches than counters");
    SsTimingRec *tm = ss_timing_start(SS_KERNEL_MEMORY, ps);
    hipLaunchKernelGGL(G.peak_narrow ? fast_peaks<true> : fast_peaks<false>,
                       dim3((unsigned)std::min<int64_t>(nj, M.nslots)), dim3(kWave), 0, ps, G, j0, nj,
                       static_cast<const Rec *>(own), static_cast<const Rec *>(cp),
                       static_cast<const int32_t *>(meta), M.wk, M.wb, M.slot_cap, M.ticket + M.it, peak, violation);
    ss_timing_stop(tm, ps);
    err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(err, "fast_peaks launch");
    if (!M.single) {
      err = hipEventRecord(M.pk_done[set], M.aux);
      if (err != hipSuccess) return hip_fail(err, "hipEventRecord");
    }
  }
  return SS_OK;
}

}  // namespace

size_t ss_fast_schedule_lds(const ss_gmg *g) {
  return (size_t)g->n_dev * kWave * 4 + (size_t)g->n_req * kWave * 4 + (size_t)(g->n_dev + 1) * 8 +
         (size_t)(g->n_dev + 3) / 4 * 4;
}


// Scratch of one fast-path call, laid out for a chunk of `chunk` candidates
// and memory-pass sub-chunks of `sub`.
struct FastPlan {
  int64_t chunk = 0, sub = 0, nslots = 0, n_ticket = 0;
  int sets = kRecSets;
  size_t sz_pt = 0, sz_fin = 0, sz_own = 0, sz_cp = 0, sz_meta = 0, sz_rank = 0, sz_wk = 0, sz_wb = 0, sz_tk = 0,
         total = 0;
};

hipError_t ss_rows_from_op_major(const uint8_t *P, int64_t n_ops, int64_t B, int64_t b0, int64_t nb, uint8_t *rows,
                                 hipStream_t stream) {
  if (n_ops == 0 || nb == 0) return hipSuccess;
  const dim3 tg((unsigned)((nb + 63) / 64), (unsigned)((n_ops + 63) / 64));
  hipLaunchKernelGGL(transpose_tiles<uint8_t>, tg, dim3(256), 0, stream, P + b0, n_ops, nb, B, rows);
  return hipGetLastError();
}

int ss_run_simulate_fast(const ss_gmg *g, SsPlace src, int64_t *makespan, int64_t *peak, uint8_t *violation,
                         int64_t *slack, int64_t *sumfin, hipStream_t stream, SsWork &W) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev, R = g->n_req, B = src.B;
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  int lds_cu = 0;
  err = hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  // the schedule writes the candidates' finish-time rows itself (no
  // transpose) when each row is 16-byte aligned
  const bool sched_rows = N > 0 && N % 4 == 0;
  const size_t sched_lds = ss_fast_schedule_lds(g);
  // kernel variant: link classes from device groups, a bit table or (more
  // than two classes) xfer32; in-degrees above the pipelined count go
  // through the predecessor CSR
  const int link_mode = G.link_shift >= 0 ? 3 : G.link_grp ? 0 : g->n_link <= 2 ? 1 : 2;
  const bool overflow = g->max_indeg > kPipePre;
  const bool one_class = g->n_class == 1;
  const void *const sched_fn = link_mode == 0   ? schedule_fn<0>(overflow, one_class)
                               : link_mode == 1 ? schedule_fn<1>(overflow, one_class)
                               : link_mode == 2 ? schedule_fn<2>(overflow, one_class)
                                                : schedule_fn<3>(overflow, one_class);
  const bool iv_fast = g->n_class == 1 && g->n_link <= 2 && g->max_outdeg <= 2;
  // chunk: placements (op-major for the schedule from row-major input, rows
  // for the memory passes from op-major input), op-major and row-major finish
  // times
  const int64_t per_cand = N * (1 + 4 + 4);
  // A schedule launch is best a whole number of rounds of the waves the chip
  // holds at once (every wave runs about as long as any other).
  const int64_t round =
      (int64_t)cus * std::max<int64_t>(1, lds_cu / (int64_t)std::max<size_t>(sched_lds, 1)) * kWave;
  // sub-chunk: interval records of each candidate (own N, copies <= E)
  const int64_t rec_per_cand = (own_stride(N) + cp_stride(E)) * (int64_t)sizeof(Rec) + 3 * (D + 1) * 4 + N * 2;
  const int64_t slot_cap = N + E + 1;  // most allocations one device can hold
  const int sets = W.single ? 1 : kRecSets;
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  // the layout for a chunk and a sub-chunk cap (equal sub-chunks, at least
  // two for a large chunk so the peak pass of one overlaps the interval pass
  // of the next)
  auto plan_of = [&](int64_t chunk, int64_t sub_cap) {
    FastPlan q;
    q.sets = sets;
    q.chunk = chunk = std::min<int64_t>(chunk, B);
    int64_t sub = std::min<int64_t>(std::max<int64_t>(1, sub_cap), chunk);
    const int64_t n = std::max<int64_t>((chunk + sub - 1) / sub, chunk >= 8192 && !W.single ? 2 : 1);
    q.sub = sub = (chunk + n - 1) / n;
    q.nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kPeakBlocksPerCU, sub));
    q.sz_pt = align((size_t)chunk * N + 1);
    q.sz_fin = align((size_t)chunk * N * 4 + 4);
    q.sz_own = align((size_t)sub * own_stride(N) * sizeof(Rec));
    q.sz_cp = align((size_t)sub * cp_stride(E) * sizeof(Rec));
    q.sz_meta = align((size_t)sub * 3 * (D + 1) * 4);
    q.sz_rank = align(((size_t)sub * N + 1) * 2);
    q.sz_wk = align((size_t)q.nslots * 2 * (slot_cap + 2) * 4);
    q.sz_wb = align((size_t)q.nslots * slot_cap * 8);
    q.n_ticket = (B + chunk - 1) / chunk * ((chunk + sub - 1) / sub);
    q.sz_tk = align((size_t)q.n_ticket * 4);
    q.total = q.sz_pt + 2 * q.sz_fin + (size_t)sets * (q.sz_own + q.sz_cp + q.sz_meta) +
              q.sz_rank + q.sz_wk + q.sz_wb + q.sz_tk;
    return q;
  };
  // the largest chunk within a budget, in whole rounds of schedule waves
  auto plan_for_budget = [&](int64_t budget) {
    int64_t chunk = budget / std::max<int64_t>(1, per_cand);
    chunk = chunk >= round ? chunk / round * round : std::max<int64_t>(kWave, chunk / kWave * kWave);
    chunk = std::min<int64_t>(chunk, int64_t(65535) * 64);  // transpose grids index 64-candidate tiles in y
    return plan_of(chunk, std::max<int64_t>(1, kRecordBudget / std::max<int64_t>(1, rec_per_cand)));
  };
  const FastPlan pmin = plan_of(kWave, 1), pref = plan_for_budget(kFastScratchBudget);
  // the largest layout within `bytes`: the preferred chunk with sub-chunks as
  // large as fit (down to a sixteenth of the chunk), else smaller chunks (by
  // whole rounds, then halves), down to the smallest layout
  auto plan_fit = [&](int64_t bytes) {
    if ((int64_t)pref.total <= bytes) return pref;
    int64_t chunk = pref.chunk;
    for (;;) {
      const int64_t lo0 = chunk > kWave ? std::max<int64_t>(1, std::min<int64_t>(pref.sub, chunk / 16)) : 1;
      if ((int64_t)plan_of(chunk, lo0).total <= bytes) {
        int64_t lo = lo0, hi = std::max<int64_t>(lo0, pref.sub);  // the largest sub-chunk cap that fits
        while (lo < hi) {
          const int64_t mid = lo + (hi - lo + 1) / 2;
          if ((int64_t)plan_of(chunk, mid).total <= bytes)
            lo = mid;
          else
            hi = mid - 1;
        }
        return plan_of(chunk, lo);
      }
      if (chunk <= kWave) return plan_of(chunk, 1);
      chunk = chunk > round ? chunk - round : std::max<int64_t>(kWave, chunk / 2 / kWave * kWave);
    }
  };
  // the pool path's budget: up to the preferred layout, within seven eighths
  // of the memory the call can get now
  auto pool_budget = [&] { return ss_scratch_budget(g->device, g->pool, (int64_t)pref.total, 7); };
  if (W.query) {
    W.need_min = pmin.total;
    W.need_pref = pref.total;
    const FastPlan pq = W.single ? pref : plan_fit(pool_budget());
    W.chunk = pq.chunk;
    W.sub = pq.sub;
    return SS_OK;
  }
  err = hipFuncSetAttribute(sched_fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sched_lds);
  if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");
  FastPlan pl;
  SsScratch scr;
  void *scratch = nullptr;
  if (W.ptr) {  // the caller's workspace: the largest layout that fits, nothing allocated
    if (pmin.total > W.bytes)
      return ss_set_error(SS_ERR_INVALID_ARG, "workspace of " + std::to_string(W.bytes) +
                                                   " bytes is smaller than this call's minimum of " +
                                                   std::to_string(pmin.total));
    pl = plan_fit((int64_t)W.bytes);
    scratch = W.ptr;
  } else {
    // the largest layout within the budget; while its scratch cannot be
    // had, half the budget (down to the smallest layout)
    for (int64_t budget = pool_budget();; budget /= 2) {
      pl = plan_fit(budget);
      err = ss_scratch_get(g->device, g->pool, pl.total, stream, &scr);
      if (err != hipErrorOutOfMemory || pl.total <= pmin.total) break;
    }
    if (err != hipSuccess) return hip_fail(err, "allocating the simulation scratch");
    scratch = scr.p;
  }
  const int64_t chunk = pl.chunk;
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *PT = reinterpret_cast<uint8_t *>(take(pl.sz_pt));  // op-major copy, or candidate rows of op-major input
  auto *finT = reinterpret_cast<uint32_t *>(take(pl.sz_fin));
  auto *fin = reinterpret_cast<uint32_t *>(take(pl.sz_fin));
  MemPass M{};
  for (int k = 0; k < pl.sets; ++k) {
    M.own[k] = reinterpret_cast<Rec *>(take(pl.sz_own));
    M.cp[k] = reinterpret_cast<Rec *>(take(pl.sz_cp));
    M.meta[k] = reinterpret_cast<int32_t *>(take(pl.sz_meta));
  }
  M.rank = reinterpret_cast<uint16_t *>(take(pl.sz_rank));
  M.wk = reinterpret_cast<uint32_t *>(take(pl.sz_wk));
  M.wb = reinterpret_cast<int64_t *>(take(pl.sz_wb));
  M.ticket = reinterpret_cast<uint32_t *>(take(pl.sz_tk));
  M.n_ticket = pl.n_ticket;
  M.sub = pl.sub;
  M.nslots = pl.nslots;
  M.slot_cap = slot_cap;
  M.iv_fast = iv_fast;
  M.single = W.single;
  M.sets = pl.sets;
  M.aux = g->aux;

  int rc = mem_pass_events(M);
  if (rc == SS_OK) {
    hipLaunchKernelGGL(fill_zero_u32, dim3((unsigned)std::min<int64_t>((pl.n_ticket + 255) / 256, 1024)), dim3(256),
                       0, stream, M.ticket, pl.n_ticket);
    const hipError_t fe = hipGetLastError();
    if (fe != hipSuccess) rc = hip_fail(fe, "fill_zero_u32 launch");
  }
  auto check = [&](const char *what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess && rc == SS_OK) rc = hip_fail(e, what);
    return rc == SS_OK;
  };
  for (int64_t b0 = 0; b0 < B && rc == SS_OK; b0 += chunk) {
    const int64_t nb = std::min(chunk, B - b0);
    // the schedule reads op-major placements (the caller's own, or a copy of
    // the chunk's rows); the memory passes read candidate rows (the caller's
    // own, or a copy of the chunk from the op-major input)
    const uint8_t *sched_P = PT;
    int64_t ppitch = nb;
    const uint8_t *Pc = PT;
    SsTimingRec *tp = ss_timing_start(SS_KERNEL_TRANSPOSE, stream);
    if (src.op_major) {
      sched_P = src.p + b0;
      ppitch = B;
      const hipError_t te = ss_rows_from_op_major(src.p, N, B, b0, nb, PT, stream);
      if (te != hipSuccess && rc == SS_OK) rc = hip_fail(te, "transpose launch");
    } else {
      Pc = src.p + b0 * N;
      if (N > 0) {  // candidates' placement rows -> op-major [op][candidate]
        if (N % 4 == 0 && nb % 4 == 0 && (reinterpret_cast<uintptr_t>(Pc) & 3) == 0) {
          const dim3 tg((unsigned)((N + 127) / 128), (unsigned)((nb + 127) / 128));
          hipLaunchKernelGGL(transpose_u8_words, tg, dim3(256), 0, stream, Pc, nb, (int64_t)N, (int64_t)N, PT);
        } else {
          const dim3 tg((unsigned)((N + 63) / 64), (unsigned)((nb + 63) / 64));
          hipLaunchKernelGGL(transpose_tiles<uint8_t>, tg, dim3(256), 0, stream, Pc, nb, (int64_t)N, (int64_t)N,
                             PT);
        }
      }
    }
    ss_timing_stop(tp, stream);
    if (!check("transpose launch")) break;
    if (!M.single && M.it > 0) {  // the schedule runs with no peak pass beside it
      const hipError_t we = hipStreamWaitEvent(stream, M.pk_done[(M.it - 1) % M.sets], 0);
      if (we != hipSuccess && rc == SS_OK) rc = hip_fail(we, "hipStreamWaitEvent");
    }
    SsTimingRec *ts = ss_timing_start(SS_KERNEL_SCHEDULE, stream);
    {
      int64_t *ms_out = makespan + b0, *sf_out = sumfin ? sumfin + b0 : nullptr,
              *sl_out = slack ? slack + b0 * R : nullptr;
      uint8_t *vi_out = violation + b0;
      uint32_t *rows_out = sched_rows ? fin : nullptr;
      void *args[] = {const_cast<GmgView *>(&G), &sched_P, &ppitch, const_cast<int64_t *>(&nb), &finT, &ms_out,
                      &sf_out, &sl_out, &vi_out, &rows_out};
      const hipError_t le = hipLaunchKernel(sched_fn, dim3((unsigned)((nb + kWave - 1) / kWave)), dim3(kWave), args,
                                            sched_lds, stream);
      if (le != hipSuccess && rc == SS_OK) rc = hip_fail(le, "fast_schedule launch");
    }
    ss_timing_stop(ts, stream);
    if (!check("fast_schedule launch")) break;
    if (N > 0 && !sched_rows) {  // op-major -> candidates' rows for the memory passes
      SsTimingRec *tt = ss_timing_start(SS_KERNEL_TRANSPOSE, stream);
      if (N % 4 == 0 && nb % 4 == 0) {  // scratch buffers are 256-byte aligned
        const dim3 tg((unsigned)((nb + 63) / 64), (unsigned)((N + 64 * kStripTiles - 1) / (64 * kStripTiles)));
        hipLaunchKernelGGL(transpose_u32_strips, tg, dim3(256), 0, stream, static_cast<const uint32_t *>(finT),
                           (int64_t)N, nb, nb, fin);
      } else {
        const dim3 tg((unsigned)((nb + 63) / 64), (unsigned)((N + 63) / 64));
        hipLaunchKernelGGL(transpose_tiles<uint32_t>, tg, dim3(256), 0, stream, static_cast<const uint32_t *>(finT),
                           (int64_t)N, nb, nb, fin);
      }
      ss_timing_stop(tt, stream);
      if (!check("transpose launch")) break;
    }
    rc = memory_passes(g, M, Pc, fin, nb, false, peak ? peak + b0 * D : nullptr, violation + b0, stream);
  }
  const int jrc = mem_pass_join(M, stream);
  if (rc == SS_OK) rc = jrc;
  if (!W.ptr) {
    err = ss_scratch_put(g->device, &scr, stream);
    if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "releasing the scratch");
  }
  return rc;
}


size_t ss_ready_schedule_lds(const ss_gmg *g) { return ready_schedule_lds((int)g->n_dev, (int)g->n_req); }

int ss_run_simulate_ready(const ss_gmg *g, SsPlace src, int64_t *makespan, int64_t *peak, uint8_t *violation,
                          int64_t *slack, int64_t *sumfin, hipStream_t stream, SsWork &W) {
  const GmgView &G = g->view;
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev, R = g->n_req, B = src.B;
  const size_t lds = ss_ready_schedule_lds(g);
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  const bool iv_fast = g->n_class == 1 && g->n_link <= 2 && g->max_outdeg <= 2;
  // chunk: finish times, ranks, missing-predecessor counts and the spill list
  // of each candidate (candidate rows), and with op-major input the chunk's
  // placement rows
  const int64_t per_cand = N * (4 + 2 + 2 + 8 + (src.op_major ? 1 : 0));
  const int64_t rec_per_cand = (own_stride(N) + cp_stride(E)) * (int64_t)sizeof(Rec) + 3 * (D + 1) * 4;
  const int64_t slot_cap = N + E + 1;
  const int sets = W.single ? 1 : kRecSets;
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  // one lane per candidate (ready_lanes) unless SS_READY=wave; its per-device
  // ranks and per-request completions, and the flags of the candidates it
  // hands to ready_schedule
  const char *rmode = std::getenv("SS_READY");
  const bool lanes_env = !(rmode && std::strcmp(rmode, "wave") == 0);
  const size_t lane_lds = (size_t)(D + R) * kWave * 4;
  int lds_blk = 0;
  err = hipDeviceGetAttribute(&lds_blk, hipDeviceAttributeMaxSharedMemoryPerBlock, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  const bool lanes = lanes_env && lane_lds <= (size_t)lds_blk;  // else one wave per candidate throughout
  struct Plan {
    int64_t chunk, sub, nslots, n_ticket;
    size_t sz_fin, sz_rank, sz_miss, sz_spill, sz_rows, sz_own, sz_cp, sz_meta, sz_wk, sz_wb, sz_tk, sz_lane, total;
  };
  auto plan_of = [&](int64_t chunk, int64_t sub_cap) {
    Plan q{};
    q.chunk = chunk = std::min<int64_t>(std::max<int64_t>(1, chunk), B);
    int64_t sub = std::min<int64_t>(std::max<int64_t>(1, sub_cap), chunk);
    const int64_t n = std::max<int64_t>((chunk + sub - 1) / sub, chunk >= 8192 && !W.single ? 2 : 1);
    q.sub = sub = (chunk + n - 1) / n;
    q.nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kPeakBlocksPerCU, sub));
    q.sz_fin = align((size_t)chunk * N * 4 + 4);
    q.sz_rank = align(((size_t)chunk * N + 1) * 2);
    q.sz_miss = align(((size_t)chunk * N + 1) * 2);
    q.sz_spill = align((size_t)chunk * N * 8 + 8);
    q.sz_rows = src.op_major ? align((size_t)chunk * N + 1) : 0;
    q.sz_own = align((size_t)sub * own_stride(N) * sizeof(Rec));
    q.sz_cp = align((size_t)sub * cp_stride(E) * sizeof(Rec));
    q.sz_meta = align((size_t)sub * 3 * (D + 1) * 4);
    q.sz_wk = align((size_t)q.nslots * 2 * (slot_cap + 2) * 4);
    q.sz_wb = align((size_t)q.nslots * slot_cap * 8);
    q.n_ticket = (B + chunk - 1) / chunk * ((chunk + sub - 1) / sub);
    q.sz_tk = align((size_t)q.n_ticket * 4);
    q.sz_lane = lanes ? align((size_t)chunk * D * 2) + align((size_t)chunk * 4) : 0;
    q.total = q.sz_fin + q.sz_rank + q.sz_miss + q.sz_spill + q.sz_rows +
              (size_t)sets * (q.sz_own + q.sz_cp + q.sz_meta) + q.sz_wk + q.sz_wb + q.sz_tk + q.sz_lane;
    return q;
  };
  const int64_t sub_pref = std::max<int64_t>(1, kRecordBudget / std::max<int64_t>(1, rec_per_cand));
  // the lane kernel keeps one wave per 64 candidates resident: large chunks
  // (the fast path's chunk budget) fill the chip.  That is the preferred
  // layout (a caller's workspace of that size gets it); the pool path fits
  // the whole layout, record sets included, to seven eighths of the memory
  // the call can get now: sub-chunks shrink first (down to a sixteenth of the
  // chunk), then the chunk halves.
  const int64_t budget_pref = lanes ? kFastScratchBudget : kScratchBudget;
  const Plan ppref = plan_of(budget_pref / std::max<int64_t>(1, per_cand), sub_pref);
  const Plan pmin = plan_of(1, 1);
  auto plan_fit = [&](int64_t bytes) {
    if ((int64_t)ppref.total <= bytes) return ppref;
    int64_t chunk = ppref.chunk;
    for (;;) {
      const int64_t lo0 = chunk > kWave ? std::max<int64_t>(1, std::min<int64_t>(ppref.sub, chunk / 16)) : 1;
      if ((int64_t)plan_of(chunk, lo0).total <= bytes) {
        int64_t lo = lo0, hi = std::max<int64_t>(lo0, ppref.sub);  // the largest sub-chunk cap that fits
        while (lo < hi) {
          const int64_t mid = lo + (hi - lo + 1) / 2;
          if ((int64_t)plan_of(chunk, mid).total <= bytes)
            lo = mid;
          else
            hi = mid - 1;
        }
        return plan_of(chunk, lo);
      }
      if (chunk <= 1) return pmin;
      chunk = chunk > kWave ? chunk / 2 / kWave * kWave : chunk / 2;
    }
  };
  const int64_t budget0 = ss_scratch_budget(g->device, g->pool, (int64_t)ppref.total, 7);
  if (W.query) {
    W.need_min = pmin.total;
    W.need_pref = ppref.total;
    const Plan pq = W.single ? ppref : plan_fit(budget0);
    W.chunk = pq.chunk;
    W.sub = pq.sub;
    return SS_OK;
  }
  err = hipFuncSetAttribute(reinterpret_cast<const void *>(&ready_schedule), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");
  const int packed = G.succ2 && g->n_link <= 2 ? (g->max_indeg <= 2 ? 2 : g->max_indeg <= 4 ? 4 : 0) : 0;
  const void *lane_fn = packed == 2   ? reinterpret_cast<const void *>(&ready_lanes<2>)
                        : packed == 4 ? reinterpret_cast<const void *>(&ready_lanes<4>)
                                      : reinterpret_cast<const void *>(&ready_lanes<0>);
  if (lanes) {
    err = hipFuncSetAttribute(lane_fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lane_lds);
    if (err != hipSuccess) return hip_fail(err, "hipFuncSetAttribute");
  }
  Plan pl = ppref;
  SsScratch scr;
  void *scratch = nullptr;
  if (W.ptr) {
    if (pmin.total > W.bytes)
      return ss_set_error(SS_ERR_INVALID_ARG, "workspace of " + std::to_string(W.bytes) +
                                                   " bytes is smaller than this call's minimum of " +
                                                   std::to_string(pmin.total));
    pl = plan_fit((int64_t)W.bytes);
    scratch = W.ptr;
  } else {
    for (int64_t budget = budget0;; budget /= 2) {
      pl = plan_fit(budget);
      err = ss_scratch_get(g->device, g->pool, pl.total, stream, &scr);
      if (err != hipErrorOutOfMemory || pl.total <= pmin.total) break;
    }
    if (err != hipSuccess) return hip_fail(err, "allocating the simulation scratch");
    scratch = scr.p;
  }
  const int64_t chunk = pl.chunk;
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *fin = reinterpret_cast<uint32_t *>(take(pl.sz_fin));
  auto *rank = reinterpret_cast<uint16_t *>(take(pl.sz_rank));
  auto *miss = reinterpret_cast<uint16_t *>(take(pl.sz_miss));
  auto *spill = reinterpret_cast<uint64_t *>(take(pl.sz_spill));
  auto *rows = reinterpret_cast<uint8_t *>(take(pl.sz_rows));
  uint16_t *lcnt = nullptr;
  uint32_t *lovf = nullptr;
  if (lanes) {
    lcnt = reinterpret_cast<uint16_t *>(take(align((size_t)chunk * D * 2)));
    lovf = reinterpret_cast<uint32_t *>(take(align((size_t)chunk * 4)));
  }
  MemPass M{};
  for (int k = 0; k < sets; ++k) {
    M.own[k] = reinterpret_cast<Rec *>(take(pl.sz_own));
    M.cp[k] = reinterpret_cast<Rec *>(take(pl.sz_cp));
    M.meta[k] = reinterpret_cast<int32_t *>(take(pl.sz_meta));
  }
  M.rank = rank;
  M.wk = reinterpret_cast<uint32_t *>(take(pl.sz_wk));
  M.wb = reinterpret_cast<int64_t *>(take(pl.sz_wb));
  M.ticket = reinterpret_cast<uint32_t *>(take(pl.sz_tk));
  M.n_ticket = pl.n_ticket;
  M.sub = pl.sub;
  M.nslots = pl.nslots;
  M.slot_cap = slot_cap;
  M.iv_fast = iv_fast;
  M.single = W.single;
  M.sets = sets;
  M.aux = g->aux;

  int rc = mem_pass_events(M);
  if (rc == SS_OK) {
    hipLaunchKernelGGL(fill_zero_u32, dim3((unsigned)std::min<int64_t>((pl.n_ticket + 255) / 256, 1024)), dim3(256),
                       0, stream, M.ticket, pl.n_ticket);
    const hipError_t fe = hipGetLastError();
    if (fe != hipSuccess) rc = hip_fail(fe, "fill_zero_u32 launch");
  }
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
    SsTimingRec *ts = ss_timing_start(SS_KERNEL_SCHEDULE, stream);
    if (lanes) {
      int64_t *ms_out = makespan + b0, *sf_out = sumfin ? sumfin + b0 : nullptr,
              *sl_out = slack ? slack + b0 * R : nullptr;
      uint8_t *vi_out = violation + b0;
      const uint8_t *pc = Pc;
      int64_t nbv = nb;
      void *args[] = {const_cast<GmgView *>(&G), &pc, &nbv, &fin, &rank, &lcnt, &lovf, &ms_out, &sf_out, &sl_out,
                      &vi_out};
      err = hipLaunchKernel(lane_fn, dim3((unsigned)((nb + kWave - 1) / kWave)), dim3(kWave), args, lane_lds, stream);
      if (err == hipSuccess) err = hipGetLastError();
      if (err != hipSuccess) {
        rc = hip_fail(err, "ready_lanes launch");
        break;
      }
    }
    // the candidates ready_lanes flagged (all of them without it), one wave each
    hipLaunchKernelGGL(ready_schedule, dim3((unsigned)nb), dim3(kWave), lds, stream, G, Pc, fin, rank, miss, spill,
                       makespan + b0, sumfin ? sumfin + b0 : nullptr, slack ? slack + b0 * R : nullptr,
                       violation + b0, static_cast<const uint32_t *>(lovf));
    ss_timing_stop(ts, stream);
    err = hipGetLastError();
    if (err != hipSuccess) {
      rc = hip_fail(err, "ready_schedule launch");
      break;
    }
    rc = memory_passes(g, M, Pc, fin, nb, true, peak ? peak + b0 * D : nullptr, violation + b0, stream);
  }
  const int jrc = mem_pass_join(M, stream);
  if (rc == SS_OK) rc = jrc;
  if (!W.ptr) {
    err = ss_scratch_put(g->device, &scr, stream);
    if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "releasing the scratch");
  }
  return rc;
}

// The memory passes of the 32-bit path (fast_intervals, fast_peaks) for
// schedules computed elsewhere: candidate rows of placements P[B][N] and int64
// finish times fin[B][N] (every time below 2^32, which the loader proved when
// it enabled the 32-bit path).  Candidates already marked invalid are skipped.
namespace {
// Arrivals of one chunk, [edge][stride] int64 (candidate-minor, as the port
// schedule writes them), to candidate rows [nb][E] of u32 through 64 x 64
// LDS tiles (times fit 32 bits on this path).
__global__ __launch_bounds__(256) void arrival_rows(const int64_t *__restrict__ arr, int64_t stride, int64_t E,
                                                    int64_t nb, uint32_t *__restrict__ out) {
  __shared__ uint32_t tile[64][65];
  const int64_t c0 = (int64_t)blockIdx.x * 64, e0 = (int64_t)blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t e = e0 + i, c = c0 + tx;
    if (e < E && c < nb) tile[i][tx] = (uint32_t)arr[e * stride + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, e = e0 + tx;
    if (c < nb && e < E) out[c * E + e] = tile[tx][i];
  }
}

__global__ __launch_bounds__(256) void narrow_times(const int64_t *__restrict__ in, int64_t n, uint32_t *__restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = (uint32_t)in[i];
}
}  // namespace

int ss_run_memory_fast(const ss_gmg *g, const uint8_t *P, const int64_t *fin64, int64_t B, int64_t *peak,
                       uint8_t *violation, hipStream_t stream, const int64_t *arr64, int64_t arr_stride) {
  const int64_t N = g->n_ops, E = g->n_edges, D = g->n_dev;
  if (!g->view.time32 || N == 0) return ss_set_error(SS_ERR_UNSUPPORTED, "the 32-bit memory passes need ops and a 32-bit horizon");
  if (B == 0) return SS_OK;
  int cus = 0;
  hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, g->device);
  if (err != hipSuccess) return hip_fail(err, "hipDeviceGetAttribute");
  const bool iv_fast = g->n_class == 1 && g->n_link <= 2 && g->max_outdeg <= 2;
  const bool ports = arr64 != nullptr && E > 0;
  if (ports && (!iv_fast || !g->view.succ2_pe))
    return ss_set_error(SS_ERR_UNSUPPORTED, "port arrivals need the branch-free interval writer");
  const int64_t rec_per_cand = (own_stride(N) + cp_stride(E)) * (int64_t)sizeof(Rec) + 3 * (D + 1) * 4 + N * 2;
  const int64_t sub = std::min<int64_t>(B, std::max<int64_t>(1, kRecordBudget / std::max<int64_t>(1, rec_per_cand)));
  const int64_t chunk = std::min<int64_t>(B, std::max<int64_t>(1, kScratchBudget / ((N + (ports ? E : 0)) * 4)));
  const int64_t nslots = std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * kPeakBlocksPerCU, sub));
  const int64_t slot_cap = N + E + 1;
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t sz_fin = align((size_t)chunk * N * 4 + 4);
  const size_t sz_own = align((size_t)sub * own_stride(N) * sizeof(Rec));
  const size_t sz_cp = align((size_t)sub * cp_stride(E) * sizeof(Rec));
  const size_t sz_meta = align((size_t)sub * 3 * (D + 1) * 4);
  const size_t sz_rank = align(((size_t)sub * N + 1) * 2);
  const size_t sz_wk = align((size_t)nslots * 2 * (slot_cap + 2) * 4);
  const size_t sz_wb = align((size_t)nslots * slot_cap * 8);
  const int64_t n_chunk = (B + chunk - 1) / chunk;
  const int64_t n_ticket = n_chunk * ((chunk + sub - 1) / sub);
  const size_t sz_tk = align((size_t)n_ticket * 4);
  const size_t sz_arr = ports ? align((size_t)chunk * E * 4) : 0;
  SsScratch scr;
  err = ss_scratch_get(g->device, g->pool,
                       sz_fin + sz_arr + kRecSets * (sz_own + sz_cp + sz_meta) + sz_rank + sz_wk + sz_wb + sz_tk,
                       stream, &scr);
  void *scratch = scr.p;
  if (err != hipSuccess) return hip_fail(err, "allocating the memory-pass scratch");
  unsigned char *p = static_cast<unsigned char *>(scratch);
  auto take = [&](size_t bytes) {
    unsigned char *q = p;
    p += bytes;
    return q;
  };
  auto *fin = reinterpret_cast<uint32_t *>(take(sz_fin));
  auto *arr = ports ? reinterpret_cast<uint32_t *>(take(sz_arr)) : nullptr;
  MemPass M{};
  for (int k = 0; k < kRecSets; ++k) {
    M.own[k] = reinterpret_cast<Rec *>(take(sz_own));
    M.cp[k] = reinterpret_cast<Rec *>(take(sz_cp));
    M.meta[k] = reinterpret_cast<int32_t *>(take(sz_meta));
  }
  M.rank = reinterpret_cast<uint16_t *>(take(sz_rank));
  M.wk = reinterpret_cast<uint32_t *>(take(sz_wk));
  M.wb = reinterpret_cast<int64_t *>(take(sz_wb));
  M.ticket = reinterpret_cast<uint32_t *>(take(sz_tk));
  M.n_ticket = n_ticket;
  M.sub = sub;
  M.nslots = nslots;
  M.slot_cap = slot_cap;
  M.iv_fast = iv_fast;
  M.single = false;
  M.sets = kRecSets;
  M.aux = g->aux;
  int rc = mem_pass_events(M);
  if (rc == SS_OK) {
    hipLaunchKernelGGL(fill_zero_u32, dim3((unsigned)std::min<int64_t>((n_ticket + 255) / 256, 1024)), dim3(256), 0,
                       stream, M.ticket, n_ticket);
    const hipError_t fe = hipGetLastError();
    if (fe != hipSuccess) rc = hip_fail(fe, "fill_zero_u32 launch");
  }
  for (int64_t b0 = 0; b0 < B && rc == SS_OK; b0 += chunk) {
    const int64_t nb = std::min(chunk, B - b0);
    hipLaunchKernelGGL(narrow_times, dim3((unsigned)std::min<int64_t>((nb * N + 255) / 256, 8192)), dim3(256), 0,
                       stream, fin64 + b0 * N, nb * N, fin);
    err = hipGetLastError();
    if (err != hipSuccess) {
      rc = hip_fail(err, "narrow_times launch");
      break;
    }
    if (ports) {
      const dim3 tg((unsigned)((nb + 63) / 64), (unsigned)((E + 63) / 64));
      hipLaunchKernelGGL(arrival_rows, tg, dim3(256), 0, stream, arr64 + b0, arr_stride, E, nb, arr);
      err = hipGetLastError();
      if (err != hipSuccess) {
        rc = hip_fail(err, "arrival_rows launch");
        break;
      }
    }
    rc = memory_passes(g, M, P + b0 * N, fin, nb, false, peak ? peak + b0 * D : nullptr, violation + b0, stream, arr);
  }
  const int jrc = mem_pass_join(M, stream);
  if (rc == SS_OK) rc = jrc;
  err = ss_scratch_put(g->device, &scr, stream);
  if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "releasing the scratch");
  return rc;
}
