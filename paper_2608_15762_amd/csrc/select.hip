// Best-candidate selection (Alg. 1: record feasible candidates, return the
// best; Sec. 3.4.2: discard out-of-memory placements, minimise the average
// completion time).  Lexicographic argmin of (key, index) over the feasible
// candidates: a grid-stride pass leaves one (key, index) per block, a single
// block reduces those.  The operator is associative and commutative, so the
// result does not depend on the reduction order.
#include <climits>

#include "ss_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 1024;

struct Best {
  int64_t key, idx;  // idx == INT64_MAX: nothing feasible
};

__device__ __forceinline__ Best better(Best a, Best b) {
  return (b.key < a.key || (b.key == a.key && b.idx < a.idx)) ? b : a;
}

__device__ Best block_best(Best x) {
  __shared__ int64_t sk[kThreads / 64], si[kThreads / 64];
  for (int o = 32; o >= 1; o >>= 1) {
    Best y{__shfl_xor(x.key, o, 64), __shfl_xor(x.idx, o, 64)};
    x = better(x, y);
  }
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  if (lane == 0) {
    sk[wave] = x.key;
    si[wave] = x.idx;
  }
  __syncthreads();
  Best r{INT64_MAX, INT64_MAX};
  if (threadIdx.x == 0)
    for (int w = 0; w < kThreads / 64; ++w) r = better(r, Best{sk[w], si[w]});
  return r;
}

__global__ __launch_bounds__(kThreads) void select_partial(const uint8_t *__restrict__ violation,
                                                           const int64_t *__restrict__ key,
                                                           const int64_t *__restrict__ slack, int64_t R, int64_t B,
                                                           int require_sla, int64_t *__restrict__ part) {
  Best x{INT64_MAX, INT64_MAX};
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < B; b += (int64_t)gridDim.x * kThreads) {
    if (violation[b] != 0) continue;
    if (require_sla) {
      bool ok = true;
      for (int64_t r = 0; r < R; ++r) ok = ok && slack[b * R + r] >= 0;
      if (!ok) continue;
    }
    x = better(x, Best{key[b], b});
  }
  const Best r = block_best(x);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = r.key;
    part[2 * blockIdx.x + 1] = r.idx;
  }
}

__global__ __launch_bounds__(kThreads) void select_final(const int64_t *__restrict__ part, int nparts,
                                                         int64_t *__restrict__ out) {
  Best x{INT64_MAX, INT64_MAX};
  for (int i = threadIdx.x; i < nparts; i += kThreads) x = better(x, Best{part[2 * i], part[2 * i + 1]});
  const Best r = block_best(x);
  if (threadIdx.x == 0) {
    const bool none = r.idx == INT64_MAX;
    out[0] = none ? -1 : r.idx;
    out[1] = none ? INT64_MAX : r.key;
  }
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

}  // namespace

int ss_run_select(const ss_gmg *g, const uint8_t *violation, const int64_t *key, const int64_t *slack, int64_t B,
                  int require_sla, int64_t *out_best, hipStream_t stream) {
  const int nblk = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxBlocks, (B + kThreads - 1) / kThreads));
  void *part = nullptr;
  hipError_t err = ss_pool_malloc(&part, (size_t)nblk * 2 * sizeof(int64_t), g->pool, stream);
  if (err != hipSuccess) return hip_fail(err, "allocating the selection scratch");
  int rc = SS_OK;
  SsTimingRec *t_sel = ss_timing_start(SS_KERNEL_SELECT, stream);
  hipLaunchKernelGGL(select_partial, dim3(nblk), dim3(kThreads), 0, stream, violation, key, slack, g->n_req, B,
                     require_sla, static_cast<int64_t *>(part));
  err = hipGetLastError();
  if (err != hipSuccess) rc = hip_fail(err, "select_partial launch");
  if (rc == SS_OK) {
    hipLaunchKernelGGL(select_final, dim3(1), dim3(kThreads), 0, stream, static_cast<const int64_t *>(part), nblk,
                       out_best);
    err = hipGetLastError();
    if (err != hipSuccess) rc = hip_fail(err, "select_final launch");
  }
  ss_timing_stop(t_sel, stream);
  err = hipFreeAsync(part, stream);
  if (rc == SS_OK && err != hipSuccess) rc = hip_fail(err, "hipFreeAsync");
  return rc;
}
