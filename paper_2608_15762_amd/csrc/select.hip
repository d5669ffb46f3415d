// Best-candidate selection (Alg. 1: record feasible candidates, return the
// best; Sec. 3.4.2: discard out-of-memory placements, minimise the average
// completion time).  Lexicographic argmin of (key, index) over the feasible
// candidates, with no scratch: a grid-stride pass takes the smallest feasible
// key into out[1] (one 64-bit atomic minimum per block), a second pass the
// smallest index among the feasible candidates with that key into out[0],
// and one thread turns "nothing feasible" into -1.  Minima do not depend on
// the order in which blocks combine, so the result is deterministic.
#include <climits>

#include "ss_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 1024;

__device__ __forceinline__ bool feasible(const uint8_t *violation, const int64_t *slack, int64_t R, int require_sla,
                                         int64_t b) {
  if (violation[b] != 0) return false;
  if (require_sla)
    for (int64_t r = 0; r < R; ++r)
      if (slack[b * R + r] < 0) return false;
  return true;
}

__device__ int64_t block_min(int64_t x) {
  __shared__ int64_t part[kThreads / 64];
  for (int o = 32; o >= 1; o >>= 1) {
    const int64_t y = __shfl_xor(x, o, 64);
    x = y < x ? y : x;
  }
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  if (lane == 0) part[wave] = x;
  __syncthreads();
  int64_t r = INT64_MAX;
  if (threadIdx.x == 0)
    for (int w = 0; w < kThreads / 64; ++w) r = part[w] < r ? part[w] : r;
  return r;
}

__global__ void select_init(int64_t *__restrict__ out) {
  out[0] = INT64_MAX;
  out[1] = INT64_MAX;
}

__global__ __launch_bounds__(kThreads) void select_min_key(const uint8_t *__restrict__ violation,
                                                           const int64_t *__restrict__ key,
                                                           const int64_t *__restrict__ slack, int64_t R, int64_t B,
                                                           int require_sla, int64_t *__restrict__ out) {
  int64_t x = INT64_MAX;
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < B; b += (int64_t)gridDim.x * kThreads)
    if (feasible(violation, slack, R, require_sla, b) && key[b] < x) x = key[b];
  const int64_t r = block_min(x);
  if (threadIdx.x == 0 && r != INT64_MAX) atomicMin(reinterpret_cast<long long *>(&out[1]), (long long)r);
}

__global__ __launch_bounds__(kThreads) void select_min_index(const uint8_t *__restrict__ violation,
                                                             const int64_t *__restrict__ key,
                                                             const int64_t *__restrict__ slack, int64_t R, int64_t B,
                                                             int require_sla, int64_t *__restrict__ out) {
  const int64_t best = out[1];
  int64_t x = INT64_MAX;
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < B; b += (int64_t)gridDim.x * kThreads)
    if (key[b] == best && b < x && feasible(violation, slack, R, require_sla, b)) x = b;
  const int64_t r = block_min(x);
  if (threadIdx.x == 0 && r != INT64_MAX) atomicMin(reinterpret_cast<long long *>(&out[0]), (long long)r);
}

__global__ void select_finish(int64_t *__restrict__ out) {
  if (out[0] == INT64_MAX) out[0] = -1;  // nothing feasible: {-1, INT64_MAX}
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

}  // namespace

int ss_run_select(const ss_gmg *g, const uint8_t *violation, const int64_t *key, const int64_t *slack, int64_t B,
                  int require_sla, int64_t *out_best, hipStream_t stream) {
  const int nblk = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxBlocks, (B + kThreads - 1) / kThreads));
  SsTimingRec *t_sel = ss_timing_start(SS_KERNEL_SELECT, stream);
  hipLaunchKernelGGL(select_init, dim3(1), dim3(1), 0, stream, out_best);
  hipLaunchKernelGGL(select_min_key, dim3(nblk), dim3(kThreads), 0, stream, violation, key, slack, g->n_req, B,
                     require_sla, out_best);
  hipLaunchKernelGGL(select_min_index, dim3(nblk), dim3(kThreads), 0, stream, violation, key, slack, g->n_req, B,
                     require_sla, out_best);
  hipLaunchKernelGGL(select_finish, dim3(1), dim3(1), 0, stream, out_best);
  ss_timing_stop(t_sel, stream);
  const hipError_t err = hipGetLastError();
  return err != hipSuccess ? hip_fail(err, "selection launch") : SS_OK;
}
