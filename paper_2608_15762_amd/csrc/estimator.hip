// Online linear estimators (Sec. 3.3.1) for gfx950: ordinary least-squares
// fits refined as samples are fed back.  The state of an estimator set is the
// sufficient statistics of every fit, in device memory, float64:
//   gram[e][F][F] = sum x x^T,  mom[e][F] = sum x y,  count[e].
//
// est_accumulate  a group of lanes per estimator (sized to the batch's average
//                 samples per estimator): its lanes stride over the estimator's
//                 samples (grouped by estimator), sum in registers, and reduce
//                 across the group in a fixed order (results do not depend on
//                 scheduling), then add to the state.
// est_solve       one lane per estimator: Cholesky factorisation of the Gram
//                 matrix and two triangular solves for the coefficients.
// est_predict     one lane per query: integer microseconds for the simulator.
#include <climits>
#include <cmath>

#include "ss_internal.h"

struct ss_est {
  int device = 0;
  int64_t n_est = 0, n_feat = 0;
  double *gram = nullptr, *mom = nullptr;  // [n_est][F][F], [n_est][F]
  int64_t *count = nullptr;                // [n_est]
};

namespace {

constexpr int kWave = 64;
constexpr double kPivotRtol = 1e-12;  // relative pivot below which a Gram matrix is singular

// kL lanes per estimator (a power of two dividing 64): each wave serves
// 64 / kL estimators, lane t of a group takes samples t, t + kL, ...; the
// group then reduces by a fixed butterfly, so the sums do not depend on how
// the device schedules the work.
template <int F, int kL>
__global__ __launch_bounds__(kWave) void est_accumulate(int64_t n_est, const int64_t *__restrict__ ptr,
                                                        int64_t n_samples, const double *__restrict__ x,
                                                        const double *__restrict__ y, double *__restrict__ gram,
                                                        double *__restrict__ mom, int64_t *__restrict__ count) {
  const int lane = threadIdx.x, t = lane & (kL - 1);
  const int64_t e = (int64_t)blockIdx.x * (kWave / kL) + lane / kL;
  const bool live = e < n_est;
  const int64_t ec = live ? e : n_est - 1;
  // the estimator's samples, clamped to [0, n_samples)
  const int64_t s0 = min(max(ptr[ec], (int64_t)0), n_samples);
  const int64_t s1 = live ? min(max(ptr[ec + 1], s0), n_samples) : s0;
  double g[F * (F + 1) / 2], m[F];
#pragma unroll
  for (int i = 0; i < F * (F + 1) / 2; ++i) g[i] = 0.0;
#pragma unroll
  for (int i = 0; i < F; ++i) m[i] = 0.0;
  for (int64_t s = s0 + t; s < s1; s += kL) {
    double v[F];
#pragma unroll
    for (int i = 0; i < F; ++i) v[i] = x[s * F + i];
    const double yt = y[s];
    int k = 0;
#pragma unroll
    for (int i = 0; i < F; ++i) {
      m[i] = fma(v[i], yt, m[i]);
#pragma unroll
      for (int j = i; j < F; ++j, ++k) g[k] = fma(v[i], v[j], g[k]);
    }
  }
  auto group_sum = [&](double v) {
#pragma unroll
    for (int o = kL / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
  };
  double *ge = gram + ec * F * F, *me = mom + ec * F;
  const bool writer = live && t == 0;
  int k = 0;
#pragma unroll
  for (int i = 0; i < F; ++i) {
    const double mi = group_sum(m[i]);
    if (writer) me[i] += mi;
#pragma unroll
    for (int j = i; j < F; ++j, ++k) {
      const double gij = group_sum(g[k]);
      if (writer) {
        ge[i * F + j] += gij;
        if (j != i) ge[j * F + i] += gij;
      }
    }
  }
  if (writer) count[ec] += s1 - s0;
}

template <int F>
__global__ __launch_bounds__(256) void est_solve(int64_t n_est, const double *__restrict__ gram,
                                                 const double *__restrict__ mom, const int64_t *__restrict__ count,
                                                 double *__restrict__ coef, int32_t *__restrict__ status) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_est) return;
  double L[F][F], z[F], beta[F];
  const double *a = gram + e * F * F, *b = mom + e * F;
  int st = SS_EST_FITTED;
  if (count[e] < F) st = SS_EST_UNDERDETERMINED;
  for (int j = 0; j < F && st == SS_EST_FITTED; ++j) {
    double d = a[j * F + j];
    for (int k = 0; k < j; ++k) d -= L[j][k] * L[j][k];
    if (!(d > kPivotRtol * fabs(a[j * F + j])) || a[j * F + j] <= 0.0) {
      st = SS_EST_SINGULAR;
      break;
    }
    L[j][j] = sqrt(d);
    for (int i = j + 1; i < F; ++i) {
      double s = a[i * F + j];
      for (int k = 0; k < j; ++k) s -= L[i][k] * L[j][k];
      L[i][j] = s / L[j][j];
    }
  }
  if (st == SS_EST_FITTED) {
    for (int i = 0; i < F; ++i) {  // L z = mom
      double s = b[i];
      for (int k = 0; k < i; ++k) s -= L[i][k] * z[k];
      z[i] = s / L[i][i];
    }
    for (int i = F - 1; i >= 0; --i) {  // L^T beta = z
      double s = z[i];
      for (int k = i + 1; k < F; ++k) s -= L[k][i] * beta[k];
      beta[i] = s / L[i][i];
    }
  }
  for (int i = 0; i < F; ++i) coef[e * F + i] = st == SS_EST_FITTED ? beta[i] : 0.0;
  status[e] = st;
}

__global__ __launch_bounds__(256) void est_predict(const double *__restrict__ coef, int64_t n_est, int F,
                                                   const int32_t *__restrict__ est_of, const double *__restrict__ x,
                                                   int64_t M, int64_t *__restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const int32_t e = est_of[i];
  if (e < 0 || e >= n_est) {
    out[i] = 0;  // unknown estimator
    return;
  }
  // products and sums rounded one by one, in feature order (no fused
  // multiply-add): the integer decision below is then reproducible bit for bit
  double t = 0.0;
  for (int j = 0; j < F; ++j) t = __dadd_rn(t, __dmul_rn(x[i * F + j], coef[(int64_t)e * F + j]));
  const double c = ceil(t);
  out[i] = !(c < 4.611686018427388e18) ? 0 : c < 1.0 ? 1 : (int64_t)c;  // not finite or >= 2^62: 0
}

int hip_fail(hipError_t err, const char *what) {
  return ss_set_error(err == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                      std::string(what) + ": " + hipGetErrorString(err));
}

template <int F, int kL>
void launch_group(const ss_est *E, const int64_t *ptr, int64_t S, const double *x, const double *y,
                  hipStream_t stream) {
  constexpr int64_t per = kWave / kL;  // estimators per wave
  hipLaunchKernelGGL((est_accumulate<F, kL>), dim3((unsigned)((E->n_est + per - 1) / per)), dim3(kWave), 0, stream,
                     E->n_est, ptr, S, x, y, E->gram, E->mom, E->count);
}

// Lanes per estimator from the average samples per estimator of the batch
// (4 .. 64), so that most lanes have a sample.
template <int F>
void launch_accumulate(const ss_est *E, const int64_t *ptr, int64_t S, const double *x, const double *y,
                       hipStream_t stream) {
  const int64_t avg = S / E->n_est;
  if (avg >= 48)
    launch_group<F, 64>(E, ptr, S, x, y, stream);
  else if (avg >= 24)
    launch_group<F, 32>(E, ptr, S, x, y, stream);
  else if (avg >= 12)
    launch_group<F, 16>(E, ptr, S, x, y, stream);
  else if (avg >= 6)
    launch_group<F, 8>(E, ptr, S, x, y, stream);
  else
    launch_group<F, 4>(E, ptr, S, x, y, stream);
}

template <int F>
void launch_solve(const ss_est *E, double *coef, int32_t *status, hipStream_t stream) {
  hipLaunchKernelGGL(est_solve<F>, dim3((unsigned)((E->n_est + 255) / 256)), dim3(256), 0, stream, E->n_est, E->gram,
                     E->mom, E->count, coef, status);
}

}  // namespace

int ss_run_est_create(int64_t n_est, int64_t n_feat, ss_est **out) {
  auto *E = new ss_est();
  E->n_est = n_est;
  E->n_feat = n_feat;
  hipError_t err = hipGetDevice(&E->device);
  const size_t g = (size_t)n_est * n_feat * n_feat * sizeof(double), m = (size_t)n_est * n_feat * sizeof(double),
               c = (size_t)n_est * sizeof(int64_t);
  void *mem = nullptr;
  if (err == hipSuccess) err = hipMalloc(&mem, g + m + c + 8);
  if (err == hipSuccess) err = hipMemset(mem, 0, g + m + c + 8);
  if (err == hipSuccess) err = hipDeviceSynchronize();
  if (err != hipSuccess) {
    if (mem) (void)hipFree(mem);
    delete E;
    return hip_fail(err, "allocating the estimator state");
  }
  E->gram = static_cast<double *>(mem);
  E->mom = E->gram + (size_t)n_est * n_feat * n_feat;
  E->count = reinterpret_cast<int64_t *>(E->mom + (size_t)n_est * n_feat);
  *out = E;
  return SS_OK;
}

void ss_run_est_free(ss_est *E) {
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(E->device);
  (void)hipDeviceSynchronize();
  (void)hipFree(E->gram);
  (void)hipSetDevice(prev);
  delete E;
}

int ss_run_est_info(const ss_est *E, int64_t *n_est, int64_t *n_feat, int *device) {
  if (n_est) *n_est = E->n_est;
  if (n_feat) *n_feat = E->n_feat;
  if (device) *device = E->device;
  return SS_OK;
}

int ss_run_est_add(const ss_est *E, const int64_t *ptr, int64_t S, const double *x, const double *y,
                   hipStream_t stream) {
  if (E->n_est == 0) return SS_OK;
  using L = void (*)(const ss_est *, const int64_t *, int64_t, const double *, const double *, hipStream_t);
  static const L table[SS_EST_MAX_FEAT] = {launch_accumulate<1>, launch_accumulate<2>, launch_accumulate<3>,
                                           launch_accumulate<4>, launch_accumulate<5>, launch_accumulate<6>,
                                           launch_accumulate<7>, launch_accumulate<8>};
  SsTimingRec *t = ss_timing_start(SS_KERNEL_ESTIMATOR, stream);
  table[E->n_feat - 1](E, ptr, S, x, y, stream);
  ss_timing_stop(t, stream);
  const hipError_t err = hipGetLastError();
  return err == hipSuccess ? SS_OK : hip_fail(err, "est_accumulate launch");
}

int ss_run_est_solve(const ss_est *E, double *coef, int32_t *status, hipStream_t stream) {
  if (E->n_est == 0) return SS_OK;
  using L = void (*)(const ss_est *, double *, int32_t *, hipStream_t);
  static const L table[SS_EST_MAX_FEAT] = {launch_solve<1>, launch_solve<2>, launch_solve<3>, launch_solve<4>,
                                           launch_solve<5>, launch_solve<6>, launch_solve<7>, launch_solve<8>};
  SsTimingRec *t = ss_timing_start(SS_KERNEL_ESTIMATOR, stream);
  table[E->n_feat - 1](E, coef, status, stream);
  ss_timing_stop(t, stream);
  const hipError_t err = hipGetLastError();
  return err == hipSuccess ? SS_OK : hip_fail(err, "est_solve launch");
}

int ss_run_est_predict(const double *coef, int64_t n_est, int64_t n_feat, const int32_t *est_of, const double *x,
                       int64_t M, int64_t *out, hipStream_t stream) {
  if (M == 0) return SS_OK;
  SsTimingRec *t = ss_timing_start(SS_KERNEL_ESTIMATOR, stream);
  hipLaunchKernelGGL(est_predict, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, stream, coef, n_est, (int)n_feat,
                     est_of, x, M, out);
  ss_timing_stop(t, stream);
  const hipError_t err = hipGetLastError();
  return err == hipSuccess ? SS_OK : hip_fail(err, "est_predict launch");
}
