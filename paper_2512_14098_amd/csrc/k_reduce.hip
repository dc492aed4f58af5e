// k_reduce.hip -- cf_goodput_reduce, cf_select_best and the diagnostic
// element-wise evaluators of the device primitives.
//
// Goodput of a type is the throughput of its requests that meet their
// latency target (Sec. 3.2); a plan is credited with its maximum achievable
// goodput, at the highest rate it supports (Sec. 6.1); the selected plan
// maximises the sum over types (Alg. 2).  One wavefront per plan: lane k
// pools rate k's counts over seeds (u64, exact), a ballot of the infeasible
// rates gives the first failure (what bisection over a monotone predicate
// returns), and lanes t compute the per-type goodput at that rate.  A rate
// at which some seed's simulation ended with a nonzero status word (invalid
// plan or rate, exceeded capacity, deadlock) is infeasible: its counts are
// truncated and say nothing about attainment.
#include "cf_internal.h"

namespace cf {
namespace {

__global__ void __launch_bounds__(64) k_goodput(const uint32_t *met, const uint32_t *cnt, const uint32_t *status,
                                               int K, int S, int T, const double *rates, uint32_t tn, uint32_t td,
                                               double denom, int32_t *kstar, double *goodput_t, double *goodput) {
  const int i = blockIdx.x, lane = threadIdx.x;
  bool infeasible = false;
  if (lane < K) {
    for (int s = 0; s < S; s++) infeasible |= status[((size_t)i * K + lane) * S + s] != 0u;
    for (int t = 0; t < T; t++) {
      uint64_t M = 0, N = 0;
      for (int s = 0; s < S; s++) {
        const size_t o = (((size_t)i * K + lane) * S + s) * T + t;
        M += met[o];
        N += cnt[o];
      }
      if (N > 0 && (uint64_t)td * M < (uint64_t)tn * N) infeasible = true;
    }
  }
  const uint64_t bad = __ballot(infeasible);
  const int ks = bad ? (__ffsll((long long)bad) - 2) : K - 1;
  double gt = 0.0;
  if (lane < T && ks >= 0) {
    uint64_t M = 0;
    for (int s = 0; s < S; s++) M += met[(((size_t)i * K + ks) * S + s) * T + lane];
    gt = (rates[(size_t)i * K + ks] * (double)M) / denom;
  }
  if (lane < T) goodput_t[(size_t)i * T + lane] = gt;
  double g = 0.0;
  for (int t = 0; t < T; t++) g = g + __shfl(gt, t, 64);
  if (lane == 0) {
    kstar[i] = ks;
    goodput[i] = g;
  }
}

// The same computation per latency-target bin b: block (i, b), lane k pools
// rate k's requests in bins 0..b over seeds.
__global__ void __launch_bounds__(64) k_goodput_curve(const uint32_t *hist, const uint32_t *cnt,
                                                     const uint32_t *status, int K, int S, int T, int nb,
                                                     const double *rates, uint32_t tn, uint32_t td, double denom,
                                                     int32_t *kstar, double *goodput_t, double *goodput) {
  const int i = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int hw = nb + 1;
  auto pooled = [&](int k, int t) {
    uint64_t M = 0;
    for (int s = 0; s < S; s++) {
      const uint32_t *h = hist + ((((size_t)i * K + k) * S + s) * T + t) * hw;
      for (int q = 0; q <= b; q++) M += h[q];
    }
    return M;
  };
  bool infeasible = false;
  if (lane < K) {
    for (int s = 0; s < S; s++) infeasible |= status[((size_t)i * K + lane) * S + s] != 0u;
    for (int t = 0; t < T; t++) {
      uint64_t N = 0;
      for (int s = 0; s < S; s++) N += cnt[(((size_t)i * K + lane) * S + s) * T + t];
      const uint64_t M = pooled(lane, t);
      if (N > 0 && (uint64_t)td * M < (uint64_t)tn * N) infeasible = true;
    }
  }
  const uint64_t bad = __ballot(infeasible);
  const int ks = bad ? (__ffsll((long long)bad) - 2) : K - 1;
  double gt = 0.0;
  if (lane < T && ks >= 0) gt = (rates[(size_t)i * K + ks] * (double)pooled(ks, lane)) / denom;
  const size_t ob = (size_t)i * nb + b;
  if (lane < T) goodput_t[ob * T + lane] = gt;
  double g = 0.0;
  for (int t = 0; t < T; t++) g = g + __shfl(gt, t, 64);
  if (lane == 0) {
    kstar[ob] = ks;
    goodput[ob] = g;
  }
}

__global__ void __launch_bounds__(256) k_best(const double *g, int n, int32_t *best) {
  __shared__ double bv[256];
  __shared__ int bi[256];
  double v = 0.0;
  int idx = -1;
  for (int j = threadIdx.x; j < n; j += 256) {
    const double x = g[j];
    if (idx < 0 || x > v) { v = x; idx = j; }  // strided: j increases, so ties keep the lower index
  }
  bv[threadIdx.x] = v;
  bi[threadIdx.x] = idx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      const double ov = bv[threadIdx.x + w];
      const int oi = bi[threadIdx.x + w];
      const int mi = bi[threadIdx.x];
      if (oi >= 0 && (mi < 0 || ov > bv[threadIdx.x] || (ov == bv[threadIdx.x] && oi < mi))) {
        bv[threadIdx.x] = ov;
        bi[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) best[0] = bi[0];
}

__global__ void k_math(int op, const double *x, const double *y, double *out, long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double a = x[i];
  double r = 0.0;
  switch (op) {
    case 0: r = dev_log(a); break;
    case 1: r = dev_exp(a); break;
    case 2: r = sqrt(a); break;
    case 3: r = a / y[i]; break;
    case 4: r = u01((uint64_t)__double_as_longlong(a)); break;
    default: break;
  }
  out[i] = r;
}

__global__ void k_philox(const uint64_t *ctr, const uint64_t *key, uint64_t *out, long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint64_t o[4];
  philox4x64_10(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3], key[2 * i], key[2 * i + 1], o);
  for (int j = 0; j < 4; j++) out[4 * i + j] = o[j];
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_goodput_reduce(const cf_fine_out *fine, int32_t n_plans, int32_t K, int32_t S, int32_t T,
                                       const double *rates_dev, uint32_t theta_num, uint32_t theta_den,
                                       int32_t n_req, int32_t *kstar_dev, double *goodput_t_dev,
                                       double *goodput_dev, void *stream) {
  using namespace cf;
  if (!fine || !fine->met_dev || !fine->cnt_dev || !fine->status_dev || !rates_dev || !kstar_dev ||
      !goodput_t_dev || !goodput_dev)
    return set_error(CF_EINVAL, "NULL argument");
  if (n_plans < 0 || K < 1 || S < 1 || T < 1 || T > CF_MAX_TYPES || n_req < 0 || theta_den == 0)
    return set_error(CF_EINVAL, "sizes");
  if (K > 64) return set_error(CF_ECAPACITY, "K above 64 (one lane per rate)");
  if (n_plans == 0) return CF_OK;
  const double denom = (double)((uint64_t)S * (uint64_t)n_req);
  hipLaunchKernelGGL(k_goodput, dim3((unsigned)n_plans), dim3(64), 0, as_stream(stream), fine->met_dev,
                     fine->cnt_dev, fine->status_dev, K, S, T, rates_dev, theta_num, theta_den, denom, kstar_dev,
                     goodput_t_dev, goodput_dev);
  return hip_check(hipGetLastError(), "cf_goodput_reduce launch");
}

extern "C" cf_status cf_goodput_curve(const cf_fine_out *fine, int32_t n_plans, int32_t K, int32_t S, int32_t T,
                                      const double *rates_dev, uint32_t theta_num, uint32_t theta_den,
                                      int32_t n_req, int32_t *kstar_dev, double *goodput_t_dev, double *goodput_dev,
                                      void *stream) {
  using namespace cf;
  if (!fine) return set_error(CF_EINVAL, "NULL argument");
  const int32_t n_bins = fine->n_bins;
  if (n_plans < 0 || K < 1 || S < 1 || T < 1 || T > CF_MAX_TYPES || n_req < 0 || theta_den == 0)
    return set_error(CF_EINVAL, "sizes");
  if (n_bins < 1 || n_bins > 64) return set_error(CF_EINVAL, "n_bins must be in 1..64");
  if (K > 64) return set_error(CF_ECAPACITY, "K above 64 (one lane per rate)");
  if (n_plans == 0) return CF_OK;
  if (!fine->hist_dev || !fine->cnt_dev || !fine->status_dev || !rates_dev || !kstar_dev || !goodput_t_dev ||
      !goodput_dev)
    return set_error(CF_EINVAL, "NULL device array");
  const double denom = (double)((uint64_t)S * (uint64_t)n_req);
  hipLaunchKernelGGL(k_goodput_curve, dim3((unsigned)n_plans, (unsigned)n_bins), dim3(64), 0, as_stream(stream),
                     fine->hist_dev, fine->cnt_dev, fine->status_dev, K, S, T, n_bins, rates_dev, theta_num,
                     theta_den, denom, kstar_dev, goodput_t_dev, goodput_dev);
  return hip_check(hipGetLastError(), "cf_goodput_curve launch");
}

extern "C" cf_status cf_select_best(const double *goodput_dev, int32_t n, int32_t *best_dev, void *stream) {
  using namespace cf;
  if (!goodput_dev || !best_dev || n < 1) return set_error(CF_EINVAL, "arguments");
  hipLaunchKernelGGL(k_best, dim3(1), dim3(256), 0, as_stream(stream), goodput_dev, n, best_dev);
  return hip_check(hipGetLastError(), "cf_select_best launch");
}

extern "C" cf_status cf_math_eval(int32_t op, const double *x_dev, const double *y_dev, double *out_dev,
                                  int64_t n, void *stream) {
  using namespace cf;
  if (!x_dev || !out_dev || op < 0 || op > 4 || (op == 3 && !y_dev) || n < 0)
    return set_error(CF_EINVAL, "arguments");
  if (n == 0) return CF_OK;
  hipLaunchKernelGGL(k_math, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, as_stream(stream), op, x_dev, y_dev,
                     out_dev, (long long)n);
  return hip_check(hipGetLastError(), "cf_math_eval launch");
}

extern "C" cf_status cf_philox_eval(const uint64_t *ctr_dev, const uint64_t *key_dev, uint64_t *out_dev, int64_t n,
                                    void *stream) {
  using namespace cf;
  if (!ctr_dev || !key_dev || !out_dev || n < 0) return set_error(CF_EINVAL, "arguments");
  if (n == 0) return CF_OK;
  hipLaunchKernelGGL(k_philox, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, as_stream(stream), ctr_dev, key_dev,
                     out_dev, (long long)n);
  return hip_check(hipGetLastError(), "cf_philox_eval launch");
}
