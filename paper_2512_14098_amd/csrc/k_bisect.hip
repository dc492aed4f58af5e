// k_bisect.hip -- cf_eval_bisect: phase 3 with the rates of each plan
// bisected over its grid instead of simulated at every grid point.
//
// A round is: compact the plans whose interval (lo, hi) is still open into
// (plan id, rate at mid) rows (one block, ordered prefix sums, so the rows
// keep plan order), simulate every seed of every row with the phase-3
// kernel, then move each row's lo or hi to mid by the pooled attainment test
// of the goodput reduction.  A grid of K rates closes after at most
// ceil(log2(K + 1)) rounds.
#include "cf_internal.h"

#include <cstring>

namespace cf {
namespace {

struct BisectState {
  int32_t *lo, *hi, *n_eval;
  uint32_t *status;
  uint64_t *events, *mlo;  // mlo: [n][T] pooled met counts at lo
  int32_t *act_idx, *act_ids;
  double *act_rates;
  uint32_t *n_act;
};

__global__ void k_bisect_init(BisectState B, int n, int K, int T) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  B.lo[i] = -1;
  B.hi[i] = K;
  B.n_eval[i] = 0;
  B.status[i] = 0;
  B.events[i] = 0;
  for (int t = 0; t < T; t++) B.mlo[(size_t)i * T + t] = 0;
}

// Plans with an open interval, in plan order: their index, plan id and the
// rate at mid.  One block of 1024 threads.
__global__ void __launch_bounds__(1024) k_bisect_next(BisectState B, int n, int K, const int32_t *plan_ids,
                                                      const double *rates) {
  __shared__ uint32_t part[1024];
  __shared__ uint32_t base_s;
  const int tid = threadIdx.x;
  if (tid == 0) base_s = 0;
  __syncthreads();
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int i = c0 + tid;
    const bool open = i < n && B.hi[i] - B.lo[i] > 1;
    part[tid] = open ? 1u : 0u;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {
      const uint32_t add = tid >= d ? part[tid - d] : 0u;
      __syncthreads();
      part[tid] += add;
      __syncthreads();
    }
    if (open) {
      const uint32_t j = base_s + part[tid] - 1u;
      const int mid = (B.lo[i] + B.hi[i]) / 2;
      B.act_idx[j] = i;
      B.act_ids[j] = plan_ids[i];
      B.act_rates[j] = rates[(size_t)i * K + mid];
    }
    __syncthreads();
    if (tid == 1023) base_s += part[1023];
    __syncthreads();
  }
  if (tid == 0) *B.n_act = base_s;
}

// One thread per simulated row: pool over seeds, test, move lo or hi.
__global__ void k_bisect_update(BisectState B, int n_act, int S, int T, uint32_t tn, uint32_t td,
                                const uint32_t *met, const uint32_t *cnt, const uint64_t *events,
                                const uint32_t *status) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n_act) return;
  const int i = B.act_idx[j];
  const int mid = (B.lo[i] + B.hi[i]) / 2;
  bool feasible = true;
  uint64_t M[CF_MAX_TYPES];
  for (int t = 0; t < T; t++) {
    uint64_t m = 0, c = 0;
    for (int s = 0; s < S; s++) {
      m += met[((size_t)j * S + s) * T + t];
      c += cnt[((size_t)j * S + s) * T + t];
    }
    M[t] = m;
    if (c > 0 && (uint64_t)td * m < (uint64_t)tn * c) feasible = false;
  }
  uint64_t ev = 0;
  uint32_t st = 0;
  for (int s = 0; s < S; s++) {
    ev += events[(size_t)j * S + s];
    st |= status[(size_t)j * S + s];
  }
  B.events[i] += ev;
  B.status[i] |= st;
  B.n_eval[i] += 1;
  if (st != 0) feasible = false;  // counts of a failed simulation are not evidence of attainment
  if (feasible) {
    B.lo[i] = mid;
    for (int t = 0; t < T; t++) B.mlo[(size_t)i * T + t] = M[t];
  } else {
    B.hi[i] = mid;
  }
}

__global__ void k_bisect_finish(BisectState B, int n, int K, int T, const double *rates, double denom,
                                int32_t *kstar, double *goodput_t, double *goodput, int32_t *n_eval,
                                uint64_t *events, uint32_t *status) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int lo = B.lo[i];
  double g = 0.0;
  for (int t = 0; t < T; t++) {
    const double gt = lo >= 0 ? (rates[(size_t)i * K + lo] * (double)B.mlo[(size_t)i * T + t]) / denom : 0.0;
    goodput_t[(size_t)i * T + t] = gt;
    g = g + gt;
  }
  kstar[i] = lo;
  goodput[i] = g;
  n_eval[i] = B.n_eval[i];
  events[i] = B.events[i];
  status[i] = B.status[i];
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace
}  // namespace cf

extern "C" cf_status cf_eval_bisect(const cf_model_desc *model, const cf_plan_table *plans,
                                    const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev, int32_t K,
                                    const cf_trace *trace, uint32_t theta_num, uint32_t theta_den, int32_t *kstar_dev,
                                    double *goodput_t_dev, double *goodput_dev, int32_t *n_eval_dev,
                                    uint64_t *events_dev, uint32_t *status_dev, void *stream) {
  using namespace cf;
  if (!model || !plans || !trace) return set_error(CF_EINVAL, "NULL argument");
  if (n_plans < 0 || K < 1 || K > 64 || theta_den == 0) return set_error(CF_EINVAL, "sizes or theta");
  const int T = model->n_types, S = trace->n_seeds;
  if (T < 1 || T > CF_MAX_TYPES || S < 1) return set_error(CF_EINVAL, "model or trace sizes");
  if (n_plans == 0) return CF_OK;
  if (!plan_ids_dev || !rates_dev || !kstar_dev || !goodput_t_dev || !goodput_dev || !n_eval_dev || !events_dev ||
      !status_dev)
    return set_error(CF_EINVAL, "NULL device array");
  const size_t n = (size_t)n_plans;
  size_t off[16], total = 0;
  const size_t sizes[] = {n * 4, n * 4, n * 4, n * 4, n * 8, n * T * 8, n * 4, n * 4, n * 8, 64,
                          n * S * T * 4, n * S * T * 4, n * S * 8, n * S * 4};
  const int nsz = (int)(sizeof sizes / sizeof sizes[0]);
  for (int k = 0; k < nsz; k++) {
    off[k] = total;
    total += align256(sizes[k]);
  }
  cf_status st = CF_OK;
  char *scr = (char *)scratch_get(SCR_BISECT, total, &st);
  if (!scr) return st;
  BisectState B;
  B.lo = (int32_t *)(scr + off[0]);
  B.hi = (int32_t *)(scr + off[1]);
  B.n_eval = (int32_t *)(scr + off[2]);
  B.status = (uint32_t *)(scr + off[3]);
  B.events = (uint64_t *)(scr + off[4]);
  B.mlo = (uint64_t *)(scr + off[5]);
  B.act_idx = (int32_t *)(scr + off[6]);
  B.act_ids = (int32_t *)(scr + off[7]);
  B.act_rates = (double *)(scr + off[8]);
  B.n_act = (uint32_t *)(scr + off[9]);
  uint32_t *met = (uint32_t *)(scr + off[10]);
  uint32_t *cnt = (uint32_t *)(scr + off[11]);
  uint64_t *events = (uint64_t *)(scr + off[12]);
  uint32_t *status = (uint32_t *)(scr + off[13]);
  hipStream_t s = as_stream(stream);
  const unsigned nb = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(k_bisect_init, dim3(nb), dim3(256), 0, s, B, n_plans, K, T);
  if ((st = hip_check(hipGetLastError(), "cf_eval_bisect init")) != CF_OK) return st;
  for (int round = 0; round <= 64; round++) {
    hipLaunchKernelGGL(k_bisect_next, dim3(1), dim3(1024), 0, s, B, n_plans, K, plan_ids_dev, rates_dev);
    if ((st = hip_check(hipGetLastError(), "cf_eval_bisect next")) != CF_OK) return st;
    uint32_t n_act = 0;
    if ((st = hip_check(hipMemcpyAsync(&n_act, B.n_act, sizeof n_act, hipMemcpyDeviceToHost, s), "bisect count")) !=
        CF_OK)
      return st;
    if ((st = hip_check(hipStreamSynchronize(s), "bisect sync")) != CF_OK) return st;
    if (n_act == 0) break;
    cf_fine_out fo;
    std::memset(&fo, 0, sizeof fo);
    fo.met_dev = met;
    fo.cnt_dev = cnt;
    fo.events_dev = events;
    fo.status_dev = status;
    st = cf_eval_fine(model, plans, B.act_ids, (int32_t)n_act, B.act_rates, 1, trace, 0, &fo, stream);
    if (st != CF_OK) return st;
    hipLaunchKernelGGL(k_bisect_update, dim3((n_act + 255) / 256), dim3(256), 0, s, B, (int)n_act, S, T, theta_num,
                       theta_den, met, cnt, events, status);
    if ((st = hip_check(hipGetLastError(), "cf_eval_bisect update")) != CF_OK) return st;
  }
  const double denom = (double)((uint64_t)S * (uint64_t)trace->n_req);
  hipLaunchKernelGGL(k_bisect_finish, dim3(nb), dim3(256), 0, s, B, n_plans, K, T, rates_dev, denom, kstar_dev,
                     goodput_t_dev, goodput_dev, n_eval_dev, events_dev, status_dev);
  return hip_check(hipGetLastError(), "cf_eval_bisect finish");
}
