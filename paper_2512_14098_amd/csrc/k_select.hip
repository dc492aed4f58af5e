// k_select.hip -- cf_select_topk and cf_rate_grid.
//
// Top-K of the plans kept by phase 1, ordered by R_d descending and plan id
// ascending (Alg. 2 evaluates the most promising survivors first; the rate
// grid scales with the headroom alpha of Sec. 4.3).  The order key is the
// 96-bit value (bits of R_d, ~id): unique per plan, so the K largest keys
// are found by an MSD radix select of 12 eight-bit digits, compacted, and
// placed by rank (number of larger keys).
//
// cf_topk_merge keeps the top-K of a plan space screened window by window:
// the window's selection and the running list are both in key order, so
// each element's place in the merged list is its index in its own list plus
// the number of elements of the other list ahead of it (a binary search).
#include <cmath>

#include "cf_internal.h"

namespace cf {
namespace {

struct SelState {
  unsigned long long pre_hi;  // decided high bits of the threshold key
  unsigned int pre_lo;
  unsigned int k_rem;         // keys still to take at or below the prefix
  unsigned int all;           // fewer candidates than k: take every kept plan
  unsigned int count;         // compacted so far
  unsigned int hist[256];
};

__device__ __forceinline__ void plan_key(const double *rd, int p, unsigned long long &hi, unsigned int &lo) {
  hi = (unsigned long long)__double_as_longlong(rd[p]);
  lo = 0xFFFFFFFFu - (unsigned int)p;
}

// digit d (0 = most significant) of the 96-bit key
__device__ __forceinline__ unsigned int key_digit(unsigned long long hi, unsigned int lo, int d) {
  return d < 8 ? (unsigned int)(hi >> (56 - 8 * d)) & 0xFFu : (lo >> (24 - 8 * (d - 8))) & 0xFFu;
}

__device__ __forceinline__ bool prefix_match(unsigned long long hi, unsigned int lo, const SelState *st, int d) {
  // compares the first d digits with the prefix decided so far
  if (d <= 8) {
    if (d == 0) return true;
    const unsigned long long mask = ~0ull << (64 - 8 * d);
    return (hi & mask) == (st->pre_hi & mask);
  }
  if (hi != st->pre_hi) return false;
  const unsigned int mask = ~0u << (32 - 8 * (d - 8));
  return (lo & mask) == (st->pre_lo & mask);
}

__global__ void k_sel_init(SelState *st, unsigned int k) {
  const int t = threadIdx.x;
  if (t == 0) { st->pre_hi = 0; st->pre_lo = 0; st->k_rem = k; st->all = 0; st->count = 0; }
  st->hist[t] = 0;
}

__global__ void __launch_bounds__(256) k_sel_hist(const double *rd, const uint8_t *flags, int P, SelState *st, int d) {
  __shared__ unsigned int h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  if (!st->all) {
    for (long long p = (long long)blockIdx.x * 256 + threadIdx.x; p < P; p += (long long)gridDim.x * 256) {
      if (!(flags[p] & CF_FLAG_KEEP)) continue;
      unsigned long long hi;
      unsigned int lo;
      plan_key(rd, (int)p, hi, lo);
      if (prefix_match(hi, lo, st, d)) atomicAdd(&h[key_digit(hi, lo, d)], 1u);
    }
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&st->hist[threadIdx.x], h[threadIdx.x]);
}

__global__ void k_sel_pick(SelState *st, int d) {
  if (threadIdx.x == 0 && !st->all) {
    unsigned int cum = 0;
    int b = 255;
    for (; b >= 0; b--) {
      if (cum + st->hist[b] >= st->k_rem) break;
      cum += st->hist[b];
    }
    if (b < 0) {
      st->all = 1;  // only possible at the first digit: fewer kept plans than k
    } else {
      st->k_rem -= cum;
      if (d < 8) st->pre_hi |= (unsigned long long)b << (56 - 8 * d);
      else st->pre_lo |= (unsigned int)b << (24 - 8 * (d - 8));
    }
  }
  __syncthreads();
  st->hist[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(256) k_sel_compact(const double *rd, const uint8_t *flags, int P, SelState *st,
                                                    unsigned long long *khi, unsigned int *klo, int cap) {
  for (long long p = (long long)blockIdx.x * 256 + threadIdx.x; p < P; p += (long long)gridDim.x * 256) {
    if (!(flags[p] & CF_FLAG_KEEP)) continue;
    unsigned long long hi;
    unsigned int lo;
    plan_key(rd, (int)p, hi, lo);
    const bool take = st->all || hi > st->pre_hi || (hi == st->pre_hi && lo >= st->pre_lo);
    if (take) {
      const unsigned int i = atomicAdd(&st->count, 1u);
      if ((int)i < cap) { khi[i] = hi; klo[i] = lo; }
    }
  }
}

constexpr int kTile = 1024;

__global__ void __launch_bounds__(256) k_sel_rank(const unsigned long long *khi, const unsigned int *klo,
                                                 const SelState *st, int cap, int32_t *ids) {
  __shared__ unsigned long long th[kTile];
  __shared__ unsigned int tl[kTile];
  const int n = (int)(st->count < (unsigned)cap ? st->count : (unsigned)cap);
  const int i = blockIdx.x * 256 + threadIdx.x;
  unsigned long long hi = 0;
  unsigned int lo = 0;
  if (i < n) { hi = khi[i]; lo = klo[i]; }
  int rank = 0;
  for (int j0 = 0; j0 < n; j0 += kTile) {
    __syncthreads();
    for (int j = threadIdx.x; j < kTile; j += 256) {
      if (j0 + j < n) { th[j] = khi[j0 + j]; tl[j] = klo[j0 + j]; }
    }
    __syncthreads();
    const int m = n - j0 < kTile ? n - j0 : kTile;
    for (int j = 0; j < m; j++) rank += (th[j] > hi || (th[j] == hi && tl[j] > lo)) ? 1 : 0;
  }
  if (i < n) ids[rank] = (int32_t)(0xFFFFFFFFu - lo);
}

// (R_d bits, plan number) of a precedes b: larger R_d, or equal R_d and a
// smaller plan number (the order of cf_select_topk, with 64-bit numbers)
__device__ __forceinline__ bool key_ahead(unsigned long long ra, uint64_t ga, unsigned long long rb, uint64_t gb) {
  return ra > rb || (ra == rb && ga < gb);
}

__global__ void k_topk_merge(const double *rd_run, const uint64_t *gid_run, int n_run, const double *rd_win,
                             const int32_t *ids_win, int n_win, uint64_t first, int k, double *rd_out,
                             uint64_t *gid_out) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n_run + n_win) return;
  const bool in_run = i < n_run;
  const int own = in_run ? i : i - n_run;
  double r;
  uint64_t g;
  if (in_run) {
    r = rd_run[own];
    g = gid_run[own];
  } else {
    const int32_t id = ids_win[own];
    r = rd_win[id];
    g = first + (uint64_t)id;
  }
  const unsigned long long rb = (unsigned long long)__double_as_longlong(r);
  // elements of the other list ahead of this one: a prefix of that list
  int lo = 0, hi = in_run ? n_win : n_run;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    unsigned long long ro;
    uint64_t go;
    if (in_run) {
      const int32_t id = ids_win[mid];
      ro = (unsigned long long)__double_as_longlong(rd_win[id]);
      go = first + (uint64_t)id;
    } else {
      ro = (unsigned long long)__double_as_longlong(rd_run[mid]);
      go = gid_run[mid];
    }
    if (key_ahead(ro, go, rb, g)) lo = mid + 1;
    else hi = mid;
  }
  const int pos = own + lo;
  if (pos < k) {
    rd_out[pos] = r;
    gid_out[pos] = g;
  }
}

__global__ void k_rate_grid(const double *rd, const int32_t *ids, int n, int K, double alpha, double *rates) {
  const long long j = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= (long long)n * K) return;
  const int i = (int)(j / K), k = (int)(j % K);
  const double A = rd[ids[i]] * alpha;
  rates[j] = (A * (double)(k + 1)) / (double)K;
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_select_topk(const double *rd_dev, const uint8_t *flags_dev, int32_t P, int32_t k,
                                    int32_t *ids_dev, int32_t *n_selected_host, void *stream) {
  using namespace cf;
  if (!rd_dev || !flags_dev || !ids_dev || !n_selected_host) return set_error(CF_EINVAL, "NULL argument");
  if (P < 0 || P > (1 << 24)) return set_error(CF_ECAPACITY, "P out of 0..2^24");
  if (k < 1 || k > 65536) return set_error(CF_ECAPACITY, "k out of 1..65536");
  hipStream_t s = as_stream(stream);
  cf_status st = CF_OK;
  const size_t bytes = 256 + sizeof(SelState) + (size_t)k * (sizeof(unsigned long long) + sizeof(unsigned int));
  char *scr = (char *)scratch_get(SCR_SELECT, bytes, &st);
  if (!scr) return st;
  SelState *ss = (SelState *)scr;
  unsigned long long *khi = (unsigned long long *)(scr + ((sizeof(SelState) + 255) & ~(size_t)255));
  unsigned int *klo = (unsigned int *)(khi + k);
  hipLaunchKernelGGL(k_sel_init, dim3(1), dim3(256), 0, s, ss, (unsigned)k);
  const unsigned grid = (unsigned)((P + 255) / 256 < 2048 ? (P + 255) / 256 : 2048);
  if (P > 0) {
    for (int d = 0; d < 12; d++) {
      hipLaunchKernelGGL(k_sel_hist, dim3(grid), dim3(256), 0, s, rd_dev, flags_dev, P, ss, d);
      hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(256), 0, s, ss, d);
    }
    hipLaunchKernelGGL(k_sel_compact, dim3(grid), dim3(256), 0, s, rd_dev, flags_dev, P, ss, khi, klo, k);
    hipLaunchKernelGGL(k_sel_rank, dim3((unsigned)((k + 255) / 256)), dim3(256), 0, s, khi, klo, ss, k, ids_dev);
  }
  st = hip_check(hipGetLastError(), "cf_select_topk launch");
  if (st != CF_OK) return st;
  unsigned int cnt = 0;
  st = hip_check(hipMemcpyAsync(&cnt, &ss->count, sizeof cnt, hipMemcpyDeviceToHost, s), "copy count");
  if (st != CF_OK) return st;
  st = hip_check(hipStreamSynchronize(s), "cf_select_topk sync");
  if (st != CF_OK) return st;
  *n_selected_host = (int32_t)(cnt < (unsigned)k ? cnt : (unsigned)k);
  return CF_OK;
}

extern "C" cf_status cf_rate_grid(const double *rd_dev, const int32_t *ids_dev, int32_t n, int32_t K,
                                  double alpha_max, double *rates_dev, void *stream) {
  using namespace cf;
  if (!rd_dev || !ids_dev || !rates_dev) return set_error(CF_EINVAL, "NULL argument");
  if (n < 0 || K < 1) return set_error(CF_EINVAL, "n >= 0 and K >= 1 required");
  if (!(alpha_max > 0.0) || !std::isfinite(alpha_max)) return set_error(CF_EINVAL, "alpha_max must be > 0");
  if (n == 0) return CF_OK;
  const long long tot = (long long)n * K;
  hipLaunchKernelGGL(k_rate_grid, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, as_stream(stream), rd_dev,
                     ids_dev, n, K, alpha_max, rates_dev);
  return hip_check(hipGetLastError(), "cf_rate_grid launch");
}

extern "C" cf_status cf_topk_merge(const double *rd_run_dev, const uint64_t *gid_run_dev, int32_t n_run,
                                   const double *rd_win_dev, const int32_t *ids_win_dev, int32_t n_win,
                                   uint64_t win_first, int32_t k, double *rd_out_dev, uint64_t *gid_out_dev,
                                   void *stream) {
  using namespace cf;
  if (k < 1 || k > 65536) return set_error(CF_ECAPACITY, "k out of 1..65536");
  if (n_run < 0 || n_run > 65536 || n_win < 0 || n_win > 65536)
    return set_error(CF_EINVAL, "n_run and n_win must be in 0..65536");
  if (!rd_out_dev || !gid_out_dev) return set_error(CF_EINVAL, "NULL output");
  if (n_run > 0 && (!rd_run_dev || !gid_run_dev)) return set_error(CF_EINVAL, "NULL running list");
  if (n_win > 0 && (!rd_win_dev || !ids_win_dev)) return set_error(CF_EINVAL, "NULL window");
  if ((const void *)rd_out_dev == (const void *)rd_run_dev || (const void *)gid_out_dev == (const void *)gid_run_dev)
    return set_error(CF_EINVAL, "outputs alias the running list");
  const int n = n_run + n_win;
  if (n == 0) return CF_OK;
  hipLaunchKernelGGL(k_topk_merge, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, as_stream(stream), rd_run_dev,
                     gid_run_dev, n_run, rd_win_dev, ids_win_dev, n_win, win_first, k, rd_out_dev, gid_out_dev);
  return hip_check(hipGetLastError(), "cf_topk_merge launch");
}
