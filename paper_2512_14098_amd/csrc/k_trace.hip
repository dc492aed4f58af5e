// k_trace.hip -- cf_trace_gen: synthetic Any-to-Any request traces.
//
// The workload of Sec. 3.1 (request types with fractions pi_t) with Poisson
// arrivals.  One thread per (seed, request) draws Philox4x64-10 blocks keyed
// by (seed, 0) with counter (request, field, attempt, 0); the gap ticks are
// then turned into arrival ticks by an exact u64 inclusive scan per seed.
// Per-type moments are u64 sums (order-free integer atomics).
#include "cf_internal.h"

namespace cf {
namespace {

constexpr int kSeedsPerLaunch = 64;
struct SeedChunk { uint64_t v[kSeedsPerLaunch]; };

enum { F_ARRIVAL = 0, F_PROMPT = 1, F_OUT = 2, F_PATCH = 3, F_AUDIN = 4, F_AUDOUT = 5, F_ROUTE = 6 };

__device__ __forceinline__ int64_t uni_int(uint64_t x, int64_t lo, int64_t hi) {
  return lo + (int64_t)(((x >> 32) * (uint64_t)(hi - lo + 1)) >> 32);
}

// Marsaglia polar method on blocks (req, field, k), pairs (x0,x1) then (x2,x3).
__device__ double normal_polar(uint64_t seed, uint64_t req, uint64_t field) {
  for (uint64_t k = 0; k < 32; k++) {
    uint64_t x[4];
    philox4x64_10(req, field, k, 0, seed, 0, x);
    for (int h = 0; h < 2; h++) {
      double v1 = 2.0 * u01(x[2 * h]) - 1.0;
      double v2 = 2.0 * u01(x[2 * h + 1]) - 1.0;
      double w = v1 * v1 + v2 * v2;
      if (w > 0.0 && w < 1.0) return v1 * sqrt((-2.0 * dev_log(w)) / w);
    }
  }
  return 0.0;
}

__device__ __forceinline__ int64_t clamp_round(double v, int64_t lo, int64_t hi) {
  double r = rint(v);
  if (r <= (double)lo) return lo;
  if (r >= (double)hi) return hi;
  return (int64_t)r;
}

__device__ int64_t draw_len(const cf_dist &d, uint64_t seed, uint64_t req, uint64_t field) {
  if (d.kind == CF_DIST_CONST) return (int64_t)d.p0;
  if (d.kind == CF_DIST_LOGNORMAL) {
    double z = normal_polar(seed, req, field);
    return clamp_round(d.scale * dev_exp(d.p0 + d.p1 * z), d.lo, d.hi);
  }
  if (d.kind == CF_DIST_EXP) {
    uint64_t x[4];
    philox4x64_10(req, field, 0, 0, seed, 0, x);
    return clamp_round(d.p0 * (-dev_log(u01(x[0]))), d.lo, d.hi);
  }
  return 0;
}

__global__ void k_zero_u64(uint64_t *p, long long n) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

__global__ void __launch_bounds__(256) k_trace_draw(KModel m, SeedChunk seeds, int s0, int n,
                                                    cf_trace tr, uint64_t *moments) {
  __shared__ unsigned long long mom[CF_MAX_TYPES * 8];
  const int tid = threadIdx.x;
  if (tid < CF_MAX_TYPES * 8) mom[tid] = 0;
  __syncthreads();
  const int sl = blockIdx.y;
  const int s = s0 + sl;
  const long long i = (long long)blockIdx.x * blockDim.x + tid;
  if (i < n) {
    const uint64_t seed = seeds.v[sl];
    const size_t o = (size_t)s * (size_t)n + (size_t)i;
    uint64_t x[4];
    philox4x64_10((uint64_t)i, F_ARRIVAL, 0, 0, seed, 0, x);
    const double g = -dev_log(u01(x[0])) * 0x1p32;
    tr.arr_ticks_dev[o] = (uint64_t)rint(g);  // gap; the scan makes it a prefix sum
    const uint64_t v = ((x[1] >> 32) * m.wsum) >> 32;
    int t = 0;
    uint64_t cum = m.weight[0];
    while (cum <= v && t + 1 < m.nt) { t++; cum += m.weight[t]; }
    int nimg = 0;
    if (m.img_kind[t] == CF_IMG_CONST) nimg = m.img_lo[t];
    else if (m.img_kind[t] == CF_IMG_UNIFORM) nimg = (int)uni_int(x[2], m.img_lo[t], m.img_hi[t]);
    uint32_t patches = 0;
    if (nimg > 0) {
      uint64_t y[4];
      philox4x64_10((uint64_t)i, F_PATCH, 0, 0, seed, 0, y);
      for (int k = 0; k < nimg; k++) patches += (uint32_t)uni_int(y[k], m.patch_lo, m.patch_hi);
    }
    const uint32_t prompt = (uint32_t)draw_len(m.len[t][0], seed, (uint64_t)i, F_PROMPT);
    const uint32_t out = (uint32_t)draw_len(m.len[t][1], seed, (uint64_t)i, F_OUT);
    const uint32_t ain = (uint32_t)draw_len(m.len[t][2], seed, (uint64_t)i, F_AUDIN);
    const uint32_t aout = (uint32_t)draw_len(m.len[t][3], seed, (uint64_t)i, F_AUDOUT);
    uint64_t y[4];
    philox4x64_10((uint64_t)i, F_ROUTE, 0, 0, seed, 0, y);
    tr.type_dev[o] = (uint8_t)t;
    tr.n_img_dev[o] = (uint8_t)nimg;
    tr.patches_dev[o] = (uint16_t)patches;
    tr.prompt_dev[o] = (uint16_t)prompt;
    tr.out_dev[o] = (uint16_t)out;
    tr.aud_in_ms_dev[o] = ain;
    tr.aud_out_ms_dev[o] = aout;
    tr.rkey0_dev[o] = y[0];
    tr.rkey1_dev[o] = y[1];
    tr.akey_dev[o] = (uint32_t)(y[2] >> 32);
    unsigned long long *mt = mom + t * 8;
    atomicAdd(mt + 0, 1ull);
    atomicAdd(mt + 1, (unsigned long long)prompt);
    atomicAdd(mt + 2, (unsigned long long)out);
    atomicAdd(mt + 3, (unsigned long long)patches);
    atomicAdd(mt + 4, (unsigned long long)ain);
    atomicAdd(mt + 5, (unsigned long long)aout);
    atomicAdd(mt + 6, (unsigned long long)((ain + 79u) / 80u));
    atomicAdd(mt + 7, (unsigned long long)((aout + 79u) / 80u));
  }
  __syncthreads();
  if (tid < m.nt * 8 && mom[tid] != 0)
    atomicAdd((unsigned long long *)(moments + (size_t)s * m.nt * 8 + tid), mom[tid]);
}

// ---- exact u64 inclusive scan of each seed's gaps: blocks of 1024, block
// totals scanned per seed, offsets added back.
constexpr int kScanBlock = 1024;

__device__ __forceinline__ uint64_t wave_incl_scan(uint64_t v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint64_t o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

__global__ void __launch_bounds__(256) k_scan_blocks(uint64_t *a, int n, uint64_t *tot, int nb) {
  __shared__ uint64_t wsum[4];
  const int s = blockIdx.y, b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  uint64_t *base = a + (size_t)s * n;
  const long long i0 = (long long)b * kScanBlock + tid * 4;
  uint64_t v[4];
  for (int j = 0; j < 4; j++) v[j] = (i0 + j < n) ? base[i0 + j] : 0;
  v[1] += v[0]; v[2] += v[1]; v[3] += v[2];
  uint64_t incl = wave_incl_scan(v[3], lane);
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  uint64_t off = incl - v[3];
  for (int k = 0; k < w; k++) off += wsum[k];
  for (int j = 0; j < 4; j++)
    if (i0 + j < n) base[i0 + j] = v[j] + off;
  if (tid == 255) tot[(size_t)s * nb + b] = off + v[3];
}

__global__ void __launch_bounds__(64) k_scan_totals(uint64_t *tot, int nb) {
  const int s = blockIdx.x, lane = threadIdx.x;
  uint64_t carry = 0;
  uint64_t *t = tot + (size_t)s * nb;
  for (int b0 = 0; b0 < nb; b0 += 64) {
    uint64_t v = (b0 + lane < nb) ? t[b0 + lane] : 0;
    uint64_t incl = wave_incl_scan(v, lane);
    if (b0 + lane < nb) t[b0 + lane] = carry + incl - v;  // exclusive
    carry += __shfl(incl, 63, 64);
  }
}

__global__ void __launch_bounds__(256) k_scan_add(uint64_t *a, int n, const uint64_t *tot, int nb) {
  const int s = blockIdx.y, b = blockIdx.x;
  const uint64_t off = tot[(size_t)s * nb + b];
  uint64_t *base = a + (size_t)s * n;
  for (int j = threadIdx.x; j < kScanBlock; j += 256) {
    long long i = (long long)b * kScanBlock + j;
    if (i < n) base[i] += off;
  }
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_trace_gen(const cf_model_desc *model, const uint64_t *seeds_host,
                                  int32_t n_seeds, int32_t n_req, const cf_trace *out,
                                  uint64_t *moments_dev, void *stream) {
  using namespace cf;
  KModel m;
  cf_status st = lower_model(model, &m);
  if (st != CF_OK) return st;
  if (!seeds_host || !out || !moments_dev) return set_error(CF_EINVAL, "NULL argument");
  if (n_seeds < 1 || n_req < 0) return set_error(CF_EINVAL, "n_seeds >= 1 and n_req >= 0 required");
  if (out->n_seeds != n_seeds || out->n_req != n_req)
    return set_error(CF_EINVAL, "trace descriptor sizes differ from the call's");
  if (n_req > (1 << 26)) return set_error(CF_ECAPACITY, "n_req above 2^26");
  if (n_req > 0 && (!out->arr_ticks_dev || !out->type_dev || !out->n_img_dev || !out->patches_dev ||
                    !out->prompt_dev || !out->out_dev || !out->aud_in_ms_dev || !out->aud_out_ms_dev ||
                    !out->rkey0_dev || !out->rkey1_dev || !out->akey_dev))
    return set_error(CF_EINVAL, "NULL trace array");
  hipStream_t s = as_stream(stream);
  const long long nmom = (long long)n_seeds * m.nt * 8;
  hipLaunchKernelGGL(k_zero_u64, dim3((unsigned)((nmom + 255) / 256)), dim3(256), 0, s, moments_dev, nmom);
  if (n_req == 0) return hip_check(hipGetLastError(), "cf_trace_gen launch");
  const int nb = (n_req + kScanBlock - 1) / kScanBlock;
  uint64_t *tot = (uint64_t *)scratch_get(SCR_TRACE, sizeof(uint64_t) * (size_t)nb * n_seeds, &st);
  if (!tot) return st;
  for (int s0 = 0; s0 < n_seeds; s0 += kSeedsPerLaunch) {
    SeedChunk sc;
    const int ns = n_seeds - s0 < kSeedsPerLaunch ? n_seeds - s0 : kSeedsPerLaunch;
    for (int j = 0; j < kSeedsPerLaunch; j++) sc.v[j] = j < ns ? seeds_host[s0 + j] : 0;
    hipLaunchKernelGGL(k_trace_draw, dim3((unsigned)((n_req + 255) / 256), (unsigned)ns), dim3(256), 0, s,
                       m, sc, s0, n_req, *out, moments_dev);
  }
  hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)nb, (unsigned)n_seeds), dim3(256), 0, s,
                     out->arr_ticks_dev, n_req, tot, nb);
  hipLaunchKernelGGL(k_scan_totals, dim3((unsigned)n_seeds), dim3(64), 0, s, tot, nb);
  hipLaunchKernelGGL(k_scan_add, dim3((unsigned)nb, (unsigned)n_seeds), dim3(256), 0, s,
                     out->arr_ticks_dev, n_req, tot, nb);
  return hip_check(hipGetLastError(), "cf_trace_gen launch");
}
