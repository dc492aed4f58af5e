// cf_internal.h -- internal definitions of libcf (HIP, gfx950).
//
// Device primitives (Philox4x64-10, the pinned log/exp, samplers) and the
// lowered model description that every kernel receives.  Written for this
// library only; the CPU oracle used by the tests has its own independent
// implementation of the same published definitions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cf.h"

namespace cf {

// ------------------------------------------------------------------ model
// The descriptor lowered for the kernels: the caller's cf_model_desc plus
// per-type structure derived once on the host (children, parent counts,
// source components, TTFT stage, gating pair).
struct KModel {
  int32_t nc, nt;
  int32_t kind[CF_MAX_COMP];
  double k0[CF_MAX_COMP], k1[CF_MAX_COMP], k2[CF_MAX_COMP], d0[CF_MAX_COMP], d1[CF_MAX_COMP];
  uint32_t xsel[CF_MAX_COMP];
  int32_t nout_attr[CF_MAX_COMP];
  int32_t cap[CF_MAX_COMP];
  double comm, cpu_pre;
  uint32_t weight[CF_MAX_TYPES];
  uint64_t wsum;
  uint32_t path[CF_MAX_TYPES], outm[CF_MAX_TYPES], pfo[CF_MAX_TYPES], srcm[CF_MAX_TYPES];
  uint8_t child[CF_MAX_TYPES][CF_MAX_COMP];  // non-streaming children of c on the path
  uint8_t npar[CF_MAX_TYPES][CF_MAX_COMP];   // parents of c on the path
  int8_t ttft_c[CF_MAX_TYPES];               // first LLM on the path, or -1
  int8_t th_c[CF_MAX_TYPES];                 // gate source (thinker) of the type, or -1
  int8_t ta_c[CF_MAX_TYPES];                 // gated component (talker) of the type, or -1
  uint8_t gen_out[CF_MAX_TYPES];             // a GEN component is an output
  uint32_t gate_src_mask;                    // components that are a gate source
  uint32_t gated_mask;                       // components that are gated
  int32_t img_kind[CF_MAX_TYPES], img_lo[CF_MAX_TYPES], img_hi[CF_MAX_TYPES];
  int32_t patch_lo, patch_hi;
  cf_dist len[CF_MAX_TYPES][4];
  double slo[CF_MAX_TYPES][4];
  uint32_t theta_num, theta_den;
  int32_t max_path;                          // most components on one path
  double tps[CF_MAX_COMP][8];                // iteration-time multiplier on executors of g GPUs, [c][min(g,8)-1]
  int32_t tp_any;                            // some multiplier is not 1
};

// Host: validate a descriptor and lower it.  Returns CF_OK or sets the
// thread's error text and returns CF_EINVAL.
cf_status lower_model(const cf_model_desc *d, KModel *k);
cf_status set_error(cf_status s, const char *fmt, ...);
cf_status hip_check(hipError_t e, const char *what);
hipStream_t as_stream(void *s);

// ------------------------------------------------------------------ device primitives
__device__ __forceinline__ void philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                              uint64_t k0, uint64_t k1, uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int i = 0; i < 10; i++) {
    uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += W0; k1 += W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

__device__ __forceinline__ double u01(uint64_t x) {
  return (double)(((x >> 12) << 1) | 1ull) * 0x1p-53;
}

// log: x = 2^e m, m in (sqrt2/2, sqrt2]; f = m-1, s = f/(2+f), z = s^2;
// log m = f - (h - s (h + R)), h = f^2/2, R = sum_{k=1..10} 2 z^k/(2k+1).
__device__ __forceinline__ double dev_log(double x) {
  uint64_t b = (uint64_t)__double_as_longlong(x);
  int e = (int)((b >> 52) & 0x7ff) - 1023;
  double m = __longlong_as_double((long long)((b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull));
  if (m > 0x1.6a09e667f3bcdp+0) { m = m * 0.5; e = e + 1; }
  double f = m - 1.0;
  double s = f / (2.0 + f);
  double z = s * s;
  constexpr double c1 = 2.0 / 3.0, c2 = 2.0 / 5.0, c3 = 2.0 / 7.0, c4 = 2.0 / 9.0, c5 = 2.0 / 11.0,
                   c6 = 2.0 / 13.0, c7 = 2.0 / 15.0, c8 = 2.0 / 17.0, c9 = 2.0 / 19.0, c10 = 2.0 / 21.0;
  double p = c10;
  p = p * z + c9; p = p * z + c8; p = p * z + c7; p = p * z + c6; p = p * z + c5;
  p = p * z + c4; p = p * z + c3; p = p * z + c2; p = p * z + c1;
  double R = z * p;
  double h = 0.5 * f * f;
  double de = (double)e;
  return de * 0x1.62e42ff000000p-1 - ((h - (s * (h + R) + de * (-0x1.718432a1b0e26p-35))) - f);
}

// exp for |x| <= 700: n = rint(x/ln2), r = (x - n LN2_HI) - n LN2_LO, Taylor to degree 14.
__device__ __forceinline__ double dev_exp(double x) {
  double n = rint(x * 0x1.71547652b82fep+0);
  double r = (x - n * 0x1.62e42ff000000p-1) - n * (-0x1.718432a1b0e26p-35);
  constexpr double f2 = 2.0, f3 = f2 * 3, f4 = f3 * 4, f5 = f4 * 5, f6 = f5 * 6, f7 = f6 * 7,
                   f8 = f7 * 8, f9 = f8 * 9, f10 = f9 * 10, f11 = f10 * 11, f12 = f11 * 12,
                   f13 = f12 * 13, f14 = f13 * 14;
  double p = 1.0 / f14;
  p = p * r + 1.0 / f13; p = p * r + 1.0 / f12; p = p * r + 1.0 / f11; p = p * r + 1.0 / f10;
  p = p * r + 1.0 / f9; p = p * r + 1.0 / f8; p = p * r + 1.0 / f7; p = p * r + 1.0 / f6;
  p = p * r + 1.0 / f5; p = p * r + 1.0 / f4; p = p * r + 1.0 / f3; p = p * r + 1.0 / f2;
  p = p * r + 1.0; p = p * r + 1.0;
  int ni = (int)n;
  double sc = __longlong_as_double((long long)((uint64_t)(ni + 1023) << 52));
  return p * sc;
}

}  // namespace cf

namespace cf {
// Per-device scratch owned by the library, grown on demand, one region per
// purpose.  Calls that use the same region must not overlap on one device.
// A latency-target table [T][n_bins][4] (TTFT, TPOT, E2E, MEDIA bounds, not
// decreasing with the bin) checked on the host and copied to device scratch.
cf_status load_targets(int T, int n_bins, const double *host, const double **dev, hipStream_t s);
// Host: validation alone of a target table [T][n_bins][4] (load_targets also copies it
// to library scratch).
cf_status check_targets(int T, int n_bins, const double *host);

// The first bin b whose four bounds the latencies meet (n_bins if none), by
// bisection: the bounds do not decrease with b, so meeting them is monotone.
__device__ __forceinline__ int target_bin(const double *tg, int n_bins, int t, double l0, double l1, double l2,
                                          double l3) {
  int lo = 0, hi = n_bins;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const double *b = tg + ((size_t)t * n_bins + mid) * 4;
    if (l0 <= b[0] && l1 <= b[1] && l2 <= b[2] && l3 <= b[3]) hi = mid; else lo = mid + 1;
  }
  return lo;
}

enum ScratchSlot { SCR_TRACE = 0, SCR_SELECT = 1, SCR_FINE = 2, SCR_MC = 3, SCR_PARETO = 4, SCR_ENUM = 5, SCR_TARGETS = 6, SCR_BISECT = 7, SCR_NSLOTS = 8 };
void *scratch_get(int slot, size_t bytes, cf_status *st);
}  // namespace cf

namespace cf {
// The executor, among a node's executors (those of its first configuration
// first), that serves a request whose 16-bit replica key for the node is key.
// A node of one configuration (w == 0) cuts the key range into rep1 equal
// parts.  A node with rep2 executors of a second configuration gives the keys
// below w * 2^16 / 10 to the first configuration and the rest to the second,
// each part cut into equal parts for its executors (every product stays below
// 10 * 2^16 * 64 < 2^32).
__device__ __forceinline__ int node_exec(uint32_t key, uint32_t rep1, uint32_t rep2, uint32_t w) {
  if (w == 0) return (int)((key * rep1) >> 16);
  const uint32_t pos = key * 10u, cut = w << 16;
  if (pos < cut) return (int)((pos * rep1) / cut);
  return (int)rep1 + (int)(((pos - cut) * rep2) / ((10u - w) << 16));
}
}  // namespace cf
