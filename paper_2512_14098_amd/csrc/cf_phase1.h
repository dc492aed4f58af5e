// cf_phase1.h -- the arithmetic of phase 1 (Sec. 4.3, Alg. 2: flow-based
// throughput, redundancy pruning, the GPU budget of Eq. 1) shared by the
// kernels that screen plans from a plan table (k_coarse) and from plan
// numbers (k_enum_screen), so both compute the same values in the same
// order.
#pragma once
#include "cf_internal.h"

namespace cf {

// Per-type means of X and of the output length from the per-type moments,
// one (t, c) pair per thread of the block.
__device__ __forceinline__ void phase1_means(const KModel &m, const uint64_t *moments, int tid,
                                             double (*ex_s)[CF_MAX_COMP], double (*en_s)[CF_MAX_COMP]) {
  if (tid < m.nt * m.nc) {
    const int t = tid / m.nc, c = tid % m.nc;
    const uint64_t *mo = moments + (size_t)t * 8;
    double ex = 0.0, en = 1.0;
    if (mo[0] > 0) {
      uint64_t xs = 0;
      for (int a = 0; a < 7; a++)
        if ((m.xsel[c] >> a) & 1u) xs += mo[1 + a];
      ex = (double)xs / (double)mo[0];
      if (m.kind[c] == CF_LLM && !((m.pfo[t] >> c) & 1u)) {
        en = (double)mo[1 + m.nout_attr[c]] / (double)mo[0];
        if (en < 1.0) en = 1.0;
      }
    }
    ex_s[t][c] = ex;
    en_s[t][c] = en;
  }
}

// Seconds of executor time per type-t request at component c on a node of
// batch bn whose executors have the multiplier tps.
__device__ __forceinline__ double phase1_work(const KModel &m, int c, int bn, double ex, double en, double tps) {
  const double B = (double)(bn < m.cap[c] ? bn : m.cap[c]);
  double w = ((m.k0[c] / B) + m.k1[c] * ex) + m.k2[c];
  if (m.kind[c] == CF_LLM) w = w + (en - 1.0) * ((m.d0[c] / B) + m.d1[c]);
  // on executors of g GPUs every iteration takes tp_scale times as long
  if (m.tp_any) w = tps * w;
  return w;
}

// R_d = min_v m_v / u_v (lowest bottleneck on ties), redundancy and budget
// flags from the per-node demands; rep, gp and u_at(v) for v < nv.
template <class U>
__device__ __forceinline__ void phase1_result(int nv, const uint32_t *rep, const uint32_t *gp, U u_at, int n_gpus,
                                              double *rd, int32_t *bott, uint8_t *flags) {
  double best = __builtin_inf();
  int bn = -1;
  bool redundant = false;
  uint64_t gpus = 0;
#pragma unroll
  for (int v = 0; v < CF_MAX_NODES; v++) {
    if (v < nv) {
      const double u = u_at(v);
      if (u > 0.0) {
        const double r = (double)rep[v] / u;
        if (r < best) { best = r; bn = v; }
      }
    }
  }
#pragma unroll
  for (int v = 0; v < CF_MAX_NODES; v++) {
    if (v < nv) {
      const double u = u_at(v);
      gpus += (uint64_t)rep[v] * gp[v];
      if (u == 0.0) redundant = true;
      else if (rep[v] >= 2 && (double)(rep[v] - 1) / u >= best) redundant = true;
    }
  }
  const bool over = gpus > (uint64_t)n_gpus;
  *rd = best;
  *bott = bn;
  *flags = (uint8_t)(((!over && !redundant) ? CF_FLAG_KEEP : 0u) | (over ? CF_FLAG_OVER_BUDGET : 0u) |
                     (redundant ? CF_FLAG_REDUNDANT : 0u));
}

// phase1_result for plans whose nodes may hold a second executor
// configuration: the capacity m/u of every executor group, in node order and a
// node's first configuration before its second (rep2[v] = 0: none), gives R_d
// and the bottleneck node; the budget counts both configurations; a group
// receiving no work, or keeping R_d without one of its executors, makes the
// plan redundant.
template <class U, class U2>
__device__ __forceinline__ void phase1_result_groups(int nv, const uint32_t *rep, const uint32_t *gp,
                                                     const uint32_t *rep2, const uint32_t *gp2, U u_at, U2 u2_at,
                                                     int n_gpus, double *rd, int32_t *bott, uint8_t *flags) {
  double best = __builtin_inf();
  int bn = -1;
  bool redundant = false;
  uint64_t gpus = 0;
  for (int v = 0; v < nv; v++) {
    const double u = u_at(v);
    if (u > 0.0) {
      const double r = (double)rep[v] / u;
      if (r < best) { best = r; bn = v; }
    }
    if (rep2[v] > 0) {
      const double u2 = u2_at(v);
      if (u2 > 0.0) {
        const double r = (double)rep2[v] / u2;
        if (r < best) { best = r; bn = v; }
      }
    }
  }
  for (int v = 0; v < nv; v++) {
    const double u = u_at(v);
    gpus += (uint64_t)rep[v] * gp[v];
    if (u == 0.0) redundant = true;
    else if (rep[v] >= 2 && (double)(rep[v] - 1) / u >= best) redundant = true;
    if (rep2[v] > 0) {
      const double u2 = u2_at(v);
      gpus += (uint64_t)rep2[v] * gp2[v];
      if (u2 == 0.0) redundant = true;
      else if (rep2[v] >= 2 && (double)(rep2[v] - 1) / u2 >= best) redundant = true;
    }
  }
  const bool over = gpus > (uint64_t)n_gpus;
  *rd = best;
  *bott = bn;
  *flags = (uint8_t)(((!over && !redundant) ? CF_FLAG_KEEP : 0u) | (over ? CF_FLAG_OVER_BUDGET : 0u) |
                     (redundant ? CF_FLAG_REDUNDANT : 0u));
}

}  // namespace cf
