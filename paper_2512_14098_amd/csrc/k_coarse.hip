// k_coarse.hip -- cf_eval_coarse: phase 1 of the plan evaluation
// (Sec. 4.3, Alg. 2): flow-based throughput estimation with redundancy
// pruning and the GPU budget of Eq. (1).
//
// One thread per plan streams the plan's structure-of-arrays record
// (coalesced across the wave), accumulates the per-node demand u_v in LDS in
// the fixed order (type, alternative, component), and writes R_d, the
// bottleneck node and the flag bits.  Per-type means of X and of the output
// length are computed once per block from the moments.
#include "cf_internal.h"

namespace cf {
namespace {

constexpr int kBlock = 256;

struct PlanView {
  int P;
  const uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  const uint16_t *node_batch;
};

__global__ void __launch_bounds__(kBlock) k_coarse(KModel m, PlanView pv, const uint64_t *moments,
                                                   int n_gpus, double *rd, int32_t *bott, uint8_t *flags) {
  __shared__ double ex_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double en_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double u_s[CF_MAX_NODES][kBlock];
  const int tid = threadIdx.x;
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
  __syncthreads();
  const long long p = (long long)blockIdx.x * kBlock + tid;
  if (p >= pv.P) return;
  const size_t P = (size_t)pv.P;
#define AT(arr, slot) (arr)[(size_t)(slot) * P + (size_t)p]
  const int nv = pv.n_nodes[p];
  bool valid = nv >= 1 && nv <= CF_MAX_NODES;
  int execs = 0;
  uint32_t cm[CF_MAX_NODES];
  for (int v = 0; v < CF_MAX_NODES; v++) {
    cm[v] = 0;
    if (v < nv) {
      cm[v] = AT(pv.node_comp, v);
      const int rep = AT(pv.node_rep, v), b = AT(pv.node_batch, v);
      if (cm[v] == 0 || (cm[v] >> m.nc) || rep < 1 || b < 1 || b > CF_MAX_BATCH || AT(pv.node_gpus, v) < 1)
        valid = false;
      execs += rep;
    }
  }
  if (execs > CF_MAX_EXEC) valid = false;
  for (int t = 0; t < m.nt && valid; t++) {
    const int na = AT(pv.n_alt, t);
    if (na < 1 || na > 2) { valid = false; break; }
    for (int a = 0; a < na && valid; a++) {
      if (na > 1 && AT(pv.alt_w, 2 * t + a) < 1) valid = false;
      uint32_t path = m.path[t];
      while (path) {
        const int c = __ffs(path) - 1;
        path &= path - 1;
        const int v = AT(pv.alt_node, (2 * t + a) * 8 + c);
        if (v >= nv || !((cm[v] >> c) & 1u)) { valid = false; break; }
      }
    }
  }
  if (!valid) {
    rd[p] = 0.0;
    bott[p] = -1;
    flags[p] = CF_FLAG_INVALID;
    return;
  }
  for (int v = 0; v < nv; v++) u_s[v][tid] = 0.0;
  const double wsum = (double)m.wsum;
  for (int t = 0; t < m.nt; t++) {
    const double pi = (double)m.weight[t] / wsum;
    const int na = AT(pv.n_alt, t);
    uint32_t wtot = 0;
    for (int a = 0; a < na; a++) wtot += na > 1 ? AT(pv.alt_w, 2 * t + a) : 1u;
    for (int a = 0; a < na; a++) {
      const uint32_t wa = na > 1 ? AT(pv.alt_w, 2 * t + a) : 1u;
      const double q = (double)wa / (double)wtot;
      const double pq = pi * q;
      uint32_t path = m.path[t];
      while (path) {
        const int c = __ffs(path) - 1;
        path &= path - 1;
        const int v = AT(pv.alt_node, (2 * t + a) * 8 + c);
        const int bn = AT(pv.node_batch, v);
        const double B = (double)(bn < m.cap[c] ? bn : m.cap[c]);
        double w = ((m.k0[c] / B) + m.k1[c] * ex_s[t][c]) + m.k2[c];
        if (m.kind[c] == CF_LLM) w = w + (en_s[t][c] - 1.0) * ((m.d0[c] / B) + m.d1[c]);
        u_s[v][tid] = u_s[v][tid] + pq * w;
      }
    }
  }
  double best = __builtin_inf();
  int bn = -1;
  for (int v = 0; v < nv; v++) {
    const double u = u_s[v][tid];
    if (u > 0.0) {
      const double r = (double)AT(pv.node_rep, v) / u;
      if (r < best) { best = r; bn = v; }
    }
  }
  bool redundant = false;
  uint64_t gpus = 0;
  for (int v = 0; v < nv; v++) {
    const int rep = AT(pv.node_rep, v);
    const double u = u_s[v][tid];
    gpus += (uint64_t)rep * AT(pv.node_gpus, v);
    if (u == 0.0) redundant = true;
    else if (rep >= 2 && (double)(rep - 1) / u >= best) redundant = true;
  }
  const bool over = gpus > (uint64_t)n_gpus;
  rd[p] = best;
  bott[p] = bn;
  flags[p] = (uint8_t)(((!over && !redundant) ? CF_FLAG_KEEP : 0u) | (over ? CF_FLAG_OVER_BUDGET : 0u) |
                       (redundant ? CF_FLAG_REDUNDANT : 0u));
#undef AT
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_eval_coarse(const cf_model_desc *model, const cf_plan_table *plans,
                                    const uint64_t *moments_dev, int32_t n_gpus, double *rd_dev,
                                    int32_t *bottleneck_dev, uint8_t *flags_dev, void *stream) {
  using namespace cf;
  KModel m;
  cf_status st = lower_model(model, &m);
  if (st != CF_OK) return st;
  if (!plans || !moments_dev || !rd_dev || !bottleneck_dev || !flags_dev)
    return set_error(CF_EINVAL, "NULL argument");
  if (plans->P < 0) return set_error(CF_EINVAL, "P < 0");
  if (plans->P == 0) return CF_OK;
  if (!plans->n_nodes_dev || !plans->node_comp_dev || !plans->node_rep_dev || !plans->node_batch_dev ||
      !plans->node_gpus_dev || !plans->n_alt_dev || !plans->alt_w_dev || !plans->alt_node_dev)
    return set_error(CF_EINVAL, "NULL plan array");
  PlanView pv{plans->P, plans->n_nodes_dev, plans->node_comp_dev, plans->node_rep_dev, plans->node_gpus_dev,
              plans->n_alt_dev, plans->alt_w_dev, plans->alt_node_dev, plans->node_batch_dev};
  hipLaunchKernelGGL(k_coarse, dim3((unsigned)((plans->P + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                     as_stream(stream), m, pv, moments_dev, n_gpus, rd_dev, bottleneck_dev, flags_dev);
  return hip_check(hipGetLastError(), "cf_eval_coarse launch");
}
