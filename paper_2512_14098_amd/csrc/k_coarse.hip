// k_coarse.hip -- cf_eval_coarse: phase 1 of the plan evaluation
// (Sec. 4.3, Alg. 2): flow-based throughput estimation with redundancy
// pruning and the GPU budget of Eq. (1).
//
// One thread per plan loads the fields of the plan's structure-of-arrays
// record it needs (coalesced across the wave, all loads independent),
// accumulates the per-node demand u_v in LDS in the fixed order (type,
// alternative, component), and writes R_d, the bottleneck node and the flag
// bits.  Per-type means of X and of the output
// length are computed once per block from the moments.
#include "cf_internal.h"
#include "cf_phase1.h"

namespace cf {
namespace {

constexpr int kBlock = 256;
// plans whose nodes may hold a second executor configuration: a smaller block
// for the second set of per-node LDS arrays
constexpr int kBlockGroups = 128;

struct PlanView {
  int P;
  const uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  const uint16_t *node_batch;
  const uint8_t *node_rep2, *node_gpus2, *node_w;  // second configurations (HET kernel only)
  const uint16_t *node_batch2;
};

template <bool HET>
__global__ void __launch_bounds__(HET ? kBlockGroups : kBlock)
    k_coarse(KModel m, PlanView pv, const uint64_t *moments, int n_gpus, double *rd, int32_t *bott, uint8_t *flags) {
  constexpr int NB = HET ? kBlockGroups : kBlock;
  __shared__ double ex_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double en_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double u_s[CF_MAX_NODES][NB];
  __shared__ uint16_t b_s[CF_MAX_NODES][NB];  // node batch
  __shared__ uint8_t c_s[CF_MAX_NODES][NB];   // node component set
  __shared__ uint8_t g_s[CF_MAX_NODES][NB];   // node GPUs per executor, as min(g, 8) - 1
  __shared__ double tps_s[CF_MAX_COMP][8];    // iteration-time multipliers by GPUs per executor
  // second configuration of a node (HET): demand, batch, GPUs index, tenths to the first
  __shared__ double u2_s[HET ? CF_MAX_NODES : 1][HET ? NB : 1];
  __shared__ uint16_t b2_s[HET ? CF_MAX_NODES : 1][HET ? NB : 1];
  __shared__ uint8_t g2_s[HET ? CF_MAX_NODES : 1][HET ? NB : 1];
  __shared__ uint8_t w_s[HET ? CF_MAX_NODES : 1][HET ? NB : 1];
  const int tid = threadIdx.x;
  if (tid < CF_MAX_COMP * 8) (&tps_s[0][0])[tid] = (&m.tps[0][0])[tid];
  phase1_means(m, moments, tid, ex_s, en_s);
  __syncthreads();
  const long long p = (long long)blockIdx.x * NB + tid;
  if (p >= pv.P) return;
  const size_t P = (size_t)pv.P;
#define AT(arr, slot) (arr)[(size_t)(slot) * P + (size_t)p]
  // Every field the plan's evaluation needs is loaded first, with no load
  // depending on another (one memory latency per plan instead of one per
  // field); slots past the plan's node count and alternatives past its
  // count are not fetched.
  const int nv = pv.n_nodes[p];
  uint32_t rep[CF_MAX_NODES], gp[CF_MAX_NODES];
  uint32_t rep2[HET ? CF_MAX_NODES : 1], gp2[HET ? CF_MAX_NODES : 1];
#pragma unroll
  for (int v = 0; v < CF_MAX_NODES; v++) {
    uint32_t cm = 0, b = 0;
    rep[v] = 0;
    gp[v] = 0;
    if (v < nv) {
      cm = AT(pv.node_comp, v);
      rep[v] = AT(pv.node_rep, v);
      b = AT(pv.node_batch, v);
      gp[v] = AT(pv.node_gpus, v);
    }
    c_s[v][tid] = (uint8_t)cm;
    b_s[v][tid] = (uint16_t)b;
    if (m.tp_any) g_s[v][tid] = (uint8_t)(gp[v] < 1 ? 0 : (gp[v] > 8 ? 7 : gp[v] - 1));
    if constexpr (HET) {
      uint32_t b2 = 0, w = 0;
      rep2[v] = 0;
      gp2[v] = 0;
      if (v < nv) {
        rep2[v] = AT(pv.node_rep2, v);
        b2 = AT(pv.node_batch2, v);
        gp2[v] = AT(pv.node_gpus2, v);
        w = AT(pv.node_w, v);
      }
      b2_s[v][tid] = (uint16_t)b2;
      w_s[v][tid] = (uint8_t)(rep2[v] > 0 ? w : 0u);
      if (m.tp_any) g2_s[v][tid] = (uint8_t)(gp2[v] < 1 ? 0 : (gp2[v] > 8 ? 7 : gp2[v] - 1));
    }
  }
  bool valid = nv >= 1 && nv <= CF_MAX_NODES;
  int execs = 0;
#pragma unroll
  for (int v = 0; v < CF_MAX_NODES; v++) {
    if (v < nv) {
      const uint32_t cm = c_s[v][tid], b = b_s[v][tid];
      if (cm == 0 || (cm >> m.nc) || rep[v] < 1 || b < 1 || b > CF_MAX_BATCH || gp[v] < 1) valid = false;
      execs += (int)rep[v];
      if constexpr (HET) {
        if (rep2[v] > 0) {
          const uint32_t b2 = b2_s[v][tid], w = w_s[v][tid];
          if (b2 < 1 || b2 > CF_MAX_BATCH || gp2[v] < 1 || w < 1 || w > 9) valid = false;
          execs += (int)rep2[v];
        }
      }
    }
  }
  if (execs > CF_MAX_EXEC) valid = false;
  if (!valid) {
    rd[p] = 0.0;
    bott[p] = -1;
    flags[p] = CF_FLAG_INVALID;
    return;
  }
  // per type: the routes of both alternatives are loaded together, then
  // checked and accumulated: u_v += (pi_t q_a) w in the order t, a, c (and,
  // for a node of two configurations, u_v += ((pi_t q_a) s) w for each
  // configuration, s its share of the node's requests)
  for (int v = 0; v < nv; v++) {
    u_s[v][tid] = 0.0;
    if constexpr (HET) u2_s[v][tid] = 0.0;
  }
  const double wsum = (double)m.wsum;
  for (int t = 0; t < m.nt; t++) {
    const uint32_t path = m.path[t];
    const uint32_t na = AT(pv.n_alt, t);
    uint32_t wl[2], nd[2][CF_MAX_COMP];
#pragma unroll
    for (int a = 0; a < 2; a++) {
      wl[a] = AT(pv.alt_w, 2 * t + a);
#pragma unroll
      for (int c = 0; c < CF_MAX_COMP; c++) nd[a][c] = ((path >> c) & 1u) ? AT(pv.alt_node, (2 * t + a) * 8 + c) : 0u;
    }
    if (na < 1 || na > 2) {
      valid = false;
      break;
    }
    const double pi = (double)m.weight[t] / wsum;
    const uint32_t wtot = na > 1 ? wl[0] + wl[1] : 1u;
#pragma unroll
    for (int a = 0; a < 2; a++) {
      if (a < (int)na) {
        if (na > 1 && wl[a] < 1) valid = false;
        const uint32_t wa = na > 1 ? wl[a] : 1u;
        const double q = (double)wa / (double)wtot;
        const double pq = pi * q;
#pragma unroll
        for (int c = 0; c < CF_MAX_COMP; c++) {
          if (!((path >> c) & 1u)) continue;
          const int v = (int)nd[a][c];
          if (v >= nv || !((c_s[v][tid] >> c) & 1u)) {
            valid = false;
            continue;
          }
          const double w =
              phase1_work(m, c, b_s[v][tid], ex_s[t][c], en_s[t][c], m.tp_any ? tps_s[c][g_s[v][tid]] : 1.0);
          if constexpr (HET) {
            const uint32_t ws = w_s[v][tid];
            if (ws) {
              const double w2 = phase1_work(m, c, b2_s[v][tid], ex_s[t][c], en_s[t][c],
                                            m.tp_any ? tps_s[c][g2_s[v][tid]] : 1.0);
              u_s[v][tid] = u_s[v][tid] + (pq * ((double)ws / 10.0)) * w;
              u2_s[v][tid] = u2_s[v][tid] + (pq * ((double)(10u - ws) / 10.0)) * w2;
              continue;
            }
          }
          u_s[v][tid] = u_s[v][tid] + pq * w;
        }
      }
    }
  }
  if (!valid) {
    rd[p] = 0.0;
    bott[p] = -1;
    flags[p] = CF_FLAG_INVALID;
    return;
  }
  if constexpr (HET)
    phase1_result_groups(nv, rep, gp, rep2, gp2, [&](int v) { return u_s[v][tid]; },
                         [&](int v) { return u2_s[v][tid]; }, n_gpus, &rd[p], &bott[p], &flags[p]);
  else
    phase1_result(nv, rep, gp, [&](int v) { return u_s[v][tid]; }, n_gpus, &rd[p], &bott[p], &flags[p]);
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
  const int ngroups = (plans->node_rep2_dev != nullptr) + (plans->node_batch2_dev != nullptr) +
                      (plans->node_gpus2_dev != nullptr) + (plans->node_w_dev != nullptr);
  if (ngroups != 0 && ngroups != 4) return set_error(CF_EINVAL, "second-configuration arrays: all four or none");
  PlanView pv{plans->P,          plans->n_nodes_dev,  plans->node_comp_dev,  plans->node_rep_dev,
              plans->node_gpus_dev, plans->n_alt_dev,   plans->alt_w_dev,      plans->alt_node_dev,
              plans->node_batch_dev, plans->node_rep2_dev, plans->node_gpus2_dev, plans->node_w_dev,
              plans->node_batch2_dev};
  if (ngroups)
    hipLaunchKernelGGL(k_coarse<true>, dim3((unsigned)((plans->P + kBlockGroups - 1) / kBlockGroups)),
                       dim3(kBlockGroups), 0, as_stream(stream), m, pv, moments_dev, n_gpus, rd_dev, bottleneck_dev,
                       flags_dev);
  else
    hipLaunchKernelGGL(k_coarse<false>, dim3((unsigned)((plans->P + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                       as_stream(stream), m, pv, moments_dev, n_gpus, rd_dev, bottleneck_dev, flags_dev);
  return hip_check(hipGetLastError(), "cf_eval_coarse launch");
}
