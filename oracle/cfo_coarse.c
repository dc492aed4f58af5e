/*
 * cfo_coarse.c -- oracle (test infrastructure only): phase 1 of the plan
 * evaluation (Sec. 4.3, Alg. 2 phase 1), top-K selection, the rate grid and
 * the goodput reduction with argmax selection (Sec. 3.2, Sec. 6.1, Alg. 2
 * final step).
 *
 * Phase 1 (flow-based throughput): each request type t contributes R*pi_t
 * to every node on its path, split between alternative paths by the routing
 * probabilities; at each node the demands of all types are summed and
 * compared with the node's capacity.  The node whose aggregate demand first
 * reaches its capacity is the bottleneck and the aggregate rate at which
 * that happens is R_d.  Plans with more capacity than demand at some node
 * are pruned.  The paper takes per-executor, per-type capacities from
 * profiles; here the per-request work of a component comes from its latency
 * model at the node's configured batch and the per-type means of seed 0's
 * trace.
 */
#include "cfo.h"
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define P_AT(arr, slot, P, p) ((arr)[(size_t)(slot) * (size_t)(P) + (size_t)(p)])

/* structural validity of plan p against model m (Eq. 1's ">= 1 executor
 * per node", routes that name a node hosting the component). */
int cfo_plan_valid(const cfo_model *m, const cfo_plans *pl, int p) {
  int P = pl->P;
  int nv = pl->n_nodes[p];
  if (nv < 1 || nv > CFO_MAXV) return 0;
  int execs = 0;
  for (int v = 0; v < nv; v++) {
    int cm = P_AT(pl->node_comp, v, P, p);
    if (cm == 0 || (cm >> m->n_comp) != 0) return 0;
    cfo_group g[2];
    int ng = cfo_node_groups(pl, v, p, g);
    if (ng == 2) {
      int w = P_AT(pl->node_w, v, P, p);
      if (w < 1 || w > 9) return 0;
    }
    for (int k = 0; k < ng; k++) {
      if (g[k].rep < 1 || g[k].batch < 1 || g[k].batch > CFO_MAXB || g[k].gpus < 1) return 0;
      execs += g[k].rep;
    }
  }
  if (execs > CFO_MAXX) return 0;
  for (int t = 0; t < m->n_types; t++) {
    int na = P_AT(pl->n_alt, t, P, p);
    if (na < 1 || na > CFO_MAXA) return 0;
    for (int a = 0; a < na; a++) {
      if (na > 1 && P_AT(pl->alt_w, t * 2 + a, P, p) < 1) return 0;
      for (int c = 0; c < m->n_comp; c++) {
        if (!((m->path_mask[t] >> c) & 1u)) continue;
        int v = P_AT(pl->alt_node, (t * 2 + a) * 8 + c, P, p);
        if (v >= nv) return 0;
        if (!((P_AT(pl->node_comp, v, P, p) >> c) & 1)) return 0;
      }
    }
  }
  return 1;
}

/* u[v][g]: seconds of executor time that one request of the workload mix puts
 * on executor group g of node v (summed over its executors) at the group's
 * configured batch: u[v][g] += ((pi_t * q_a) * s_g) * w(c, t, B_g) in the
 * order t, a, c, g ascending, s_g the group's share of the node's requests
 * (1 for a node of one configuration). */
void cfo_node_demand(const cfo_model *m, const cfo_plans *pl, int p, const uint64_t *moments,
                     double u[CFO_MAXV][2]) {
  int P = pl->P;
  uint64_t wsum_i = 0;
  for (int t = 0; t < m->n_types; t++) wsum_i += m->weight[t];
  double wsum = (double)wsum_i;
  for (int v = 0; v < CFO_MAXV; v++) u[v][0] = u[v][1] = 0.0;
  for (int t = 0; t < m->n_types; t++) {
    const uint64_t *mo = moments + (size_t)t * 8;
    double pi = (double)m->weight[t] / wsum;
    int na = P_AT(pl->n_alt, t, P, p);
    uint64_t wa_sum = 0;
    for (int a = 0; a < na; a++) wa_sum += (na > 1) ? P_AT(pl->alt_w, t * 2 + a, P, p) : 1u;
    for (int a = 0; a < na; a++) {
      uint64_t wa = (na > 1) ? P_AT(pl->alt_w, t * 2 + a, P, p) : 1u;
      double q = (double)wa / (double)wa_sum;
      for (int c = 0; c < m->n_comp; c++) {
        if (!((m->path_mask[t] >> c) & 1u)) continue;
        int v = P_AT(pl->alt_node, (t * 2 + a) * 8 + c, P, p);
        /* per-type mean of X and of the output length */
        double ex = 0.0, en = 1.0;
        if (mo[0] > 0) {
          uint64_t xs = 0;
          for (int at = 0; at < CFO_NATTR; at++)
            if ((m->x_sel[c] >> at) & 1u) xs += mo[1 + at];
          ex = (double)xs / (double)mo[0];
          if (m->kind[c] == CFO_LLM && !((m->prefill_only[t] >> c) & 1u)) {
            en = (double)mo[1 + m->nout_attr[c]] / (double)mo[0];
            if (en < 1.0) en = 1.0;
          }
        }
        cfo_group grp[2];
        int ng = cfo_node_groups(pl, v, p, grp);
        for (int k = 0; k < ng; k++) {
          int beff = grp[k].batch < m->batch_cap[c] ? grp[k].batch : m->batch_cap[c];
          double B = (double)beff;
          /* seconds of executor time per request at batch B */
          double w = ((m->k0[c] / B) + m->k1[c] * ex) + m->k2[c];
          if (m->kind[c] == CFO_LLM) w = w + (en - 1.0) * ((m->d0[c] / B) + m->d1[c]);
          /* on executors of g GPUs every iteration takes tp_scale times as long */
          w = cfo_tp(m, c, grp[k].gpus) * w;
          u[v][k] = u[v][k] + ((pi * q) * grp[k].share) * w;
        }
      }
    }
  }
}

int cfo_eval_coarse(const cfo_model *m, const cfo_plans *pl, const uint64_t *moments,
                    int32_t n_gpus, double *rd, int32_t *bottleneck, uint8_t *flags) {
  int P = pl->P;
  for (int p = 0; p < P; p++) {
    if (!cfo_plan_valid(m, pl, p)) {
      rd[p] = 0.0; bottleneck[p] = -1; flags[p] = 4;
      continue;
    }
    int nv = pl->n_nodes[p];
    double u[CFO_MAXV][2];
    cfo_node_demand(m, pl, p, moments, u);
    /* capacity m/u of every executor group; R_d is the smallest, its node the bottleneck */
    double best = INFINITY;
    int bn = -1;
    for (int v = 0; v < nv; v++) {
      cfo_group g[2];
      int ng = cfo_node_groups(pl, v, p, g);
      for (int k = 0; k < ng; k++) {
        if (u[v][k] > 0.0) {
          double r = (double)g[k].rep / u[v][k];
          if (r < best) { best = r; bn = v; }
        }
      }
    }
    /* Eq. (1) budget over every configuration; redundant: a group that receives no work, or
     * one whose capacity without one executor still reaches R_d */
    int redundant = 0;
    uint64_t gpus = 0;
    for (int v = 0; v < nv; v++) {
      cfo_group g[2];
      int ng = cfo_node_groups(pl, v, p, g);
      for (int k = 0; k < ng; k++) {
        gpus += (uint64_t)g[k].rep * (uint64_t)g[k].gpus;
        if (u[v][k] == 0.0) redundant = 1;
        else if (g[k].rep >= 2 && (double)(g[k].rep - 1) / u[v][k] >= best) redundant = 1;
      }
    }
    int over = gpus > (uint64_t)n_gpus;
    rd[p] = best;
    bottleneck[p] = bn;
    flags[p] = (uint8_t)(((!over && !redundant) ? 1 : 0) | (over ? 2 : 0) | (redundant ? 8 : 0));
  }
  return 0;
}

/* ---------------- top-K by R_d ---------------- */
static const double *g_sort_rd;
static int cmp_plan(const void *a, const void *b) {
  int i = *(const int32_t *)a, j = *(const int32_t *)b;
  if (g_sort_rd[i] > g_sort_rd[j]) return -1;
  if (g_sort_rd[i] < g_sort_rd[j]) return 1;
  return (i < j) ? -1 : (i > j);
}

int cfo_select_topk(const double *rd, const uint8_t *flags, int32_t P, int32_t k, int32_t *ids,
                    int32_t *n_selected) {
  int32_t *all = (int32_t *)malloc(sizeof(int32_t) * (size_t)(P > 0 ? P : 1));
  int n = 0;
  for (int p = 0; p < P; p++)
    if (flags[p] & 1u) all[n++] = p;
  g_sort_rd = rd;
  qsort(all, (size_t)n, sizeof(int32_t), cmp_plan);
  int take = n < k ? n : k;
  for (int i = 0; i < take; i++) ids[i] = all[i];
  *n_selected = take;
  free(all);
  return 0;
}

/* rate grid: r_k = (A * (k+1)) / K with A = R_d * alpha_max */
int cfo_rate_grid(const double *rd, const int32_t *ids, int32_t n, int32_t K, double alpha_max,
                  double *rates) {
  for (int i = 0; i < n; i++) {
    double A = rd[ids[i]] * alpha_max;
    for (int k = 0; k < K; k++) rates[(size_t)i * K + k] = (A * (double)(k + 1)) / (double)K;
  }
  return 0;
}

/* ---------------- goodput ---------------- */
int cfo_goodput_reduce(const uint32_t *met, const uint32_t *cnt, const uint32_t *status, int32_t n_plans,
                       int32_t K, int32_t S, int32_t T, const double *rates, uint32_t theta_num,
                       uint32_t theta_den, int32_t n_req, int32_t *kstar, double *goodput_t,
                       double *goodput) {
  double denom = (double)((uint64_t)S * (uint64_t)n_req);
  for (int i = 0; i < n_plans; i++) {
    int ks = K - 1;
    for (int k = 0; k < K; k++) {
      int feasible = 1;
      /* a simulation that failed (nonzero status) leaves counts that prove nothing */
      for (int s = 0; s < S; s++)
        if (status[((size_t)i * K + k) * S + s] != 0) feasible = 0;
      for (int t = 0; t < T; t++) {
        uint64_t M = 0, N = 0;
        for (int s = 0; s < S; s++) {
          size_t o = (((size_t)i * K + k) * S + s) * T + t;
          M += met[o];
          N += cnt[o];
        }
        if (N > 0 && (uint64_t)theta_den * M < (uint64_t)theta_num * N) feasible = 0;
      }
      if (!feasible) { ks = k - 1; break; }
    }
    kstar[i] = ks;
    double g = 0.0;
    for (int t = 0; t < T; t++) {
      double gt = 0.0;
      if (ks >= 0) {
        uint64_t M = 0;
        for (int s = 0; s < S; s++) M += met[(((size_t)i * K + ks) * S + s) * T + t];
        gt = (rates[(size_t)i * K + ks] * (double)M) / denom;
      }
      goodput_t[(size_t)i * T + t] = gt;
      g = g + gt;
    }
    goodput[i] = g;
  }
  return 0;
}

int32_t cfo_argmax(const double *goodput, int32_t n) {
  int32_t best = -1;
  for (int32_t i = 0; i < n; i++)
    if (best < 0 || goodput[i] > goodput[best]) best = i;
  return best;
}
