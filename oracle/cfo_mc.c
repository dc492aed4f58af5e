/*
 * cfo_mc.c -- oracle (test infrastructure only): phase 2 of the plan
 * evaluation (Sec. 4.3, Alg. 2 phase 2), Monte Carlo latency estimation with
 * occupancy-aware latency scaling (Sec. 5.2), and Pareto pruning of the
 * per-type goodput vectors (Alg. 2).
 *
 * For a plan d, K requests are drawn from the workload (the first K of one
 * trace seed: the trace is a seeded sample of the workload) and each is
 * routed through d alone, without queueing: each component it visits takes
 * one iteration of that component's latency model, at the component's
 * effective batch size on its node.  The per-type fraction of sampled
 * requests meeting the latency targets is F_t(L_t) and the per-type goodput
 * estimate is G_t = alpha R_d pi_t F_t(L_t).
 *
 * Readings (where the paper gives no formula):
 *   - effective batch: the bottleneck node runs at its configured batch B;
 *     a node with capacity R_v = m_v / u_v (phase 1) runs at
 *     b = clamp(ceil(B * (R_d / R_v)), 1, B), its share of the bottleneck's
 *     load;
 *   - an encoder or generator iteration is a static batch of b requests
 *     like this one: (k0 + k1 * (b * x)) + k2 * b (every iteration time
 *     times the component's multiplier for the node's GPUs per executor); an LLM admits a request's
 *     prefill as soon as it arrives (with prefill priority the prefill batch
 *     holds the few requests that arrived during one iteration), so the
 *     prefill is this request alone, (k0 + k1 * x) + k2, and the decode
 *     steps are shared with the running set of size b: d0 + d1 * b;
 *   - a component starts when its last input arrives: a parent's finish (a
 *     gate source's first token for a gated LLM) plus comm when the parent
 *     runs on another executor; token k+1 of a gated LLM needs the gate
 *     source's token min(k+1, n_src) (visible comm later across
 *     executors) and its own previous token; no CPU preprocessing time;
 *   - no sampled request of a type: F_t = 0.
 * Every fp64 formula is evaluated in the written order.
 */
#include "cfo.h"
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define P_AT(arr, slot, P, p) ((arr)[(size_t)(slot) * (size_t)(P) + (size_t)(p)])

static uint64_t attr(const cfo_trace *tr, size_t o, int a) {
  switch (a) {
  case CFO_A_PROMPT: return tr->prompt[o];
  case CFO_A_OUT: return tr->out[o];
  case CFO_A_PATCHES: return tr->patches[o];
  case CFO_A_AUDIN_MS: return tr->aud_in_ms[o];
  case CFO_A_AUDOUT_MS: return tr->aud_out_ms[o];
  case CFO_A_AUDIN_TOK: return (tr->aud_in_ms[o] + 79u) / 80u;
  case CFO_A_AUDOUT_TOK: return (tr->aud_out_ms[o] + 79u) / 80u;
  default: return 0;
  }
}

int cfo_eval_mc(const cfo_model *m, const cfo_plans *pl, const int32_t *ids, int32_t n,
                const double *rd, const uint64_t *moments, double alpha, const cfo_trace *tr,
                int32_t seed_idx, int32_t n_sample, uint32_t *met, uint32_t *cnt, double *gt,
                double *lat) {
  const int P = pl->P, T = m->n_types, NC = m->n_comp;
  uint64_t wsum_i = 0;
  for (int t = 0; t < T; t++) wsum_i += m->weight[t];
  const double wsum = (double)wsum_i;
  for (int i = 0; i < n; i++) {
    const int p = ids[i];
    uint32_t *mt = met + (size_t)i * T, *ct = cnt + (size_t)i * T;
    for (int t = 0; t < T; t++) { mt[t] = 0; ct[t] = 0; gt[(size_t)i * T + t] = 0.0; }
    if (p < 0 || p >= P || !cfo_plan_valid(m, pl, p)) continue;
    const int nv = pl->n_nodes[p];
    const double R_d = rd[p];
    /* capacities and effective batches */
    double u[CFO_MAXV][2];
    cfo_node_demand(m, pl, p, moments, u);
    /* effective batch of component c on executor group g of node v: the group's share of
     * the bottleneck's load */
    int beff[CFO_MAXV][2][CFO_MAXC];
    cfo_group grp[CFO_MAXV][2];
    int ngrp[CFO_MAXV];
    int base[CFO_MAXV + 1];
    base[0] = 0;
    for (int v = 0; v < nv; v++) {
      ngrp[v] = cfo_node_groups(pl, v, p, grp[v]);
      base[v + 1] = base[v];
      for (int k = 0; k < ngrp[v]; k++) {
        const int rep = grp[v][k].rep;
        base[v + 1] += rep;
        const double Rv = u[v][k] > 0.0 ? (double)rep / u[v][k] : INFINITY;
        const double q = R_d / Rv;
        for (int c = 0; c < NC; c++) {
          const int bnode = grp[v][k].batch;
          const int B = bnode < m->batch_cap[c] ? bnode : m->batch_cap[c];
          double bb = ceil((double)B * q);
          int b = bb < 1.0 ? 1 : (bb > (double)B ? B : (int)bb);
          beff[v][k][c] = b;
        }
      }
    }
    /* the sampled requests */
    for (int r = 0; r < n_sample; r++) {
      const size_t o = (size_t)seed_idx * (size_t)tr->n_req + (size_t)r;
      const int ty = tr->type[o];
      if (ty >= T) continue;
      const int na = P_AT(pl->n_alt, ty, P, p);
      int alt = 0;
      if (na == 2) {
        uint64_t w0 = P_AT(pl->alt_w, ty * 2 + 0, P, p), w1 = P_AT(pl->alt_w, ty * 2 + 1, P, p);
        alt = ((((uint64_t)tr->akey[o]) * (w0 + w1)) >> 32) < w0 ? 0 : 1;
      }
      int ex[CFO_MAXC], node[CFO_MAXC], nout[CFO_MAXC];
      double fin[CFO_MAXC], first[CFO_MAXC], dstep[CFO_MAXC];
      int ttft_c = -1;
      double completion = 0.0, media = 0.0;
      int has_gen = 0;
      for (int c = 0; c < NC; c++) {
        if (!((m->path_mask[ty] >> c) & 1u)) continue;
        const int v = P_AT(pl->alt_node, (ty * 2 + alt) * 8 + c, P, p);
        const int cm = P_AT(pl->node_comp, v, P, p);
        const int minc = __builtin_ctz(cm);
        const uint64_t word = minc < 4 ? tr->rkey0[o] : tr->rkey1[o];
        const uint64_t key = (word >> (16 * (minc & 3))) & 0xFFFFu;
        const int j = cfo_node_pick(key, grp[v], ngrp[v], pl, v, p);
        const int gk = j < grp[v][0].rep ? 0 : 1;  /* the executor's group */
        ex[c] = base[v] + j;
        node[c] = v;
        /* start: the last input to arrive */
        const int src = m->gate_src[c];
        const int gated_here = src >= 0 && ((m->path_mask[ty] >> src) & 1u) && ((m->parents[ty][c] >> src) & 1u);
        double start = 0.0;
        for (int pc = 0; pc < c; pc++) {
          if (!((m->parents[ty][c] >> pc) & 1u)) continue;
          const double hop = ex[pc] == ex[c] ? 0.0 : m->comm_s;
          const double ready = (gated_here && pc == src) ? first[pc] + hop : fin[pc] + hop;
          if (ready > start) start = ready;
        }
        const int b = beff[v][gk][c];
        const double tps = cfo_tp(m, c, grp[v][gk].gpus);
        uint64_t x = 0;
        for (int at = 0; at < CFO_NATTR; at++)
          if ((m->x_sel[c] >> at) & 1u) x += attr(tr, o, at);
        if (m->kind[c] != CFO_LLM) {
          const double dur = tps * ((m->k0[c] + m->k1[c] * (double)((uint64_t)b * x)) + m->k2[c] * (double)b);
          fin[c] = start + dur;
          first[c] = fin[c];
        } else {
          const double dur = tps * ((m->k0[c] + m->k1[c] * (double)x) + m->k2[c] * 1.0);
          uint64_t no = ((m->prefill_only[ty] >> c) & 1u) ? 1u : attr(tr, o, m->nout_attr[c]);
          nout[c] = no < 1 ? 1 : (int)no;
          const double D = tps * (m->d0[c] + m->d1[c] * (double)b);
          dstep[c] = D;
          first[c] = start + dur;
          double e = first[c];
          if (!gated_here) {
            for (int k = 2; k <= nout[c]; k++) e = e + D;
          } else {
            /* token k+1 waits for the gate source's token min(k+1, n_src) */
            const double hop = ex[src] == ex[c] ? 0.0 : m->comm_s;
            double eg = first[src];
            int jg = 1;
            for (int k = 1; k < nout[c]; k++) {
              const int need = k + 1 < nout[src] ? k + 1 : nout[src];
              while (jg < need) { eg = eg + dstep[src]; jg++; }
              const double vis = eg + hop;
              const double s = e < vis ? vis : e;
              e = s + D;
            }
          }
          fin[c] = e;
          if (ttft_c < 0) ttft_c = c;
        }
        if ((m->out_mask[ty] >> c) & 1u) {
          if (fin[c] > completion) completion = fin[c];
          if (m->kind[c] == CFO_GEN) {
            has_gen = 1;
            if (fin[c] > media) media = fin[c];
          }
        }
      }
      (void)node;
      double ttft = 0.0, tpot = 0.0;
      if (ttft_c >= 0) {
        ttft = first[ttft_c];
        if (nout[ttft_c] > 1) tpot = (fin[ttft_c] - first[ttft_c]) / (double)(nout[ttft_c] - 1);
      }
      const double e2e = completion, md = has_gen ? media : 0.0;
      const int ok = ttft <= m->slo[ty][0] && tpot <= m->slo[ty][1] && e2e <= m->slo[ty][2] &&
                     md <= m->slo[ty][3];
      ct[ty]++;
      if (ok) mt[ty]++;
      if (lat) {
        double *L = lat + ((size_t)i * n_sample + r) * 4;
        L[0] = ttft; L[1] = tpot; L[2] = e2e; L[3] = md;
      }
    }
    for (int t = 0; t < T; t++) {
      const double pi = (double)m->weight[t] / wsum;
      gt[(size_t)i * T + t] = ct[t] > 0 ? ((alpha * R_d) * pi) * ((double)mt[t] / (double)ct[t]) : 0.0;
    }
  }
  return 0;
}

int cfo_pareto(const double *g, int32_t n, int32_t T, uint8_t *keep) {
  for (int i = 0; i < n; i++) {
    int dominated = 0;
    for (int j = 0; j < n && !dominated; j++) {
      if (j == i) continue;
      int ge = 1, gt = 0;
      for (int t = 0; t < T; t++) {
        const double a = g[(size_t)j * T + t], b = g[(size_t)i * T + t];
        if (a < b) { ge = 0; break; }
        if (a > b) gt = 1;
      }
      if (ge && gt) dominated = 1;
    }
    keep[i] = dominated ? 0 : 1;
  }
  return 0;
}

/* The bin of one request: the first bin whose four bounds its latencies
 * meet, by a scan from bin 0 (n_bins if none). */
static int first_bin(const double *targets, int n_bins, int t, const double *lat) {
  for (int b = 0; b < n_bins; b++) {
    const double *g = targets + ((size_t)t * n_bins + b) * 4;
    if (lat[0] <= g[0] && lat[1] <= g[1] && lat[2] <= g[2] && lat[3] <= g[3]) return b;
  }
  return n_bins;
}

int cfo_latency_hist(const double *lat, const uint8_t *type, int32_t n, int32_t T, int32_t n_bins,
                     const double *targets, uint32_t *hist) {
  for (int q = 0; q < T * (n_bins + 1); q++) hist[q] = 0;
  for (int r = 0; r < n; r++) {
    const int t = type[r];
    if (t >= T) continue;
    hist[t * (n_bins + 1) + first_bin(targets, n_bins, t, lat + (size_t)r * 4)]++;
  }
  return 0;
}

int cfo_mc_curve(const cfo_model *m, const cfo_plans *pl, const int32_t *ids, int32_t n, const double *rd,
                 const uint64_t *moments, double alpha, const cfo_trace *tr, int32_t seed_idx, int32_t n_sample,
                 int32_t n_bins, const double *targets, uint32_t *met, uint32_t *cnt, double *gt, uint32_t *hist,
                 double *curve) {
  const int T = m->n_types;
  double *lat = (double *)malloc(sizeof(double) * 4 * (size_t)(n_sample > 0 ? n_sample : 1));
  if (!lat) return -1;
  uint64_t wsum_i = 0;
  for (int t = 0; t < T; t++) wsum_i += m->weight[t];
  const double wsum = (double)wsum_i;
  for (int i = 0; i < n; i++) {
    cfo_eval_mc(m, pl, ids + i, 1, rd, moments, alpha, tr, seed_idx, n_sample, met + (size_t)i * T,
                cnt + (size_t)i * T, gt + (size_t)i * T, lat);
    uint32_t *h = hist + (size_t)i * T * (n_bins + 1);
    const int p = ids[i];
    const int valid = p >= 0 && p < pl->P && cfo_plan_valid(m, pl, p);
    if (valid)
      cfo_latency_hist(lat, tr->type + (size_t)seed_idx * (size_t)tr->n_req, n_sample, T, n_bins, targets, h);
    else
      for (int q = 0; q < T * (n_bins + 1); q++) h[q] = 0;
    /* F_t at bin b: the requests in bins 0..b over the type's count */
    for (int b = 0; b < n_bins; b++)
      for (int t = 0; t < T; t++) {
        uint32_t below = 0;
        for (int k = 0; k <= b; k++) below += h[t * (n_bins + 1) + k];
        const uint32_t ct = cnt[(size_t)i * T + t];
        const double pi = (double)m->weight[t] / wsum;
        curve[((size_t)i * n_bins + b) * T + t] =
            (valid && ct > 0) ? ((alpha * rd[p]) * pi) * ((double)below / (double)ct) : 0.0;
      }
  }
  free(lat);
  return 0;
}
