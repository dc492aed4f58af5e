/*
 * cfo_enum.c -- oracle (test infrastructure only): plan enumeration
 * (Sec. 4.2, Alg. 1) and the executor partitions of Eq. (1).
 *
 * Logical plans, in this order:
 *   - subgraphs: for every non-empty set of request types, the union cs of
 *     their paths; the distinct unions in ascending bitmask order.  A
 *     subgraph covers every type whose path lies inside it;
 *   - simple subplans of cs (Alg. 1, Keep/Merge): the edges of the covered
 *     types that may be colocated, in ascending (parent, child) order; for
 *     every Keep/Merge vector m = 0 .. 2^k - 1 (bit i: merge edge i) the
 *     connected groups of cs under the merged edges are the nodes, listed
 *     by ascending bitmask; a grouping already produced for cs is skipped;
 *   - logical plans: every simple subplan covering all types alone; then,
 *     with k_s = 2, every pair i <= j of simple subplans that together cover
 *     all types, once per set s of shared nodes (compound subplans: a node
 *     of subplan j whose mask equals a node of subplan i may be the same
 *     node; s runs over the subsets of those nodes in ascending bitmask
 *     order, only the empty set when sharing is off, never all of subplan
 *     j's nodes).  Nodes: subplan i's, then subplan j's unshared ones.  A
 *     type covered by both has two alternatives (i's path first) unless both
 *     map every component of its path to the same nodes; plans with more
 *     than 16 nodes, and repeats of an earlier plan, are dropped.
 * Physical plans of a logical plan (Eq. 1): node v takes one configuration
 * k (GPUs per executor from the options of its lowest component, then the
 * batch from that component's knobs; GPU option major) and n_v >= 1
 * executors, with sum_v gpus_v n_v <= N; every type with two alternatives
 * takes a routing weight w in 1..9 tenths for its first alternative (10 - w
 * for the second).  Order: the executor assignments lexicographically in
 * ((k_0, n_0), (k_1, n_1), ...), the routing weights lexicographically
 * (lowest type most significant) inside each.
 */
#include "cfo.h"
#include <stdlib.h>
#include <string.h>

/* groups of cs under the merged edges, ascending masks; returns the count */
static int groups_of(uint32_t cs, const int *ea, const int *eb, int ne, uint32_t m, uint32_t *out) {
  uint32_t group[CFO_MAXC];
  for (int c = 0; c < CFO_MAXC; c++) group[c] = 1u << c;
  /* repeat until stable: each merged edge joins the groups of its ends */
  int changed = 1;
  while (changed) {
    changed = 0;
    for (int i = 0; i < ne; i++) {
      if (!((m >> i) & 1u)) continue;
      const uint32_t u = group[ea[i]] | group[eb[i]];
      for (int c = 0; c < CFO_MAXC; c++)
        if ((u >> c) & 1u && group[c] != u) {
          group[c] = u;
          changed = 1;
        }
    }
  }
  int n = 0;
  for (int c = 0; c < CFO_MAXC; c++) {
    if (!((cs >> c) & 1u)) continue;
    int seen = 0;
    for (int k = 0; k < n; k++)
      if (out[k] == group[c]) seen = 1;
    if (!seen) out[n++] = group[c];
  }
  /* ascending masks (insertion sort) */
  for (int a = 1; a < n; a++)
    for (int b = a; b > 0 && out[b - 1] > out[b]; b--) {
      const uint32_t t = out[b];
      out[b] = out[b - 1];
      out[b - 1] = t;
    }
  return n;
}

typedef struct {
  uint32_t cs, cov;
  int nn;
  uint32_t mask[CFO_MAXC];
} simple_t;

static int same_plan(const cfo_logical *a, const cfo_logical *b, int T) {
  if (a->n_nodes != b->n_nodes) return 0;
  for (int v = 0; v < a->n_nodes; v++)
    if (a->node_comp[v] != b->node_comp[v]) return 0;
  for (int t = 0; t < T; t++) {
    if (a->n_alt[t] != b->n_alt[t]) return 0;
    for (int k = 0; k < a->n_alt[t]; k++)
      for (int c = 0; c < CFO_MAXC; c++)
        if (a->alt_node[t][k][c] != b->alt_node[t][k][c]) return 0;
  }
  return 1;
}

/* the node of subplan s holding component c (index into its mask list) */
static int holder(const simple_t *s, int c) {
  for (int k = 0; k < s->nn; k++)
    if ((s->mask[k] >> c) & 1u) return k;
  return -1;
}

int cfo_enum_logical(const cfo_model *m, const cfo_enum_opts *o, cfo_logical *out, int32_t cap,
                     int32_t *n_out) {
  const int T = m->n_types, C = m->n_comp;
  const uint32_t all = (T >= 32) ? 0xFFFFFFFFu : ((1u << T) - 1u);
  *n_out = 0;
  /* distinct subgraphs */
  uint32_t css[256];
  int ncs = 0;
  for (uint32_t u = 1; u <= all && u < (1u << CFO_MAXT); u++) {
    uint32_t cs = 0;
    for (int t = 0; t < T; t++)
      if ((u >> t) & 1u) cs |= m->path_mask[t];
    int seen = 0;
    for (int k = 0; k < ncs; k++)
      if (css[k] == cs) seen = 1;
    if (!seen) css[ncs++] = cs;
  }
  for (int a = 1; a < ncs; a++)
    for (int b = a; b > 0 && css[b - 1] > css[b]; b--) {
      const uint32_t t = css[b];
      css[b] = css[b - 1];
      css[b - 1] = t;
    }
  /* simple subplans */
  simple_t *S = (simple_t *)malloc(sizeof(simple_t) * 65536);
  if (!S) return -1;
  int ns = 0;
  for (int k = 0; k < ncs; k++) {
    const uint32_t cs = css[k];
    uint32_t cov = 0;
    for (int t = 0; t < T; t++)
      if ((m->path_mask[t] & ~cs) == 0) cov |= 1u << t;
    int ea[64], eb[64], ne = 0;
    for (int p = 0; p < C; p++)
      for (int c = 0; c < C; c++) {
        if (!((o->colocatable[p] >> c) & 1u)) continue;
        int used = 0;
        for (int t = 0; t < T; t++)
          if (((cov >> t) & 1u) && ((m->parents[t][c] >> p) & 1u)) used = 1;
        if (used) {
          ea[ne] = p;
          eb[ne] = c;
          ne++;
        }
      }
    if (ne > 16) {
      free(S);
      return -2;
    }
    const int first = ns;
    for (uint32_t mm = 0; mm < (1u << ne); mm++) {
      simple_t s;
      s.cs = cs;
      s.cov = cov;
      s.nn = groups_of(cs, ea, eb, ne, mm, s.mask);
      int dup = 0;
      for (int q = first; q < ns && !dup; q++) {
        if (S[q].nn != s.nn) continue;
        int eq = 1;
        for (int v = 0; v < s.nn; v++)
          if (S[q].mask[v] != s.mask[v]) eq = 0;
        dup = eq;
      }
      if (dup) continue;
      if (ns >= 65536) {
        free(S);
        return -3;
      }
      S[ns++] = s;
    }
  }
  /* logical plans */
  int n = 0;
#define EMIT(Lp)                                                          \
  do {                                                                    \
    int dup_ = 0;                                                         \
    for (int q_ = 0; q_ < n && !dup_; q_++) dup_ = same_plan(&out[q_], (Lp), T); \
    if (!dup_) {                                                          \
      if (n >= cap) { free(S); return -4; }                               \
      out[n++] = *(Lp);                                                   \
    }                                                                     \
  } while (0)
  for (int i = 0; i < ns; i++) {
    if (S[i].cov != all) continue;
    cfo_logical L;
    memset(&L, 0, sizeof L);
    memset(L.alt_node, 255, sizeof L.alt_node);
    L.n_nodes = (uint8_t)S[i].nn;
    for (int v = 0; v < S[i].nn; v++) L.node_comp[v] = (uint8_t)S[i].mask[v];
    for (int t = 0; t < T; t++) {
      L.n_alt[t] = 1;
      for (int c = 0; c < C; c++)
        if ((m->path_mask[t] >> c) & 1u) L.alt_node[t][0][c] = (uint8_t)holder(&S[i], c);
    }
    EMIT(&L);
  }
  if (o->k_s >= 2) {
    for (int i = 0; i < ns; i++)
      for (int j = i; j < ns; j++) {
        if ((S[i].cov | S[j].cov) != all) continue;
        /* the nodes of j that may be shared, in j's order, and their partner in i */
        int cand[CFO_MAXC], partner[CFO_MAXC], nc = 0;
        for (int v = 0; v < S[j].nn; v++)
          for (int w = 0; w < S[i].nn; w++)
            if (S[j].mask[v] == S[i].mask[w]) {
              cand[nc] = v;
              partner[nc] = w;
              nc++;
            }
        const uint32_t nsets = o->share ? (1u << nc) : 1u;
        for (uint32_t sset = 0; sset < nsets; sset++) {
          if (nc == S[j].nn && sset == nsets - 1 && o->share) continue; /* all of j shared */
          int jmap[CFO_MAXC];
          const int nv_i = S[i].nn;
          int nv = nv_i;
          for (int v = 0; v < S[j].nn; v++) {
            jmap[v] = -1;
            for (int k = 0; k < nc; k++)
              if (cand[k] == v && ((sset >> k) & 1u)) jmap[v] = partner[k];
            if (jmap[v] < 0) jmap[v] = nv++;
          }
          if (nv > CFO_MAXV) continue;
          cfo_logical L;
          memset(&L, 0, sizeof L);
          memset(L.alt_node, 255, sizeof L.alt_node);
          L.n_nodes = (uint8_t)nv;
          for (int v = 0; v < nv_i; v++) L.node_comp[v] = (uint8_t)S[i].mask[v];
          for (int v = 0; v < S[j].nn; v++) L.node_comp[jmap[v]] = (uint8_t)S[j].mask[v];
          for (int t = 0; t < T; t++) {
            int na = 0;
            if ((S[i].cov >> t) & 1u) {
              for (int c = 0; c < C; c++)
                if ((m->path_mask[t] >> c) & 1u) L.alt_node[t][na][c] = (uint8_t)holder(&S[i], c);
              na++;
            }
            if ((S[j].cov >> t) & 1u) {
              for (int c = 0; c < C; c++)
                if ((m->path_mask[t] >> c) & 1u) L.alt_node[t][na][c] = (uint8_t)jmap[holder(&S[j], c)];
              if (na == 1 && memcmp(L.alt_node[t][0], L.alt_node[t][1], CFO_MAXC) == 0)
                memset(L.alt_node[t][1], 255, CFO_MAXC);
              else
                na++;
            }
            L.n_alt[t] = (uint8_t)na;
          }
          EMIT(&L);
        }
      }
  }
#undef EMIT
  free(S);
  *n_out = n;
  return 0;
}

/* node v's configurations: GPU option major, batch minor */
static int n_configs(const cfo_enum_opts *o, int c0) { return o->n_gpu_opt[c0] * o->n_batch[c0]; }
static int config_gpus(const cfo_enum_opts *o, int c0, int k) { return o->gpu_opt[c0][k / o->n_batch[c0]]; }
static int config_batch(const cfo_enum_opts *o, int c0, int k) { return o->batch[c0][k % o->n_batch[c0]]; }

static int lowest(uint32_t mask) {
  for (int c = 0; c < 32; c++)
    if ((mask >> c) & 1u) return c;
  return -1;
}

/* cnt[v][b]: executor assignments of nodes v.. within budget b, by the
 * recursion over node v's configuration and executor count (saturating at
 * UINT64_MAX) */
#define CFO_MAXN 256
typedef uint64_t count_table[CFO_MAXV + 1][CFO_MAXN + 1];

static uint64_t sat_add(uint64_t a, uint64_t b) { return a > UINT64_MAX - b ? UINT64_MAX : a + b; }
static uint64_t sat_mul(uint64_t a, uint64_t b) { return (b != 0 && a > UINT64_MAX / b) ? UINT64_MAX : a * b; }

/* A node's executor assignments, in this order: one configuration k with n >= 1
 * executors (k, then n ascending); then, with het, two configurations k1 < k2 with
 * n1, n2 >= 1 executors and w = 1..9 tenths of the node's requests for k1 (k1, k2,
 * n1, n2, w ascending). */
static void fill_counts(const cfo_logical *L, const cfo_enum_opts *o, count_table cnt) {
  const int N = o->n_gpus, V = L->n_nodes;
  for (int b = 0; b <= N; b++) cnt[V][b] = 1;
  for (int v = V - 1; v >= 0; v--) {
    const int c0 = lowest(L->node_comp[v]);
    const int K = n_configs(o, c0);
    for (int b = 0; b <= N; b++) {
      uint64_t total = 0;
      for (int k = 0; k < K; k++) {
        const int g = config_gpus(o, c0, k);
        for (int n = 1; g * n <= b; n++) total = sat_add(total, cnt[v + 1][b - g * n]);
      }
      if (o->het)
        for (int k1 = 0; k1 < K; k1++)
          for (int k2 = k1 + 1; k2 < K; k2++) {
            const int g1 = config_gpus(o, c0, k1), g2 = config_gpus(o, c0, k2);
            for (int n1 = 1; g1 * n1 + g2 <= b; n1++)
              for (int n2 = 1; g1 * n1 + g2 * n2 <= b; n2++)
                total = sat_add(total, sat_mul(9, cnt[v + 1][b - g1 * n1 - g2 * n2]));
          }
      cnt[v][b] = total;
    }
  }
}

static int two_alt_types(const cfo_logical *L, int T) {
  int a = 0;
  for (int t = 0; t < T; t++) a += L->n_alt[t] == 2;
  return a;
}

static uint64_t routings(const cfo_logical *L, int T) {
  uint64_t R = 1;
  for (int i = 0; i < two_alt_types(L, T); i++) R *= 9;
  return R;
}

uint64_t cfo_enum_count(const cfo_model *m, const cfo_enum_opts *o, const cfo_logical *L) {
  static count_table cnt;
  fill_counts(L, o, cnt);
  return sat_mul(cnt[0][o->n_gpus], routings(L, m->n_types));
}

typedef struct {
  const cfo_model *m;
  const cfo_enum_opts *o;
  const cfo_logical *L;
  uint64_t idx, first, end; /* running index, output window [first, end) */
  int32_t P;                /* output columns */
  uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  uint16_t *node_batch;
  uint8_t *node_rep2, *node_gpus2, *node_w;
  uint16_t *node_batch2;
  int kk[CFO_MAXV], nn[CFO_MAXV];
  int kk2[CFO_MAXV], nn2[CFO_MAXV], ww[CFO_MAXV]; /* second configuration (nn2 = 0: none) */
  uint64_t R;
  uint64_t (*cnt)[CFO_MAXN + 1];
} walk_t;

static void emit_routes(walk_t *w) {
  const cfo_logical *L = w->L;
  const int T = w->m->n_types;
  const int a = two_alt_types(L, T);
  const uint64_t R = w->R;
  for (uint64_t r = 0; r < R; r++, w->idx++) {
    if (w->idx < w->first || w->idx >= w->end) continue;
    const size_t p = (size_t)(w->idx - w->first), P = (size_t)w->P;
    w->n_nodes[p] = L->n_nodes;
    for (int v = 0; v < CFO_MAXV; v++) {
      if (v < L->n_nodes) {
        const int c0 = lowest(L->node_comp[v]);
        w->node_comp[v * P + p] = L->node_comp[v];
        w->node_rep[v * P + p] = (uint8_t)w->nn[v];
        w->node_gpus[v * P + p] = (uint8_t)config_gpus(w->o, c0, w->kk[v]);
        w->node_batch[v * P + p] = (uint16_t)config_batch(w->o, c0, w->kk[v]);
        w->node_rep2[v * P + p] = (uint8_t)w->nn2[v];
        w->node_gpus2[v * P + p] = (uint8_t)(w->nn2[v] ? config_gpus(w->o, c0, w->kk2[v]) : 0);
        w->node_batch2[v * P + p] = (uint16_t)(w->nn2[v] ? config_batch(w->o, c0, w->kk2[v]) : 0);
        w->node_w[v * P + p] = (uint8_t)(w->nn2[v] ? w->ww[v] : 10);
      } else {
        w->node_comp[v * P + p] = 0;
        w->node_rep[v * P + p] = 0;
        w->node_gpus[v * P + p] = 0;
        w->node_batch[v * P + p] = 0;
        w->node_rep2[v * P + p] = 0;
        w->node_gpus2[v * P + p] = 0;
        w->node_batch2[v * P + p] = 0;
        w->node_w[v * P + p] = 10;
      }
    }
    /* routing digits: the lowest type is the most significant */
    uint64_t rem = r;
    int wt[CFO_MAXT];
    for (int i = a - 1; i >= 0; i--) {
      wt[i] = (int)(rem % 9) + 1;
      rem /= 9;
    }
    int i2 = 0;
    for (int t = 0; t < CFO_MAXT; t++) {
      const int na = t < T ? L->n_alt[t] : 0;
      w->n_alt[t * P + p] = (uint8_t)na;
      int w0 = 0, w1 = 0;
      if (na == 1) w0 = 10;
      if (na == 2) {
        w0 = wt[i2++];
        w1 = 10 - w0;
      }
      w->alt_w[(2 * t) * P + p] = (uint8_t)w0;
      w->alt_w[(2 * t + 1) * P + p] = (uint8_t)w1;
      for (int k = 0; k < 2; k++)
        for (int c = 0; c < CFO_MAXC; c++)
          w->alt_node[((2 * t + k) * CFO_MAXC + c) * P + p] = t < T ? L->alt_node[t][k][c] : 255;
    }
  }
}

/* every assignment in order; a subtree wholly before the window is skipped
 * by its count */
static void walk_nodes(walk_t *w, int v, int b) {
  if (w->idx >= w->end) return;
  if (v == w->L->n_nodes) {
    emit_routes(w);
    return;
  }
  const int c0 = lowest(w->L->node_comp[v]);
  for (int k = 0; k < n_configs(w->o, c0); k++) {
    const int g = config_gpus(w->o, c0, k);
    for (int n = 1; g * n <= b; n++) {
      if (w->idx >= w->end) return;
      const uint64_t sub = sat_mul(w->cnt[v + 1][b - g * n], w->R);
      if (w->idx + sub <= w->first) {
        w->idx += sub;
        continue;
      }
      w->kk[v] = k;
      w->nn[v] = n;
      w->nn2[v] = 0;
      walk_nodes(w, v + 1, b - g * n);
    }
  }
  if (!w->o->het) return;
  const int K = n_configs(w->o, c0);
  for (int k1 = 0; k1 < K; k1++)
    for (int k2 = k1 + 1; k2 < K; k2++) {
      const int g1 = config_gpus(w->o, c0, k1), g2 = config_gpus(w->o, c0, k2);
      for (int n1 = 1; g1 * n1 + g2 <= b; n1++)
        for (int n2 = 1; g1 * n1 + g2 * n2 <= b; n2++)
          for (int ws = 1; ws <= 9; ws++) {
            if (w->idx >= w->end) return;
            const int rest = b - g1 * n1 - g2 * n2;
            const uint64_t sub = sat_mul(w->cnt[v + 1][rest], w->R);
            if (w->idx + sub <= w->first) {
              w->idx += sub;
              continue;
            }
            w->kk[v] = k1;
            w->nn[v] = n1;
            w->kk2[v] = k2;
            w->nn2[v] = n2;
            w->ww[v] = ws;
            walk_nodes(w, v + 1, rest);
          }
    }
}

int cfo_enum_plans(const cfo_model *m, const cfo_enum_opts *o, const cfo_logical *L, int32_t n_logical,
                   uint64_t first, int32_t count, uint8_t *n_nodes, uint8_t *node_comp, uint8_t *node_rep,
                   uint16_t *node_batch, uint8_t *node_gpus, uint8_t *n_alt, uint8_t *alt_w,
                   uint8_t *alt_node, uint8_t *node_rep2, uint16_t *node_batch2, uint8_t *node_gpus2,
                   uint8_t *node_w) {
  static count_table table;
  uint64_t base = 0;
  const uint64_t end = first + (uint64_t)count;
  if (o->n_gpus < 1 || o->n_gpus > CFO_MAXN) return -3;
  for (int i = 0; i < n_logical && base < end; i++) {
    fill_counts(&L[i], o, table);
    const uint64_t cnt = sat_mul(table[0][o->n_gpus], routings(&L[i], m->n_types));
    if (cnt == UINT64_MAX) return -1;
    if (base + cnt > first) {
      walk_t w;
      memset(&w, 0, sizeof w);
      w.m = m;
      w.o = o;
      w.L = &L[i];
      w.idx = base;
      w.first = first;
      w.end = end;
      w.P = count;
      w.n_nodes = n_nodes;
      w.node_comp = node_comp;
      w.node_rep = node_rep;
      w.node_batch = node_batch;
      w.node_gpus = node_gpus;
      w.n_alt = n_alt;
      w.alt_w = alt_w;
      w.alt_node = alt_node;
      w.node_rep2 = node_rep2;
      w.node_batch2 = node_batch2;
      w.node_gpus2 = node_gpus2;
      w.node_w = node_w;
      w.R = routings(&L[i], m->n_types);
      w.cnt = table;
      walk_nodes(&w, 0, o->n_gpus);
    }
    base += cnt;
  }
  return base >= end ? 0 : -2;
}
