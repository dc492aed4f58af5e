/*
 * cfo.h -- the oracle: a plain, slow, single-threaded CPU implementation of
 * the statistical plan evaluation of Cornfigurator (arXiv 2512.14098), used
 * ONLY as test infrastructure (pytest, the smoke check and the CPU-baseline
 * leg of the benchmark).  Nothing in the product path may link or call it.
 *
 * It shares no code, header, table or helper with the HIP library: every
 * structure below is the oracle's own.  All floating point is IEEE fp64,
 * compiled with -ffp-contract=off, and every formula is evaluated in the
 * written order with one rounding per operation.
 *
 * What is computed, and where the paper defines it:
 *   - request traces (workload with per-type fractions pi_t, Sec. 3.1);
 *   - phase 1 flow-based throughput R_d, bottleneck and redundancy pruning
 *     (Sec. 4.3, Alg. 2 phase 1);
 *   - phase 2 Monte Carlo latency with occupancy-aware latency scaling and
 *     Pareto pruning (Sec. 4.3, Alg. 2 phase 2; Sec. 5.2);
 *   - phase 3 request-level simulation of a physical plan at a given rate
 *     (Sec. 4.3, Alg. 2 phase 3; Sec. 5.2 CPU-GPU overlap and communication
 *     overhead);
 *   - plan enumeration: logical plans from simple and compound subplans,
 *     physical plans by the executor partitions of Eq. (1) and routing
 *     weights (Sec. 4.2, Alg. 1);
 *   - per-type goodput = throughput of requests meeting their latency target
 *     (Sec. 3.2), maximum achievable goodput over a rate grid (Sec. 6.1),
 *     argmax selection (Alg. 2, final step).
 * Where the paper is silent, the readings are the ones listed in the design
 * notes of this repository (scheduling policy, tie-breaking, gating).
 */
#ifndef CFO_H
#define CFO_H
#include <stdint.h>
#include <stddef.h>

#define CFO_MAXC 8   /* components */
#define CFO_MAXT 8   /* request types */
#define CFO_MAXV 16  /* nodes per plan */
#define CFO_MAXA 2   /* alternative paths per type (k_s = 2, Sec. 4.2) */
#define CFO_MAXX 64  /* executors per plan */
#define CFO_MAXB 256 /* max batch */

enum { CFO_ENC = 0, CFO_LLM = 1, CFO_GEN = 2 };

/* per-request attributes (index into the attribute vector) */
enum {
  CFO_A_PROMPT = 0, CFO_A_OUT = 1, CFO_A_PATCHES = 2, CFO_A_AUDIN_MS = 3,
  CFO_A_AUDOUT_MS = 4, CFO_A_AUDIN_TOK = 5, CFO_A_AUDOUT_TOK = 6, CFO_NATTR = 7
};

/* length distributions */
enum { CFO_D_NONE = 0, CFO_D_CONST = 1, CFO_D_LOGNORMAL = 2, CFO_D_EXP = 3 };
/* image-count distributions */
enum { CFO_I_NONE = 0, CFO_I_CONST = 1, CFO_I_UNIFORM = 2 };

/* per-triple status bits */
#define CFO_ST_INVALID 1u   /* route does not fit the plan */
#define CFO_ST_DEADLOCK 2u  /* event queue drained with requests unfinished */

typedef struct {
  int32_t kind;      /* CFO_D_* */
  int32_t pad;
  double p0, p1;     /* CONST: value p0; LOGNORMAL: mu=p0 sigma=p1; EXP: mean p0 */
  double scale;      /* multiplier applied before rounding (1 tokens, 1000 ms) */
  int64_t lo, hi;    /* clamp */
} cfo_dist;

typedef struct {
  int32_t n_comp, n_types;
  int32_t kind[CFO_MAXC];
  double k0[CFO_MAXC], k1[CFO_MAXC], k2[CFO_MAXC]; /* batch: (k0 + k1*X) + k2*n */
  double d0[CFO_MAXC], d1[CFO_MAXC];               /* LLM decode: d0 + d1*n   */
  uint32_t x_sel[CFO_MAXC];     /* bitmask of attributes summed into X     */
  int32_t nout_attr[CFO_MAXC];  /* LLM: attribute giving the output length */
  int32_t gate_src[CFO_MAXC];   /* LLM gated by this component, or -1      */
  int32_t batch_cap[CFO_MAXC];  /* stage batch = min(node batch, cap)      */
  double comm_s, cpu_pre_s;
  uint32_t weight[CFO_MAXT];
  uint32_t path_mask[CFO_MAXT], out_mask[CFO_MAXT], prefill_only[CFO_MAXT];
  uint32_t parents[CFO_MAXT][CFO_MAXC];
  int32_t img_kind[CFO_MAXT], img_lo[CFO_MAXT], img_hi[CFO_MAXT];
  int32_t patch_lo, patch_hi;
  cfo_dist len[CFO_MAXT][4];    /* prompt, out, aud_in_ms, aud_out_ms */
  double slo[CFO_MAXT][4];      /* ttft, tpot, e2e, media (<=; +inf = none) */
  uint32_t theta_num, theta_den;
  /* latency multiplier of component c on executors of g GPUs (tensor
   * parallelism degree), tp_scale[c][min(g, 8) - 1]; 1 = the profiled
   * single-GPU latency model */
  double tp_scale[CFO_MAXC][8];
} cfo_model;

/* the multiplier of component c's iteration time on executors of g GPUs */
static inline double cfo_tp(const cfo_model *m, int c, int g) {
  const int k = g < 1 ? 1 : (g > 8 ? 8 : g);
  return m->tp_scale[c][k - 1];
}

typedef struct {
  int32_t n_seeds, n_req;
  uint64_t *arr_ticks;            /* [S][n] inclusive prefix of gap ticks */
  uint8_t *type, *n_img;          /* [S][n] */
  uint16_t *patches, *prompt, *out;
  uint32_t *aud_in_ms, *aud_out_ms;
  uint64_t *rkey0, *rkey1;        /* 16-bit replica keys, component c at bits 16*(c%4) of word c/4 */
  uint32_t *akey;                 /* alternative-choice key */
} cfo_trace;

/* plan table: structure of arrays, field-slot major ([slot][P]) */
typedef struct {
  int32_t P;
  const uint8_t *n_nodes;     /* [P] */
  const uint8_t *node_comp;   /* [16][P] component bitmask */
  const uint8_t *node_rep;    /* [16][P] replicas m_v */
  const uint16_t *node_batch; /* [16][P] max batch B_v */
  const uint8_t *node_gpus;   /* [16][P] GPUs per replica */
  const uint8_t *n_alt;       /* [8][P] */
  const uint8_t *alt_w;       /* [8][2][P] weight in tenths */
  const uint8_t *alt_node;    /* [8][2][8][P] node per component, 255 = none */
  /* A node may hold executors of two configurations (Eq. (1): n_{v,k} executors of
   * configuration k): node_rep2 > 0 executors of batch node_batch2 and node_gpus2 GPUs next
   * to the node_rep of the first, and a request reaching the node goes to the first group
   * with probability node_w / 10, to the second with (10 - node_w) / 10 (routing between the
   * executors of a node in steps of 0.1, Sec. 4.2).  NULL arrays: every node has one
   * configuration. */
  const uint8_t *node_rep2;    /* [16][P] */
  const uint16_t *node_batch2; /* [16][P] */
  const uint8_t *node_gpus2;   /* [16][P] */
  const uint8_t *node_w;       /* [16][P] tenths for the first group (1..9 when node_rep2 > 0) */
} cfo_plans;

/* the executor groups of node v of plan p (one or two) */
typedef struct {
  int rep, batch, gpus;
  double share;  /* probability that a request reaching the node goes to this group */
} cfo_group;

static inline int cfo_node_groups(const cfo_plans *pl, int v, int p, cfo_group g[2]) {
  const size_t o = (size_t)v * (size_t)pl->P + (size_t)p;
  const int rep2 = pl->node_rep2 ? pl->node_rep2[o] : 0;
  g[0].rep = pl->node_rep[o];
  g[0].batch = pl->node_batch[o];
  g[0].gpus = pl->node_gpus[o];
  g[0].share = 1.0;
  if (rep2 == 0) return 1;
  const int w = pl->node_w[o];
  g[0].share = (double)w / 10.0;
  g[1].rep = rep2;
  g[1].batch = pl->node_batch2[o];
  g[1].gpus = pl->node_gpus2[o];
  g[1].share = (double)(10 - w) / 10.0;
  return 2;
}

/* The executor of node v (index among its executors, the first group's first) that serves
 * a request with 16-bit replica key `key` for that node: the key space [0, 2^16) is cut at
 * w/10 between the two groups, and a group's part into equal parts for its executors. */
static inline int cfo_node_pick(uint64_t key, const cfo_group *g, int ng, const cfo_plans *pl, int v, int p) {
  if (ng == 1) return (int)((key * (uint64_t)g[0].rep) >> 16);
  const uint64_t w = pl->node_w[(size_t)v * (size_t)pl->P + (size_t)p];
  const uint64_t pos = key * 10u;  /* the key's place in [0, 10 * 2^16) */
  const uint64_t cut = w << 16;
  if (pos < cut) return (int)((pos * (uint64_t)g[0].rep) / cut);
  return g[0].rep + (int)(((pos - cut) * (uint64_t)g[1].rep) / ((10u - w) << 16));
}

/* --- primitives (exposed for the tests that pin them) --- */
void cfo_philox(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
double cfo_log(double x);
double cfo_exp(double x);
double cfo_uniform(uint64_t x);

/* --- hot-path steps --- */
int cfo_trace_gen(const cfo_model *m, const uint64_t *seeds, int32_t n_seeds, int32_t n_req,
                  cfo_trace *tr, uint64_t *moments /* [S][T][8] */);

int cfo_eval_coarse(const cfo_model *m, const cfo_plans *pl, const uint64_t *moments /* [T][8] */,
                    int32_t n_gpus, double *rd, int32_t *bottleneck, uint8_t *flags);

/* phase-1 helpers shared inside the oracle: structural validity of plan p,
 * and the demand u[v][g] of every executor group (seconds of executor time
 * per request). */
int cfo_plan_valid(const cfo_model *m, const cfo_plans *pl, int p);
void cfo_node_demand(const cfo_model *m, const cfo_plans *pl, int p, const uint64_t *moments,
                     double u[CFO_MAXV][2]);

/* Phase 2 (Monte Carlo latency with occupancy-aware scaling) for plans
 * ids[0..n): the first n_sample requests of trace seed seed_idx, routed
 * through each plan without queueing.  met/cnt are [n][T], gt [n][T] the
 * per-type goodput alpha R_d pi_t F_t; lat (optional) [n][n_sample][4] =
 * ttft, tpot, e2e, media of every sampled request. */
int cfo_eval_mc(const cfo_model *m, const cfo_plans *pl, const int32_t *ids, int32_t n,
                const double *rd, const uint64_t *moments, double alpha, const cfo_trace *tr,
                int32_t seed_idx, int32_t n_sample, uint32_t *met, uint32_t *cnt, double *gt,
                double *lat);

/* Latency histogram over a target table targets[T][n_bins][4] (bounds on
 * TTFT, TPOT, E2E, MEDIA): hist[T][n_bins + 1], request r of type type[r]
 * in the first bin whose bounds its latencies lat[r][4] meet, n_bins if
 * none. */
int cfo_latency_hist(const double *lat, const uint8_t *type, int32_t n, int32_t T, int32_t n_bins,
                     const double *targets, uint32_t *hist);

/* Phase 2 with the CDF of the accumulated latencies over a target table
 * (Alg. 2: F_{t,d}): cfo_eval_mc's outputs plus hist [n][T][n_bins + 1] and
 * curve [n][n_bins][T] = ((alpha R_d) pi_t) (requests in bins 0..b / cnt_t). */
int cfo_mc_curve(const cfo_model *m, const cfo_plans *pl, const int32_t *ids, int32_t n, const double *rd,
                 const uint64_t *moments, double alpha, const cfo_trace *tr, int32_t seed_idx, int32_t n_sample,
                 int32_t n_bins, const double *targets, uint32_t *met, uint32_t *cnt, double *gt, uint32_t *hist,
                 double *curve);

/* Pareto pruning: keep[i] = 0 iff some other vector of g[n][T] is >= in
 * every component and > in one. */
int cfo_pareto(const double *g, int32_t n, int32_t T, uint8_t *keep);

/* Plan enumeration (Sec. 4.2, Alg. 1; Eq. 1).  Options: GPU budget N,
 * subplans per logical plan (1 or 2), node sharing between the two
 * subplans, colocatable edges (colocatable[p] bit c: edge p -> c may be
 * merged), per component its batch knobs and GPUs-per-executor options
 * (a node takes those of its lowest component), and het: a node may also
 * hold executors of two of its configurations (Eq. 1's n_{v,k} for two k),
 * with the share of its requests for the first in tenths. */
typedef struct {
  int32_t n_gpus, k_s, share;
  uint32_t colocatable[CFO_MAXC];
  int32_t n_batch[CFO_MAXC];
  uint16_t batch[CFO_MAXC][8];
  int32_t n_gpu_opt[CFO_MAXC];
  uint8_t gpu_opt[CFO_MAXC][4];
  int32_t het;
} cfo_enum_opts;

/* a logical plan: nodes (component masks) and per type one or two
 * alternatives mapping each path component to a node (255 = off the path) */
typedef struct {
  uint8_t n_nodes;
  uint8_t node_comp[CFO_MAXV];
  uint8_t n_alt[CFO_MAXT];
  uint8_t alt_node[CFO_MAXT][2][CFO_MAXC];
} cfo_logical;

int cfo_enum_logical(const cfo_model *m, const cfo_enum_opts *o, cfo_logical *out, int32_t cap,
                     int32_t *n_out);
/* physical plans of one logical plan (UINT64_MAX if that overflows) */
uint64_t cfo_enum_count(const cfo_model *m, const cfo_enum_opts *o, const cfo_logical *L);
/* physical plans first .. first+count-1 of the concatenation over L[0..n),
 * written as plan-table columns 0..count-1 ([slot][count] arrays) */
int cfo_enum_plans(const cfo_model *m, const cfo_enum_opts *o, const cfo_logical *L, int32_t n_logical,
                   uint64_t first, int32_t count, uint8_t *n_nodes, uint8_t *node_comp, uint8_t *node_rep,
                   uint16_t *node_batch, uint8_t *node_gpus, uint8_t *n_alt, uint8_t *alt_w,
                   uint8_t *alt_node, uint8_t *node_rep2, uint16_t *node_batch2, uint8_t *node_gpus2,
                   uint8_t *node_w);

int cfo_select_topk(const double *rd, const uint8_t *flags, int32_t P, int32_t k,
                    int32_t *ids, int32_t *n_selected);

int cfo_rate_grid(const double *rd, const int32_t *ids, int32_t n, int32_t K,
                  double alpha_max, double *rates);

/* One (plan, rate, seed) simulation.  met/cnt are [T]; lat (optional, may be
 * NULL) is [n_req][4] = ttft, tpot, e2e, media; diag (optional) is
 * [4] = integral of number-in-system over time, last completion time,
 * number of instants, total executor busy time. */
int cfo_sim_triple(const cfo_model *m, const cfo_plans *pl, int32_t plan_id, double rate,
                   const cfo_trace *tr, int32_t seed_idx, uint32_t *met, uint32_t *cnt,
                   uint64_t *events, uint32_t *status, double *lat, double *diag);

/* Rate bisection over each plan's grid (seeds pooled, the attainment test
 * of cfo_goodput_reduce; a rate where some seed's simulation fails is
 * infeasible): kstar, goodput_t [n][T], goodput [n], n_eval
 * (rates simulated per plan), events (request-events simulated per plan). */
int cfo_bisect(const cfo_model *m, const cfo_plans *pl, const int32_t *plan_ids, int32_t n_plans,
               const double *rates, int32_t K, const cfo_trace *tr, uint32_t theta_num, uint32_t theta_den,
               int32_t *kstar, double *goodput_t, double *goodput, int32_t *n_eval, uint64_t *events);

/* Goodput at the highest feasible grid rate (Sec. 3.2, Sec. 6.1): met, cnt
 * [n][K][S][T], status [n][K][S]; rate k is feasible iff every seed's
 * simulation ended with status 0 and theta_den M_t >= theta_num N_t for
 * every type with N_t > 0 (counts pooled over seeds). */
int cfo_goodput_reduce(const uint32_t *met, const uint32_t *cnt, const uint32_t *status, int32_t n_plans, int32_t K,
                       int32_t S, int32_t T, const double *rates, uint32_t theta_num,
                       uint32_t theta_den, int32_t n_req, int32_t *kstar, double *goodput_t,
                       double *goodput);

int32_t cfo_argmax(const double *goodput, int32_t n);

/* element-wise helpers for the tests: op 0 log, 1 exp, 2 sqrt, 3 x/y, 4 uniform(bits of x) */
void cfo_math_n(int32_t op, const double *x, const double *y, double *out, int64_t n);
void cfo_philox_n(const uint64_t *ctr, const uint64_t *key, uint64_t *out, int64_t n);

#endif
