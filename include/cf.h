/*
 * cf.h -- C ABI of libcf, the MI355X (gfx950) implementation of the
 * statistical plan evaluation of Cornfigurator (arXiv 2512.14098):
 * request traces, flow-based screening (Sec. 4.3, Alg. 2 phase 1),
 * request-level simulation (Alg. 2 phase 3) and goodput selection
 * (Sec. 3.2, Sec. 6.1).
 *
 * Conventions
 *  - Pointers named *_dev are device pointers (HIP global memory), owned and
 *    allocated by the caller; the library never frees them.  Pointers named
 *    *_host, and every descriptor struct, live in host memory and are read
 *    during the call only.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the
 *    default stream) unless its comment says it synchronises.
 *  - Errors detectable on the host (bad descriptor, sizes, capacity limits)
 *    are returned before anything is launched; nothing is written then.
 *    Conditions found on the device are reported in per-triple status words
 *    and never trap.  cf_last_error() returns the text of the calling
 *    thread's last error.
 *  - Layouts are structure-of-arrays; every multi-dimensional array is
 *    row-major with the last index fastest.
 *  - The library allocates internal scratch (per-wave simulation state) on
 *    first use and keeps it for later calls; cf_release_scratch() frees it.
 *    Scratch is per device and shared by every call on that device: calls
 *    that overlap in time on one device (from other streams or host threads)
 *    race on it and must be serialised by the caller.  Growing a scratch
 *    region synchronises the device.
 */
#ifndef CF_H
#define CF_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cf_status;
#define CF_OK 0
#define CF_EINVAL (-1)        /* invalid descriptor or argument */
#define CF_ENOMEM (-2)        /* device allocation of scratch failed */
#define CF_EHIP (-3)          /* HIP runtime error */
#define CF_ECAPACITY (-4)     /* static limit exceeded (see CF_MAX_*) */
#define CF_EUNSUPPORTED (-6)  /* feature combination not supported */

#define CF_MAX_COMP 8     /* model components */
#define CF_MAX_TYPES 8    /* request types */
#define CF_MAX_NODES 16   /* nodes per plan */
#define CF_MAX_EXEC 64    /* executors (replicas) per plan */
#define CF_MAX_BATCH 256  /* max batch of a node */

/* component kinds */
#define CF_ENC 0
#define CF_LLM 1
#define CF_GEN 2

/* per-request attributes, used as bit positions of cf_model_desc.x_sel and
 * as values of cf_model_desc.nout_attr */
#define CF_ATTR_PROMPT 0
#define CF_ATTR_OUT 1
#define CF_ATTR_PATCHES 2
#define CF_ATTR_AUDIN_MS 3
#define CF_ATTR_AUDOUT_MS 4
#define CF_ATTR_AUDIN_TOK 5  /* ceil(aud_in_ms / 80) */
#define CF_ATTR_AUDOUT_TOK 6 /* ceil(aud_out_ms / 80) */

/* length distributions */
#define CF_DIST_NONE 0
#define CF_DIST_CONST 1     /* value p0 */
#define CF_DIST_LOGNORMAL 2 /* clamp(rint(scale * exp(p0 + p1 Z)), lo, hi) */
#define CF_DIST_EXP 3       /* clamp(rint(p0 * Exp(1)), lo, hi) */

/* image-count distributions */
#define CF_IMG_NONE 0
#define CF_IMG_CONST 1
#define CF_IMG_UNIFORM 2

/* cf_eval_coarse flag bits */
#define CF_FLAG_KEEP 1u
#define CF_FLAG_OVER_BUDGET 2u
#define CF_FLAG_INVALID 4u
#define CF_FLAG_REDUNDANT 8u

/* cf_eval_fine flags (request-level simulation, Alg. 2 phase 3) */
#define CF_FULL 0u        /* every triple is simulated until its last request completes */
#define CF_DUMP_LAT 1u    /* also write per-request latencies of the listed triples (cf_fine_out.lat_dev) */
#define CF_EARLY_EXIT 2u  /* stop a (plan, rate) once its attainment is certainly below theta: not built */

/* cf_eval_fine per-triple status bits */
#define CF_ST_INVALID 1u   /* a request's route does not fit the plan */
#define CF_ST_DEADLOCK 2u  /* nothing pending but requests unfinished */
#define CF_ST_OVERFLOW 4u  /* an internal capacity of the simulator was exceeded */

typedef struct cf_dist {
  int32_t kind;        /* CF_DIST_* */
  int32_t reserved;
  double p0, p1;       /* parameters (see CF_DIST_*) */
  double scale;        /* LOGNORMAL: multiplier before rounding (1 tokens, 1000 ms) */
  int64_t lo, hi;      /* clamp after rounding */
} cf_dist;

/* Model definition, configuration space and workload (Sec. 3.1): the
 * component graph with one latency model per component, request types with
 * their weight (pi_t proportional to weight), path, outputs, lengths and
 * latency targets.  Host memory, copied by every call that takes it. */
typedef struct cf_model_desc {
  int32_t n_comp;                    /* 1..CF_MAX_COMP, topological index order */
  int32_t n_types;                   /* 1..CF_MAX_TYPES */
  int32_t kind[CF_MAX_COMP];         /* CF_ENC / CF_LLM / CF_GEN */
  double k0[CF_MAX_COMP];            /* batch iteration: (k0 + k1*X) + k2*n seconds */
  double k1[CF_MAX_COMP];
  double k2[CF_MAX_COMP];
  double d0[CF_MAX_COMP];            /* LLM decode step: d0 + d1*n seconds */
  double d1[CF_MAX_COMP];
  uint32_t x_sel[CF_MAX_COMP];       /* bitmask of CF_ATTR_* summed into X */
  int32_t nout_attr[CF_MAX_COMP];    /* LLM: CF_ATTR_* giving the output length */
  int32_t gate_src[CF_MAX_COMP];     /* LLM gated by that component's tokens, or -1 */
  int32_t batch_cap[CF_MAX_COMP];    /* stage batch = min(node batch, cap) */
  double comm_s;                     /* delay of every inter-executor edge (Sec. 5.2) */
  double cpu_pre_s;                  /* CPU preprocessing of an idle-start encoder batch */
  uint32_t weight[CF_MAX_TYPES];     /* type weights (>= 0, sum >= 1) */
  uint32_t path_mask[CF_MAX_TYPES];  /* components on the type's path */
  uint32_t out_mask[CF_MAX_TYPES];   /* output components of the type */
  uint32_t prefill_only[CF_MAX_TYPES]; /* LLM components with one output token */
  uint32_t parents[CF_MAX_TYPES][CF_MAX_COMP]; /* parent mask of each component on the path */
  int32_t img_kind[CF_MAX_TYPES];    /* CF_IMG_* */
  int32_t img_lo[CF_MAX_TYPES], img_hi[CF_MAX_TYPES]; /* images per request (<= 4) */
  int32_t patch_lo, patch_hi;        /* patches per image, uniform integer */
  cf_dist len[CF_MAX_TYPES][4];      /* prompt, out, aud_in_ms, aud_out_ms */
  double slo[CF_MAX_TYPES][4];       /* bounds on TTFT, TPOT, E2E, MEDIA (<=; +inf = none) */
  uint32_t theta_num, theta_den;     /* attainment threshold (e.g. 9/10) */
  /* Latency multiplier of component c on executors of g GPUs (the tensor
   * parallelism degree of the configuration space): every iteration time
   * of c (batch, prefill, decode step) on such an executor is
   * tp_scale[c][min(g, 8) - 1] times its latency model, the product
   * rounded once; CPU preprocessing is not scaled.  0 means 1. */
  double tp_scale[CF_MAX_COMP][8];
} cf_model_desc;

/* Request trace: device arrays of n_seeds * n_req elements, seed-major. */
typedef struct cf_trace {
  int32_t n_seeds, n_req;
  uint64_t *arr_ticks_dev;  /* inclusive prefix sum of gaps, 2^-32 s at rate 1 */
  uint8_t *type_dev;
  uint8_t *n_img_dev;
  uint16_t *patches_dev;    /* sum over the request's images */
  uint16_t *prompt_dev;
  uint16_t *out_dev;
  uint32_t *aud_in_ms_dev;
  uint32_t *aud_out_ms_dev;
  uint64_t *rkey0_dev;      /* 16-bit replica keys of components 0..3 */
  uint64_t *rkey1_dev;      /* 16-bit replica keys of components 4..7 */
  uint32_t *akey_dev;       /* alternative-choice key */
} cf_trace;

/* Physical plans (Sec. 4.2): device arrays, field-slot major [slot][P]. */
typedef struct cf_plan_table {
  int32_t P;
  const uint8_t *n_nodes_dev;    /* [P] */
  const uint8_t *node_comp_dev;  /* [16][P] component bitmask */
  const uint8_t *node_rep_dev;   /* [16][P] executors of the node */
  const uint16_t *node_batch_dev;/* [16][P] max batch */
  const uint8_t *node_gpus_dev;  /* [16][P] GPUs per executor */
  const uint8_t *n_alt_dev;      /* [8][P] alternatives per type (1 or 2) */
  const uint8_t *alt_w_dev;      /* [16][P] slot 2t+a: routing weight in tenths */
  const uint8_t *alt_node_dev;   /* [128][P] slot (2t+a)*8+c: node serving c */
  /* Optional second executor configuration of each node (Eq. (1): n_{v,k} executors of
   * each configuration k of a node): node_rep2 more executors (0: none) of max batch
   * node_batch2 and node_gpus2 GPUs, and node_w, the tenths of the node's requests that go
   * to the first configuration (1..9 where node_rep2 > 0; routing between the executors
   * of a node in steps of 0.1, Sec. 4.2).  A request's replica key for the node (16 bits)
   * picks the executor: keys below node_w * 2^16 / 10 go to the first configuration, the
   * others to the second, each part cut into equal parts for that configuration's
   * executors, numbered after the first's.  All four NULL: one configuration per node. */
  const uint8_t *node_rep2_dev;   /* [16][P] */
  const uint16_t *node_batch2_dev;/* [16][P] */
  const uint8_t *node_gpus2_dev;  /* [16][P] */
  const uint8_t *node_w_dev;      /* [16][P] */
} cf_plan_table;

/* Outputs of cf_eval_fine, device arrays, triple (i, k, s) = plan i, rate k,
 * seed s. */
typedef struct cf_fine_out {
  uint32_t *met_dev;      /* [n_plans][K][S][T] requests meeting every bound */
  uint32_t *cnt_dev;      /* [n_plans][K][S][T] requests of the type */
  uint64_t *events_dev;   /* [n_plans][K][S] request-events simulated */
  uint32_t *status_dev;   /* [n_plans][K][S] CF_ST_* bits */
  double *lat_dev;        /* optional [n_lat][n_req][4]: TTFT, TPOT, E2E, MEDIA; NULL = off */
  const int32_t *lat_triples_dev; /* [n_lat] linear triple ids ((i*K)+k)*S+s to dump */
  int32_t n_lat;
  /* Optional latency histograms (goodput against a range of latency
   * targets, Sec. 6.2 and Appendix B): with n_bins > 0, a completed request of type
   * t counts in bin b = the first bin whose four bounds
   * hist_targets_host[t][b][0..3] (TTFT, TPOT, E2E, MEDIA, inclusive) it
   * meets, or n_bins if none; the bounds must not decrease with b (1 <=
   * n_bins <= 64).  hist_dev: [n_plans][K][S][T][n_bins + 1] (device). */
  uint32_t *hist_dev;
  const double *hist_targets_host;
  int32_t n_bins;
  /* Capacity limits for tests (0 = the capacity the library sizes): every
   * simulation of the call may hold at most lim_chunks queue chunks of 64
   * entries, lim_delay entries in its delay line (a power of two, >= 2) and
   * take at most lim_instants instants.  A simulation that needs more stops
   * and reports CF_ST_OVERFLOW (chunks, delay line) or CF_ST_DEADLOCK
   * (instants) in its status word; the kernel exits normally.  Limits above
   * the library's own capacity are clamped to it.  Lets tests force the
   * failure statuses from the host. */
  int32_t lim_chunks, lim_delay;
  uint64_t lim_instants;
} cf_fine_out;

/* Error text of the calling thread's last failed call (empty if none);
 * writes at most n bytes including the terminator, returns the full length. */
size_t cf_last_error(char *buf, size_t n);
const char *cf_status_str(cf_status s);
const char *cf_version(void);

/* Synthetic Any-to-Any trace (workload of Sec. 3.1, Poisson arrivals).
 * For seed seeds_host[s] and request i: Philox4x64-10 blocks keyed
 * (seeds_host[s], 0) with counter (i, field, attempt, 0) give the gap, type,
 * image count, patches, lengths and route keys.  moments_dev receives
 * [n_seeds][n_types][8] u64: count, then sums of prompt, out, patches,
 * aud_in_ms, aud_out_ms, aud_in tokens, aud_out tokens.
 * Errors: CF_EINVAL for a bad descriptor, n_seeds < 1 or n_req < 0. */
cf_status cf_trace_gen(const cf_model_desc *model, const uint64_t *seeds_host, int32_t n_seeds,
                       int32_t n_req, const cf_trace *out, uint64_t *moments_dev, void *stream);

/* Phase 1 of the plan evaluation (Sec. 4.3, Alg. 2): per plan, the
 * per-node demand u_v from the latency models at the node's batch and the
 * per-type means in moments_dev ([n_types][8], one seed), R_d = min_v
 * m_v/u_v, the bottleneck node (-1 if invalid) and CF_FLAG_* bits (budget of
 * Eq. (1) is n_gpus).  Output arrays have P elements. */
cf_status cf_eval_coarse(const cf_model_desc *model, const cf_plan_table *plans,
                         const uint64_t *moments_dev, int32_t n_gpus, double *rd_dev,
                         int32_t *bottleneck_dev, uint8_t *flags_dev, void *stream);

/* The candidates phase 1 passes on (Alg. 2: plans not pruned as redundant
 * or over budget, i.e. with CF_FLAG_KEEP, ranked by their flow-based
 * throughput R_d; the top K go to the finer phases): plans with CF_FLAG_KEEP
 * ordered by R_d descending, ties by plan id ascending; the first min(k,
 * kept) ids go to ids_dev[k] (device).  rd_dev, flags_dev: cf_eval_coarse's
 * outputs, P elements each (device).  Synchronises the stream and writes the
 * number selected to *n_selected_host.
 * Limits: 1 <= k <= 65536, P <= 2^24.  Errors: CF_EINVAL (NULL arrays,
 * sizes), CF_ECAPACITY (k or P above the limits). */
cf_status cf_select_topk(const double *rd_dev, const uint8_t *flags_dev, int32_t P, int32_t k,
                         int32_t *ids_dev, int32_t *n_selected_host, void *stream);

/* Running top-k over a plan space screened window by window (Alg. 2 phase 1
 * keeps the plans with the largest R_d; cf_enum_screen screens one window of
 * an enumerated space at a time).  Running list: rd_run_dev[n_run] and plan
 * numbers gid_run_dev[n_run], in the order of cf_select_topk (R_d descending,
 * ties by plan number ascending; R_d compared by its bits, as there).
 * Window: ids_win_dev[n_win], the ids cf_select_topk returned for the
 * window's rd_win_dev, plan number win_first + id.  Writes the first
 * min(k, n_run + n_win) plans of the merged order to rd_out_dev[k] and
 * gid_out_dev[k], which must not alias the running list.  The two lists
 * must hold distinct plan numbers (windows that do not overlap).
 * Asynchronous on stream.  Limits: 1 <= k <= 65536, 0 <= n_run, n_win <= 65536.
 * Errors: CF_ECAPACITY (k), CF_EINVAL (sizes, NULL pointers, aliasing). */
cf_status cf_topk_merge(const double *rd_run_dev, const uint64_t *gid_run_dev, int32_t n_run,
                        const double *rd_win_dev, const int32_t *ids_win_dev, int32_t n_win, uint64_t win_first,
                        int32_t k, double *rd_out_dev, uint64_t *gid_out_dev, void *stream);

/* Arrival-rate grid of phase 3: R_d is an ideal upper bound, so the planner
 * simulates a plan at alpha R_d with headroom alpha <= 1 (Sec. 4.3, Alg. 2
 * phase 3; alpha in 0.5..0.8 in Table 5); here K rates up to alpha_max R_d:
 * rates_dev[i][k] = ((R_d[ids_dev[i]] * alpha_max) * (k+1)) / K, i < n, k < K
 * (device arrays; rd_dev indexed by plan id).  alpha_max > 0, 1 <= K.
 * Asynchronous on stream.  Errors: CF_EINVAL (NULL arrays, sizes, alpha). */
cf_status cf_rate_grid(const double *rd_dev, const int32_t *ids_dev, int32_t n, int32_t K,
                       double alpha_max, double *rates_dev, void *stream);

/* Phase 3 (Sec. 4.3, Alg. 2): request-level simulation of every triple
 * (plan plan_ids_dev[i], rate rates_dev[i][k], trace seed s) for i <
 * n_plans, k < K, s < trace->n_seeds, one wavefront per triple.  Outputs in
 * *out (device arrays, caller-owned).  flags: CF_FULL, or CF_DUMP_LAT to
 * also write out->lat_dev for the out->n_lat triples listed in
 * out->lat_triples_dev (both required with the flag, ignored without it);
 * CF_EARLY_EXIT is not built and returns CF_EUNSUPPORTED.  Every array of
 * *trace but n_img_dev is read (a request's lengths are copied beside its
 * record when it arrives).  Synchronises the stream (the argument block is
 * copied from host memory).
 * Errors: CF_EINVAL (descriptor, sizes, flags, NULL trace arrays),
 * CF_ECAPACITY, CF_ENOMEM, CF_EUNSUPPORTED. */
cf_status cf_eval_fine(const cf_model_desc *model, const cf_plan_table *plans,
                       const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev,
                       int32_t K, const cf_trace *trace, uint32_t flags, const cf_fine_out *out,
                       void *stream);

/* cf_eval_fine for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, checks, outputs and status words, bit for bit, but
 * the per-wavefront simulation state lives in one fixed array of 64 MiB
 * per device (held from the library's load on that device until the
 * process ends) instead of the library's cached allocations, and no
 * hipMalloc, hipFree or allocating library routine is called.  The array
 * bounds the number of wavefronts (64 MiB, less the launch's (plan, rate)
 * order of 4 bytes per pair, over the state of one simulation, about
 * 0.9 MiB at 3,000 requests); a call whose single simulation does not fit
 * (about 60,000 requests and more) returns CF_ECAPACITY before any launch.  Every call on a device shares that device's array and leaves its
 * contents behind (the call clears what must start at zero itself): calls
 * that overlap in time on one device race and must be serialised by the
 * caller.  Synchronises the stream, as cf_eval_fine does.
 * Errors: those of cf_eval_fine; CF_ECAPACITY as above; CF_EHIP if the
 * array's device address cannot be obtained. */
cf_status cf_eval_fine_noalloc(const cf_model_desc *model, const cf_plan_table *plans,
                               const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev,
                               int32_t K, const cf_trace *trace, uint32_t flags, const cf_fine_out *out,
                               void *stream);

/* Phase 2 (Sec. 4.3, Alg. 2 phase 2) with occupancy-aware latency scaling
 * (Sec. 5.2): plan plan_ids_dev[i], i < n_plans, is evaluated on the first
 * n_sample requests of trace seed seed_idx, each routed through the plan
 * alone (no queueing).  Every component a request visits costs one
 * iteration at its effective batch b = clamp(ceil(B * (R_d / R_v)), 1, B)
 * (B = min(node batch, cap), R_v = m_v / u_v the node's phase-1 capacity):
 * an encoder or generator a static batch of b such requests, an LLM the
 * request's own prefill then decode steps d0 + d1 b; a component starts
 * when its last input arrives (comm later across executors; a gated LLM
 * after its gate source's first token, each further token after the gate
 * source's matching token).
 * rd_dev: phase 1's R_d indexed by plan id ([P]); moments_dev: the [T][8]
 * moments phase 1 used; alpha in (0, 1].  Outputs (device, caller-owned):
 * met_dev, cnt_dev [n_plans][T] (sampled requests of each type meeting every
 * target / in all), goodput_t_dev [n_plans][T] = (alpha R_d) pi_t met/cnt
 * (0 when cnt = 0), lat_dev optional [n_plans][n_sample][4] = TTFT, TPOT,
 * E2E, MEDIA of every sampled request (NULL = off).  An invalid plan gets
 * zeros.  Asynchronous on stream.
 * Errors: CF_EINVAL (descriptor, sizes, seed_idx or n_sample outside the
 * trace, alpha). */
cf_status cf_eval_mc(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev,
                     int32_t n_plans, const double *rd_dev, const uint64_t *moments_dev, double alpha,
                     const cf_trace *trace, int32_t seed_idx, int32_t n_sample, uint32_t *met_dev,
                     uint32_t *cnt_dev, double *goodput_t_dev, double *lat_dev, void *stream);

/* Phase 2 with its latency CDFs (Alg. 2: F_{t,d} is the CDF of the
 * accumulated latencies; G_{t,d} = alpha R_d pi_t F_{t,d}(L_t)) evaluated
 * over a table of targets: everything cf_eval_mc computes, plus hist_dev
 * [n_plans][T][n_bins + 1] (a sampled request of type t in the first bin b
 * whose bounds hist_targets_host[t][b][0..3] it meets, n_bins if none; the
 * bounds must not decrease with b; 1 <= n_bins <= 64) and curve_dev
 * [n_plans][n_bins][T] = ((alpha R_d) pi_t) (H_t(b) / cnt_t), H_t(b) the
 * requests in bins 0..b (0 if cnt_t = 0 or the plan is invalid).
 * Errors: those of cf_eval_mc, CF_EINVAL for the target table. */
cf_status cf_eval_mc_curve(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev,
                           int32_t n_plans, const double *rd_dev, const uint64_t *moments_dev, double alpha,
                           const cf_trace *trace, int32_t seed_idx, int32_t n_sample, int32_t n_bins,
                           const double *hist_targets_host, uint32_t *met_dev, uint32_t *cnt_dev,
                           double *goodput_t_dev, uint32_t *hist_dev, double *curve_dev, void *stream);

/* Pareto pruning (Alg. 2, after phases 2 and 3): keep_dev[i] = 0 iff some
 * other row of goodput_t_dev [n][T] (device) is >= in every component and >
 * in at least one, else 1.  1 <= T <= 8.  Rows given in decreasing R_d
 * order (as cf_select_topk returns them) are the fast case.
 * Optionally (plan_ids_dev and flags_dev both non-NULL, both device): row i
 * is plan plan_ids_dev[i], and a dominated row clears CF_FLAG_KEEP in
 * flags_dev[plan] (flags_dev has n_flags entries; ids outside [0, n_flags)
 * are left alone), so that cf_select_topk then returns the survivors.
 * Plan ids must be distinct.  Asynchronous on stream.
 * Errors: CF_EINVAL (sizes, NULL arrays, only one of plan_ids_dev/flags_dev). */
cf_status cf_pareto(const double *goodput_t_dev, int32_t n, int32_t T, uint8_t *keep_dev,
                    const int32_t *plan_ids_dev, uint8_t *flags_dev, int32_t n_flags, void *stream);

/* ------------------------------------------------------------------ plan enumeration
 * Plan enumeration (Sec. 4.2, Alg. 1) and the executor partitions of
 * Eq. (1).  Options: GPU budget N (1..64), subplans per logical plan k_s (1
 * or 2), node sharing between the two subplans (compound subplans), the
 * colocatable edges (bit c of colocatable[p]: the edge p -> c may be
 * merged), and per component its batch knobs (1..8 values in 1..256) and
 * GPUs-per-executor options (1..4 values in 1..N); a node takes the options
 * of its lowest component. */
typedef struct cf_enum_opts {
  int32_t n_gpus;
  int32_t k_s;
  int32_t share;
  uint32_t colocatable[CF_MAX_COMP];
  int32_t n_batch[CF_MAX_COMP];
  uint16_t batch[CF_MAX_COMP][8];
  int32_t n_gpu_opt[CF_MAX_COMP];
  uint8_t gpu_opt[CF_MAX_COMP][4];
  /* 1: a node may also hold executors of two of its configurations (Eq. 1's
   * n_{v,k} for two k), with 1..9 tenths of its requests for the first (the
   * plan table's second-configuration arrays); 0: one configuration per node */
  int32_t het;
} cf_enum_opts;

/* A logical plan (Alg. 1): nodes as component masks, and per type one or
 * two alternative paths mapping each component of the type's path to a
 * node (255 off the path).  153 bytes, no padding. */
typedef struct cf_logical {
  uint8_t n_nodes;
  uint8_t node_comp[CF_MAX_NODES];
  uint8_t n_alt[CF_MAX_TYPES];
  uint8_t alt_node[CF_MAX_TYPES][2][CF_MAX_COMP];
} cf_logical;

/* Logical plans (host only, no device work), in this order: subgraphs are
 * the distinct unions of type paths, ascending as bitmasks, each covering
 * the types whose paths it contains; the simple subplans of a subgraph come
 * from the Keep/Merge vectors m = 0 .. 2^k - 1 over its covered types'
 * colocatable edges in ascending (parent, child) order (bit i merges edge
 * i), nodes = connected groups in ascending mask order, a repeated grouping
 * skipped.  Logical plans: each simple subplan covering every type alone;
 * then, if k_s = 2, each pair i <= j covering every type together, once per
 * set of shared nodes (a node of j equal to a node of i; subsets in
 * ascending bitmask order; none without sharing; never all of j's nodes);
 * nodes = i's, then j's unshared; a type covered by both gets two
 * alternatives (i's first) unless they map its path to the same nodes.
 * Plans over 16 nodes and exact repeats are dropped.  Writes up to cap
 * plans to out_host and their number to *n_out.
 * Errors: CF_EINVAL (descriptor, options), CF_ECAPACITY (more than cap
 * plans, or over 16 colocatable edges in one subgraph). */
cf_status cf_enum_logical(const cf_model_desc *model, const cf_enum_opts *opts, cf_logical *out_host,
                          int32_t cap, int32_t *n_out);

/* Physical plans per logical plan (Eq. 1): node v takes a configuration k
 * (GPU option major, batch knob minor) and n_v >= 1 executors with
 * sum_v gpus_v n_v <= N; each type with two alternatives takes a weight w in
 * 1..9 tenths for its first (10 - w for the second).  With opts->het a node
 * may instead take two configurations k1 < k2 with n1, n2 >= 1 executors and
 * 1..9 tenths w of its requests for k1; a node's assignments are ordered
 * (k, n) first, then (k1, k2, n1, n2, w), each lexicographically.  The plans
 * of logical plan l are numbered offsets[l] .. offsets[l+1]-1: executor
 * assignments lexicographically over the nodes in that per-node order,
 * routing weights lexicographically inside each (lowest type most
 * significant).
 * logical_dev: n_logical plans in device memory; writes offsets_dev[n_logical
 * + 1] (device) and the total to *total_host (synchronises the stream).
 * Errors: CF_EINVAL, CF_ECAPACITY (the total does not fit 64 bits). */
cf_status cf_enum_count(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                        int32_t n_logical, uint64_t *offsets_dev, uint64_t *total_host, void *stream);

/* Physical plans first .. first+count-1 (numbered as cf_enum_count numbers
 * them; offsets_dev and total from it, with the same options and logical
 * plans) into columns 0..count-1 of the device plan table *out (out->P >=
 * count; its arrays are written, unused node slots 0, unused route entries
 * 255; the second-configuration arrays, required with opts->het, are written
 * when present: 0 executors and 10 tenths for a node of one configuration).
 * One thread per plan, asynchronous on stream.
 * Errors: CF_EINVAL (options, sizes, first + count > total, het without the
 * second-configuration arrays). */
cf_status cf_enum_plans(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                        int32_t n_logical, const uint64_t *offsets_dev, uint64_t total, uint64_t first,
                        int32_t count, const cf_plan_table *out, void *stream);

/* Goodput (Sec. 3.2) at the highest feasible rate (Sec. 6.1) from the
 * outputs of cf_eval_fine: fine->met_dev, cnt_dev [n_plans][K][S][T] and
 * status_dev [n_plans][K][S] (device; the other fields are not read).
 * M_t, N_t pooled over seeds; rate k is feasible iff every seed's
 * simulation ended with status 0 and theta_den*M_t >= theta_num*N_t for
 * every type with N_t > 0; kstar = first infeasible - 1; goodput_t =
 * (rates[i][kstar] * M_t) / (S * n_req) (0 if kstar < 0); goodput = sum_t.
 * Outputs: kstar_dev[n_plans], goodput_t_dev[n_plans][T], goodput_dev[n_plans].
 * Asynchronous on stream.  Limits: K <= 64.  Errors: CF_EINVAL (NULL
 * arrays, sizes, theta_den = 0), CF_ECAPACITY (K). */
cf_status cf_goodput_reduce(const cf_fine_out *fine, int32_t n_plans, int32_t K, int32_t S, int32_t T,
                            const double *rates_dev, uint32_t theta_num, uint32_t theta_den, int32_t n_req,
                            int32_t *kstar_dev, double *goodput_t_dev, double *goodput_dev, void *stream);

/* Enumeration fused with phase 1 (one configuration per node: opts->het
 * returns CF_EUNSUPPORTED; cf_enum_plans then cf_eval_coarse screen such
 * plans): for physical plans first .. first+count-1
 * (numbered as cf_enum_plans numbers them), exactly what cf_eval_coarse
 * writes for those plans' table columns -- rd_dev[count], bottleneck_dev
 * [count], flags_dev[count] (device) -- without writing the plan table.
 * moments_dev: the [T][8] per-type moments of one trace seed; n_gpus: the
 * budget for the over-budget flag.  Asynchronous on stream.
 * Errors: those of cf_enum_plans and cf_eval_coarse. */
cf_status cf_enum_screen(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                         int32_t n_logical, const uint64_t *offsets_dev, uint64_t total, uint64_t first,
                         int32_t count, const uint64_t *moments_dev, int32_t n_gpus, double *rd_dev,
                         int32_t *bottleneck_dev, uint8_t *flags_dev, void *stream);

/* Phase 3 with rate bisection (the workload descriptions bisect rates over
 * a grid; Alg. 2 phase 3 simulates each plan at its rate): for plan
 * plan_ids_dev[i] and its grid rates_dev[i][0..K), lo = -1 and hi = K;
 * each round simulates every seed of the trace at mid = (lo + hi) / 2 for
 * every plan with hi > lo + 1, and moves lo to mid if the pooled counts
 * pass the attainment test of cf_goodput_reduce (theta), else hi.  At the
 * end kstar = lo, goodput_t = (rates[lo] M_t) / (S n_req) with M_t the
 * pooled met counts of the round at lo (0 if lo < 0), goodput = sum_t.  On
 * a monotone feasibility this is cf_goodput_reduce's result with
 * ceil(log2(K + 1)) rates simulated instead of K.
 * Outputs (device): kstar_dev[n], goodput_t_dev[n][T], goodput_dev[n],
 * n_eval_dev[n] (rates simulated), events_dev[n] (request-events simulated),
 * status_dev[n] (CF_ST_* bits OR-ed over the plan's simulations).
 * Synchronises the stream once per round.  Limits: K <= 64.
 * Errors: those of cf_eval_fine; CF_EINVAL (sizes, theta). */
cf_status cf_eval_bisect(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev,
                         int32_t n_plans, const double *rates_dev, int32_t K, const cf_trace *trace,
                         uint32_t theta_num, uint32_t theta_den, int32_t *kstar_dev, double *goodput_t_dev,
                         double *goodput_dev, int32_t *n_eval_dev, uint64_t *events_dev, uint32_t *status_dev,
                         void *stream);

/* Goodput against a range of latency targets (Sec. 6.2 and Appendix B, per-type goodput
 * vs. latency target): for every plan and bin b, cf_goodput_reduce's
 * computation with M_t = the requests in bins 0..b of fine->hist_dev (the
 * cf_eval_fine histogram [n_plans][K][S][T][fine->n_bins + 1]), N_t from
 * fine->cnt_dev and the status words fine->status_dev.  Outputs:
 * kstar_dev[n_plans][n_bins], goodput_t_dev[n_plans][n_bins][T],
 * goodput_dev[n_plans][n_bins].  Limits: K <= 64, 1 <= n_bins <= 64. */
cf_status cf_goodput_curve(const cf_fine_out *fine, int32_t n_plans, int32_t K, int32_t S, int32_t T,
                           const double *rates_dev, uint32_t theta_num, uint32_t theta_den, int32_t n_req,
                           int32_t *kstar_dev, double *goodput_t_dev, double *goodput_dev, void *stream);

/* Selection (Alg. 2, last step): index of the largest goodput, ties to the
 * lowest index, written to best_dev[0]. */
cf_status cf_select_best(const double *goodput_dev, int32_t n, int32_t *best_dev, void *stream);

/* Diagnostics for tests: the device primitives applied element-wise.
 * op 0: cf_log(x)  1: cf_exp(x)  2: sqrt(x)  3: x / y  4: uniform(bits of x)
 * y_dev is only read by op 3; out_dev[n]. */
cf_status cf_math_eval(int32_t op, const double *x_dev, const double *y_dev, double *out_dev,
                       int64_t n, void *stream);
/* Philox4x64-10 blocks: ctr_dev[n][4], key_dev[n][2] -> out_dev[n][4]. */
cf_status cf_philox_eval(const uint64_t *ctr_dev, const uint64_t *key_dev, uint64_t *out_dev,
                         int64_t n, void *stream);

/* Frees the internal scratch (synchronises the device). */
cf_status cf_release_scratch(void);

#ifdef __cplusplus
}
#endif
#endif
