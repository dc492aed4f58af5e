// k_enum.hip -- cf_enum_logical, cf_enum_count, cf_enum_plans: plan
// enumeration (Sec. 4.2, Alg. 1) and the executor partitions of Eq. (1).
//
// Logical plans are few (hundreds to thousands) and are built on the host.
// Physical plans are many (a logical plan of five nodes on 64 GPUs has
// billions), so they are numbered and produced on the device by unranking:
//   - per logical plan, a table cnt[v][b] = number of executor assignments
//     of nodes v.. within b GPUs (one block per logical plan, the budgets
//     across threads, the nodes from the last to the first);
//   - offsets = exclusive prefix sum of cnt[0][N] * 9^(types with two
//     alternatives);
//   - four consecutive plan indices per thread: for each, the logical plan by
//     binary search in the offsets, the routing weights as base-9 digits of
//     the index within it, the executor assignment by walking the table (at
//     node v with budget b, the candidates (k, n) in order each own
//     cnt[v+1][b - gpus_k n] consecutive numbers); the plan-table columns
//     are written slot-major, four plans per 32-bit store, so a wavefront
//     fills 256 consecutive bytes of a slot row per store instruction.
#include "cf_internal.h"
#include "cf_phase1.h"

#include <algorithm>
#include <cstring>
#include <map>
#include <set>
#include <string>
#include <vector>

namespace cf {
namespace {

constexpr int kEnumMaxN = 64;                       // GPU budget limit (executors per plan)
constexpr int kTabStride = kEnumMaxN + 1;           // budgets 0..N
constexpr int kTabSize = (CF_MAX_NODES + 1) * kTabStride;  // u64 entries per logical plan

cf_status check_opts(const cf_model_desc *d, const cf_enum_opts *o) {
  if (!d || !o) return set_error(CF_EINVAL, "NULL argument");
  if (d->n_comp < 1 || d->n_comp > CF_MAX_COMP || d->n_types < 1 || d->n_types > CF_MAX_TYPES)
    return set_error(CF_EINVAL, "model sizes");
  if (o->n_gpus < 1 || o->n_gpus > kEnumMaxN) return set_error(CF_EINVAL, "n_gpus must be in 1..%d", kEnumMaxN);
  if (o->k_s < 1 || o->k_s > 2) return set_error(CF_EINVAL, "k_s must be 1 or 2");
  if (o->het != 0 && o->het != 1) return set_error(CF_EINVAL, "het must be 0 or 1");
  for (int c = 0; c < d->n_comp; c++) {
    if (o->n_batch[c] < 1 || o->n_batch[c] > 8) return set_error(CF_EINVAL, "n_batch[%d]", c);
    for (int k = 0; k < o->n_batch[c]; k++)
      if (o->batch[c][k] < 1 || o->batch[c][k] > CF_MAX_BATCH) return set_error(CF_EINVAL, "batch[%d][%d]", c, k);
    if (o->n_gpu_opt[c] < 1 || o->n_gpu_opt[c] > 4) return set_error(CF_EINVAL, "n_gpu_opt[%d]", c);
    for (int k = 0; k < o->n_gpu_opt[c]; k++)
      if (o->gpu_opt[c][k] < 1 || o->gpu_opt[c][k] > o->n_gpus) return set_error(CF_EINVAL, "gpu_opt[%d][%d]", c, k);
  }
  return CF_OK;
}

// ------------------------------------------------------------------ host: logical plans
struct Subplan {
  uint32_t cs, cov;
  std::vector<uint8_t> nodes;  // ascending masks
  int node_of(int c) const {
    for (size_t k = 0; k < nodes.size(); k++)
      if ((nodes[k] >> c) & 1u) return (int)k;
    return -1;
  }
};

int uf_find(int *par, int x) {
  while (par[x] != x) {
    par[x] = par[par[x]];
    x = par[x];
  }
  return x;
}

std::string plan_key(const cf_logical &L, int T) {
  std::string k;
  k.push_back((char)L.n_nodes);
  for (int v = 0; v < L.n_nodes; v++) k.push_back((char)L.node_comp[v]);
  for (int t = 0; t < T; t++) {
    k.push_back((char)L.n_alt[t]);
    for (int a = 0; a < L.n_alt[t]; a++)
      for (int c = 0; c < CF_MAX_COMP; c++) k.push_back((char)L.alt_node[t][a][c]);
  }
  return k;
}

void route_type(cf_logical &L, int t, int a, uint32_t path, const Subplan &s, const int *node_map) {
  for (int c = 0; c < CF_MAX_COMP; c++)
    if ((path >> c) & 1u) L.alt_node[t][a][c] = (uint8_t)node_map[s.node_of(c)];
}

// ------------------------------------------------------------------ device
struct EnumView {
  int N;
  const cf_logical *logical;
  int n_logical;
  uint64_t *tab;      // [n_logical][kTabSize]
  uint64_t *totals;   // [n_logical]
};

__device__ __forceinline__ uint64_t sat_add(uint64_t a, uint64_t b) { return a > ~0ull - b ? ~0ull : a + b; }
__device__ __forceinline__ uint64_t sat_mul(uint64_t a, uint64_t b) { return (b && a > ~0ull / b) ? ~0ull : a * b; }

// The option tables a node indexes by its lowest component, staged in LDS.
struct OptsLds {
  uint8_t n_batch[CF_MAX_COMP], n_gpu[CF_MAX_COMP];
  uint8_t gpu[CF_MAX_COMP][4];
  uint16_t batch[CF_MAX_COMP][8];
};

__device__ void stage_opts(OptsLds &s, const cf_enum_opts &o, int tid, int nthreads) {
  for (int i = tid; i < CF_MAX_COMP; i += nthreads) {
    s.n_batch[i] = (uint8_t)o.n_batch[i];
    s.n_gpu[i] = (uint8_t)o.n_gpu_opt[i];
    for (int k = 0; k < 4; k++) s.gpu[i][k] = o.gpu_opt[i][k];
    for (int k = 0; k < 8; k++) s.batch[i][k] = o.batch[i][k];
  }
}

// One block per logical plan: cnt[v][b], then the plan's total.
__global__ void __launch_bounds__(128) k_enum_table(cf_enum_opts o, EnumView V) {
  __shared__ OptsLds so;
  __shared__ uint64_t cnt[CF_MAX_NODES + 1][kTabStride];
  const int l = blockIdx.x, b = threadIdx.x;
  stage_opts(so, o, threadIdx.x, blockDim.x);
  const cf_logical &L = V.logical[l];
  const int nv = L.n_nodes <= CF_MAX_NODES ? L.n_nodes : CF_MAX_NODES;
  if (b <= V.N) cnt[nv][b] = 1;
  __syncthreads();
  for (int v = nv - 1; v >= 0; v--) {
    if (b <= V.N) {
      const int c0 = L.node_comp[v] ? __ffs(L.node_comp[v]) - 1 : 0;
      uint64_t tot = 0;
      for (int gi = 0; gi < so.n_gpu[c0]; gi++) {
        const int g = so.gpu[c0][gi];
        uint64_t per_cfg = 0;
        for (int n = 1; g * n <= b; n++) per_cfg = sat_add(per_cfg, cnt[v + 1][b - g * n]);
        for (int bi = 0; bi < so.n_batch[c0]; bi++) tot = sat_add(tot, per_cfg);
      }
      if (o.het) {
        // two configurations k1 < k2 (GPU option major, batch minor), n1, n2 >= 1, 9 weights
        const int nb = so.n_batch[c0], K = so.n_gpu[c0] * nb;
        for (int k1 = 0; k1 < K; k1++)
          for (int k2 = k1 + 1; k2 < K; k2++) {
            const int g1 = so.gpu[c0][k1 / nb], g2 = so.gpu[c0][k2 / nb];
            for (int n1 = 1; g1 * n1 + g2 <= b; n1++)
              for (int n2 = 1; g1 * n1 + g2 * n2 <= b; n2++)
                tot = sat_add(tot, sat_mul(9, cnt[v + 1][b - g1 * n1 - g2 * n2]));
          }
      }
      cnt[v][b] = tot;
    }
    __syncthreads();
  }
  uint64_t *out = V.tab + (size_t)l * kTabSize;
  for (int i = threadIdx.x; i < (nv + 1) * kTabStride; i += blockDim.x) out[i] = (&cnt[0][0])[i];
  if (threadIdx.x == 0) {
    uint64_t tot = cnt[0][V.N];
    for (int t = 0; t < CF_MAX_TYPES; t++)
      if (L.n_alt[t] == 2) tot = sat_mul(tot, 9);
    V.totals[l] = tot;
  }
}

// offsets[0] = 0, offsets[l+1] = offsets[l] + totals[l] (saturating); one block.
__global__ void __launch_bounds__(1024) k_enum_offsets(const uint64_t *totals, int n, uint64_t *offsets) {
  __shared__ uint64_t part[1024];
  __shared__ uint64_t carry_s;
  const int tid = threadIdx.x;
  if (tid == 0) {
    carry_s = 0;
    offsets[0] = 0;
  }
  __syncthreads();
  for (int base = 0; base < n; base += 1024) {
    const uint64_t x = base + tid < n ? totals[base + tid] : 0;
    part[tid] = x;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {
      const uint64_t add = tid >= d ? part[tid - d] : 0;
      __syncthreads();
      part[tid] = sat_add(part[tid], add);
      __syncthreads();
    }
    if (base + tid < n) offsets[base + tid + 1] = sat_add(carry_s, part[tid]);
    __syncthreads();
    if (tid == 1023) carry_s = sat_add(carry_s, part[1023]);
    __syncthreads();
  }
}

struct PlanOut {
  int P;
  uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  uint16_t *node_batch;
  uint8_t *node_rep2, *node_gpus2, *node_w;  // second configurations (NULL: not written)
  uint16_t *node_batch2;
};

// The position of plan idx: its logical plan, routing digits and the cursor
// of the executor-assignment walk.
struct Cursor {
  int l, nv;
  bool ok;
  uint64_t q;   // rank among the executor assignments still to place
  int b;        // GPUs left
  uint32_t w;   // routing weights, 4 bits per type with two alternatives, in type order
};

__device__ Cursor locate(const EnumView &V, const uint64_t *offsets, uint64_t idx, bool valid) {
  Cursor c;
  c.ok = valid && idx < offsets[V.n_logical];
  int lo = 0, hi = V.n_logical;  // offsets[lo] <= idx < offsets[hi]
  if (c.ok) {
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (offsets[mid] <= idx) lo = mid; else hi = mid;
    }
  }
  c.l = lo;
  const cf_logical &L = V.logical[lo];
  c.nv = c.ok ? L.n_nodes : 0;
  const uint64_t local = c.ok ? idx - offsets[lo] : 0;
  int na2 = 0;
  for (int t = 0; t < CF_MAX_TYPES; t++) na2 += L.n_alt[t] == 2;
  uint64_t R = 1;
  for (int i = 0; i < na2; i++) R *= 9;
  uint64_t r = local % R;
  c.q = local / R;
  c.w = 0;
  for (int i = na2 - 1; i >= 0; i--) {  // lowest type is the most significant digit
    c.w |= (uint32_t)(r % 9 + 1) << (4 * i);
    r /= 9;
  }
  c.b = V.N;
  return c;
}

struct NodeCfg {
  uint8_t comp, rep, gpus;
  uint16_t batch;
  uint8_t rep2, gpus2, w;  // a second configuration (rep2 = 0: none, w = 10)
  uint16_t batch2;
};

// Node v of the plan at cursor c: the candidates (k, n) in order own
// cnt[v+1][b - gpus_k n] consecutive ranks each; with het, then the
// candidates (k1, k2, n1, n2, w) own cnt[v+1][b - gpus_k1 n1 - gpus_k2 n2]
// each.
__device__ NodeCfg place(const EnumView &V, const OptsLds &so, Cursor &c, int v, bool het) {
  NodeCfg r = {0, 0, 0, 0, 0, 0, 10, 0};
  if (v >= c.nv) return r;
  const cf_logical &L = V.logical[c.l];
  const uint64_t *tab = V.tab + (size_t)c.l * kTabSize + (size_t)(v + 1) * kTabStride;
  r.comp = L.node_comp[v];
  const int c0 = r.comp ? __ffs(r.comp) - 1 : 0;
  const int nb = so.n_batch[c0];
  for (int gi = 0; gi < so.n_gpu[c0]; gi++) {
    const int g = so.gpu[c0][gi];
    for (int bi = 0; bi < nb; bi++) {
      for (int n = 1; g * n <= c.b; n++) {
        const uint64_t k = tab[c.b - g * n];
        if (c.q < k) {
          r.rep = (uint8_t)n;
          r.gpus = (uint8_t)g;
          r.batch = so.batch[c0][bi];
          c.b -= g * n;
          return r;
        }
        c.q -= k;
      }
    }
  }
  if (het) {
    const int K = so.n_gpu[c0] * nb;
    for (int k1 = 0; k1 < K; k1++)
      for (int k2 = k1 + 1; k2 < K; k2++) {
        const int g1 = so.gpu[c0][k1 / nb], g2 = so.gpu[c0][k2 / nb];
        for (int n1 = 1; g1 * n1 + g2 <= c.b; n1++)
          for (int n2 = 1; g1 * n1 + g2 * n2 <= c.b; n2++) {
            const uint64_t k = tab[c.b - g1 * n1 - g2 * n2];
            const uint64_t k9 = sat_mul(k, 9);  // the nine weights, k ranks each
            if (c.q < k9) {
              const uint64_t wi = c.q / k;
              c.q -= wi * k;
              r.rep = (uint8_t)n1;
              r.gpus = (uint8_t)g1;
              r.batch = so.batch[c0][k1 % nb];
              r.rep2 = (uint8_t)n2;
              r.gpus2 = (uint8_t)g2;
              r.batch2 = so.batch[c0][k2 % nb];
              r.w = (uint8_t)(wi + 1);
              c.b -= g1 * n1 + g2 * n2;
              return r;
            }
            c.q -= k9;
          }
      }
  }
  return r;
}

// Four consecutive plans per thread, each slot row written with one 32-bit
// store (64-bit for the batch row): a wavefront writes 256 bytes of a row
// per instruction.  Needs out.P % 4 == 0; the last thread writes bytes.
// HET: the space has nodes of two configurations (o.het); without them the
// walk over configuration pairs is not compiled in.
constexpr int kPlansPerThread = 4;
template <bool HET>
__global__ void __launch_bounds__(256) k_enum_unrank(cf_enum_opts o, EnumView V, const uint64_t *offsets,
                                                    uint64_t first, int count, PlanOut out) {
  __shared__ OptsLds so;
  stage_opts(so, o, threadIdx.x, blockDim.x);
  __syncthreads();
  const int p0 = (blockIdx.x * blockDim.x + threadIdx.x) * kPlansPerThread;
  if (p0 >= count) return;
  const size_t P = (size_t)out.P;
  const bool packed = p0 + kPlansPerThread <= count && (out.P % kPlansPerThread) == 0;
  // consecutive plans of one logical plan that differ only in their routing
  // weights share the executor assignment: it is walked once
  Cursor cur[kPlansPerThread];
  bool same[kPlansPerThread];
#pragma unroll
  for (int j = 0; j < kPlansPerThread; j++) {
    cur[j] = locate(V, offsets, first + (uint64_t)(p0 + j), p0 + j < count);
    same[j] = j > 0 && cur[j].ok && cur[j - 1].ok && cur[j].l == cur[j - 1].l && cur[j].q == cur[j - 1].q;
  }
  auto put8 = [&](uint8_t *row, const uint8_t *x) {
    if (packed) {
      *(uint32_t *)(row + p0) = (uint32_t)x[0] | ((uint32_t)x[1] << 8) | ((uint32_t)x[2] << 16) | ((uint32_t)x[3] << 24);
    } else {
      for (int j = 0; j < kPlansPerThread; j++)
        if (p0 + j < count) row[p0 + j] = x[j];
    }
  };
  uint8_t b8[kPlansPerThread];
#pragma unroll
  for (int j = 0; j < kPlansPerThread; j++) b8[j] = (uint8_t)cur[j].nv;
  put8(out.n_nodes, b8);
  for (int v = 0; v < CF_MAX_NODES; v++) {
    NodeCfg nc[kPlansPerThread];
#pragma unroll
    for (int j = 0; j < kPlansPerThread; j++) nc[j] = same[j] ? nc[j - 1] : place(V, so, cur[j], v, HET);
#pragma unroll
    for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].comp;
    put8(out.node_comp + v * P, b8);
#pragma unroll
    for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].rep;
    put8(out.node_rep + v * P, b8);
#pragma unroll
    for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].gpus;
    put8(out.node_gpus + v * P, b8);
    uint16_t *brow = out.node_batch + v * P;
    if (packed) {
      *(uint64_t *)(brow + p0) = (uint64_t)nc[0].batch | ((uint64_t)nc[1].batch << 16) |
                                 ((uint64_t)nc[2].batch << 32) | ((uint64_t)nc[3].batch << 48);
    } else {
      for (int j = 0; j < kPlansPerThread; j++)
        if (p0 + j < count) brow[p0 + j] = nc[j].batch;
    }
    if (out.node_rep2) {
#pragma unroll
      for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].rep2;
      put8(out.node_rep2 + v * P, b8);
#pragma unroll
      for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].gpus2;
      put8(out.node_gpus2 + v * P, b8);
#pragma unroll
      for (int j = 0; j < kPlansPerThread; j++) b8[j] = nc[j].w;
      put8(out.node_w + v * P, b8);
      uint16_t *b2row = out.node_batch2 + v * P;
      for (int j = 0; j < kPlansPerThread; j++)
        if (p0 + j < count) b2row[p0 + j] = nc[j].batch2;
    }
  }
  int i2[kPlansPerThread] = {0, 0, 0, 0};
  for (int t = 0; t < CF_MAX_TYPES; t++) {
    uint8_t na[kPlansPerThread], w0[kPlansPerThread], w1[kPlansPerThread];
#pragma unroll
    for (int j = 0; j < kPlansPerThread; j++) {
      na[j] = cur[j].ok ? V.logical[cur[j].l].n_alt[t] : 0;
      w0[j] = na[j] == 1 ? 10 : 0;
      w1[j] = 0;
      if (na[j] == 2) {
        w0[j] = (uint8_t)((cur[j].w >> (4 * i2[j])) & 15u);
        w1[j] = (uint8_t)(10 - w0[j]);
        i2[j]++;
      }
    }
    put8(out.n_alt + t * P, na);
    put8(out.alt_w + (2 * t) * P, w0);
    put8(out.alt_w + (2 * t + 1) * P, w1);
    for (int a = 0; a < 2; a++)
      for (int c = 0; c < CF_MAX_COMP; c++) {
#pragma unroll
        for (int j = 0; j < kPlansPerThread; j++)
          b8[j] = cur[j].ok ? V.logical[cur[j].l].alt_node[t][a][c] : (uint8_t)255;
        put8(out.alt_node + ((2 * t + a) * CF_MAX_COMP + c) * P, b8);
      }
  }
}

// Enumeration fused with phase 1: a thread numbers its plan, builds the
// plan's nodes and routes in registers and LDS exactly as k_enum_unrank
// would write them, and screens it as k_coarse would read them, writing only
// R_d, the bottleneck and the flags (13 B per plan instead of the 233 B
// table written and read back).
constexpr int kScrBlock = 256;
__global__ void __launch_bounds__(kScrBlock) k_enum_screen(cf_enum_opts o, EnumView V, const uint64_t *offsets,
                                                          uint64_t first, int count, KModel m, const uint64_t *moments,
                                                          int n_gpus, double *rd, int32_t *bott, uint8_t *flags) {
  __shared__ OptsLds so;
  __shared__ double ex_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double en_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double tps_s[CF_MAX_COMP][8];
  __shared__ double u_s[CF_MAX_NODES][kScrBlock];
  __shared__ uint16_t b_s[CF_MAX_NODES][kScrBlock];
  __shared__ uint8_t g_s[CF_MAX_NODES][kScrBlock];
  const int tid = threadIdx.x;
  stage_opts(so, o, tid, blockDim.x);
  if (tid < CF_MAX_COMP * 8) (&tps_s[0][0])[tid] = (&m.tps[0][0])[tid];
  phase1_means(m, moments, tid, ex_s, en_s);
  __syncthreads();
  const int p = blockIdx.x * kScrBlock + tid;
  if (p >= count) return;
  Cursor cur = locate(V, offsets, first + (uint64_t)p, true);
  const int nv = cur.nv;
  uint32_t rep[CF_MAX_NODES], gp[CF_MAX_NODES];
#pragma unroll
  for (int v = 0; v < CF_MAX_NODES; v++) {
    const NodeCfg nc = place(V, so, cur, v, false);
    rep[v] = nc.rep;
    gp[v] = nc.gpus;
    b_s[v][tid] = nc.batch;
    if (m.tp_any) g_s[v][tid] = (uint8_t)(nc.gpus < 1 ? 0 : (nc.gpus > 8 ? 7 : nc.gpus - 1));
    u_s[v][tid] = 0.0;
  }
  if (!cur.ok || nv < 1) {
    rd[p] = 0.0;
    bott[p] = -1;
    flags[p] = CF_FLAG_INVALID;
    return;
  }
  const cf_logical &L = V.logical[cur.l];
  const double wsum = (double)m.wsum;
  int i2 = 0;
  for (int t = 0; t < m.nt; t++) {
    const uint32_t path = m.path[t];
    const uint32_t na = L.n_alt[t];
    uint32_t wl[2] = {10u, 0u};
    if (na == 2) {
      wl[0] = (cur.w >> (4 * i2)) & 15u;
      wl[1] = 10u - wl[0];
      i2++;
    }
    const double pi = (double)m.weight[t] / wsum;
    const uint32_t wtot = na > 1 ? wl[0] + wl[1] : 1u;
#pragma unroll
    for (int a = 0; a < 2; a++) {
      if (a < (int)na) {
        const uint32_t wa = na > 1 ? wl[a] : 1u;
        const double q = (double)wa / (double)wtot;
        const double pq = pi * q;
#pragma unroll
        for (int c = 0; c < CF_MAX_COMP; c++) {
          if (!((path >> c) & 1u)) continue;
          const int v = L.alt_node[t][a][c];
          const double w =
              phase1_work(m, c, b_s[v][tid], ex_s[t][c], en_s[t][c], m.tp_any ? tps_s[c][g_s[v][tid]] : 1.0);
          u_s[v][tid] = u_s[v][tid] + pq * w;
        }
      }
    }
  }
  phase1_result(nv, rep, gp, [&](int v) { return u_s[v][tid]; }, n_gpus, &rd[p], &bott[p], &flags[p]);
}

cf_status run_tables(const cf_enum_opts *opts, const cf_logical *logical_dev, int n_logical, uint64_t **tab_out,
                     uint64_t **totals_out, hipStream_t s) {
  cf_status st = CF_OK;
  const size_t bytes = sizeof(uint64_t) * ((size_t)n_logical * kTabSize + (size_t)n_logical);
  uint64_t *scr = (uint64_t *)scratch_get(SCR_ENUM, bytes, &st);
  if (!scr) return st;
  EnumView V;
  V.N = opts->n_gpus;
  V.logical = logical_dev;
  V.n_logical = n_logical;
  V.tab = scr;
  V.totals = scr + (size_t)n_logical * kTabSize;
  hipLaunchKernelGGL(k_enum_table, dim3((unsigned)n_logical), dim3(128), 0, s, *opts, V);
  st = hip_check(hipGetLastError(), "cf_enum table launch");
  *tab_out = V.tab;
  *totals_out = V.totals;
  return st;
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_enum_logical(const cf_model_desc *model, const cf_enum_opts *opts, cf_logical *out_host,
                                     int32_t cap, int32_t *n_out) {
  using namespace cf;
  cf_status st = check_opts(model, opts);
  if (st != CF_OK) return st;
  if (!out_host || !n_out || cap < 0) return set_error(CF_EINVAL, "NULL output or cap < 0");
  *n_out = 0;
  const int T = model->n_types, C = model->n_comp;
  const uint32_t all_types = (1u << T) - 1u;
  // subgraphs: distinct unions of type paths, ascending
  std::set<uint32_t> subgraphs;
  for (uint32_t u = 1; u <= all_types; u++) {
    uint32_t cs = 0;
    for (int t = 0; t < T; t++)
      if ((u >> t) & 1u) cs |= model->path_mask[t];
    subgraphs.insert(cs);
  }
  // simple subplans
  std::vector<Subplan> S;
  for (uint32_t cs : subgraphs) {
    uint32_t cov = 0;
    for (int t = 0; t < T; t++)
      if (!(model->path_mask[t] & ~cs)) cov |= 1u << t;
    std::vector<std::pair<int, int>> edges;
    for (int p = 0; p < C; p++)
      for (int c = 0; c < C; c++) {
        if (!((opts->colocatable[p] >> c) & 1u)) continue;
        bool on = false;
        for (int t = 0; t < T && !on; t++) on = ((cov >> t) & 1u) && ((model->parents[t][c] >> p) & 1u);
        if (on) edges.emplace_back(p, c);
      }
    if (edges.size() > 16) return set_error(CF_ECAPACITY, "more than 16 colocatable edges in a subgraph");
    std::set<std::vector<uint8_t>> seen;
    for (uint32_t m = 0; m < (1u << edges.size()); m++) {
      int par[CF_MAX_COMP];
      for (int c = 0; c < CF_MAX_COMP; c++) par[c] = c;
      for (size_t i = 0; i < edges.size(); i++)
        if ((m >> i) & 1u) {
          const int ra = uf_find(par, edges[i].first), rb = uf_find(par, edges[i].second);
          if (ra != rb) par[std::max(ra, rb)] = std::min(ra, rb);
        }
      std::map<int, uint8_t> groups;
      for (int c = 0; c < CF_MAX_COMP; c++)
        if ((cs >> c) & 1u) groups[uf_find(par, c)] |= (uint8_t)(1u << c);
      std::vector<uint8_t> nodes;
      for (auto &g : groups) nodes.push_back(g.second);
      std::sort(nodes.begin(), nodes.end());
      if (!seen.insert(nodes).second) continue;
      S.push_back(Subplan{cs, cov, nodes});
    }
  }
  // logical plans
  std::set<std::string> emitted;
  int n = 0;
  auto emit = [&](const cf_logical &L) -> cf_status {
    if (!emitted.insert(plan_key(L, T)).second) return CF_OK;
    if (n >= cap) return set_error(CF_ECAPACITY, "more than %d logical plans", cap);
    out_host[n++] = L;
    return CF_OK;
  };
  auto blank = []() {
    cf_logical L;
    memset(&L, 0, sizeof L);
    memset(L.alt_node, 255, sizeof L.alt_node);
    return L;
  };
  for (const Subplan &s : S) {
    if (s.cov != all_types) continue;
    cf_logical L = blank();
    L.n_nodes = (uint8_t)s.nodes.size();
    int ident[CF_MAX_COMP];
    for (size_t v = 0; v < s.nodes.size(); v++) {
      L.node_comp[v] = s.nodes[v];
      ident[v] = (int)v;
    }
    for (int t = 0; t < T; t++) {
      L.n_alt[t] = 1;
      route_type(L, t, 0, model->path_mask[t], s, ident);
    }
    if ((st = emit(L)) != CF_OK) return st;
  }
  if (opts->k_s == 2) {
    for (size_t i = 0; i < S.size(); i++)
      for (size_t j = i; j < S.size(); j++) {
        const Subplan &A = S[i], &B = S[j];
        if ((A.cov | B.cov) != all_types) continue;
        std::vector<std::pair<int, int>> matchable;  // (node of B, equal node of A), in B's order
        for (size_t v = 0; v < B.nodes.size(); v++)
          for (size_t w = 0; w < A.nodes.size(); w++)
            if (B.nodes[v] == A.nodes[w]) matchable.emplace_back((int)v, (int)w);
        const uint32_t n_sets = opts->share ? (1u << matchable.size()) : 1u;
        for (uint32_t sh = 0; sh < n_sets; sh++) {
          if (opts->share && matchable.size() == B.nodes.size() && sh == n_sets - 1) continue;
          int amap[CF_MAX_COMP], bmap[CF_MAX_COMP];
          int nv = (int)A.nodes.size();
          for (int v = 0; v < nv; v++) amap[v] = v;
          for (size_t v = 0; v < B.nodes.size(); v++) bmap[v] = -1;
          for (size_t k = 0; k < matchable.size(); k++)
            if ((sh >> k) & 1u) bmap[matchable[k].first] = matchable[k].second;
          for (size_t v = 0; v < B.nodes.size(); v++)
            if (bmap[v] < 0) bmap[v] = nv++;
          if (nv > CF_MAX_NODES) continue;
          cf_logical L = blank();
          L.n_nodes = (uint8_t)nv;
          for (size_t v = 0; v < A.nodes.size(); v++) L.node_comp[v] = A.nodes[v];
          for (size_t v = 0; v < B.nodes.size(); v++) L.node_comp[bmap[v]] = B.nodes[v];
          for (int t = 0; t < T; t++) {
            const bool inA = (A.cov >> t) & 1u, inB = (B.cov >> t) & 1u;
            int na = 0;
            if (inA) route_type(L, t, na++, model->path_mask[t], A, amap);
            if (inB) {
              route_type(L, t, na, model->path_mask[t], B, bmap);
              if (na == 1 && !memcmp(L.alt_node[t][0], L.alt_node[t][1], CF_MAX_COMP))
                memset(L.alt_node[t][1], 255, CF_MAX_COMP);
              else
                na++;
            }
            L.n_alt[t] = (uint8_t)na;
          }
          if ((st = emit(L)) != CF_OK) return st;
        }
      }
  }
  *n_out = n;
  return CF_OK;
}

extern "C" cf_status cf_enum_count(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                                   int32_t n_logical, uint64_t *offsets_dev, uint64_t *total_host, void *stream) {
  using namespace cf;
  cf_status st = check_opts(model, opts);
  if (st != CF_OK) return st;
  if (n_logical < 0 || !offsets_dev || !total_host || (n_logical > 0 && !logical_dev))
    return set_error(CF_EINVAL, "NULL array or n_logical < 0");
  hipStream_t s = as_stream(stream);
  *total_host = 0;
  if (n_logical == 0) {
    const uint64_t zero = 0;
    st = hip_check(hipMemcpyAsync(offsets_dev, &zero, sizeof zero, hipMemcpyHostToDevice, s), "cf_enum_count copy");
    if (st != CF_OK) return st;
    return hip_check(hipStreamSynchronize(s), "cf_enum_count sync");
  }
  uint64_t *tab = nullptr, *totals = nullptr;
  if ((st = run_tables(opts, logical_dev, n_logical, &tab, &totals, s)) != CF_OK) return st;
  hipLaunchKernelGGL(k_enum_offsets, dim3(1), dim3(1024), 0, s, totals, n_logical, offsets_dev);
  if ((st = hip_check(hipGetLastError(), "cf_enum offsets launch")) != CF_OK) return st;
  st = hip_check(hipMemcpyAsync(total_host, offsets_dev + n_logical, sizeof(uint64_t), hipMemcpyDeviceToHost, s),
                 "cf_enum_count copy");
  if (st != CF_OK) return st;
  if ((st = hip_check(hipStreamSynchronize(s), "cf_enum_count sync")) != CF_OK) return st;
  if (*total_host == ~0ull) return set_error(CF_ECAPACITY, "the number of physical plans does not fit 64 bits");
  return CF_OK;
}

extern "C" cf_status cf_enum_plans(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                                   int32_t n_logical, const uint64_t *offsets_dev, uint64_t total, uint64_t first,
                                   int32_t count, const cf_plan_table *out, void *stream) {
  using namespace cf;
  cf_status st = check_opts(model, opts);
  if (st != CF_OK) return st;
  if (!out || count < 0 || out->P < count) return set_error(CF_EINVAL, "output table smaller than count");
  if (count == 0) return CF_OK;
  if (n_logical < 1 || !logical_dev || !offsets_dev) return set_error(CF_EINVAL, "no logical plans");
  if (first > total || (uint64_t)count > total - first) return set_error(CF_EINVAL, "first + count > total");
  if (!out->n_nodes_dev || !out->node_comp_dev || !out->node_rep_dev || !out->node_batch_dev ||
      !out->node_gpus_dev || !out->n_alt_dev || !out->alt_w_dev || !out->alt_node_dev)
    return set_error(CF_EINVAL, "NULL plan-table array");
  const int ng = (out->node_rep2_dev != nullptr) + (out->node_batch2_dev != nullptr) +
                 (out->node_gpus2_dev != nullptr) + (out->node_w_dev != nullptr);
  if (ng != 0 && ng != 4) return set_error(CF_EINVAL, "second-configuration arrays: all four or none");
  if (opts->het && ng == 0) return set_error(CF_EINVAL, "het plans need the second-configuration arrays");
  hipStream_t s = as_stream(stream);
  uint64_t *tab = nullptr, *totals = nullptr;
  if ((st = run_tables(opts, logical_dev, n_logical, &tab, &totals, s)) != CF_OK) return st;
  EnumView V;
  V.N = opts->n_gpus;
  V.logical = logical_dev;
  V.n_logical = n_logical;
  V.tab = tab;
  V.totals = totals;
  PlanOut o;
  o.P = out->P;
  o.n_nodes = const_cast<uint8_t *>(out->n_nodes_dev);
  o.node_comp = const_cast<uint8_t *>(out->node_comp_dev);
  o.node_rep = const_cast<uint8_t *>(out->node_rep_dev);
  o.node_batch = const_cast<uint16_t *>(out->node_batch_dev);
  o.node_gpus = const_cast<uint8_t *>(out->node_gpus_dev);
  o.n_alt = const_cast<uint8_t *>(out->n_alt_dev);
  o.alt_w = const_cast<uint8_t *>(out->alt_w_dev);
  o.alt_node = const_cast<uint8_t *>(out->alt_node_dev);
  o.node_rep2 = const_cast<uint8_t *>(out->node_rep2_dev);
  o.node_batch2 = const_cast<uint16_t *>(out->node_batch2_dev);
  o.node_gpus2 = const_cast<uint8_t *>(out->node_gpus2_dev);
  o.node_w = const_cast<uint8_t *>(out->node_w_dev);
  const unsigned threads = (unsigned)((count + kPlansPerThread - 1) / kPlansPerThread);
  if (opts->het)
    hipLaunchKernelGGL(k_enum_unrank<true>, dim3((threads + 255) / 256), dim3(256), 0, s, *opts, V, offsets_dev, first,
                       count, o);
  else
    hipLaunchKernelGGL(k_enum_unrank<false>, dim3((threads + 255) / 256), dim3(256), 0, s, *opts, V, offsets_dev,
                       first, count, o);
  return hip_check(hipGetLastError(), "cf_enum_plans launch");
}

extern "C" cf_status cf_enum_screen(const cf_model_desc *model, const cf_enum_opts *opts, const cf_logical *logical_dev,
                                    int32_t n_logical, const uint64_t *offsets_dev, uint64_t total, uint64_t first,
                                    int32_t count, const uint64_t *moments_dev, int32_t n_gpus, double *rd_dev,
                                    int32_t *bottleneck_dev, uint8_t *flags_dev, void *stream) {
  using namespace cf;
  cf_status st = check_opts(model, opts);
  if (st != CF_OK) return st;
  if (opts->het) return set_error(CF_EUNSUPPORTED, "cf_enum_screen takes one configuration per node");
  KModel m;
  if ((st = lower_model(model, &m)) != CF_OK) return st;
  if (count < 0) return set_error(CF_EINVAL, "count < 0");
  if (count == 0) return CF_OK;
  if (n_logical < 1 || !logical_dev || !offsets_dev || !moments_dev || !rd_dev || !bottleneck_dev || !flags_dev)
    return set_error(CF_EINVAL, "NULL argument");
  if (first > total || (uint64_t)count > total - first) return set_error(CF_EINVAL, "first + count > total");
  hipStream_t s = as_stream(stream);
  uint64_t *tab = nullptr, *totals = nullptr;
  if ((st = run_tables(opts, logical_dev, n_logical, &tab, &totals, s)) != CF_OK) return st;
  EnumView V;
  V.N = opts->n_gpus;
  V.logical = logical_dev;
  V.n_logical = n_logical;
  V.tab = tab;
  V.totals = totals;
  hipLaunchKernelGGL(k_enum_screen, dim3((unsigned)((count + kScrBlock - 1) / kScrBlock)), dim3(kScrBlock), 0, s,
                     *opts, V, offsets_dev, first, count, m, moments_dev, n_gpus, rd_dev, bottleneck_dev, flags_dev);
  return hip_check(hipGetLastError(), "cf_enum_screen launch");
}
