// k_mc.hip -- cf_eval_mc and cf_pareto: phase 2 of the plan evaluation
// (Sec. 4.3, Alg. 2 phase 2) with occupancy-aware latency scaling
// (Sec. 5.2), and Pareto pruning of per-type goodput vectors (Alg. 2).
//
// Phase 2 draws K requests from the workload and routes each through a plan
// alone, without queueing; every component it visits costs one iteration of
// its latency model at the component's effective batch on its node.  The
// fraction of sampled requests of type t meeting the targets is F_t and the
// goodput estimate G_t = alpha R_d pi_t F_t.
//   - effective batch: node v, whose phase-1 capacity is R_v = m_v / u_v,
//     runs at b = clamp(ceil(B (R_d / R_v)), 1, B), B = min(node batch, cap)
//     (the bottleneck at its configured batch);
//   - encoder / generator iteration: a static batch of b requests like this
//     one, (k0 + k1 (b x)) + k2 b; LLM: the request's own prefill,
//     (k0 + k1 x) + k2, then decode steps d0 + d1 b shared with the running set;
//   - a component starts at the last arrival of its inputs (a parent's finish,
//     a gate source's first token for a gated LLM, plus comm across
//     executors); token k+1 of a gated LLM waits for the gate source's token
//     min(k+1, n_src) (comm later across executors) and for its own token k.
//
// One wavefront per plan: the plan's nodes, routes and effective batches are
// set up in LDS (the per-node demand u_v is summed by one lane in the order
// phase 1 uses), then the lanes take the sampled requests, 64 at a time;
// each lane walks its request's path in component order with the whole
// timeline in registers (a decode run in closed form, a gated decode one
// token at a time), and SLO counts are LDS atomics per type.
#include "cf_internal.h"
#include "cf_run.h"

namespace cf {
namespace {

struct McView {
  int P;
  const uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  const uint16_t *node_batch;
  const uint8_t *node_rep2, *node_gpus2, *node_w;  // a node's second configuration (NULL: none)
  const uint16_t *node_batch2;
  const int32_t *ids;
  const double *rd;
  const uint64_t *moments;
  double alpha;
  const uint64_t *ticks, *rkey0, *rkey1;
  const uint8_t *type;
  const uint16_t *patches, *prompt, *out;
  const uint32_t *aud_in, *aud_out, *akey;
  size_t toff;  // first sampled request: seed_idx * n_req
  int n_sample;
  const uint32_t *order;  // the sampled requests in walking order (a permutation of 0..n_sample-1)
  // optional latency CDF over a target table [T][nb][4]: hist [n_plans][T][nb+1], curve [n_plans][nb][T]
  const double *tg;
  int nb;
  uint32_t *hist;
  double *curve;
  uint32_t *met, *cnt;
  double *gt, *lat;
};

// the request's attributes, loaded together once per request
struct McReq {
  uint32_t prompt, out, patches, aud_in, aud_out;
};

__device__ __forceinline__ uint32_t mc_attr(const McReq &q, int a) {
  switch (a) {
    case CF_ATTR_PROMPT: return q.prompt;
    case CF_ATTR_OUT: return q.out;
    case CF_ATTR_PATCHES: return q.patches;
    case CF_ATTR_AUDIN_MS: return q.aud_in;
    case CF_ATTR_AUDOUT_MS: return q.aud_out;
    case CF_ATTR_AUDIN_TOK: return (q.aud_in + 79u) / 80u;
    case CF_ATTR_AUDOUT_TOK: return (q.aud_out + 79u) / 80u;
    default: return 0;
  }
}

// The order the lanes take the sampled requests in.  Every request's walk
// is independent of the others and the counts are sums, so any order gives
// the same results; this one groups requests by type and then by the token
// count of the type's gated decode, so that a wavefront mostly walks one
// path and its gated decode loops have nearly equal lengths.  One workgroup:
// a histogram over (type, min(tokens, 255)), an exclusive scan, a scatter.
constexpr int kOrdThreads = 1024, kOrdBuckets = CF_MAX_TYPES * 256;
__global__ void __launch_bounds__(kOrdThreads) k_mc_order(KModel m, McView V, uint32_t *order) {
  __shared__ uint32_t hist[kOrdBuckets];
  __shared__ uint32_t part[kOrdThreads];
  __shared__ int8_t tok_attr[CF_MAX_TYPES];
  const int tid = threadIdx.x;
  for (int b = tid; b < kOrdBuckets; b += kOrdThreads) hist[b] = 0;
  if (tid < CF_MAX_TYPES) {
    const int ta = tid < m.nt ? m.ta_c[tid] : -1;
    tok_attr[tid] = (int8_t)(ta >= 0 && !((m.pfo[tid] >> ta) & 1u) ? m.nout_attr[ta] : -1);
  }
  __syncthreads();
  auto bucket = [&](int r) -> uint32_t {
    const size_t o = V.toff + (size_t)r;
    const uint32_t t = V.type[o] < CF_MAX_TYPES ? V.type[o] : CF_MAX_TYPES - 1;
    uint32_t tok = 0;
    if (tok_attr[t] >= 0) {
      McReq q;
      q.prompt = V.prompt[o];
      q.out = V.out[o];
      q.patches = V.patches[o];
      q.aud_in = V.aud_in[o];
      q.aud_out = V.aud_out[o];
      tok = mc_attr(q, tok_attr[t]);
      tok = tok < 255u ? tok : 255u;
    }
    return t * 256u + tok;
  };
  for (int r = tid; r < V.n_sample; r += kOrdThreads) atomicAdd(&hist[bucket(r)], 1u);
  __syncthreads();
  // exclusive scan: each thread owns kOrdBuckets / kOrdThreads consecutive buckets
  constexpr int per = kOrdBuckets / kOrdThreads;
  uint32_t mine = 0;
  for (int k = 0; k < per; k++) mine += hist[tid * per + k];
  part[tid] = mine;
  __syncthreads();
  for (int d = 1; d < kOrdThreads; d <<= 1) {
    const uint32_t add = tid >= d ? part[tid - d] : 0u;
    __syncthreads();
    part[tid] += add;
    __syncthreads();
  }
  uint32_t run = part[tid] - mine;
  for (int k = 0; k < per; k++) {
    const uint32_t h = hist[tid * per + k];
    hist[tid * per + k] = run;
    run += h;
  }
  __syncthreads();
  for (int r = tid; r < V.n_sample; r += kOrdThreads) order[atomicAdd(&hist[bucket(r)], 1u)] = (uint32_t)r;
}

__global__ void __launch_bounds__(64) k_mc(KModel m, McView V) {
  __shared__ uint8_t vcomp[CF_MAX_NODES], vrep[CF_MAX_NODES], vminc[CF_MAX_NODES], vbase[CF_MAX_NODES];
  __shared__ uint8_t vtp[CF_MAX_NODES];            // GPUs per executor, as min(g, 8) - 1
  __shared__ double tps_s[CF_MAX_COMP][8];         // iteration-time multipliers by GPUs per executor
  __shared__ uint16_t vbatch[CF_MAX_NODES];
  __shared__ uint16_t beff[CF_MAX_NODES][CF_MAX_COMP];
  // a node's second configuration: executors vrep - vrep1 of batch vbatch2 and GPUs index vtp2,
  // tenths vw of its requests to the first (0: one configuration), its demand and effective batches
  __shared__ uint8_t vrep1[CF_MAX_NODES], vw[CF_MAX_NODES], vtp2[CF_MAX_NODES];
  __shared__ uint16_t vbatch2[CF_MAX_NODES];
  __shared__ uint16_t beff2[CF_MAX_NODES][CF_MAX_COMP];
  __shared__ double u2_s[CF_MAX_NODES];
  __shared__ int groups_bad;
  __shared__ uint8_t route[CF_MAX_TYPES][2][CF_MAX_COMP];
  __shared__ uint8_t nalt[CF_MAX_TYPES], aw[CF_MAX_TYPES][2];
  __shared__ double ex_s[CF_MAX_TYPES][CF_MAX_COMP], en_s[CF_MAX_TYPES][CF_MAX_COMP];
  __shared__ double u_s[CF_MAX_NODES];
  __shared__ uint32_t met_s[CF_MAX_TYPES], cnt_s[CF_MAX_TYPES];
  __shared__ int valid_s;
  // per-type model fields indexed by a lane's request type (kernel arguments
  // indexed per lane would be one memory round trip each)
  __shared__ uint64_t child_s[CF_MAX_TYPES];  // byte c: the non-streaming children of c
  __shared__ uint32_t tinfo_s[CF_MAX_TYPES];  // path | outm << 8 | pfo << 16 | gen_out << 24
  __shared__ int8_t ta_s[CF_MAX_TYPES], th_s[CF_MAX_TYPES];
  __shared__ double slo_s[CF_MAX_TYPES][4];
  __shared__ uint32_t hist_s[CF_MAX_TYPES * 65];
  const int i = blockIdx.x, lane = threadIdx.x;
  const int p = V.ids[i];
  const size_t P = (size_t)V.P;
  if (lane < CF_MAX_TYPES) {
    met_s[lane] = 0;
    cnt_s[lane] = 0;
  }
  if (lane == 0) valid_s = 0;
  if (lane < CF_MAX_TYPES) {
    uint64_t ch = 0;
#pragma unroll
    for (int c = 0; c < CF_MAX_COMP; c++) ch |= (uint64_t)m.child[lane][c] << (8 * c);
    child_s[lane] = ch;
    tinfo_s[lane] = (m.path[lane] & 0xFFu) | ((m.outm[lane] & 0xFFu) << 8) | ((m.pfo[lane] & 0xFFu) << 16) |
                    ((uint32_t)(m.gen_out[lane] ? 1 : 0) << 24);
    ta_s[lane] = m.ta_c[lane];
    th_s[lane] = m.th_c[lane];
  }
  if (lane < CF_MAX_TYPES * 4) (&slo_s[0][0])[lane] = (&m.slo[0][0])[lane];
  (&tps_s[0][0])[lane] = (&m.tps[0][0])[lane];
  const int hw = V.nb + 1;  // histogram row width
  if (V.hist)
    for (int q = lane; q < m.nt * hw; q += 64) hist_s[q] = 0;
  // per-type means of X and of the output length (phase 1's work per request)
  if (lane < m.nt * m.nc) {
    const int t = lane / m.nc, c = lane % m.nc;
    const uint64_t *mo = V.moments + (size_t)t * 8;
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
  const bool in_range = p >= 0 && p < V.P;
  const int nv = in_range ? V.n_nodes[p] : 0;
  if (lane == 0) groups_bad = 0;
  __syncthreads();
  if (in_range && lane < CF_MAX_NODES) {
    const uint32_t rep = lane < nv ? V.node_rep[lane * P + p] : 0;
    const uint32_t rep2 = (lane < nv && V.node_rep2) ? V.node_rep2[lane * P + p] : 0;
    vcomp[lane] = lane < nv ? V.node_comp[lane * P + p] : 0;
    vrep[lane] = (uint8_t)(rep + rep2 < 255 ? rep + rep2 : 255);
    vrep1[lane] = (uint8_t)rep;
    vbatch[lane] = lane < nv ? V.node_batch[lane * P + p] : 0;
    const uint32_t g = lane < nv ? V.node_gpus[lane * P + p] : 1u;
    vtp[lane] = (uint8_t)(g < 1 ? 0 : (g > 8 ? 7 : g - 1));
    const uint32_t w = rep2 ? V.node_w[lane * P + p] : 0u;
    const uint32_t b2 = rep2 ? V.node_batch2[lane * P + p] : 0u;
    const uint32_t g2 = rep2 ? V.node_gpus2[lane * P + p] : 1u;
    vw[lane] = (uint8_t)w;
    vbatch2[lane] = (uint16_t)b2;
    vtp2[lane] = (uint8_t)(g2 < 1 ? 0 : (g2 > 8 ? 7 : g2 - 1));
    if (rep2 && (rep < 1 || w < 1 || w > 9 || b2 < 1 || b2 > CF_MAX_BATCH || g2 < 1)) atomicOr(&groups_bad, 1);
  }
  if (in_range) {
    for (int j = lane; j < CF_MAX_TYPES * 2 * CF_MAX_COMP; j += 64) (&route[0][0][0])[j] = V.alt_node[j * P + p];
    if (lane < CF_MAX_TYPES) nalt[lane] = lane < m.nt ? V.n_alt[lane * P + p] : 0;
    if (lane < 2 * CF_MAX_TYPES) (&aw[0][0])[lane] = V.alt_w[lane * P + p];
  }
  __syncthreads();
  // validity (phase 1's), capacities, effective batches: one lane, phase 1's order
  if (lane == 0 && in_range) {
    bool ok = nv >= 1 && nv <= CF_MAX_NODES && !groups_bad;
    int execs = 0;
    for (int v = 0; v < nv && ok; v++) {
      const int cm = vcomp[v], rep = vrep[v], b = vbatch[v];
      if (cm == 0 || (cm >> m.nc) || rep < 1 || b < 1 || b > CF_MAX_BATCH || V.node_gpus[v * P + p] < 1) ok = false;
      vminc[v] = (uint8_t)(cm ? __ffs(cm) - 1 : 0);
      vbase[v] = (uint8_t)(execs < 255 ? execs : 255);
      execs += rep;
    }
    if (execs > CF_MAX_EXEC) ok = false;
    for (int t = 0; t < m.nt && ok; t++) {
      const int na = nalt[t];
      if (na < 1 || na > 2) { ok = false; break; }
      for (int a = 0; a < na && ok; a++) {
        if (na > 1 && aw[t][a] < 1) ok = false;
        for (int c = 0; c < m.nc; c++) {
          if (!((m.path[t] >> c) & 1u)) continue;
          const int v = route[t][a][c];
          if (v >= nv || !((vcomp[v] >> c) & 1u)) { ok = false; break; }
        }
      }
    }
    if (ok) {
      for (int v = 0; v < CF_MAX_NODES; v++) u_s[v] = u2_s[v] = 0.0;
      const double wsum = (double)m.wsum;
      for (int t = 0; t < m.nt; t++) {
        const double pi = (double)m.weight[t] / wsum;
        const int na = nalt[t];
        uint32_t wtot = 0;
        for (int a = 0; a < na; a++) wtot += na > 1 ? aw[t][a] : 1u;
        for (int a = 0; a < na; a++) {
          const uint32_t wa = na > 1 ? aw[t][a] : 1u;
          const double q = (double)wa / (double)wtot;
          const double pq = pi * q;
          for (int c = 0; c < m.nc; c++) {
            if (!((m.path[t] >> c) & 1u)) continue;
            const int v = route[t][a][c];
            // seconds of executor time per request on each configuration of the node
            for (int k = 0; k < (vw[v] ? 2 : 1); k++) {
              const int bn = k ? vbatch2[v] : vbatch[v];
              const double B = (double)(bn < m.cap[c] ? bn : m.cap[c]);
              double w = ((m.k0[c] / B) + m.k1[c] * ex_s[t][c]) + m.k2[c];
              if (m.kind[c] == CF_LLM) w = w + (en_s[t][c] - 1.0) * ((m.d0[c] / B) + m.d1[c]);
              if (m.tp_any) w = tps_s[c][k ? vtp2[v] : vtp[v]] * w;
              if (!vw[v]) u_s[v] = u_s[v] + pq * w;
              else if (k == 0) u_s[v] = u_s[v] + (pq * ((double)vw[v] / 10.0)) * w;
              else u2_s[v] = u2_s[v] + (pq * ((double)(10u - vw[v]) / 10.0)) * w;
            }
          }
        }
      }
      const double R_d = V.rd[p];
      for (int v = 0; v < nv; v++) {
        // effective batch per configuration: its share of the bottleneck's load
        for (int k = 0; k < (vw[v] ? 2 : 1); k++) {
          const double u = k ? u2_s[v] : u_s[v];
          const double Rv = u > 0.0 ? (double)(k ? vrep[v] - vrep1[v] : vrep1[v]) / u : __builtin_inf();
          const double q = R_d / Rv;
          for (int c = 0; c < m.nc; c++) {
            const int bn = k ? vbatch2[v] : vbatch[v];
            const int B = bn < m.cap[c] ? bn : m.cap[c];
            const double bb = ceil((double)B * q);
            (k ? beff2 : beff)[v][c] = (uint16_t)(bb < 1.0 ? 1 : (bb > (double)B ? B : (int)bb));
          }
        }
      }
      valid_s = 1;
    }
  }
  __syncthreads();
  if (valid_s) {
    const double comm = m.comm;
    for (int j = lane; j < V.n_sample; j += 64) {
      const int r = (int)V.order[j];
      const size_t o = V.toff + (size_t)r;
      const int t = V.type[o];
      if (t >= m.nt) continue;
      int alt = 0;
      if (nalt[t] == 2) {
        const uint64_t w0 = aw[t][0], w1 = aw[t][1];
        alt = ((((uint64_t)V.akey[o]) * (w0 + w1)) >> 32) < w0 ? 0 : 1;
      }
      const uint64_t k0 = V.rkey0[o], k1 = V.rkey1[o];
      McReq q;
      q.prompt = V.prompt[o];
      q.out = V.out[o];
      q.patches = V.patches[o];
      q.aud_in = V.aud_in[o];
      q.aud_out = V.aud_out[o];
      const int ta = ta_s[t], th = th_s[t];
      const uint64_t child = child_s[t];
      const uint32_t tinfo = tinfo_s[t];
      const uint32_t path = tinfo & 0xFFu, outm = (tinfo >> 8) & 0xFFu, pfo = (tinfo >> 16) & 0xFFu;
      int ex[CF_MAX_COMP], nout[CF_MAX_COMP];
      double fin[CF_MAX_COMP], first[CF_MAX_COMP], dstep[CF_MAX_COMP];
      int ttft_c = -1;
      double completion = 0.0, media = 0.0;
#pragma unroll
      for (int c = 0; c < CF_MAX_COMP; c++) {
        ex[c] = 0;
        nout[c] = 1;
        fin[c] = 0.0;
        first[c] = 0.0;
        dstep[c] = 0.0;
      }
#pragma unroll
      for (int c = 0; c < CF_MAX_COMP; c++) {
        if (c >= m.nc || !((path >> c) & 1u)) continue;
        const int v = route[t][alt][c];
        const int mc = vminc[v];
        const uint64_t key = ((mc < 4 ? k0 : k1) >> (16 * (mc & 3))) & 0xFFFFull;
        const int j = node_exec((uint32_t)key, vrep1[v], (uint32_t)(vrep[v] - vrep1[v]), vw[v]);
        const bool second = j >= vrep1[v];  // an executor of the node's second configuration
        ex[c] = vbase[v] + j;
        // the last input to arrive
        double start = 0.0;
#pragma unroll
        for (int pc = 0; pc < c; pc++) {
          const bool gate_edge = c == ta && pc == th;
          if (!(((child >> (8 * pc + c)) & 1u) || gate_edge)) continue;
          const double hop = ex[pc] == ex[c] ? 0.0 : comm;
          const double ready = gate_edge ? first[pc] + hop : fin[pc] + hop;
          start = ready > start ? ready : start;
        }
        const int b = second ? beff2[v][c] : beff[v][c];
        const double tps = tps_s[c][second ? vtp2[v] : vtp[v]];
        uint32_t x = 0;
        for (uint32_t sel = m.xsel[c]; sel; sel &= sel - 1) x += mc_attr(q, __ffs(sel) - 1);
        if (m.kind[c] != CF_LLM) {
          double dur = (m.k0[c] + m.k1[c] * (double)((uint64_t)b * x)) + m.k2[c] * (double)b;
          if (m.tp_any) dur = tps * dur;
          fin[c] = start + dur;
          first[c] = fin[c];
        } else {
          double dur = (m.k0[c] + m.k1[c] * (double)x) + m.k2[c] * 1.0;
          if (m.tp_any) dur = tps * dur;
          uint32_t no = ((pfo >> c) & 1u) ? 1u : mc_attr(q, m.nout_attr[c]);
          no = no < 1 ? 1u : no;
          nout[c] = (int)no;
          double D = m.d0[c] + m.d1[c] * (double)b;
          if (m.tp_any) D = tps * D;
          dstep[c] = D;
          first[c] = start + dur;
          double e = first[c];
          if (c != ta) {
            uint32_t taken = 0;
            e = run_walk(e, D, no - 1u, __builtin_inf(), &taken);
          } else {
            // the gate source's tokens: its first token, then one step of dstep each
            double eg = 0.0, dg = 0.0, hop = 0.0;
            int ng = 1;
#pragma unroll
            for (int s2 = 0; s2 < c; s2++) {
              if (s2 == th) {
                eg = first[s2];
                dg = dstep[s2];
                ng = nout[s2];
                hop = ex[s2] == ex[c] ? 0.0 : comm;
              }
            }
            int jg = 1;
            for (int k = 1; k < (int)no; k++) {
              const int need = k + 1 < ng ? k + 1 : ng;
              if (jg < need) {
                eg = eg + dg;
                jg++;
              }
              const double vis = eg + hop;
              const double s = e < vis ? vis : e;
              e = s + D;
            }
          }
          fin[c] = e;
          if (ttft_c < 0) ttft_c = c;
        }
        if ((outm >> c) & 1u) {
          completion = fin[c] > completion ? fin[c] : completion;
          if (m.kind[c] == CF_GEN) media = fin[c] > media ? fin[c] : media;
        }
      }
      double ttft = 0.0, tpot = 0.0;
#pragma unroll
      for (int c = 0; c < CF_MAX_COMP; c++) {
        if (c == ttft_c) {
          ttft = first[c];
          if (nout[c] > 1) tpot = (fin[c] - first[c]) / (double)(nout[c] - 1);
        }
      }
      const double md = (tinfo >> 24) ? media : 0.0;
      const bool ok = ttft <= slo_s[t][0] && tpot <= slo_s[t][1] && completion <= slo_s[t][2] && md <= slo_s[t][3];
      atomicAdd(&cnt_s[t], 1u);
      if (ok) atomicAdd(&met_s[t], 1u);
      if (V.hist) atomicAdd(&hist_s[t * hw + target_bin(V.tg, V.nb, t, ttft, tpot, completion, md)], 1u);
      if (V.lat) {
        double *L = V.lat + ((size_t)i * V.n_sample + r) * 4;
        L[0] = ttft;
        L[1] = tpot;
        L[2] = completion;
        L[3] = md;
      }
    }
  }
  __syncthreads();
  if (lane < m.nt) {
    const size_t oi = (size_t)i * m.nt + lane;
    const uint32_t mt = met_s[lane], ct = cnt_s[lane];
    V.met[oi] = mt;
    V.cnt[oi] = ct;
    double g = 0.0;
    if (valid_s && ct > 0) {
      const double pi = (double)m.weight[lane] / (double)m.wsum;
      g = ((V.alpha * V.rd[p]) * pi) * ((double)mt / (double)ct);
    }
    V.gt[oi] = g;
  }
  if (V.hist) {
    for (int q = lane; q < m.nt * hw; q += 64) V.hist[(size_t)i * m.nt * hw + q] = hist_s[q];
    // the CDF at each bin: requests in bins 0..b over the type's count
    for (int q = lane; q < V.nb * m.nt; q += 64) {
      const int b = q / m.nt, t = q - b * m.nt;
      uint32_t h = 0;
      for (int k = 0; k <= b; k++) h += hist_s[t * hw + k];
      const uint32_t ct = cnt_s[t];
      double g = 0.0;
      if (valid_s && ct > 0) {
        const double pi = (double)m.weight[t] / (double)m.wsum;
        g = ((V.alpha * V.rd[p]) * pi) * ((double)h / (double)ct);
      }
      V.curve[((size_t)i * V.nb + b) * m.nt + t] = g;
    }
  }
}

// Pareto pruning, keep[i] = 0 iff another row j of g[n][T] is >= in every
// component and > in one.  Dominance is a strict partial order on finitely
// many rows, so a dominated row is dominated by some row that nothing
// dominates, and such a row is never pruned.  Two passes use this:
//   1. each block of kParBlock consecutive rows prunes the rows another row
//      of the same block dominates and lists its survivors;
//   2. each survivor is tested against the survivors of every block (which
//      include every undominated row), a block stopping once all of its
//      survivors are dominated.
// The result is the plain all-pairs definition; the work is n * kParBlock
// plus (survivors)^2 comparisons instead of n^2.
constexpr int kParBlock = 256;

__device__ __forceinline__ bool dominates(const double *a, const double *b, int T) {
  bool ge = true, gt = false;
#pragma unroll
  for (int t = 0; t < CF_MAX_TYPES; t++) {
    if (t < T) {
      ge = ge && !(a[t] < b[t]);
      gt = gt || a[t] > b[t];
    }
  }
  return ge && gt;
}

__device__ __forceinline__ void prune(int i, uint8_t *keep, const int32_t *plan_ids, uint8_t *flags, int n_flags,
                                      bool dominated) {
  keep[i] = dominated ? 0 : 1;
  if (flags && dominated) {
    const int p = plan_ids[i];
    if (p >= 0 && p < n_flags) flags[p] = (uint8_t)(flags[p] & ~CF_FLAG_KEEP);
  }
}

__global__ void __launch_bounds__(kParBlock) k_pareto_local(const double *g, int n, int T, uint8_t *keep,
                                                            const int32_t *plan_ids, uint8_t *flags, int n_flags,
                                                            int32_t *surv, int32_t *surv_n) {
  __shared__ double tile[kParBlock * CF_MAX_TYPES];
  __shared__ int cnt_s;
  const int i0 = blockIdx.x * kParBlock, i = i0 + threadIdx.x;
  const int cnt = n - i0 < kParBlock ? n - i0 : kParBlock;
  if (threadIdx.x == 0) cnt_s = 0;
  for (int q = threadIdx.x; q < cnt * T; q += kParBlock) tile[q] = g[(size_t)i0 * T + q];
  __syncthreads();
  if (i < n) {
    double mine[CF_MAX_TYPES];
#pragma unroll
    for (int t = 0; t < CF_MAX_TYPES; t++) mine[t] = t < T ? tile[threadIdx.x * T + t] : 0.0;
    bool dominated = false;
    for (int jj = 0; jj < cnt && !dominated; jj++) {
      double other[CF_MAX_TYPES];
#pragma unroll
      for (int t = 0; t < CF_MAX_TYPES; t++) other[t] = t < T ? tile[jj * T + t] : 0.0;
      dominated = jj != (int)threadIdx.x && dominates(other, mine, T);
    }
    if (dominated)
      prune(i, keep, plan_ids, flags, n_flags, true);
    else
      surv[i0 + atomicAdd(&cnt_s, 1)] = i;
  }
  __syncthreads();
  if (threadIdx.x == 0) surv_n[blockIdx.x] = cnt_s;
}

__global__ void __launch_bounds__(kParBlock) k_pareto_global(const double *g, int n, int T, uint8_t *keep,
                                                             const int32_t *plan_ids, uint8_t *flags, int n_flags,
                                                             const int32_t *surv, const int32_t *surv_n) {
  __shared__ double tile[kParBlock * CF_MAX_TYPES];
  const int nb = (n + kParBlock - 1) / kParBlock;
  const int b = blockIdx.x, ns = surv_n[b];
  const int i = (int)threadIdx.x < ns ? surv[b * kParBlock + threadIdx.x] : -1;
  double mine[CF_MAX_TYPES];
#pragma unroll
  for (int t = 0; t < CF_MAX_TYPES; t++) mine[t] = (i >= 0 && t < T) ? g[(size_t)i * T + t] : 0.0;
  bool dominated = false;
  for (int b2 = 0; b2 < nb; b2++) {
    const int n2 = surv_n[b2];
    for (int q = threadIdx.x; q < n2 * T; q += kParBlock) {
      const int k = q / T, t = q - k * T;
      tile[q] = g[(size_t)surv[b2 * kParBlock + k] * T + t];
    }
    __syncthreads();
    if (i >= 0 && !dominated) {
      for (int k = 0; k < n2; k++) {
        double other[CF_MAX_TYPES];
#pragma unroll
        for (int t = 0; t < CF_MAX_TYPES; t++) other[t] = t < T ? tile[k * T + t] : 0.0;
        if (dominates(other, mine, T)) {
          dominated = true;
          break;
        }
      }
    }
    // also the barrier before the next tile overwrites this one
    if (!__syncthreads_or(i >= 0 && !dominated)) break;
  }
  if (i >= 0) prune(i, keep, plan_ids, flags, n_flags, dominated);
}

}  // namespace
}  // namespace cf

namespace cf {
namespace {
cf_status eval_mc(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev, int32_t n_plans,
                  const double *rd_dev, const uint64_t *moments_dev, double alpha, const cf_trace *trace,
                  int32_t seed_idx, int32_t n_sample, uint32_t *met_dev, uint32_t *cnt_dev, double *goodput_t_dev,
                  double *lat_dev, int32_t n_bins, const double *targets_host, uint32_t *hist_dev, double *curve_dev,
                  void *stream) {
  KModel m;
  cf_status st = lower_model(model, &m);
  if (st != CF_OK) return st;
  if (!plans || !trace) return set_error(CF_EINVAL, "NULL argument");
  if (n_plans < 0 || n_sample < 0 || plans->P < 0) return set_error(CF_EINVAL, "sizes");
  if (n_plans == 0) return CF_OK;
  if (!plan_ids_dev || !rd_dev || !moments_dev || !met_dev || !cnt_dev || !goodput_t_dev)
    return set_error(CF_EINVAL, "NULL device array");
  if (!(alpha > 0.0) || !(alpha <= 1.0)) return set_error(CF_EINVAL, "alpha must be in (0, 1]");
  if (seed_idx < 0 || seed_idx >= trace->n_seeds || n_sample > trace->n_req)
    return set_error(CF_EINVAL, "seed_idx or n_sample outside the trace");
  McView V;
  V.P = plans->P;
  V.n_nodes = plans->n_nodes_dev;
  V.node_comp = plans->node_comp_dev;
  V.node_rep = plans->node_rep_dev;
  V.node_gpus = plans->node_gpus_dev;
  V.n_alt = plans->n_alt_dev;
  V.alt_w = plans->alt_w_dev;
  V.alt_node = plans->alt_node_dev;
  V.node_batch = plans->node_batch_dev;
  {
    const int ng = (plans->node_rep2_dev != nullptr) + (plans->node_batch2_dev != nullptr) +
                   (plans->node_gpus2_dev != nullptr) + (plans->node_w_dev != nullptr);
    if (ng != 0 && ng != 4) return set_error(CF_EINVAL, "second-configuration arrays: all four or none");
  }
  V.node_rep2 = plans->node_rep2_dev;
  V.node_batch2 = plans->node_batch2_dev;
  V.node_gpus2 = plans->node_gpus2_dev;
  V.node_w = plans->node_w_dev;
  V.ids = plan_ids_dev;
  V.rd = rd_dev;
  V.moments = moments_dev;
  V.alpha = alpha;
  V.ticks = trace->arr_ticks_dev;
  V.rkey0 = trace->rkey0_dev;
  V.rkey1 = trace->rkey1_dev;
  V.type = trace->type_dev;
  V.patches = trace->patches_dev;
  V.prompt = trace->prompt_dev;
  V.out = trace->out_dev;
  V.aud_in = trace->aud_in_ms_dev;
  V.aud_out = trace->aud_out_ms_dev;
  V.akey = trace->akey_dev;
  V.toff = (size_t)seed_idx * (size_t)trace->n_req;
  V.n_sample = n_sample;
  V.met = met_dev;
  V.cnt = cnt_dev;
  V.gt = goodput_t_dev;
  V.lat = lat_dev;
  V.order = nullptr;
  V.tg = nullptr;
  V.nb = 0;
  V.hist = nullptr;
  V.curve = nullptr;
  if (n_bins > 0) {
    if (!hist_dev || !curve_dev) return set_error(CF_EINVAL, "NULL histogram or curve array");
    if ((st = load_targets(m.nt, n_bins, targets_host, &V.tg, as_stream(stream))) != CF_OK) return st;
    V.nb = n_bins;
    V.hist = hist_dev;
    V.curve = curve_dev;
  }
  if (n_sample > 0) {
    uint32_t *order = (uint32_t *)scratch_get(SCR_MC, sizeof(uint32_t) * (size_t)n_sample, &st);
    if (!order) return st;
    hipLaunchKernelGGL(k_mc_order, dim3(1), dim3(kOrdThreads), 0, as_stream(stream), m, V, order);
    st = hip_check(hipGetLastError(), "cf_eval_mc order launch");
    if (st != CF_OK) return st;
    V.order = order;
  }
  hipLaunchKernelGGL(k_mc, dim3((unsigned)n_plans), dim3(64), 0, as_stream(stream), m, V);
  return hip_check(hipGetLastError(), "cf_eval_mc launch");
}
}  // namespace
}  // namespace cf

extern "C" cf_status cf_eval_mc(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev,
                                int32_t n_plans, const double *rd_dev, const uint64_t *moments_dev, double alpha,
                                const cf_trace *trace, int32_t seed_idx, int32_t n_sample, uint32_t *met_dev,
                                uint32_t *cnt_dev, double *goodput_t_dev, double *lat_dev, void *stream) {
  return cf::eval_mc(model, plans, plan_ids_dev, n_plans, rd_dev, moments_dev, alpha, trace, seed_idx, n_sample,
                     met_dev, cnt_dev, goodput_t_dev, lat_dev, 0, nullptr, nullptr, nullptr, stream);
}

extern "C" cf_status cf_eval_mc_curve(const cf_model_desc *model, const cf_plan_table *plans,
                                      const int32_t *plan_ids_dev, int32_t n_plans, const double *rd_dev,
                                      const uint64_t *moments_dev, double alpha, const cf_trace *trace,
                                      int32_t seed_idx, int32_t n_sample, int32_t n_bins,
                                      const double *hist_targets_host, uint32_t *met_dev, uint32_t *cnt_dev,
                                      double *goodput_t_dev, uint32_t *hist_dev, double *curve_dev, void *stream) {
  if (n_bins < 1) return cf::set_error(CF_EINVAL, "n_bins must be in 1..64");
  return cf::eval_mc(model, plans, plan_ids_dev, n_plans, rd_dev, moments_dev, alpha, trace, seed_idx, n_sample,
                     met_dev, cnt_dev, goodput_t_dev, nullptr, n_bins, hist_targets_host, hist_dev, curve_dev,
                     stream);
}

extern "C" cf_status cf_pareto(const double *goodput_t_dev, int32_t n, int32_t T, uint8_t *keep_dev,
                               const int32_t *plan_ids_dev, uint8_t *flags_dev, int32_t n_flags, void *stream) {
  using namespace cf;
  if (n < 0 || T < 1 || T > CF_MAX_TYPES) return set_error(CF_EINVAL, "sizes");
  if ((plan_ids_dev == nullptr) != (flags_dev == nullptr))
    return set_error(CF_EINVAL, "plan_ids_dev and flags_dev are given together or not at all");
  if (flags_dev && n_flags < 0) return set_error(CF_EINVAL, "n_flags");
  if (n == 0) return CF_OK;
  if (!goodput_t_dev || !keep_dev) return set_error(CF_EINVAL, "NULL device array");
  const int nb = (n + kParBlock - 1) / kParBlock;
  cf_status st = CF_OK;
  int32_t *surv = (int32_t *)scratch_get(SCR_PARETO, sizeof(int32_t) * ((size_t)nb * kParBlock + nb), &st);
  if (!surv) return st;
  int32_t *surv_n = surv + (size_t)nb * kParBlock;
  hipLaunchKernelGGL(k_pareto_local, dim3((unsigned)nb), dim3(kParBlock), 0, as_stream(stream), goodput_t_dev, n, T,
                     keep_dev, plan_ids_dev, flags_dev, n_flags, surv, surv_n);
  st = hip_check(hipGetLastError(), "cf_pareto launch");
  if (st != CF_OK) return st;
  hipLaunchKernelGGL(k_pareto_global, dim3((unsigned)nb), dim3(kParBlock), 0, as_stream(stream), goodput_t_dev, n, T,
                     keep_dev, plan_ids_dev, flags_dev, n_flags, surv, surv_n);
  return hip_check(hipGetLastError(), "cf_pareto launch");
}
