// k_fine.hip -- cf_eval_fine: phase 3 of the plan evaluation (Sec. 4.3,
// Alg. 2), the request-level simulation of every (plan, rate, seed) triple.
//
// One wavefront simulates one triple; a persistent grid of wavefronts takes
// triples from an atomic ticket, seed-major so that concurrent wavefronts
// read the same seed's trace (L2 / MALL reuse).
//
// The event structure needs no heap.  Pending times are
//   - the end of the running iteration of each executor (lane x holds
//     executor x; the next one is a wavefront min-reduction),
//   - the next external arrival (requests arrive in id order),
//   - the head of one FIFO delay line: every remote delivery and wake-up is
//     delayed by the same comm, so production order is due-time order.
// Per instant: iterations ending at t complete in executor order, delayed
// deliveries due at t then arrivals at t are applied, and every executor
// whose state changed since it went idle may start one iteration.
//
// Memory: executor state and the plan in LDS; stage queues as chunked
// lists in a per-wavefront pool in HBM; LLM running sets as ordered slot
// arrays; per-request state in HBM, indexed by request id.
//
// Decode steps of a non-gated LLM stage cost O(1): a running request's
// token count is (decode steps of its stage since it joined) + 1, so each
// running slot stores the step index at which it finishes and only the
// finishing slots are touched.  The gated stage (talker) keeps per-request
// token counts; visibility of thinker tokens comes from the request's join
// step in the thinker's stage and a ring of that stage's recent step end
// times.
#include <stdlib.h>
#include <string.h>

#include "cf_internal.h"

namespace cf {
namespace {

constexpr int kMaxSI = CF_MAX_EXEC * CF_MAX_COMP;  // stage instances
constexpr int kChunk = 64;                          // queue chunk entries
constexpr int kHist = 64;                           // thinker step-time ring
constexpr uint32_t kNone = 0xFFFFFFFFu;

enum { IT_BATCH = 0, IT_PREFILL = 1, IT_DECODE = 2 };
enum { DL_DELIVER = 0, DL_TICK = 1 };
constexpr uint32_t FL_TH_DONE = 16u;   // rs_flags: thinker finished; low 4 bits: outputs left
constexpr uint32_t MARK = 0x80000000u; // gated running slot: in the current decode step

struct Layout {
  size_t si_comp, si_exec, si_beff, si_qhc, si_qhp, si_qtc, si_qtp, si_qn, si_roff, si_rn, si_iter, si_minfin,
      si_hist;
  size_t run_r, run_k, hist, mem, dl_t, dl_v, pool, pool_next, pool_free;
  size_t rs_ex, rs_join, rs_flags, rs_tfirst, rs_tlast, rs_tmedia, rs_thjoin;
  size_t bytes;
  int run_cap, hist_slots, n_chunks;
  uint32_t dl_mask;
};

struct FineArgs {
  KModel m;
  // plans
  int P;
  const uint8_t *n_nodes, *node_comp, *node_rep, *n_alt, *alt_w, *alt_node;
  const uint16_t *node_batch;
  const int32_t *plan_ids;
  int n_plans;
  const double *rates;
  int K;
  // trace
  const uint64_t *ticks, *rkey0, *rkey1;
  const uint8_t *type;
  const uint16_t *patches, *prompt, *out;
  const uint32_t *aud_in, *aud_out, *akey;
  int S, n;
  // outputs
  uint32_t *met, *cnt, *status;
  uint64_t *events;
  double *lat;
  const int32_t *lat_triples;
  int n_lat;
  // scratch
  char *slab;
  Layout L;
  unsigned int *ticket;
  unsigned int total;
};

struct WaveShared {
  double ex_tend[CF_MAX_EXEC];
  double ex_last[CF_MAX_EXEC];
  uint32_t ex_st[CF_MAX_EXEC];  // busy:1 ran:1 kind:2 rr:4 cur:4 nmem:9
  uint16_t ex_first[CF_MAX_EXEC];
  uint8_t ex_ns[CF_MAX_EXEC], ex_node[CF_MAX_EXEC];
  uint8_t route[CF_MAX_TYPES][2][CF_MAX_COMP];
  uint8_t nalt[CF_MAX_TYPES], aw[CF_MAX_TYPES][2];
  uint8_t vbase[CF_MAX_NODES + 1], vrep[CF_MAX_NODES], vminc[CF_MAX_NODES], vcomp[CF_MAX_NODES];
  uint16_t vbatch[CF_MAX_NODES];
  uint32_t met[CF_MAX_TYPES], cnt[CF_MAX_TYPES];
};

__device__ __forceinline__ int lane_id() { return threadIdx.x; }
__device__ __forceinline__ uint32_t ru(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int ri(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t ru64(uint64_t v) {
  return ((uint64_t)ru((uint32_t)(v >> 32)) << 32) | ru((uint32_t)v);
}
__device__ __forceinline__ double rd(double v) { return __longlong_as_double((long long)ru64((uint64_t)__double_as_longlong(v))); }

__device__ __forceinline__ double wave_min(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    double w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}
__device__ __forceinline__ uint32_t wave_min_u(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}
__device__ __forceinline__ uint32_t wave_sum_u(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ uint32_t lanes_below(uint64_t bal) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
}

// All mutable per-triple state that is not in LDS; lives in registers.
struct Sim {
  const FineArgs *A;
  WaveShared *sh;
  // slab arrays
  uint8_t *si_comp, *si_exec;
  uint16_t *si_beff;
  int *si_qhc, *si_qhp, *si_qtc, *si_qtp, *si_qn, *si_roff, *si_rn, *si_hist;
  uint32_t *si_iter, *si_minfin, *run_r, *run_k, *mem, *dl_v, *pool, *rs_join, *rs_flags, *rs_thjoin;
  int *pool_next, *pool_free;
  double *hist, *dl_t, *rs_tfirst, *rs_tlast, *rs_tmedia;
  uint64_t *rs_ex;
  // scalars
  size_t soff;
  double lam, now;
  uint64_t events, dirty, ta_exec_mask;
  uint32_t status, dl_head, dl_tail;
  int pool_top, pool_fresh, n_done, nx, lat_slot;
  bool remote_gate;
};

// ------------------------------------------------------------------ trace
__device__ __forceinline__ uint32_t attr(const Sim &S, uint32_t r, int a) {
  const size_t o = S.soff + r;
  const FineArgs &A = *S.A;
  switch (a) {
    case CF_ATTR_PROMPT: return A.prompt[o];
    case CF_ATTR_OUT: return A.out[o];
    case CF_ATTR_PATCHES: return A.patches[o];
    case CF_ATTR_AUDIN_MS: return A.aud_in[o];
    case CF_ATTR_AUDOUT_MS: return A.aud_out[o];
    case CF_ATTR_AUDIN_TOK: return (A.aud_in[o] + 79u) / 80u;
    case CF_ATTR_AUDOUT_TOK: return (A.aud_out[o] + 79u) / 80u;
    default: return 0;
  }
}

__device__ __forceinline__ uint32_t x_of(const Sim &S, uint32_t r, int c) {
  uint32_t sel = S.A->m.xsel[c], x = 0;
  while (sel) {
    const int a = __ffs(sel) - 1;
    sel &= sel - 1;
    x += attr(S, r, a);
  }
  return x;
}

__device__ __forceinline__ int type_of(const Sim &S, uint32_t r) { return S.A->type[S.soff + r]; }

__device__ __forceinline__ uint32_t nout_of(const Sim &S, uint32_t r, int t, int c) {
  if ((S.A->m.pfo[t] >> c) & 1u) return 1;
  const uint32_t v = attr(S, r, S.A->m.nout_attr[c]);
  return v < 1 ? 1 : v;
}

__device__ __forceinline__ double arrival_time(const Sim &S, uint32_t r) {
  return ((double)S.A->ticks[S.soff + r] * 0x1p-32) / S.lam;
}

__device__ __forceinline__ int exec_of(const Sim &S, uint32_t r, int c) { return (int)((S.rs_ex[r] >> (8 * c)) & 0xFFu); }

__device__ __forceinline__ int stage_of(const Sim &S, int x, int c) {
  const int v = S.sh->ex_node[x];
  return S.sh->ex_first[x] + __popc((uint32_t)S.sh->vcomp[v] & ((1u << c) - 1u));
}

// ------------------------------------------------------------------ pool / queues
__device__ __forceinline__ int chunk_alloc(Sim &S) {
  if (S.pool_top > 0) return S.pool_free[--S.pool_top];
  if (S.pool_fresh < S.A->L.n_chunks) return S.pool_fresh++;
  S.status |= CF_ST_OVERFLOW;
  return -1;
}
__device__ __forceinline__ void chunk_free(Sim &S, int c) {
  if (c >= 0 && c < S.A->L.n_chunks && S.pool_top < S.A->L.n_chunks) S.pool_free[S.pool_top++] = c;
  else S.status |= CF_ST_OVERFLOW;
}

__device__ void q_push(Sim &S, int si, uint32_t r) {
  int qn = S.si_qn[si], tc = S.si_qtc[si], tp = S.si_qtp[si];
  if (qn > 0 && (tc < 0 || tc >= S.A->L.n_chunks || tp < 0 || tp > kChunk)) {
    S.status |= CF_ST_OVERFLOW;
    return;
  }
  if (qn == 0) {
    const int c = chunk_alloc(S);
    if (c < 0) return;
    S.si_qhc[si] = c;
    S.si_qhp[si] = 0;
    tc = c;
    tp = 0;
  } else if (tp == kChunk) {
    const int c = chunk_alloc(S);
    if (c < 0) return;
    S.pool_next[tc] = c;
    tc = c;
    tp = 0;
  }
  S.pool[(size_t)tc * kChunk + tp] = r;
  S.si_qtc[si] = tc;
  S.si_qtp[si] = tp + 1;
  S.si_qn[si] = qn + 1;
}

// pops the first k entries of stage si's queue into mem[dst..dst+k)
__device__ void q_pop(Sim &S, int si, int k, uint32_t *dst) {
  int hc = S.si_qhc[si], hp = S.si_qhp[si];
  const int tc = S.si_qtc[si], tp = S.si_qtp[si];
  if (k <= 0) return;
  if (k > S.si_qn[si] || hc < 0 || hc >= S.A->L.n_chunks) {  // never on a consistent queue
    S.status |= CF_ST_OVERFLOW;
    return;
  }
  int got = 0;
  while (got < k) {
    const int lim = (hc == tc) ? tp : kChunk;
    int take = lim - hp;
    if (take > k - got) take = k - got;
    if (take <= 0 || hc < 0 || hc >= S.A->L.n_chunks) {
      S.status |= CF_ST_OVERFLOW;
      break;
    }
    if (lane_id() < take) dst[got + lane_id()] = S.pool[(size_t)hc * kChunk + hp + lane_id()];
    got += take;
    hp += take;
    if (hp == kChunk && got < k) {
      const int nx = S.pool_next[hc];
      chunk_free(S, hc);
      hc = nx;
      hp = 0;
    }
  }
  if (got < k) {
    __syncthreads();
    return;
  }
  const int qn = S.si_qn[si] - k;
  S.si_qn[si] = qn;
  if (qn == 0) {
    chunk_free(S, hc);
  } else if (hp == kChunk) {
    const int nx = S.pool_next[hc];
    if (nx < 0 || nx >= S.A->L.n_chunks) S.status |= CF_ST_OVERFLOW;
    chunk_free(S, hc);
    hc = nx;
    hp = 0;
  }
  S.si_qhc[si] = hc;
  S.si_qhp[si] = hp;
  __syncthreads();
}

__device__ __forceinline__ void dl_push(Sim &S, double due, uint32_t v) {
  if (S.dl_tail - S.dl_head > S.A->L.dl_mask) {
    S.status |= CF_ST_OVERFLOW;
    return;
  }
  S.dl_t[S.dl_tail & S.A->L.dl_mask] = due;
  S.dl_v[S.dl_tail & S.A->L.dl_mask] = v;
  S.dl_tail++;
}

// ------------------------------------------------------------------ request flow
__device__ void enqueue(Sim &S, uint32_t r, int c, int x) {
  S.events++;
  q_push(S, stage_of(S, x, c), r);
  S.dirty |= 1ull << x;
}

__device__ void join(Sim &S, uint32_t r, int c) {
  const uint32_t j = S.rs_join[r] + (1u << (4 * c));
  S.rs_join[r] = j;
  const int t = type_of(S, r);
  if (((j >> (4 * c)) & 15u) == S.A->m.npar[t][c]) enqueue(S, r, c, exec_of(S, r, c));
}

__device__ __forceinline__ void deliver(Sim &S, uint32_t r, int c2, int xfrom) {
  if (exec_of(S, r, c2) == xfrom) join(S, r, c2);
  else dl_push(S, S.now + S.A->m.comm, (r << 4) | (DL_DELIVER << 3) | (uint32_t)c2);
}

__device__ void complete_request(Sim &S, uint32_t r) {
  const KModel &m = S.A->m;
  S.events++;
  S.n_done++;
  const int t = type_of(S, r);
  const double a = arrival_time(S, r);
  double ttft = 0.0, tpot = 0.0, media = 0.0;
  const int tc = m.ttft_c[t];
  if (tc >= 0) {
    const double tf = S.rs_tfirst[r];
    ttft = tf - a;
    const uint32_t n1 = nout_of(S, r, t, tc);
    if (n1 > 1) tpot = (S.rs_tlast[r] - tf) / (double)(n1 - 1);
  }
  const double e2e = S.now - a;
  if (m.gen_out[t]) media = S.rs_tmedia[r] - a;
  const bool ok = ttft <= m.slo[t][0] && tpot <= m.slo[t][1] && e2e <= m.slo[t][2] && media <= m.slo[t][3];
  S.sh->cnt[t] += 1;
  if (ok) S.sh->met[t] += 1;
  if (S.lat_slot >= 0) {
    double *L = S.A->lat + ((size_t)S.lat_slot * S.A->n + r) * 4;
    L[0] = ttft;
    L[1] = tpot;
    L[2] = e2e;
    L[3] = media;
  }
}

// request r finishes component c on executor x at S.now
__device__ void finish(Sim &S, uint32_t r, int c, int x) {
  const KModel &m = S.A->m;
  const int t = type_of(S, r);
  uint32_t ch = m.child[t][c];
  while (ch) {
    const int c2 = __ffs(ch) - 1;
    ch &= ch - 1;
    deliver(S, r, c2, x);
  }
  if (c == m.th_c[t]) S.rs_flags[r] |= FL_TH_DONE;
  if ((m.outm[t] >> c) & 1u) {
    if (m.kind[c] == CF_GEN) S.rs_tmedia[r] = S.now;
    const uint32_t f = S.rs_flags[r] - 1u;
    S.rs_flags[r] = f;
    if ((f & 15u) == 0) complete_request(S, r);
  }
}

__device__ void arrive(Sim &S, uint32_t r) {
  const KModel &m = S.A->m;
  const FineArgs &A = *S.A;
  const WaveShared &sh = *S.sh;
  S.events++;
  const size_t o = S.soff + r;
  const int t = A.type[o];
  if (t >= m.nt) { S.status |= CF_ST_INVALID; return; }
  int alt = 0;
  if (sh.nalt[t] == 2) {
    const uint64_t w0 = sh.aw[t][0], w1 = sh.aw[t][1];
    alt = ((((uint64_t)A.akey[o]) * (w0 + w1)) >> 32) < w0 ? 0 : 1;
  }
  const uint64_t k0 = A.rkey0[o], k1 = A.rkey1[o];
  uint64_t ex = ~0ull;
  uint32_t path = m.path[t];
  while (path) {
    const int c = __ffs(path) - 1;
    path &= path - 1;
    const int v = sh.route[t][alt][c];
    const int mc = sh.vminc[v];
    const uint64_t key = ((mc < 4 ? k0 : k1) >> (16 * (mc & 3))) & 0xFFFFull;
    const int x = sh.vbase[v] + (int)((key * sh.vrep[v]) >> 16);
    ex = (ex & ~(0xFFull << (8 * c))) | ((uint64_t)x << (8 * c));
  }
  S.rs_ex[r] = ex;
  S.rs_join[r] = 0;
  S.rs_flags[r] = (uint32_t)__popc(m.outm[t]);
  uint32_t src = m.srcm[t];
  while (src) {
    const int c = __ffs(src) - 1;
    src &= src - 1;
    enqueue(S, r, c, exec_of(S, r, c));
  }
}

// ------------------------------------------------------------------ gating
// Is thinker token k of request r (gate source th on executor xth) visible
// at S.now to a talker on executor x?
__device__ __forceinline__ bool token_visible(const Sim &S, uint32_t r, int t, int th, int xth, int x, uint32_t k,
                                              uint32_t nth, bool &undecided) {
  const double delta = (xth == x) ? 0.0 : S.A->m.comm;
  double e;
  if (k <= 1) {
    e = S.rs_tfirst[r];
  } else if ((S.rs_flags[r] & FL_TH_DONE) && k == nth) {
    e = S.rs_tlast[r];
  } else {
    const int si = stage_of(S, xth, th);
    const uint32_t q = S.rs_thjoin[r] + k - 1u;
    const uint32_t it = S.si_iter[si];
    if (q > it) return false;
    const double *h = S.hist + (size_t)S.si_hist[si] * kHist;
    if (it - q < (uint32_t)kHist) {
      e = h[q & (kHist - 1)];
    } else {
      e = h[(it - (kHist - 1)) & (kHist - 1)];  // oldest kept: token k is no later
      if (!(e + delta <= S.now)) { undecided = true; return false; }
    }
  }
  return e + delta <= S.now;
}

// ------------------------------------------------------------------ iterations
__device__ void start_iter(Sim &S, int x, int l, int si, int c, int kind) {
  const KModel &m = S.A->m;
  WaveShared &sh = *S.sh;
  double dur;
  int nmem = 0;
  if (kind != IT_DECODE) {
    const int qn = S.si_qn[si];
    const int beff = S.si_beff[si];
    const int room = kind == IT_PREFILL ? beff - S.si_rn[si] : beff;
    const int n = qn < room ? qn : room;
    uint32_t *dst = S.mem + (size_t)x * CF_MAX_BATCH;
    q_pop(S, si, n, dst);
    if (S.status & CF_ST_OVERFLOW) return;  // the triple is abandoned at the end of this instant
    uint32_t xs = 0;
    for (int b = 0; b < n; b += 64) {
      const int j = b + lane_id();
      xs += (j < n) ? x_of(S, dst[j], c) : 0u;
    }
    xs = ru(wave_sum_u(xs));
    dur = (m.k0[c] + m.k1[c] * (double)xs) + m.k2[c] * (double)n;
    if (m.kind[c] == CF_ENC) {
      const bool ran = (sh.ex_st[x] >> 1) & 1u;
      if (!ran || sh.ex_last[x] < S.now) dur = dur + m.cpu_pre;
    }
    nmem = n;
  } else if (!((m.gated_mask >> c) & 1u)) {
    const int rn = S.si_rn[si];
    dur = m.d0[c] + m.d1[c] * (double)rn;
    nmem = rn;
  } else {
    // gated stage: mark the eligible running requests
    const int rn = S.si_rn[si];
    uint32_t *rr = S.run_r + S.si_roff[si];
    uint32_t *rk = S.run_k + S.si_roff[si];
    uint32_t cntm = 0;
    bool undecided = false;
    for (int b = 0; b < rn; b += 64) {
      const int j = b + lane_id();
      if (j < rn) {
        const uint32_t r = rr[j];
        const uint32_t tok = rk[j] & 0xFFFFu;
        const int t = type_of(S, r);
        bool el = true;
        if (S.A->m.ta_c[t] == c) {
          const int th = S.A->m.th_c[t];
          const uint32_t nth = nout_of(S, r, t, th);
          const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
          el = token_visible(S, r, t, th, exec_of(S, r, th), x, k, nth, undecided);
        }
        rk[j] = el ? (tok | MARK) : tok;
        cntm += el ? 1u : 0u;
      }
    }
    if (__ballot(undecided)) S.status |= CF_ST_OVERFLOW;
    cntm = ru(wave_sum_u(cntm));
    __syncthreads();
    dur = m.d0[c] + m.d1[c] * (double)cntm;
    nmem = (int)cntm;
  }
  const double tend = S.now + dur;
  sh.ex_tend[x] = tend;
  sh.ex_st[x] = (sh.ex_st[x] & 2u) | 1u | ((uint32_t)kind << 2) | ((uint32_t)l << 4) | ((uint32_t)l << 8) |
                ((uint32_t)nmem << 12);
}

// does stage si (component c) of executor x have runnable work now?
__device__ int runnable_kind(Sim &S, int x, int si, int c) {
  const KModel &m = S.A->m;
  const int qn = S.si_qn[si];
  if (m.kind[c] != CF_LLM) return qn > 0 ? IT_BATCH : -1;
  const int rn = S.si_rn[si];
  if (qn > 0 && rn < (int)S.si_beff[si]) return IT_PREFILL;
  if (rn == 0) return -1;
  if (!((m.gated_mask >> c) & 1u)) return IT_DECODE;
  const uint32_t *rr = S.run_r + S.si_roff[si];
  const uint32_t *rk = S.run_k + S.si_roff[si];
  bool any = false, undecided = false;
  for (int b = 0; b < rn && !any; b += 64) {
    const int j = b + lane_id();
    bool el = false;
    if (j < rn) {
      const uint32_t r = rr[j];
      const int t = type_of(S, r);
      el = true;
      if (m.ta_c[t] == c) {
        const int th = m.th_c[t];
        const uint32_t nth = nout_of(S, r, t, th);
        const uint32_t tok = rk[j] & 0xFFFFu;
        const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
        el = token_visible(S, r, t, th, exec_of(S, r, th), x, k, nth, undecided);
      }
    }
    any = __ballot(el) != 0;
  }
  if (__ballot(undecided)) S.status |= CF_ST_OVERFLOW;
  return any ? IT_DECODE : -1;
}

__device__ void try_start(Sim &S, int x) {
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[x];
  const int ns = sh.ex_ns[x], first = sh.ex_first[x];
  const int rr = (st >> 4) & 15u;
  for (int i = 0; i < ns; i++) {
    const int l = (rr == 15) ? i : (rr + 1 + i) % ns;
    const int si = first + l;
    const int c = S.si_comp[si];
    const int kind = runnable_kind(S, x, si, c);
    if (kind >= 0) {
      start_iter(S, x, l, si, c, kind);
      return;
    }
  }
}

__device__ void thinker_tick(Sim &S) {
  if (S.remote_gate) dl_push(S, S.now + S.A->m.comm, (DL_TICK << 3));
}

// compact the running slots of stage si, dropping slots whose key equals drop
// (compressed) or whose token count reached n_out (gated, fin flags).
__device__ void run_compact(Sim &S, int si, bool gated, uint32_t drop_key, const bool *fin_lane) {
  const int rn = S.si_rn[si];
  uint32_t *rr = S.run_r + S.si_roff[si];
  uint32_t *rk = S.run_k + S.si_roff[si];
  uint32_t vr[CF_MAX_BATCH / 64], vk[CF_MAX_BATCH / 64];
  bool keep[CF_MAX_BATCH / 64];
#pragma unroll
  for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
    const int j = p * 64 + lane_id();
    keep[p] = false;
    vr[p] = 0;
    vk[p] = 0;
    if (j < rn) {
      vr[p] = rr[j];
      vk[p] = rk[j];
      keep[p] = gated ? !fin_lane[p] : (vk[p] != drop_key);
    }
  }
  __syncthreads();
  uint32_t w = 0, mn = kNone;
#pragma unroll
  for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
    const uint64_t bal = __ballot(keep[p]);
    if (keep[p]) {
      const uint32_t d = w + lanes_below(bal);
      rr[d] = vr[p];
      rk[d] = vk[p];
      mn = vk[p] < mn ? vk[p] : mn;
    }
    w += (uint32_t)__popcll(bal);
  }
  __syncthreads();
  S.si_rn[si] = (int)ru(w);
  if (!gated) S.si_minfin[si] = ru(wave_min_u(mn));
}

__device__ void complete_iter(Sim &S, int x) {
  const KModel &m = S.A->m;
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[x];
  const int kind = (st >> 2) & 3u, l = (st >> 8) & 15u, nmem = (st >> 12) & 511u;
  const int si = sh.ex_first[x] + l;
  const int c = S.si_comp[si];
  sh.ex_st[x] = (st & ~1u) | 2u;  // idle, has run
  sh.ex_last[x] = S.now;
  S.dirty |= 1ull << x;
  const bool is_th = (m.gate_src_mask >> c) & 1u;
  if (kind == IT_BATCH) {
    const uint32_t *mem = S.mem + (size_t)x * CF_MAX_BATCH;
    for (int i = 0; i < nmem; i++) {
      const uint32_t r = ru(mem[i]);
      S.events++;
      finish(S, r, c, x);
    }
  } else if (kind == IT_PREFILL) {
    const uint32_t *mem = S.mem + (size_t)x * CF_MAX_BATCH;
    const bool gated = (m.gated_mask >> c) & 1u;
    const uint32_t iter = S.si_iter[si];
    int rn = S.si_rn[si];
    uint32_t mn = S.si_minfin[si];
    uint32_t *rr = S.run_r + S.si_roff[si];
    uint32_t *rk = S.run_k + S.si_roff[si];
    for (int i = 0; i < nmem; i++) {
      const uint32_t r = ru(mem[i]);
      const int t = type_of(S, r);
      S.events++;
      if (c == m.ttft_c[t]) {
        S.rs_tfirst[r] = S.now;
        S.rs_tlast[r] = S.now;
      }
      const uint32_t no = nout_of(S, r, t, c);
      if (c == m.th_c[t]) {
        S.rs_thjoin[r] = iter;
        deliver(S, r, m.ta_c[t], x);  // token 1: the talker receives the request
      }
      if (no == 1) {
        finish(S, r, c, x);
      } else {
        const uint32_t key = gated ? 1u : iter + no - 1u;
        rr[rn] = r;
        rk[rn] = key;
        rn++;
        if (!gated && key < mn) mn = key;
      }
    }
    S.si_rn[si] = rn;
    if (!gated) S.si_minfin[si] = mn;
    if (is_th) thinker_tick(S);
  } else if (!((m.gated_mask >> c) & 1u)) {
    const uint32_t it = S.si_iter[si] + 1u;
    S.si_iter[si] = it;
    const int rn = S.si_rn[si];
    S.events += (uint64_t)rn;
    if (is_th) S.hist[(size_t)S.si_hist[si] * kHist + (it & (kHist - 1))] = S.now;
    if (it == S.si_minfin[si]) {
      const uint32_t *rr = S.run_r + S.si_roff[si];
      const uint32_t *rk = S.run_k + S.si_roff[si];
      for (int b = 0; b < rn; b += 64) {
        const int j = b + lane_id();
        uint64_t bal = __ballot(j < rn && rk[j] == it);
        while (bal) {
          const int jj = b + __ffsll((long long)bal) - 1;
          bal &= bal - 1;
          const uint32_t r = ru(rr[jj]);
          const int t = type_of(S, r);
          if (c == m.ttft_c[t]) S.rs_tlast[r] = S.now;
          finish(S, r, c, x);
        }
      }
      run_compact(S, si, false, it, nullptr);
    }
    if (is_th) thinker_tick(S);
  } else {
    // gated decode step: every marked slot gains one token
    const int rn = S.si_rn[si];
    uint32_t *rr = S.run_r + S.si_roff[si];
    uint32_t *rk = S.run_k + S.si_roff[si];
    S.si_iter[si] = S.si_iter[si] + 1u;
    bool fin[CF_MAX_BATCH / 64];
    uint32_t part = 0;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
      const int j = p * 64 + lane_id();
      fin[p] = false;
      if (j < rn) {
        const uint32_t v = rk[j];
        if (v & MARK) {
          const uint32_t r = rr[j];
          const uint32_t tok = (v & 0xFFFFu) + 1u;
          rk[j] = tok;
          part++;
          fin[p] = tok == nout_of(S, r, type_of(S, r), c);
        }
      }
    }
    S.events += (uint64_t)ru(wave_sum_u(part));
    __syncthreads();
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
      uint64_t bal = __ballot(fin[p]);
      while (bal) {
        const int jj = p * 64 + __ffsll((long long)bal) - 1;
        bal &= bal - 1;
        const uint32_t r = ru(rr[jj]);
        const int t = type_of(S, r);
        if (c == m.ttft_c[t]) S.rs_tlast[r] = S.now;
        finish(S, r, c, x);
      }
    }
    run_compact(S, si, true, 0, fin);
    if (is_th) thinker_tick(S);
  }
}

// ------------------------------------------------------------------ setup
__device__ bool setup_plan(Sim &S, int p) {
  const FineArgs &A = *S.A;
  const KModel &m = A.m;
  WaveShared &sh = *S.sh;
  const size_t P = (size_t)A.P;
  const int lane = lane_id();
  const int nv = A.n_nodes[p];
  if (nv < 1 || nv > CF_MAX_NODES) return false;
  if (lane < CF_MAX_NODES) {
    sh.vcomp[lane] = lane < nv ? A.node_comp[lane * P + p] : 0;
    sh.vrep[lane] = lane < nv ? A.node_rep[lane * P + p] : 0;
    sh.vbatch[lane] = lane < nv ? A.node_batch[lane * P + p] : 0;
  }
  for (int j = lane; j < CF_MAX_TYPES * 2 * CF_MAX_COMP; j += 64) (&sh.route[0][0][0])[j] = A.alt_node[j * P + p];
  if (lane < CF_MAX_TYPES) sh.nalt[lane] = lane < m.nt ? A.n_alt[lane * P + p] : 0;
  if (lane < 2 * CF_MAX_TYPES) (&sh.aw[0][0])[lane] = A.alt_w[lane * P + p];
  __syncthreads();
  int base = 0;
  for (int v = 0; v < nv; v++) {
    const int cm = sh.vcomp[v], rep = sh.vrep[v], b = sh.vbatch[v];
    if (cm == 0 || (cm >> m.nc) || rep < 1 || b < 1 || b > CF_MAX_BATCH) return false;
    sh.vminc[v] = (uint8_t)(__ffs(cm) - 1);
    sh.vbase[v] = (uint8_t)(base < 255 ? base : 255);
    base += rep;
  }
  if (base > CF_MAX_EXEC) return false;
  S.nx = base;
  S.remote_gate = false;
  for (int t = 0; t < m.nt; t++) {
    const int na = sh.nalt[t];
    if (na < 1 || na > 2) return false;
    for (int a = 0; a < na; a++) {
      if (na > 1 && sh.aw[t][a] < 1) return false;
      uint32_t path = m.path[t];
      while (path) {
        const int c = __ffs(path) - 1;
        path &= path - 1;
        const int v = sh.route[t][a][c];
        if (v >= nv || !((sh.vcomp[v] >> c) & 1u)) return false;
      }
      if (m.th_c[t] >= 0 && sh.route[t][a][m.th_c[t]] != sh.route[t][a][m.ta_c[t]]) S.remote_gate = true;
    }
  }
  // executors and stage instances
  int si = 0, roff = 0, hs = 0;
  S.ta_exec_mask = 0;
  for (int v = 0; v < nv; v++) {
    const int cm = sh.vcomp[v];
    for (int j = 0; j < sh.vrep[v]; j++) {
      const int x = sh.vbase[v] + j;
      sh.ex_node[x] = (uint8_t)v;
      sh.ex_first[x] = (uint16_t)si;
      sh.ex_ns[x] = (uint8_t)__popc(cm);
      sh.ex_st[x] = 15u << 4;  // idle, never ran, no stage run yet
      sh.ex_tend[x] = __builtin_inf();
      sh.ex_last[x] = 0.0;
      if (cm & m.gated_mask) S.ta_exec_mask |= 1ull << x;
      uint32_t cc = (uint32_t)cm;
      while (cc) {
        const int c = __ffs(cc) - 1;
        cc &= cc - 1;
        if (si >= kMaxSI) return false;
        const int beff = sh.vbatch[v] < m.cap[c] ? sh.vbatch[v] : m.cap[c];
        S.si_comp[si] = (uint8_t)c;
        S.si_exec[si] = (uint8_t)x;
        S.si_beff[si] = (uint16_t)beff;
        S.si_qn[si] = 0;
        S.si_qhc[si] = -1;
        S.si_qtc[si] = -1;
        S.si_qhp[si] = 0;
        S.si_qtp[si] = 0;
        S.si_rn[si] = 0;
        S.si_iter[si] = 0;
        S.si_minfin[si] = kNone;
        S.si_roff[si] = roff;
        S.si_hist[si] = -1;
        if (m.kind[c] == CF_LLM) roff += beff;
        if ((m.gate_src_mask >> c) & 1u) S.si_hist[si] = hs++;
        si++;
      }
    }
  }
  if (roff > A.L.run_cap || hs > A.L.hist_slots) {
    S.status |= CF_ST_OVERFLOW;
    return true;
  }
  return true;
}

__global__ void __launch_bounds__(64) k_fine(const FineArgs *__restrict__ Ap) {
  __shared__ WaveShared sh;
  const FineArgs &A = *Ap;
  Sim S;
  S.A = Ap;
  S.sh = &sh;
  char *slab = A.slab + (size_t)blockIdx.x * A.L.bytes;
  const Layout &L = A.L;
  S.si_comp = (uint8_t *)(slab + L.si_comp);
  S.si_exec = (uint8_t *)(slab + L.si_exec);
  S.si_beff = (uint16_t *)(slab + L.si_beff);
  S.si_qhc = (int *)(slab + L.si_qhc);
  S.si_qhp = (int *)(slab + L.si_qhp);
  S.si_qtc = (int *)(slab + L.si_qtc);
  S.si_qtp = (int *)(slab + L.si_qtp);
  S.si_qn = (int *)(slab + L.si_qn);
  S.si_roff = (int *)(slab + L.si_roff);
  S.si_rn = (int *)(slab + L.si_rn);
  S.si_iter = (uint32_t *)(slab + L.si_iter);
  S.si_minfin = (uint32_t *)(slab + L.si_minfin);
  S.si_hist = (int *)(slab + L.si_hist);
  S.run_r = (uint32_t *)(slab + L.run_r);
  S.run_k = (uint32_t *)(slab + L.run_k);
  S.hist = (double *)(slab + L.hist);
  S.mem = (uint32_t *)(slab + L.mem);
  S.dl_t = (double *)(slab + L.dl_t);
  S.dl_v = (uint32_t *)(slab + L.dl_v);
  S.pool = (uint32_t *)(slab + L.pool);
  S.pool_next = (int *)(slab + L.pool_next);
  S.pool_free = (int *)(slab + L.pool_free);
  S.rs_ex = (uint64_t *)(slab + L.rs_ex);
  S.rs_join = (uint32_t *)(slab + L.rs_join);
  S.rs_flags = (uint32_t *)(slab + L.rs_flags);
  S.rs_tfirst = (double *)(slab + L.rs_tfirst);
  S.rs_tlast = (double *)(slab + L.rs_tlast);
  S.rs_tmedia = (double *)(slab + L.rs_tmedia);
  S.rs_thjoin = (uint32_t *)(slab + L.rs_thjoin);
  const int lane = lane_id();
  const KModel &m = A.m;
  const unsigned int per_seed = (unsigned int)A.n_plans * (unsigned int)A.K;
  for (;;) {
    unsigned int tk = 0;
    if (lane == 0) tk = atomicAdd(A.ticket, 1u);
    tk = ru(__shfl(tk, 0, 64));
    if (tk >= A.total) break;
    const int s = (int)(tk / per_seed);
    const unsigned int rem = tk % per_seed;
    const int i = (int)(rem / (unsigned)A.K), k = (int)(rem % (unsigned)A.K);
    const int p = ri(A.plan_ids[i]);
    const size_t oidx = ((size_t)i * A.K + k) * A.S + s;
    S.soff = (size_t)s * A.n;
    S.lam = rd(A.rates[(size_t)i * A.K + k]);
    S.events = 0;
    S.status = 0;
    S.dirty = 0;
    S.dl_head = S.dl_tail = 0;
    S.pool_top = 0;
    S.pool_fresh = 0;
    S.n_done = 0;
    S.now = 0.0;
    S.lat_slot = -1;
    for (int j = 0; j < A.n_lat; j++)
      if (A.lat_triples[j] == (int32_t)oidx) S.lat_slot = j;
    if (lane < CF_MAX_TYPES) { sh.met[lane] = 0; sh.cnt[lane] = 0; }
    __syncthreads();
    const bool ok = (p >= 0 && p < A.P) && S.lam > 0.0 && S.lam < __builtin_inf() && setup_plan(S, p);
    if (!ok) S.status |= CF_ST_INVALID;
    if (ok && !(S.status & CF_ST_OVERFLOW) && A.n > 0 && S.lam > 0.0) {
      uint32_t next_arr = 0;
      double t_arr = arrival_time(S, 0);
      uint64_t instants = 0;
      for (;;) {
        // --- next pending time
        double te = __builtin_inf();
        if (lane < S.nx && (sh.ex_st[lane] & 1u)) te = sh.ex_tend[lane];
        te = rd(wave_min(te));
        const double tdl = (S.dl_head != S.dl_tail) ? S.dl_t[S.dl_head & L.dl_mask] : __builtin_inf();
        double t = te < tdl ? te : tdl;
        t = t_arr < t ? t_arr : t;
        if (t == __builtin_inf()) break;
        S.now = t;
        if (++instants > 2 * S.events + 16ull * (uint64_t)A.n + 4096ull) { S.status |= CF_ST_DEADLOCK; break; }
        // --- step 1: iterations ending at t, ascending executor
        uint64_t done = __ballot(lane < S.nx && (sh.ex_st[lane] & 1u) && sh.ex_tend[lane] == t);
        __syncthreads();
        while (done) {
          const int x = __ffsll((long long)done) - 1;
          done &= done - 1;
          complete_iter(S, x);
        }
        // --- step 2: delayed deliveries due at t (production order), then arrivals at t
        while (S.dl_head != S.dl_tail && S.dl_t[S.dl_head & L.dl_mask] == t) {
          const uint32_t v = S.dl_v[S.dl_head & L.dl_mask];
          S.dl_head++;
          if (((v >> 3) & 1u) == DL_TICK) S.dirty |= S.ta_exec_mask;
          else join(S, v >> 4, (int)(v & 7u));
        }
        while (next_arr < (uint32_t)A.n && t_arr == t) {
          arrive(S, next_arr);
          next_arr++;
          t_arr = next_arr < (uint32_t)A.n ? arrival_time(S, next_arr) : __builtin_inf();
        }
        // --- step 3: idle executors whose state changed may start an iteration
        uint64_t cand = S.dirty;
        S.dirty = 0;
        __syncthreads();
        while (cand) {
          const int x = __ffsll((long long)cand) - 1;
          cand &= cand - 1;
          if (!(sh.ex_st[x] & 1u)) try_start(S, x);
        }
        __syncthreads();
        if (S.status & (CF_ST_OVERFLOW | CF_ST_INVALID)) break;
      }
      if (S.n_done < A.n && !(S.status & (CF_ST_OVERFLOW | CF_ST_INVALID))) S.status |= CF_ST_DEADLOCK;
    }
    __syncthreads();
    if (lane < m.nt) {
      A.met[oidx * m.nt + lane] = sh.met[lane];
      A.cnt[oidx * m.nt + lane] = sh.cnt[lane];
    }
    if (lane == 0) {
      A.events[oidx] = S.events;
      A.status[oidx] = S.status;
    }
  }
}

__global__ void k_fine_reset(unsigned int *ticket) { *ticket = 0u; }

Layout make_layout(const KModel &m, int n) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  L.si_comp = take(kMaxSI);
  L.si_exec = take(kMaxSI);
  L.si_beff = take(2 * kMaxSI);
  L.si_qhc = take(4 * kMaxSI);
  L.si_qhp = take(4 * kMaxSI);
  L.si_qtc = take(4 * kMaxSI);
  L.si_qtp = take(4 * kMaxSI);
  L.si_qn = take(4 * kMaxSI);
  L.si_roff = take(4 * kMaxSI);
  L.si_rn = take(4 * kMaxSI);
  L.si_iter = take(4 * kMaxSI);
  L.si_minfin = take(4 * kMaxSI);
  L.si_hist = take(4 * kMaxSI);
  int per_exec_run = 0, n_th = 0;
  for (int c = 0; c < m.nc; c++) {
    if (m.kind[c] == CF_LLM) per_exec_run += m.cap[c] < CF_MAX_BATCH ? m.cap[c] : CF_MAX_BATCH;
    if ((m.gate_src_mask >> c) & 1u) n_th++;
  }
  L.run_cap = CF_MAX_EXEC * per_exec_run;
  L.hist_slots = CF_MAX_EXEC * n_th;
  L.run_r = take(4 * (size_t)L.run_cap);
  L.run_k = take(4 * (size_t)L.run_cap);
  L.hist = take(8 * (size_t)L.hist_slots * kHist);
  L.mem = take(4 * (size_t)CF_MAX_EXEC * CF_MAX_BATCH);
  size_t dl = 4096;
  while (dl < 2 * (size_t)n + 8192) dl <<= 1;
  L.dl_mask = (uint32_t)(dl - 1);
  L.dl_t = take(8 * dl);
  L.dl_v = take(4 * dl);
  const int maxq = m.max_path > 0 ? m.max_path : 1;
  L.n_chunks = (int)(((size_t)n * maxq + kChunk - 1) / kChunk) + 2 * kMaxSI + 16;
  L.pool = take(4 * (size_t)L.n_chunks * kChunk);
  L.pool_next = take(4 * (size_t)L.n_chunks);
  L.pool_free = take(4 * (size_t)L.n_chunks);
  L.rs_ex = take(8 * (size_t)n);
  L.rs_join = take(4 * (size_t)n);
  L.rs_flags = take(4 * (size_t)n);
  L.rs_tfirst = take(8 * (size_t)n);
  L.rs_tlast = take(8 * (size_t)n);
  L.rs_tmedia = take(8 * (size_t)n);
  L.rs_thjoin = take(4 * (size_t)n);
  L.bytes = (off + 4095) & ~(size_t)4095;
  return L;
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_eval_fine(const cf_model_desc *model, const cf_plan_table *plans,
                                  const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev, int32_t K,
                                  const cf_trace *trace, uint32_t flags, const cf_fine_out *out, void *stream) {
  using namespace cf;
  FineArgs a;
  memset(&a, 0, sizeof a);
  cf_status st = lower_model(model, &a.m);
  if (st != CF_OK) return st;
  if (!plans || !trace || !out) return set_error(CF_EINVAL, "NULL argument");
  if (flags != 0) return set_error(CF_EUNSUPPORTED, "flags must be 0");
  if (n_plans < 0 || K < 1 || trace->n_seeds < 1 || trace->n_req < 0 || plans->P < 0)
    return set_error(CF_EINVAL, "sizes");
  if (n_plans == 0) return CF_OK;
  if (!plan_ids_dev || !rates_dev) return set_error(CF_EINVAL, "NULL argument");
  if (!out->met_dev || !out->cnt_dev || !out->events_dev || !out->status_dev)
    return set_error(CF_EINVAL, "NULL output array");
  if (out->lat_dev && (out->n_lat < 0 || (out->n_lat > 0 && !out->lat_triples_dev)))
    return set_error(CF_EINVAL, "latency dump arguments");
  if (trace->n_req > (1 << 26)) return set_error(CF_ECAPACITY, "n_req above 2^26");
  const unsigned long long total = (unsigned long long)n_plans * K * trace->n_seeds;
  if (total >= 0xFFFFFFFFull - 65536ull) return set_error(CF_ECAPACITY, "too many triples in one call");
  if (total == 0) return CF_OK;
  a.P = plans->P;
  a.n_nodes = plans->n_nodes_dev;
  a.node_comp = plans->node_comp_dev;
  a.node_rep = plans->node_rep_dev;
  a.node_batch = plans->node_batch_dev;
  a.n_alt = plans->n_alt_dev;
  a.alt_w = plans->alt_w_dev;
  a.alt_node = plans->alt_node_dev;
  a.plan_ids = plan_ids_dev;
  a.n_plans = n_plans;
  a.rates = rates_dev;
  a.K = K;
  a.ticks = trace->arr_ticks_dev;
  a.rkey0 = trace->rkey0_dev;
  a.rkey1 = trace->rkey1_dev;
  a.type = trace->type_dev;
  a.patches = trace->patches_dev;
  a.prompt = trace->prompt_dev;
  a.out = trace->out_dev;
  a.aud_in = trace->aud_in_ms_dev;
  a.aud_out = trace->aud_out_ms_dev;
  a.akey = trace->akey_dev;
  a.S = trace->n_seeds;
  a.n = trace->n_req;
  a.met = out->met_dev;
  a.cnt = out->cnt_dev;
  a.events = out->events_dev;
  a.status = out->status_dev;
  a.lat = out->lat_dev;
  a.lat_triples = out->lat_triples_dev;
  a.n_lat = out->lat_dev ? out->n_lat : 0;
  a.L = make_layout(a.m, trace->n_req);
  a.total = (unsigned int)total;
  long long waves = 4096;
  if (const char *e = getenv("CF_FINE_WAVES")) waves = atoll(e);
  if (waves < 1) waves = 1;
  if ((unsigned long long)waves > total) waves = (long long)total;
  // keep the per-wave state within a fixed share of device memory
  size_t free_b = 0, tot_b = 0;
  if (hipMemGetInfo(&free_b, &tot_b) == hipSuccess && free_b > 0) {
    const size_t budget = free_b / 2;
    while (waves > 64 && (size_t)waves * a.L.bytes > budget) waves /= 2;
  }
  const size_t hdr = 4096;
  char *scr = (char *)scratch_get(SCR_FINE, hdr + (size_t)waves * a.L.bytes, &st);
  if (!scr) return st;
  a.ticket = (unsigned int *)scr;
  FineArgs *args_dev = (FineArgs *)(scr + 256);
  static_assert(sizeof(FineArgs) + 256 <= 4096, "FineArgs must fit the scratch header");
  a.slab = scr + hdr;
  hipStream_t s = as_stream(stream);
  st = hip_check(hipMemcpyAsync(args_dev, &a, sizeof a, hipMemcpyHostToDevice, s), "copy fine args");
  if (st != CF_OK) return st;
  hipLaunchKernelGGL(k_fine_reset, dim3(1), dim3(1), 0, s, a.ticket);
  hipLaunchKernelGGL(k_fine, dim3((unsigned)waves), dim3(64), 0, s, (const FineArgs *)args_dev);
  st = hip_check(hipGetLastError(), "cf_eval_fine launch");
  if (st != CF_OK) return st;
  // the argument block is read by the kernel: the host copy must stay valid
  // until the copy has happened
  return hip_check(hipStreamSynchronize(s), "cf_eval_fine sync");
}
