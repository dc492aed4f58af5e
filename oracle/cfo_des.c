/*
 * cfo_des.c -- oracle (test infrastructure only): the request-level
 * simulator of phase 3 (Sec. 4.3, Alg. 2 phase 3), written as a plain
 * discrete-event simulation over one binary heap of all pending events.
 *
 * The paper states what the simulator models (the full request processing
 * pipeline with queueing and inter-type interaction at shared nodes, run at
 * a given aggregate rate, producing per-type throughput and latency CDFs),
 * plus CPU-GPU overlap in encoders and a fixed communication delay on every
 * disaggregated edge (Sec. 5.2).  It does not give a scheduling policy;
 * the rules implemented here are the repository's readings:
 *
 *  - an executor (one replica of a node) is a serial server whose stages are
 *    the node's components in index order; stages are served round-robin,
 *    starting after the stage that ran last, and the first stage with
 *    runnable work runs one iteration;
 *  - ENC/GEN: a batch of the first min(|queue|, B) queued requests,
 *    duration (k0 + k1*X) + k2*n;  an ENC batch that starts on an executor
 *    that was idle (previous iteration ended strictly earlier, or none)
 *    also pays the CPU preprocessing time;
 *  - LLM: iteration-level batching with prefill priority: if requests wait
 *    and fewer than B run, admit the first min(|wait|, B-|run|) and prefill
 *    them ((k0 + k1*X) + k2*n); otherwise one decode step over the eligible
 *    running requests (d0 + d1*n);
 *  - a request finishing a component is delivered to each child on its
 *    path: immediately on the same executor, after comm otherwise; a
 *    component with several parents starts when all have delivered;
 *  - a gated LLM (talker) receives the request when the gate source
 *    (thinker) has emitted its first token and that token is visible; a
 *    running talker request with j tokens may decode only when thinker token
 *    min(j+1, n_thinker) is visible (emitted at e, visible at e + delta,
 *    delta = 0 on the same executor, comm otherwise);
 *  - instants: at the smallest pending time t, first every iteration ending
 *    at t completes (ascending executor id), then every delayed delivery
 *    due at t (in the order produced), then every arrival at t (ascending
 *    request id), then every idle executor may start one iteration.
 *
 * The request-event count (the unit of the throughput metric) adds, per
 * request: 1 arrival, per component visited 1 enqueue plus one per batch or
 * iteration it takes part in, and 1 completion.
 */
#include "cfo.h"
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define P_AT(arr, slot, P, p) ((arr)[(size_t)(slot) * (size_t)(P) + (size_t)(p)])

/* ---------- small growable integer array used as FIFO or ordered list ---------- */
typedef struct { int *a; int head, n, cap; } ivec;

static void iv_push(ivec *v, int x) {
  if (v->head + v->n == v->cap) {
    if (v->head > 0) {
      memmove(v->a, v->a + v->head, sizeof(int) * (size_t)v->n);
      v->head = 0;
    }
    if (v->n == v->cap) {
      v->cap = v->cap ? 2 * v->cap : 16;
      v->a = (int *)realloc(v->a, sizeof(int) * (size_t)v->cap);
    }
  }
  v->a[v->head + v->n] = x;
  v->n++;
}
static int iv_at(const ivec *v, int i) { return v->a[v->head + i]; }
static int iv_pop_front(ivec *v) { int x = v->a[v->head]; v->head++; v->n--; return x; }

/* ---------- event heap: ordered by (time, class, key) ---------- */
enum { EV_DONE = 0, EV_DELAY = 1, EV_ARRIVE = 2 };
enum { DL_DELIVER = 0, DL_TICK = 1 };
typedef struct { double t; int cls; int64_t key; int kind, r, c; } ev_t;
typedef struct { ev_t *a; int n, cap; } heap_t;

static int ev_less(const ev_t *x, const ev_t *y) {
  if (x->t != y->t) return x->t < y->t;
  if (x->cls != y->cls) return x->cls < y->cls;
  return x->key < y->key;
}
static void hp_push(heap_t *h, ev_t e) {
  if (h->n == h->cap) {
    h->cap = h->cap ? 2 * h->cap : 64;
    h->a = (ev_t *)realloc(h->a, sizeof(ev_t) * (size_t)h->cap);
  }
  int i = h->n++;
  h->a[i] = e;
  while (i > 0) {
    int p = (i - 1) / 2;
    if (!ev_less(&h->a[i], &h->a[p])) break;
    ev_t tmp = h->a[i]; h->a[i] = h->a[p]; h->a[p] = tmp;
    i = p;
  }
}
static ev_t hp_pop(heap_t *h) {
  ev_t top = h->a[0];
  h->a[0] = h->a[--h->n];
  int i = 0;
  for (;;) {
    int l = 2 * i + 1, r = l + 1, m = i;
    if (l < h->n && ev_less(&h->a[l], &h->a[m])) m = l;
    if (r < h->n && ev_less(&h->a[r], &h->a[m])) m = r;
    if (m == i) break;
    ev_t tmp = h->a[i]; h->a[i] = h->a[m]; h->a[m] = tmp;
    i = m;
  }
  return top;
}

/* ---------- simulation state ---------- */
enum { IT_BATCH = 0, IT_PREFILL = 1, IT_DECODE = 2 };

typedef struct {
  int ns, comp[CFO_MAXC], beff[CFO_MAXC], stage_of[CFO_MAXC];
  double tps[CFO_MAXC];  /* iteration-time multiplier of each stage (GPUs per executor) */
  int busy, ran, rr, cur_s, cur_kind;
  double t_end, last_end;
  ivec mem;                 /* members of the running iteration, in order */
  ivec q[CFO_MAXC];         /* waiting FIFO per stage */
  ivec run[CFO_MAXC];       /* running list per LLM stage, admission order */
} exec_t;

typedef struct {
  int type, ttft_c, out_left, done;
  int ex[CFO_MAXC], join[CFO_MAXC], tok[CFO_MAXC], nout[CFO_MAXC];
  double a, t_first, t_last, t_media;
  double *emit; int n_emit, cap_emit;   /* gate-source token emission times */
} req_t;

typedef struct {
  const cfo_model *m;
  const cfo_trace *tr;
  size_t toff;             /* offset of this seed's trace */
  int n, nx;
  exec_t *x;
  req_t *rq;
  heap_t h;
  int64_t seq;
  uint64_t events;
  uint32_t *met, *cnt;
  double *lat;
  int in_system;
  double busy_time;
} sim_t;

static uint64_t attr_of(const sim_t *S, int r, int a) {
  size_t o = S->toff + (size_t)r;
  const cfo_trace *tr = S->tr;
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

static uint64_t x_of(const sim_t *S, int r, int c) {
  uint64_t s = 0;
  for (int a = 0; a < CFO_NATTR; a++)
    if ((S->m->x_sel[c] >> a) & 1u) s += attr_of(S, r, a);
  return s;
}

static int on_path(const cfo_model *m, int t, int c) { return (m->path_mask[t] >> c) & 1u; }

/* edge c -> c2 of type t carries the gate (streaming) */
static int stream_edge(const cfo_model *m, int t, int c, int c2) {
  return m->gate_src[c2] == c && on_path(m, t, c2) && ((m->parents[t][c2] >> c) & 1u);
}

static int gated(const cfo_model *m, int t, int c2) {
  int src = m->gate_src[c2];
  return src >= 0 && stream_edge(m, t, src, c2);
}

static void enqueue(sim_t *S, int r, int c) {
  req_t *q = &S->rq[r];
  exec_t *X = &S->x[q->ex[c]];
  S->events++;
  iv_push(&X->q[X->stage_of[c]], r);
}

static void join(sim_t *S, int r, int c) {
  req_t *q = &S->rq[r];
  q->join[c]++;
  if (q->join[c] == __builtin_popcount(S->m->parents[q->type][c])) enqueue(S, r, c);
}

static void deliver(sim_t *S, int r, int c2, int xfrom, double t) {
  req_t *q = &S->rq[r];
  if (q->ex[c2] == xfrom) {
    join(S, r, c2);
  } else {
    ev_t e = {t + S->m->comm_s, EV_DELAY, S->seq++, DL_DELIVER, r, c2};
    hp_push(&S->h, e);
  }
}

static void complete_request(sim_t *S, int r, double t) {
  const cfo_model *m = S->m;
  req_t *q = &S->rq[r];
  S->events++;
  S->in_system--;
  q->done = 1;
  int ty = q->type;
  double ttft = 0.0, tpot = 0.0, media = 0.0;
  if (q->ttft_c >= 0) {
    ttft = q->t_first - q->a;
    int n1 = q->nout[q->ttft_c];
    if (n1 > 1) tpot = (q->t_last - q->t_first) / (double)(n1 - 1);
  }
  double e2e = t - q->a;
  int has_gen = 0;
  for (int c = 0; c < m->n_comp; c++)
    if (((m->out_mask[ty] >> c) & 1u) && m->kind[c] == CFO_GEN) has_gen = 1;
  if (has_gen) media = q->t_media - q->a;
  int ok = ttft <= m->slo[ty][0] && tpot <= m->slo[ty][1] && e2e <= m->slo[ty][2] &&
           media <= m->slo[ty][3];
  S->cnt[ty]++;
  if (ok) S->met[ty]++;
  if (S->lat) {
    S->lat[(size_t)r * 4 + 0] = ttft;
    S->lat[(size_t)r * 4 + 1] = tpot;
    S->lat[(size_t)r * 4 + 2] = e2e;
    S->lat[(size_t)r * 4 + 3] = media;
  }
  free(q->emit);
  q->emit = NULL;
}

/* request r finishes component c on executor x at time t */
static void finish(sim_t *S, int r, int c, int x, double t) {
  const cfo_model *m = S->m;
  req_t *q = &S->rq[r];
  int ty = q->type;
  for (int c2 = 0; c2 < m->n_comp; c2++) {
    if (!on_path(m, ty, c2) || !((m->parents[ty][c2] >> c) & 1u)) continue;
    if (stream_edge(m, ty, c, c2)) continue;
    deliver(S, r, c2, x, t);
  }
  if ((m->out_mask[ty] >> c) & 1u) {
    if (m->kind[c] == CFO_GEN) q->t_media = t;
    q->out_left--;
    if (q->out_left == 0) complete_request(S, r, t);
  }
}

/* the gate source c of request r emitted a token at time t */
static void emit_token(sim_t *S, int r, int c, int x, double t) {
  const cfo_model *m = S->m;
  req_t *q = &S->rq[r];
  if (q->n_emit == q->cap_emit) {
    q->cap_emit = q->cap_emit ? 2 * q->cap_emit : 32;
    q->emit = (double *)realloc(q->emit, sizeof(double) * (size_t)q->cap_emit);
  }
  q->emit[q->n_emit++] = t;
  if (q->n_emit == 1) {
    /* first token: the request is delivered to every gated child */
    for (int c2 = 0; c2 < m->n_comp; c2++)
      if (stream_edge(m, q->type, c, c2)) deliver(S, r, c2, x, t);
  }
}

static int is_gate_source_of(const cfo_model *m, int t, int c) {
  for (int c2 = 0; c2 < m->n_comp; c2++)
    if (stream_edge(m, t, c, c2)) return 1;
  return 0;
}

static int eligible(const sim_t *S, int r, int c, int x, double t) {
  const cfo_model *m = S->m;
  const req_t *q = &S->rq[r];
  if (!gated(m, q->type, c)) return 1;
  int src = m->gate_src[c];
  int k = q->tok[c] + 1;
  if (k > q->nout[src]) k = q->nout[src];
  if (q->n_emit < k) return 0;
  double delta = (q->ex[src] == x) ? 0.0 : m->comm_s;
  return q->emit[k - 1] + delta <= t;
}

static int runnable(const sim_t *S, int xi, int s, double t) {
  const exec_t *X = &S->x[xi];
  int c = X->comp[s];
  if (S->m->kind[c] != CFO_LLM) return X->q[s].n > 0;
  if (X->q[s].n > 0 && X->run[s].n < X->beff[s]) return 1;
  for (int i = 0; i < X->run[s].n; i++)
    if (eligible(S, iv_at(&X->run[s], i), c, xi, t)) return 1;
  return 0;
}

static void start(sim_t *S, int xi, int s, double t) {
  const cfo_model *m = S->m;
  exec_t *X = &S->x[xi];
  int c = X->comp[s];
  double dur;
  X->mem.head = 0;
  X->mem.n = 0;
  if (m->kind[c] != CFO_LLM || (X->q[s].n > 0 && X->run[s].n < X->beff[s])) {
    int room = (m->kind[c] == CFO_LLM) ? X->beff[s] - X->run[s].n : X->beff[s];
    int n = X->q[s].n < room ? X->q[s].n : room;
    uint64_t xs = 0;
    for (int i = 0; i < n; i++) {
      int r = iv_pop_front(&X->q[s]);
      iv_push(&X->mem, r);
      xs += x_of(S, r, c);
    }
    dur = X->tps[s] * ((m->k0[c] + m->k1[c] * (double)xs) + m->k2[c] * (double)n);
    if (m->kind[c] == CFO_ENC && (!X->ran || X->last_end < t)) dur = dur + m->cpu_pre_s;
    X->cur_kind = (m->kind[c] == CFO_LLM) ? IT_PREFILL : IT_BATCH;
  } else {
    for (int i = 0; i < X->run[s].n; i++) {
      int r = iv_at(&X->run[s], i);
      if (eligible(S, r, c, xi, t)) iv_push(&X->mem, r);
    }
    dur = X->tps[s] * (m->d0[c] + m->d1[c] * (double)X->mem.n);
    X->cur_kind = IT_DECODE;
  }
  X->busy = 1;
  X->cur_s = s;
  X->t_end = t + dur;
  S->busy_time = S->busy_time + dur;
  ev_t e = {X->t_end, EV_DONE, xi, 0, 0, 0};
  hp_push(&S->h, e);
}

static void try_start(sim_t *S, int xi, double t) {
  exec_t *X = &S->x[xi];
  for (int i = 0; i < X->ns; i++) {
    int s = (X->rr + 1 + i) % X->ns;
    if (runnable(S, xi, s, t)) {
      start(S, xi, s, t);
      X->rr = s;
      return;
    }
  }
}

static void complete_iteration(sim_t *S, int xi, double t) {
  const cfo_model *m = S->m;
  exec_t *X = &S->x[xi];
  int s = X->cur_s, c = X->comp[s];
  X->busy = 0;
  X->ran = 1;
  X->last_end = t;
  if (X->cur_kind == IT_BATCH) {
    for (int i = 0; i < X->mem.n; i++) {
      int r = iv_at(&X->mem, i);
      S->events++;
      finish(S, r, c, xi, t);
    }
  } else if (X->cur_kind == IT_PREFILL) {
    for (int i = 0; i < X->mem.n; i++) {
      int r = iv_at(&X->mem, i);
      req_t *q = &S->rq[r];
      S->events++;
      q->tok[c] = 1;
      if (c == q->ttft_c) { q->t_first = t; q->t_last = t; }
      if (is_gate_source_of(m, q->type, c)) emit_token(S, r, c, xi, t);
      if (q->tok[c] == q->nout[c]) finish(S, r, c, xi, t);
      else iv_push(&X->run[s], r);
    }
  } else {
    for (int i = 0; i < X->mem.n; i++) {
      int r = iv_at(&X->mem, i);
      req_t *q = &S->rq[r];
      S->events++;
      q->tok[c]++;
      if (c == q->ttft_c) q->t_last = t;
      if (is_gate_source_of(m, q->type, c)) emit_token(S, r, c, xi, t);
      if (q->tok[c] == q->nout[c]) finish(S, r, c, xi, t);
    }
    /* drop finished requests from the running list, keeping order */
    ivec *run = &X->run[s];
    int w = 0;
    for (int i = 0; i < run->n; i++) {
      int r = iv_at(run, i);
      if (S->rq[r].tok[c] < S->rq[r].nout[c]) run->a[run->head + w++] = r;
    }
    run->n = w;
  }
  /* a gate source's iteration end is a wake-up point for remote gated stages */
  for (int c2 = 0; c2 < m->n_comp; c2++) {
    if (m->gate_src[c2] == c) {
      ev_t e = {t + m->comm_s, EV_DELAY, S->seq++, DL_TICK, -1, -1};
      hp_push(&S->h, e);
      break;
    }
  }
}

static void arrive(sim_t *S, int r) {
  const cfo_model *m = S->m;
  req_t *q = &S->rq[r];
  S->events++;
  S->in_system++;
  for (int c = 0; c < m->n_comp; c++)
    if (on_path(m, q->type, c) && m->parents[q->type][c] == 0) enqueue(S, r, c);
}

int cfo_sim_triple(const cfo_model *m, const cfo_plans *pl, int32_t plan_id, double rate,
                   const cfo_trace *tr, int32_t seed_idx, uint32_t *met, uint32_t *cnt,
                   uint64_t *events, uint32_t *status, double *lat, double *diag) {
  const int P = pl->P, p = plan_id;
  sim_t S;
  memset(&S, 0, sizeof S);
  S.m = m;
  S.tr = tr;
  S.n = tr->n_req;
  S.toff = (size_t)seed_idx * (size_t)tr->n_req;
  S.met = met;
  S.cnt = cnt;
  S.lat = lat;
  for (int t = 0; t < m->n_types; t++) { met[t] = 0; cnt[t] = 0; }
  *events = 0;
  *status = 0;
  if (diag) for (int i = 0; i < 4; i++) diag[i] = 0.0;
  /* a Poisson arrival rate is positive and finite; a plan id names a column of the table */
  if (p < 0 || p >= P || !(rate > 0.0) || !(rate < __builtin_inf())) { *status = CFO_ST_INVALID; return 0; }

  /* executors: those of each node numbered node by node, a node's first
   * executor group before its second */
  int nv = pl->n_nodes[p];
  if (nv < 1 || nv > CFO_MAXV) { *status = CFO_ST_INVALID; return 0; }
  int base[CFO_MAXV + 1];
  cfo_group grp[CFO_MAXV][2];
  int ngrp[CFO_MAXV];
  base[0] = 0;
  for (int v = 0; v < nv; v++) {
    /* a node hosts components of the model and has executors of valid batches; a second
     * configuration has a share in 1..9 tenths and GPUs */
    int cm = P_AT(pl->node_comp, v, P, p);
    ngrp[v] = cfo_node_groups(pl, v, p, grp[v]);
    int bad_node = cm == 0 || (cm >> m->n_comp) != 0;
    for (int k = 0; k < ngrp[v]; k++)
      if (grp[v][k].rep < 1 || grp[v][k].batch < 1 || grp[v][k].batch > CFO_MAXB) bad_node = 1;
    if (ngrp[v] == 2 && (P_AT(pl->node_w, v, P, p) < 1 || P_AT(pl->node_w, v, P, p) > 9 || grp[v][1].gpus < 1))
      bad_node = 1;
    if (bad_node) {
      *status = CFO_ST_INVALID;
      return 0;
    }
    base[v + 1] = base[v];
    for (int k = 0; k < ngrp[v]; k++) base[v + 1] += grp[v][k].rep;
  }
  S.nx = base[nv];
  if (S.nx < 1 || S.nx > CFO_MAXX) { *status = CFO_ST_INVALID; return 0; }
  S.x = (exec_t *)calloc((size_t)S.nx, sizeof(exec_t));
  for (int v = 0; v < nv; v++) {
    int cm = P_AT(pl->node_comp, v, P, p);
    for (int j = base[v]; j < base[v + 1]; j++) {
      const int k = j - base[v] < grp[v][0].rep ? 0 : 1;
      int bn = grp[v][k].batch;
      int gn = grp[v][k].gpus;
      exec_t *X = &S.x[j];
      X->rr = -1;
      for (int c = 0; c < CFO_MAXC; c++) X->stage_of[c] = -1;
      for (int c = 0; c < m->n_comp; c++) {
        if (!((cm >> c) & 1)) continue;
        X->comp[X->ns] = c;
        X->beff[X->ns] = bn < m->batch_cap[c] ? bn : m->batch_cap[c];
        X->tps[X->ns] = cfo_tp(m, c, gn);
        X->stage_of[c] = X->ns;
        X->ns++;
      }
    }
  }

  /* requests: type, route (alternative, replica per node), output lengths */
  S.rq = (req_t *)calloc((size_t)(S.n > 0 ? S.n : 1), sizeof(req_t));
  int bad = 0;
  for (int r = 0; r < S.n && !bad; r++) {
    size_t o = S.toff + (size_t)r;
    req_t *q = &S.rq[r];
    int ty = tr->type[o];
    q->type = ty;
    q->a = ((double)tr->arr_ticks[o] * 0x1p-32) / rate;
    int na = P_AT(pl->n_alt, ty, P, p);
    int alt = 0;
    if (na == 2) {
      uint64_t w0 = P_AT(pl->alt_w, ty * 2 + 0, P, p), w1 = P_AT(pl->alt_w, ty * 2 + 1, P, p);
      uint64_t v = ((uint64_t)tr->akey[o] * (w0 + w1)) >> 32;
      alt = (v < w0) ? 0 : 1;
    }
    q->ttft_c = -1;
    q->out_left = __builtin_popcount(m->out_mask[ty]);
    for (int c = 0; c < CFO_MAXC; c++) q->ex[c] = -1;
    for (int c = 0; c < m->n_comp; c++) {
      if (!on_path(m, ty, c)) continue;
      int v = P_AT(pl->alt_node, (ty * 2 + alt) * 8 + c, P, p);
      if (v >= nv || !((P_AT(pl->node_comp, v, P, p) >> c) & 1)) { bad = 1; break; }
      int minc = __builtin_ctz(P_AT(pl->node_comp, v, P, p));
      uint64_t word = minc < 4 ? tr->rkey0[o] : tr->rkey1[o];
      uint64_t key = (word >> (16 * (minc & 3))) & 0xFFFFu;
      int j = cfo_node_pick(key, grp[v], ngrp[v], pl, v, p);
      q->ex[c] = base[v] + j;
      if (m->kind[c] == CFO_LLM) {
        if (q->ttft_c < 0) q->ttft_c = c;
        uint64_t no = ((m->prefill_only[ty] >> c) & 1u) ? 1u : attr_of(&S, r, m->nout_attr[c]);
        q->nout[c] = no < 1 ? 1 : (int)no;
      }
    }
  }
  if (bad) {
    *status = CFO_ST_INVALID;
  } else {
    double t_prev = 0.0, area = 0.0;
    uint64_t instants = 0;
    if (S.n > 0) {
      ev_t e = {S.rq[0].a, EV_ARRIVE, 0, 0, 0, 0};
      hp_push(&S.h, e);
    }
    while (S.h.n > 0) {
      double t = S.h.a[0].t;
      instants++;
      area = area + (double)S.in_system * (t - t_prev);
      t_prev = t;
      while (S.h.n > 0 && S.h.a[0].t == t) {
        ev_t e = hp_pop(&S.h);
        if (e.cls == EV_DONE) {
          complete_iteration(&S, (int)e.key, t);
        } else if (e.cls == EV_DELAY) {
          if (e.kind == DL_DELIVER) join(&S, e.r, e.c);
        } else {
          int r = (int)e.key;
          arrive(&S, r);
          if (r + 1 < S.n) {
            ev_t a = {S.rq[r + 1].a, EV_ARRIVE, r + 1, 0, 0, 0};
            hp_push(&S.h, a);
          }
        }
      }
      for (int xi = 0; xi < S.nx; xi++)
        if (!S.x[xi].busy) try_start(&S, xi, t);
    }
    for (int r = 0; r < S.n; r++)
      if (!S.rq[r].done) { *status |= CFO_ST_DEADLOCK; break; }
    *events = S.events;
    if (diag) { diag[0] = area; diag[1] = t_prev; diag[2] = (double)instants; diag[3] = S.busy_time; }
  }
  for (int xi = 0; xi < S.nx; xi++) {
    free(S.x[xi].mem.a);
    for (int s = 0; s < CFO_MAXC; s++) { free(S.x[xi].q[s].a); free(S.x[xi].run[s].a); }
  }
  for (int r = 0; r < S.n; r++) free(S.rq[r].emit);
  free(S.x);
  free(S.rq);
  free(S.h.a);
  return 0;
}

/* Rate bisection (the workload descriptions bisect rates over a grid):
 * for plan plan_ids[i] and its grid rates[i][0..K), with feasible(k) the
 * attainment test of cfo_goodput_reduce on the counts pooled over the S
 * seeds at rate k, keep lo = -1 (feasible) and hi = K (infeasible), simulate
 * every seed at mid = (lo + hi) / 2 and move lo or hi to mid, until
 * hi = lo + 1.  kstar = lo, goodput_t = (rates[lo] M_t) / (S n) from the
 * simulation at lo (0 if lo < 0).  On a monotone predicate this is the
 * grid's first infeasible rate - 1, after at most ceil(log2(K + 1))
 * rounds; n_eval[i] counts the rates simulated. */
int cfo_bisect(const cfo_model *m, const cfo_plans *pl, const int32_t *plan_ids, int32_t n_plans,
               const double *rates, int32_t K, const cfo_trace *tr, uint32_t theta_num, uint32_t theta_den,
               int32_t *kstar, double *goodput_t, double *goodput, int32_t *n_eval, uint64_t *events) {
  const int T = m->n_types, S = tr->n_seeds;
  const double denom = (double)((uint64_t)S * (uint64_t)tr->n_req);
  uint32_t met[CFO_MAXT], cnt[CFO_MAXT];
  uint64_t Mlo[CFO_MAXT];
  for (int i = 0; i < n_plans; i++) {
    int lo = -1, hi = K, ne = 0;
    uint64_t ev_total = 0;
    for (int t = 0; t < T; t++) Mlo[t] = 0;
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      uint64_t M[CFO_MAXT], N[CFO_MAXT];
      for (int t = 0; t < T; t++) M[t] = N[t] = 0;
      int failed = 0;
      for (int s = 0; s < S; s++) {
        uint64_t ev = 0;
        uint32_t st = 0;
        cfo_sim_triple(m, pl, plan_ids[i], rates[(size_t)i * K + mid], tr, s, met, cnt, &ev, &st, NULL, NULL);
        ev_total += ev;
        if (st != 0) failed = 1;
        for (int t = 0; t < T; t++) {
          M[t] += met[t];
          N[t] += cnt[t];
        }
      }
      ne++;
      int feasible = !failed;
      for (int t = 0; t < T; t++)
        if (N[t] > 0 && (uint64_t)theta_den * M[t] < (uint64_t)theta_num * N[t]) feasible = 0;
      if (feasible) {
        lo = mid;
        for (int t = 0; t < T; t++) Mlo[t] = M[t];
      } else {
        hi = mid;
      }
    }
    kstar[i] = lo;
    n_eval[i] = ne;
    events[i] = ev_total;
    double g = 0.0;
    for (int t = 0; t < T; t++) {
      const double gt = lo >= 0 ? (rates[(size_t)i * K + lo] * (double)Mlo[t]) / denom : 0.0;
      goodput_t[(size_t)i * T + t] = gt;
      g = g + gt;
    }
    goodput[i] = g;
  }
  return 0;
}
