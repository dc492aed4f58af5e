// k_fine.hip -- cf_eval_fine: phase 3 of the plan evaluation (Sec. 4.3,
// Alg. 2), the request-level simulation of every (plan, rate, seed) triple.
//
// One wavefront simulates one triple; a persistent grid of wavefronts takes
// triples from an atomic ticket, seed-major so that concurrent wavefronts
// read the same seed's trace (L2 / MALL reuse), and within a seed from the
// lowest rate up (the costliest triples first).
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
// Memory: the plan, executor state and every stage's queue / running-set
// descriptor live in LDS (sized per launch from the largest plan), except
// that k_fine<true> keeps its executors' times in registers (lane x for
// executor x) to leave more LDS per CU to its larger stage tables; queue
// entries (chunked lists in a per-wavefront pool), running slots and the
// 16-byte per-request records live in HBM.  The members of a completed
// iteration are processed lane-parallel, 64 at a time: delay-line appends,
// queue appends and running-set appends keep the member order through
// wavefront prefix sums, and SLO counts are ballot + popcount per type.
//
// Decode steps of a non-gated LLM stage cost O(1): a running request's
// token count is (decode steps of its stage since it joined) + 1, so each
// running slot stores the step index at which it finishes and only the
// finishing slots are touched.  The gated stage (talker) keeps per-request
// token counts; the time of a thinker token comes from the request's join
// step in the thinker's stage and a ring of that stage's step end times.
//
// Two instantiations of the kernel: k_fine<false> simulates thinker steps
// one at a time and wakes the talker executors after every remote thinker
// step; it serves models without a gated stage, where none of that is
// reached.  k_fine<true>, used for models with a gated stage, also runs
// thinker stages in decode runs and replaces the per-step wake-ups by exact
// wake times: a talker request becomes eligible at the visibility time of
// the thinker token it waits for, the only state change not caused by an
// event of its own executor.  An executor hosting a talker stage that is
// idle (or in a decode run) keeps the earliest such time among its blocked
// requests whose thinker runs elsewhere; the thinker's ring holds the last
// completed steps and the predicted ends of the steps of its running decode
// run.  Requests whose token is not scheduled yet register the executor
// with the thinker's stage, and every start or cut of that stage's decode
// steps makes the registered executors recompute their wake time.  A
// thinker run on an executor that also hosts the talker stops at the first
// step whose token a local blocked talker request waits for.
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "cf_internal.h"
#include "cf_run.h"

namespace cf {
namespace {

constexpr int kMaxSI = CF_MAX_EXEC * CF_MAX_COMP;  // stage instances
static_assert(kMaxSI <= 512, "an LLM stage instance index fits the 9 bits of a gate word");
constexpr int kChunk = 64;                          // queue chunk entries
constexpr int kHist = 64;                           // k_fine<false>: ring of the last thinker step ends
constexpr int kRing = 256;                          // k_fine<true>: thinker step-time ring
constexpr int kKeep = 64;                           // k_fine<true>: completed steps kept in the ring
constexpr uint32_t kThRun = kRing - kKeep;          // k_fine<true>: longest thinker decode run
constexpr uint32_t kNone = 0xFFFFFFFFu;

enum { IT_BATCH = 0, IT_PREFILL = 1, IT_DECODE = 2, IT_FINISH = 3 };
enum { DL_DELIVER = 0, DL_TICK = 1 };
constexpr uint32_t MISC_OUTS = 15u;     // outputs still to finish
constexpr uint32_t MISC_TH_DONE = 16u;  // thinker finished
constexpr uint32_t MARK = 0x80000000u;  // gated running slot: in the current decode step
// A gated stage's running slot word: tokens so far (bits 0..15), the
// request's own token count at the stage (bits 16..30), MARK (bit 31).
constexpr uint32_t RK_TOK = 0xFFFFu;
__device__ __forceinline__ uint32_t rk_own(uint32_t v) { return (v >> 16) & 0x7FFFu; }
// k_fine<true>: gate word of a gated stage's running slot, fixed when the
// request joined: the request's type is gated at the stage (bit 31), the
// LLM index of its thinker's stage instance (bits 22..30), the thinker's
// executor (bits 16..21) and the thinker's token count (bits 0..15); run_q
// holds the request's join step in the thinker's stage.
constexpr uint32_t RG_GATED = 0x80000000u;
constexpr uint32_t EX_RUN = 1u << 21;   // executor state: busy with a multi-step decode run
// k_fine<true>: executor state kind of a joint thinker/talker run (IT_FINISH
// is a member kind only); the talker's stage index is in bits 22..25
constexpr uint32_t IT_JOINT = 3;
// stage flags
constexpr uint8_t SF_LLM = 1, SF_GATED = 2, SF_THINKER = 4, SF_ENC = 8, SF_GEN = 16;

struct __attribute__((aligned(16))) Rec {
  uint64_t ex;    // executor of each component of the path (byte c), 0xFF off the path
  uint32_t join;  // deliveries received per component (4 bits each)
  uint32_t misc;  // outputs left (4 bits), thinker done (bit 4), type (bits 8..10)
};

// token and media times of a request, and its join step in the thinker's stage
struct __attribute__((aligned(32))) Tim {
  double tfirst, tlast, tmedia;
  uint32_t thjoin, pad;
};
// a delay-line entry: due time and what is delivered (one 16-byte block)
struct __attribute__((aligned(16))) DlEnt {
  double t;
  uint32_t v, pad;
};
// a request's record, its length attributes (copied from the trace at its
// arrival) and its times side by side: one 64-byte block holds them all
struct __attribute__((aligned(64))) Req {
  Rec r;
  uint16_t prompt, out, patches, pad;
  uint32_t aud_in, aud_out;
  Tim t;
};
static_assert(sizeof(Req) == 64 && __builtin_offsetof(Req, t) == 32, "request block");

struct Layout {
  size_t req;
  size_t run, hist, mem, dl, pool, pool_next, pool_free;
  size_t bytes;
  int run_cap, hist_slots, n_chunks;
  uint32_t dl_mask;
};

struct FineArgs {
  KModel m;
  int P;
  const uint8_t *n_nodes, *node_comp, *node_rep, *node_gpus, *n_alt, *alt_w, *alt_node;
  const uint16_t *node_batch;
  const uint8_t *node_rep2, *node_gpus2, *node_w;  // a node's second configuration (NULL: none)
  const uint16_t *node_batch2;
  const int32_t *plan_ids;
  int n_plans;
  const double *rates;
  int K;
  const uint64_t *ticks, *rkey0, *rkey1;
  const uint8_t *type;
  const uint16_t *patches, *prompt, *out;
  const uint32_t *aud_in, *aud_out, *akey;
  int S, n;
  uint32_t *met, *cnt, *status;
  uint64_t *events;
  double *lat;
  const int32_t *lat_triples;
  int n_lat;
  uint32_t *hist;      // optional [n_plans][K][S][T][nb + 1] latency histograms
  const double *tg;    // their target table [T][nb][4]
  int nb;
  char *slab;
  Layout L;
  unsigned int *ticket;
  unsigned int total;
  int nsi_cap;  // stage instances provided in LDS
  int nl_cap, nt_cap;  // k_fine<true>: LLM stage instances and thinker ring slots provided in LDS
  uint64_t lim_instants;  // instants a simulation may take (a test limit; ~0 = none)
  // order in which a seed's (plan, rate) pairs are taken: entry j is i * K + k
  // (null: rate index first, then plan)
  const uint32_t *order;
};

// model tables read with per-lane (divergent) indices
struct ModelLds {
  uint8_t child[CF_MAX_TYPES][CF_MAX_COMP], npar[CF_MAX_TYPES][CF_MAX_COMP];
  int8_t ttft_c[CF_MAX_TYPES], th_c[CF_MAX_TYPES], ta_c[CF_MAX_TYPES];
  uint8_t outm[CF_MAX_TYPES], pfo[CF_MAX_TYPES], gen_out[CF_MAX_TYPES];
  uint8_t kind[CF_MAX_COMP], nout_attr[CF_MAX_COMP];
  double slo[CF_MAX_TYPES][4];
};

struct WaveShared {
  uint32_t ex_st[CF_MAX_EXEC];  // busy:1 ran:1 kind:2 rr:4 cur:4 nmem:9
  // an executor's first stage instance (bits 0..15), its node's component set
  // (bits 16..23: its stages in component order) and its node (bits 24..31):
  // one LDS word read at once
  uint32_t ex_geo[CF_MAX_EXEC];
  uint8_t ex_tp[CF_MAX_EXEC];  // GPUs per executor as min(g, 8) - 1 (iteration-time multiplier index)
  uint8_t route[CF_MAX_TYPES][2][CF_MAX_COMP];
  uint8_t nalt[CF_MAX_TYPES], aw[CF_MAX_TYPES][2];
  uint8_t vbase[CF_MAX_NODES + 1], vrep[CF_MAX_NODES], vminc[CF_MAX_NODES], vcomp[CF_MAX_NODES];
  uint16_t vbatch[CF_MAX_NODES];
  // a node's executors: vrep in all, the first vrep1 of batch vbatch, the
  // others of batch vbatch2; vw tenths of its requests to the first (0: one
  // configuration)
  uint8_t vrep1[CF_MAX_NODES], vw[CF_MAX_NODES];
  uint16_t vbatch2[CF_MAX_NODES];
  uint32_t met[CF_MAX_TYPES], cnt[CF_MAX_TYPES];
  ModelLds ml;
};

// stage-instance descriptors, structure of arrays in dynamic LDS
// k_fine<false> indexes every field by stage instance.  k_fine<true> keeps
// the LLM-only fields (rn, roff, iter, minfin, hist) for its LLM stage
// instances only, at index lsi[si], and the thinker-only fields (sched,
// watch) per thinker ring slot hist[lsi[si]].
struct SiLds {
  uint8_t *comp, *flags;  // k_fine<false>
  // k_fine<true>: a stage instance's constant fields in one word: flags
  // (bits 0..7), component (8..11), batch (12..20), LLM index (21..31; kNoLsi:
  // not an LLM stage)
  uint32_t *word;
  uint8_t *qhp, *qtp;  // k_fine<false>: queue head and tail positions in their chunks
  int *qhc, *qtc;      // k_fine<false>: queue head and tail chunks
  uint32_t *qh, *qt;   // k_fine<true>: queue head and tail, chunk and position packed by qend
  uint16_t *beff;   // k_fine<false>
  int16_t *hist;
  int *qn, *roff, *rn;
  uint32_t *iter, *minfin;
  uint64_t *watch;  // k_fine<true>, thinker stages: executors to notify when its decode steps are (re)scheduled
  uint32_t *sched;  // k_fine<true>, thinker stages: last step whose end is known (completed or in the running run)
};
constexpr size_t kSiBytes = 1 + 1 + 1 + 1 + 2 + 2 + 4 * 7;
// k_fine<true>: bytes per stage instance, per LLM stage instance, per thinker slot
constexpr size_t kSiBytesG = 4 * 4, kLlmBytesG = 4 * 4 + 2, kThBytesG = 8 + 4;
// a queue end, chunk c (-1: none) and position p <= kChunk in it, as one word
// (chunk indices stay below 2^25: at most 2^26 requests on 8 components)
__device__ __forceinline__ uint32_t qend(int c, int p) { return ((uint32_t)(c + 1) << 7) | (uint32_t)p; }
__device__ __forceinline__ int qend_chunk(uint32_t w) { return (int)(w >> 7) - 1; }
__device__ __forceinline__ int qend_pos(uint32_t w) { return (int)(w & 127u); }
static_assert(sizeof(WaveShared) % 8 == 0, "the dynamic LDS table after WaveShared holds 8-byte words");
// a wavefront's static LDS: k_fine<false> also holds the executors' times and
// decode-run step counters
template <bool G>
struct WaveLds {
  double xt[4 * CF_MAX_EXEC];
  uint32_t ex_itgt[CF_MAX_EXEC];  // decode run: step counter of its stage at the end of the running step
  WaveShared w;
};
template <>
struct WaveLds<true> {
  WaveShared w;
};

constexpr uint32_t kNoLsi = 0x7FFu;
static_assert(CF_MAX_COMP <= 16 && CF_MAX_BATCH < 512 && CF_MAX_EXEC * CF_MAX_COMP < (int)kNoLsi,
              "stage word fields");
// a stage instance's index in the LLM-only fields (k_fine<false>: its own)
template <bool G>
__device__ __forceinline__ int lx_of(const SiLds &si, int s) {
  if constexpr (G) return (int)(si.word[s] >> 21);
  else return s;
}
template <bool G>
__device__ __forceinline__ uint32_t si_flags(const SiLds &si, int s) {
  if constexpr (G) return si.word[s] & 0xFFu;
  else return si.flags[s];
}
template <bool G>
__device__ __forceinline__ int si_comp(const SiLds &si, int s) {
  if constexpr (G) return (int)((si.word[s] >> 8) & 15u);
  else return si.comp[s];
}
template <bool G>
__device__ __forceinline__ int si_beff(const SiLds &si, int s) {
  if constexpr (G) return (int)((si.word[s] >> 12) & 0x1FFu);
  else return si.beff[s];
}

__device__ __forceinline__ int lane_id() { return threadIdx.x; }
__device__ __forceinline__ uint32_t ru(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int ri(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t ru64(uint64_t v) {
  return ((uint64_t)ru((uint32_t)(v >> 32)) << 32) | ru((uint32_t)v);
}
__device__ __forceinline__ double rdb(double v) {
  return __longlong_as_double((long long)ru64((uint64_t)__double_as_longlong(v)));
}
// the value lane x holds (x wave-uniform)
__device__ __forceinline__ double lane_val(double v, int x) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), x);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ uint32_t lanes_below(uint64_t bal) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
}
// wavefront minimum of a u32 through DPP row shifts and row broadcasts
// (identity ~0 for lanes whose source is out of range); result in lane 63
__device__ __forceinline__ uint32_t dpp_min_u32(uint32_t v) {
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x111, 0xf, 0xf, false));  // row_shr:1
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x112, 0xf, 0xf, false));  // row_shr:2
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x113, 0xf, 0xf, false));  // row_shr:3
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x114, 0xf, 0xe, false));  // row_shr:4
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x118, 0xf, 0xc, false));  // row_shr:8
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast:15
  v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)~0u, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
// minimum of non-negative doubles (or +inf) over the wavefront: the bit
// patterns of such doubles order like the values, so the high words are
// reduced first and the low words among the lanes holding that high word
__device__ __forceinline__ double wave_min_time(double t) {
  const uint64_t b = (uint64_t)__double_as_longlong(t);
  const uint32_t hi = dpp_min_u32((uint32_t)(b >> 32));
  const uint32_t lo = dpp_min_u32((uint32_t)(b >> 32) == hi ? (uint32_t)b : ~0u);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// inclusive prefix sum over the lanes through DPP: row_shr 1, 2, 4, 8 scan
// each row of 16 lanes (identity 0 where the source is out of range), then
// row_bcast 15 and row_bcast 31 carry the row totals into the later rows.
// Needs every lane active.
__device__ __forceinline__ uint32_t dpp_scan_add(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}
// wavefront sum (uniform result)
__device__ __forceinline__ uint32_t dpp_sum_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)dpp_scan_add(v), 63);
}
// exclusive prefix sum of v over the lanes, and the total
__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t v, uint32_t &total) {
  const uint32_t x = dpp_scan_add(v);
  total = (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
  return x - v;
}

// Device memory (global address space) addressed by a 32-bit byte offset
// from a base held in scalar registers: loads and stores take the
// scalar-base + vector-offset form, with no 64-bit address arithmetic per
// lane.  Every array the kernel indexes is far below 4 GiB.
#define CF_GLOBAL __attribute__((address_space(1)))
template <typename T>
struct GPtr {
  CF_GLOBAL T *p;
  __device__ __forceinline__ CF_GLOBAL T &operator[](uint32_t i) const {
    return *(CF_GLOBAL T *)((CF_GLOBAL char *)p + i * (uint32_t)sizeof(T));
  }
  __device__ __forceinline__ GPtr operator+(uint32_t i) const { return GPtr{&(*this)[i]}; }
};
template <typename T>
__device__ __forceinline__ GPtr<T> gptr_at(char *base, size_t off) {
  return GPtr<T>{(CF_GLOBAL T *)(base + off)};
}
// One word of the running slots, which lie interleaved in the slab
// (k_fine<true>: request, key, gate word, join step; k_fine<false>: request,
// key): slot i's word is 4 << sh bytes after slot i - 1's, so a slot's words
// share a cache line.
struct SlotPtr {
  CF_GLOBAL uint32_t *p;
  uint32_t sh;
  __device__ __forceinline__ CF_GLOBAL uint32_t &operator[](uint32_t i) const {
    return *(CF_GLOBAL uint32_t *)((CF_GLOBAL char *)p + ((i << sh) << 2));
  }
  __device__ __forceinline__ SlotPtr operator+(uint32_t i) const { return SlotPtr{&(*this)[i], sh}; }
};
// k_fine<true>: the four words of a running slot, read in one 16-byte load
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
struct Slot4 {
  uint32_t r, k, g, q;
};
__device__ __forceinline__ Slot4 slot_get(const SlotPtr &rr, uint32_t j) {
  const u32x4 v = *(const CF_GLOBAL u32x4 *)((CF_GLOBAL char *)rr.p + (j << 4));
  return Slot4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ void slot_put(const SlotPtr &rr, uint32_t j, const Slot4 &w) {
  const u32x4 v = {w.r, w.k, w.g, w.q};
  *(CF_GLOBAL u32x4 *)((CF_GLOBAL char *)rr.p + (j << 4)) = v;
}
// element o of a read-only input array
template <typename T>
__device__ __forceinline__ T gload(const T *p, size_t o) {
  return *(const CF_GLOBAL T *)((const CF_GLOBAL char *)p + (uint32_t)o * (uint32_t)sizeof(T));
}

struct Sim {
  const FineArgs *A;
  WaveShared *sh;
  SiLds si;
  GPtr<Req> req;
  GPtr<double> hist;
  GPtr<DlEnt> dl;
  SlotPtr run_r, run_k, run_g, run_q;
  GPtr<uint32_t> mem, pool;
  GPtr<int> pool_next, pool_free;
  size_t soff;
  double lam, now, dl_head_t, t_arr;
  uint64_t events, dirty, ta_exec_mask;
  uint32_t status, dl_head, dl_tail;
  int pool_top, pool_fresh, n_done, nx, lat_slot;
  uint32_t *hrow;      // this triple's histogram rows, or null
  bool remote_gate;
  // Per-executor times: end of the running iteration, end of the last one,
  // and for a decode run the start of its first step and the duration of
  // every step.  k_fine<false> keeps them in LDS (xt, [4][CF_MAX_EXEC]);
  // k_fine<true> keeps them in registers, lane x holding executor x, which
  // leaves its LDS to the stage table that bounds its occupancy.
  double *xt;
  double r_tend, r_last, r_t0, r_dur;
  // decode run: step counter of the executor's stage at the end of its running
  // step (k_fine<false>: LDS; k_fine<true>: lane x's register)
  uint32_t *itgt;
  uint32_t r_itgt;
  // k_fine<true>, lane x for executor x
  double r_wake;       // next visibility time of a blocked request of a gated stage
  double r_dur2;       // in a joint run: duration of its talker steps
  uint64_t rewake;     // executors whose wake time is to be recomputed in this instant
  int gmark_si;        // gated stage whose running slots runnable_kind has just marked (-1: none)
  uint32_t gmark_n;    // the number of slots it marked eligible
};

enum { XT_END = 0, XT_LAST = 1, XT_T0 = 2, XT_DUR = 3 };
template <int F>
__device__ __forceinline__ double &xt_reg(Sim &S) {
  if constexpr (F == XT_END) return S.r_tend;
  else if constexpr (F == XT_LAST) return S.r_last;
  else if constexpr (F == XT_T0) return S.r_t0;
  else return S.r_dur;
}
template <int F>
__device__ __forceinline__ double xt_regv(const Sim &S) {
  if constexpr (F == XT_END) return S.r_tend;
  else if constexpr (F == XT_LAST) return S.r_last;
  else if constexpr (F == XT_T0) return S.r_t0;
  else return S.r_dur;
}
// time F of executor x (x wave-uniform)
template <bool G, int F>
__device__ __forceinline__ double xt_get(const Sim &S, int x) {
  if constexpr (G) return lane_val(xt_regv<F>(S), x);
  else return S.xt[F * CF_MAX_EXEC + x];
}
// set time F of executor x to the wave-uniform v (every lane active)
template <bool G, int F>
__device__ __forceinline__ void xt_set(Sim &S, int x, double v) {
  if constexpr (G) {
    double &r = xt_reg<F>(S);
    r = lane_id() == x ? v : r;
  } else {
    S.xt[F * CF_MAX_EXEC + x] = v;
  }
}
template <bool G>
__device__ __forceinline__ uint32_t itgt_get(const Sim &S, int x) {
  if constexpr (G) return (uint32_t)__builtin_amdgcn_readlane((int)S.r_itgt, x);
  else return S.itgt[x];
}
template <bool G>
__device__ __forceinline__ void itgt_set(Sim &S, int x, uint32_t v) {
  if constexpr (G) S.r_itgt = lane_id() == x ? v : S.r_itgt;
  else S.itgt[x] = v;
}
// time F of the executor this lane holds
template <bool G, int F>
__device__ __forceinline__ double xt_own(const Sim &S) {
  if constexpr (G) return xt_regv<F>(S);
  else return S.xt[F * CF_MAX_EXEC + lane_id()];
}

__device__ __forceinline__ Rec rec_get(const Sim &S, uint32_t r) {
  CF_GLOBAL Rec &q = S.req[r].r;
  Rec R;
  R.ex = q.ex;
  R.join = q.join;
  R.misc = q.misc;
  return R;
}
__device__ __forceinline__ void rec_put(const Sim &S, uint32_t r, const Rec &R) {
  CF_GLOBAL Rec &q = S.req[r].r;
  q.ex = R.ex;
  q.join = R.join;
  q.misc = R.misc;
}

// ------------------------------------------------------------------ trace
// attribute a of arrived request r, from its block
__device__ __forceinline__ uint32_t attr(const Sim &S, uint32_t r, int a) {
  const CF_GLOBAL Req &q = S.req[r];
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
__device__ __forceinline__ uint32_t x_of(const Sim &S, uint32_t r, uint32_t sel) {
  uint32_t x = 0;
  while (sel) {
    const int a = __ffs(sel) - 1;
    sel &= sel - 1;
    x += attr(S, r, a);
  }
  return x;
}
__device__ __forceinline__ uint32_t nout_of(const Sim &S, uint32_t r, int t, int c) {
  if ((S.sh->ml.pfo[t] >> c) & 1u) return 1;
  const uint32_t v = attr(S, r, S.sh->ml.nout_attr[c]);
  return v < 1 ? 1 : v;
}
__device__ __forceinline__ double arrival_time(const Sim &S, uint32_t r) {
  return ((double)gload(S.A->ticks, S.soff + r) * 0x1p-32) / S.lam;
}
__device__ __forceinline__ int ex_byte(uint64_t ex, int c) { return (int)((ex >> (8 * c)) & 0xFFu); }
__device__ __forceinline__ int rtype(uint32_t misc) { return (int)((misc >> 8) & 7u); }
__device__ __forceinline__ int stage_of(const Sim &S, int x, int c) {
  const uint32_t geo = S.sh->ex_geo[x];
  return (int)(geo & 0xFFFFu) + __popc((geo >> 16) & 0xFFu & ((1u << c) - 1u));
}

// ------------------------------------------------------------------ pool / queues
__device__ __forceinline__ int chunk_alloc(Sim &S) {
  if (S.pool_top > 0) return ri(S.pool_free[--S.pool_top]);
  if (S.pool_fresh < S.A->L.n_chunks) return S.pool_fresh++;
  S.status |= CF_ST_OVERFLOW;
  return -1;
}
__device__ __forceinline__ void chunk_free(Sim &S, int c) {
  if (c >= 0 && c < S.A->L.n_chunks && S.pool_top < S.A->L.n_chunks) {
    if (lane_id() == 0) S.pool_free[S.pool_top] = c;
    S.pool_top++;
  } else {
    S.status |= CF_ST_OVERFLOW;
  }
}

// appends, in lane order, the requests r of the lanes set in bal to stage si's queue
template <bool G>
__device__ void q_push_lanes(Sim &S, int si, uint64_t bal, uint32_t r) {
  const int cnt = __popcll(bal);
  if (cnt == 0) return;
  int qn = S.si.qn[si], tc, tp;
  if constexpr (G) {
    const uint32_t qt = S.si.qt[si];
    tc = qend_chunk(qt);
    tp = qend_pos(qt);
  } else {
    tc = S.si.qtc[si];
    tp = S.si.qtp[si];
  }
  if (qn > 0 && (tc < 0 || tc >= S.A->L.n_chunks || tp < 0 || tp > kChunk)) {
    S.status |= CF_ST_OVERFLOW;
    return;
  }
  if (qn == 0) {
    const int c = chunk_alloc(S);
    if (c < 0) return;
    if constexpr (G) {
      S.si.qh[si] = qend(c, 0);
    } else {
      S.si.qhc[si] = c;
      S.si.qhp[si] = 0;
    }
    tc = c;
    tp = 0;
  }
  // the entries fill the tail chunk, then at most one fresh chunk (cnt <= 64)
  const int room = kChunk - tp;
  int c1 = -1;
  if (cnt > room) {
    c1 = chunk_alloc(S);
    if (c1 < 0) return;
    if (lane_id() == 0) S.pool_next[tc] = c1;
  }
  if ((bal >> lane_id()) & 1ull) {
    const int k = (int)lanes_below(bal);
    const int ch = k < room ? tc : c1;
    const int pos = k < room ? tp + k : k - room;
    S.pool[(uint32_t)(ch * kChunk + pos)] = r;
  }
  if constexpr (G) {
    S.si.qt[si] = cnt <= room ? qend(tc, tp + cnt) : qend(c1, cnt - room);
  } else if (cnt <= room) {
    S.si.qtc[si] = tc;
    S.si.qtp[si] = (uint8_t)(tp + cnt);
  } else {
    S.si.qtc[si] = c1;
    S.si.qtp[si] = (uint8_t)(cnt - room);
  }
  S.si.qn[si] = qn + cnt;
}

// pops the first k entries of stage si's queue into dst[0..k)
template <bool G>
__device__ void q_pop(Sim &S, int si, int k, GPtr<uint32_t> dst) {
  int hc, hp, tc, tp;
  if constexpr (G) {
    const uint32_t qh = S.si.qh[si], qt = S.si.qt[si];
    hc = qend_chunk(qh);
    hp = qend_pos(qh);
    tc = qend_chunk(qt);
    tp = qend_pos(qt);
  } else {
    hc = S.si.qhc[si];
    hp = S.si.qhp[si];
    tc = S.si.qtc[si];
    tp = S.si.qtp[si];
  }
  if (k <= 0) return;
  if (k > S.si.qn[si] || hc < 0 || hc >= S.A->L.n_chunks) {
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
    if (lane_id() < take) dst[got + lane_id()] = S.pool[(uint32_t)(hc * kChunk + hp + lane_id())];
    got += take;
    hp += take;
    if (hp == kChunk && got < k) {
      const int nx = ri(S.pool_next[hc]);
      chunk_free(S, hc);
      hc = nx;
      hp = 0;
    }
  }
  __syncthreads();
  if (got < k) return;
  const int qn = S.si.qn[si] - k;
  S.si.qn[si] = qn;
  if (qn == 0) {
    chunk_free(S, hc);
    hc = -1;
    hp = 0;
  } else if (hp == kChunk) {
    const int nx = ri(S.pool_next[hc]);
    if (nx < 0 || nx >= S.A->L.n_chunks) S.status |= CF_ST_OVERFLOW;
    chunk_free(S, hc);
    hc = nx;
    hp = 0;
  }
  if constexpr (G) {
    S.si.qh[si] = qend(hc, hp);
  } else {
    S.si.qhc[si] = hc;
    S.si.qhp[si] = (uint8_t)hp;
  }
}

template <bool G>
__device__ __forceinline__ void enqueue1(Sim &S, uint32_t r, int c, int x) {
  S.events++;
  q_push_lanes<G>(S, stage_of(S, x, c), 1ull, r);
  S.dirty |= 1ull << x;
}

// ------------------------------------------------------------------ delay line
__device__ __forceinline__ void dl_push1(Sim &S, double due, uint32_t v) {
  if (S.dl_tail - S.dl_head > S.A->L.dl_mask) {
    S.status |= CF_ST_OVERFLOW;
    return;
  }
  if (lane_id() == 0) {
    S.dl[S.dl_tail & S.A->L.dl_mask].t = due;
    S.dl[S.dl_tail & S.A->L.dl_mask].v = v;
  }
  if (S.dl_head == S.dl_tail) S.dl_head_t = due;
  S.dl_tail++;
}

// ------------------------------------------------------------------ gating
__device__ __forceinline__ bool token_visible(const Sim &S, uint32_t r, uint32_t misc, int th, int xth, int x,
                                              uint32_t k, uint32_t nth, bool &undecided) {
  const double delta = (xth == x) ? 0.0 : S.A->m.comm;
  double e;
  if (k <= 1) {
    e = S.req[r].t.tfirst;
  } else if ((misc & MISC_TH_DONE) && k == nth) {
    e = S.req[r].t.tlast;
  } else {
    const int si = stage_of(S, xth, th);
    const uint32_t q = S.req[r].t.thjoin + k - 1u;
    const uint32_t it = S.si.iter[si];
    if (q > it) return false;
    const GPtr<double> h = S.hist + (uint32_t)(S.si.hist[si] * kHist);
    if (it - q < (uint32_t)kHist) {
      e = h[q & (kHist - 1)];
    } else {
      e = h[(it - (kHist - 1)) & (kHist - 1)];  // oldest kept step: token k is no later
      if (!(e + delta <= S.now)) {
        undecided = true;
        return false;
      }
    }
  }
  return e + delta <= S.now;
}

__device__ __forceinline__ bool slot_eligible(const Sim &S, uint32_t r, uint32_t tok, int c, int x, bool &undecided) {
  const Rec R = rec_get(S, r);
  const int t = rtype(R.misc);
  if (S.sh->ml.ta_c[t] != c) return true;
  const int th = S.sh->ml.th_c[t];
  const uint32_t nth = nout_of(S, r, t, th);
  const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
  return token_visible(S, r, R.misc, th, ex_byte(R.ex, th), x, k, nth, undecided);
}

// k_fine<true>: time at which token k of request r, emitted by its gate
// source (component th on executor xth), is visible at executor x: e_k +
// delta (+inf while the step emitting it is not scheduled).  wsi receives
// the thinker's ring slot while that time may still change (step not
// completed), else -1.
__device__ __forceinline__ double token_vis(const Sim &S, uint32_t r, uint32_t misc, int th, int xth, int x,
                                            uint32_t k, uint32_t nth, int &wsi, bool &undecided) {
  const double delta = (xth == x) ? 0.0 : S.A->m.comm;
  wsi = -1;
  double e;
  if (k <= 1) {
    e = S.req[r].t.tfirst;
  } else if ((misc & MISC_TH_DONE) && k == nth) {
    e = S.req[r].t.tlast;
  } else {
    const int lx = lx_of<true>(S.si, stage_of(S, xth, th));
    const int slot = S.si.hist[lx];
    const uint32_t q = S.req[r].t.thjoin + k - 1u;
    if (q > S.si.sched[slot]) {
      wsi = slot;
      return __builtin_inf();
    }
    const uint32_t it = S.si.iter[lx];
    const GPtr<double> h = S.hist + (uint32_t)(slot * kRing);
    if (q > it) {
      wsi = slot;  // predicted end of a step of the running decode run
      e = h[q & (kRing - 1)];
    } else if (it - q < (uint32_t)kKeep) {
      e = h[q & (kRing - 1)];
    } else {
      e = h[(it - (kKeep - 1)) & (kRing - 1)];  // oldest kept step: token k is no later
      if (!(e + delta <= S.now)) {
        undecided = true;
        return __builtin_inf();
      }
    }
  }
  return e + delta;
}

// k_fine<true>: visibility time of the thinker token that the running slot
// (request r, tok tokens) of gated stage component c on executor x waits for
// (-inf for requests whose type is not gated at c); xth receives the
// thinker's executor
__device__ __forceinline__ double slot_vis(const Sim &S, uint32_t r, uint32_t tok, int c, int x, int &xth, int &wsi,
                                           bool &undecided) {
  const Rec R = rec_get(S, r);
  const int t = rtype(R.misc);
  xth = x;
  wsi = -1;
  if (S.sh->ml.ta_c[t] != c) return -__builtin_inf();
  const int th = S.sh->ml.th_c[t];
  const uint32_t nth = nout_of(S, r, t, th);
  const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
  xth = ex_byte(R.ex, th);
  return token_vis(S, r, R.misc, th, xth, x, k, nth, wsi, undecided);
}

// k_fine<true>: slot_vis from the slot's gate word g and thinker join step
// q0, without reading the request's record or trace: the step's ring entry
// is the time of its token (for a finished thinker's last token too, while
// that step is kept in the ring).  The thinker's ring slot, step counter,
// schedule and ring entry are read before the case is known, so the reads
// overlap; comm is the model's transfer delay.
__device__ __forceinline__ double slot_vis_g(const Sim &S, uint32_t r, uint32_t g, uint32_t q0, uint32_t tok, int x,
                                             double comm, int &xth, int &wsi, bool &undecided) {
  xth = x;
  wsi = -1;
  if (!(g & RG_GATED)) return -__builtin_inf();
  xth = (int)((g >> 16) & 63u);
  const uint32_t nth = g & 0xFFFFu;
  const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
  const double delta = (xth == x) ? 0.0 : comm;
  if (k <= 1) return S.req[r].t.tfirst + delta;
  const int lx = (int)((g >> 22) & 511u);
  const int slot = S.si.hist[lx];
  const uint32_t it = S.si.iter[lx];
  const uint32_t q = q0 + k - 1u;
  const GPtr<double> h = S.hist + (uint32_t)(slot * kRing);
  const double hq = h[q & (kRing - 1)];  // every kept or scheduled step's entry
  const bool pend = q > S.si.sched[slot];  // the step is not scheduled yet
  const bool pred = q > it;                // predicted end of a step of the running decode run
  wsi = (pend || pred) ? slot : -1;
  double e = hq;
  if (!pend && !pred && it - q >= (uint32_t)kKeep) {
    if (k == nth && (S.req[r].r.misc & MISC_TH_DONE)) {
      e = S.req[r].t.tlast;
    } else {
      e = h[(it - (kKeep - 1)) & (kRing - 1)];  // oldest kept step: token k is no later
      if (!(e + delta <= S.now)) {
        undecided = true;
        return __builtin_inf();
      }
    }
  }
  return pend ? __builtin_inf() : e + delta;
}

template <bool G>
__device__ __forceinline__ bool eligible(const Sim &S, uint32_t r, uint32_t tok, int c, int x, bool &undecided) {
  if constexpr (G) {
    int xth, wsi;
    return slot_vis(S, r, tok, c, x, xth, wsi, undecided) <= S.now;
  } else {
    return slot_eligible(S, r, tok, c, x, undecided);
  }
}

// k_fine<true>: the decode steps of the thinker stage with ring slot `slot`
// were (re)scheduled; the registered executors recompute their wake time
__device__ __forceinline__ void notify(Sim &S, int slot) {
  const uint64_t w = S.si.watch[slot];
  if (w) {
    S.rewake |= w;
    S.si.watch[slot] = 0;
  }
}

// ------------------------------------------------------------------ requests
template <bool G>
__device__ void arrive(Sim &S, uint32_t r) {
  const KModel &m = S.A->m;
  const FineArgs &A = *S.A;
  const WaveShared &sh = *S.sh;
  S.events++;
  const size_t o = S.soff + r;
  // every field of the request is loaded before any is used (one memory latency)
  const uint8_t tv = gload(A.type, o);
  const uint64_t k0v = gload(A.rkey0, o), k1v = gload(A.rkey1, o);
  const uint32_t akv = gload(A.akey, o);
  const uint16_t prv = gload(A.prompt, o), ouv = gload(A.out, o), pav = gload(A.patches, o);
  const uint32_t aiv = gload(A.aud_in, o), aov = gload(A.aud_out, o);
  const int t = ri(tv);
  if (t >= m.nt) {
    S.status |= CF_ST_INVALID;
    return;
  }
  const uint64_t k0 = ru64(k0v), k1 = ru64(k1v);
  const uint32_t ak = ru(akv);
  int alt = 0;
  if (sh.nalt[t] == 2) {
    const uint64_t w0 = sh.aw[t][0], w1 = sh.aw[t][1];
    alt = ((((uint64_t)ak) * (w0 + w1)) >> 32) < w0 ? 0 : 1;
  }
  // the executor of every component of the path at once, lane c for component c
  const uint32_t path = m.path[t];
  uint32_t xl = 0xFFu;
  if (lane_id() < CF_MAX_COMP && ((path >> lane_id()) & 1u)) {
    const int v = sh.route[t][alt][lane_id()];
    const int mc = sh.vminc[v];
    const uint64_t key = ((mc < 4 ? k0 : k1) >> (16 * (mc & 3))) & 0xFFFFull;
    xl = sh.vbase[v] + node_exec((uint32_t)key, sh.vrep1[v], (uint32_t)(sh.vrep[v] - sh.vrep1[v]), sh.vw[v]);
  }
  uint64_t ex = ~0ull;
  for (uint32_t pc = path; pc; pc &= pc - 1) {
    const int c = __ffs(pc) - 1;
    const uint64_t x = (uint32_t)__builtin_amdgcn_readlane((int)xl, c);
    ex = (ex & ~(0xFFull << (8 * c))) | (x << (8 * c));
  }
  Rec R;
  R.ex = ex;
  R.join = 0;
  R.misc = (uint32_t)__popc(m.outm[t]) | ((uint32_t)t << 8);
  if (lane_id() == 0) {
    rec_put(S, r, R);
    // the length attributes, read by the stages from the request's block
    CF_GLOBAL Req &q = S.req[r];
    q.prompt = prv;
    q.out = ouv;
    q.patches = pav;
    q.aud_in = aiv;
    q.aud_out = aov;
  }
  uint32_t src = m.srcm[t];
  while (src) {
    const int c = __ffs(src) - 1;
    src &= src - 1;
    enqueue1<G>(S, r, c, ex_byte(ex, c));
  }
}

// step 2: a delayed delivery of request r to component c2
template <bool G>
__device__ void dl_deliver(Sim &S, uint32_t r, int c2) {
  const Rec R = rec_get(S, r);
  const uint64_t ex = ru64(R.ex);
  const uint32_t join = ru(R.join) + (1u << (4 * c2));
  const uint32_t misc = ru(R.misc);
  if (lane_id() == 0) S.req[r].r.join = join;
  const int t = rtype(misc);
  if (((join >> (4 * c2)) & 15u) == S.A->m.npar[t][c2]) enqueue1<G>(S, r, c2, ex_byte(ex, c2));
}

// Lane-parallel processing of the n members mem[0..n) of a completed
// iteration of stage si (component c) on executor x, in member order.  With
// rs, the members are instead the running slots j < n of rs whose page bit
// j / 64 is set in fbits (the slot order is the member order).
//   IT_BATCH:   ENC/GEN members finish c;
//   IT_PREFILL: members get their first token (TTFT stamps, thinker's
//               streaming delivery to the talker) and finish or join Run;
//   IT_FINISH:  decode members that produced their last token finish c.
template <bool G>
__device__ void members_done(Sim &S, int x, int si, int c, int kind, int n, GPtr<uint32_t> mem,
                             const SlotPtr *rs = nullptr, uint32_t fbits = 0u) {
  const KModel &m = S.A->m;
  const ModelLds &ml = S.sh->ml;
  const bool gated = si_flags<G>(S.si, si) & SF_GATED;
  const int lx = (G && kind != IT_PREFILL) ? 0 : lx_of<G>(S.si, si);  // LLM fields: prefill only
  const uint32_t iter_s = S.si.iter[lx];
  const double now = S.now;
  for (int b = 0; b < n; b += 64) {
    const int j = b + lane_id();
    const bool valid = j < n && (!rs || ((fbits >> (b >> 6)) & 1u));
    if (rs && !__ballot(valid)) continue;  // a page of slots with none finishing
    uint32_t r = 0;
    Rec R = {0, 0, 0};
    uint32_t a_no = 0;  // prefill: the request's output-length attribute at c
    uint64_t tkv = 0;   // the request's arrival tick
    if (valid) {
      r = rs ? (*rs)[j] : mem[j];
      // loads that depend on the request id only, issued with its record
      R = rec_get(S, r);
      tkv = gload(S.A->ticks, S.soff + r);
      if (kind == IT_PREFILL) a_no = attr(S, r, ml.nout_attr[c]);
    }
    const int t = rtype(R.misc);
    bool fin = valid;
    bool stream = false;  // thinker: deliver to the talker now
    int ta = 0;
    uint32_t key = 0, gw = 0, gq = 0;
    if (valid && kind == IT_PREFILL) {
      const uint32_t no = ((ml.pfo[t] >> c) & 1u) ? 1u : (a_no < 1u ? 1u : a_no);  // nout_of(S, r, t, c)
      if (c == ml.ttft_c[t]) {
        S.req[r].t.tfirst = now;
        S.req[r].t.tlast = now;
      }
      if (c == ml.th_c[t]) {
        S.req[r].t.thjoin = iter_s;
        stream = true;
        ta = ml.ta_c[t];
      }
      fin = no == 1;
      key = gated ? (1u | (no << 16)) : iter_s + no - 1u;
      if (gated && ml.ta_c[t] == c) {
        const int th = ml.th_c[t], xth = ex_byte(R.ex, th);
        gw = RG_GATED | ((uint32_t)lx_of<G>(S.si, stage_of(S, xth, th)) << 22) | ((uint32_t)xth << 16) |
             nout_of(S, r, t, th);
        gq = S.req[r].t.thjoin;
      }
    } else if (valid && kind == IT_FINISH) {
      if (c == ml.ttft_c[t]) S.req[r].t.tlast = now;
    }
    const bool append = valid && kind == IT_PREFILL && !fin;
    // delayed deliveries: the streaming one first, then remote children
    const uint32_t ch = fin ? ml.child[t][c] : 0u;
    uint32_t rc = 0, lc = 0;
    for (uint32_t cc = ch; cc;) {
      const int c2 = __ffs(cc) - 1;
      cc &= cc - 1;
      if (ex_byte(R.ex, c2) == x) lc |= 1u << c2;
      else rc |= 1u << c2;
    }
    const bool stream_remote = stream && ex_byte(R.ex, ta) != x;
    if (stream && !stream_remote) lc |= 1u << ta;
    const uint32_t ndl = (stream_remote ? 1u : 0u) + (uint32_t)__popc(rc);
    uint32_t dl_total, dl_off;
    const uint64_t dl_any = __ballot(ndl > 0);
    if (__ballot(ndl > 1) == 0) {
      dl_off = lanes_below(dl_any);
      dl_total = (uint32_t)__popcll(dl_any);
    } else {
      dl_off = wave_excl_scan(ndl, dl_total);
    }
    if (dl_total) {
      if (S.dl_tail - S.dl_head + dl_total > S.A->L.dl_mask + 1u) {
        S.status |= CF_ST_OVERFLOW;
        return;
      }
      const double due = now + m.comm;
      uint32_t pos = S.dl_tail + dl_off;
      if (stream_remote) {
        S.dl[pos & S.A->L.dl_mask].t = due;
        S.dl[pos & S.A->L.dl_mask].v = (r << 4) | (DL_DELIVER << 3) | (uint32_t)ta;
        pos++;
      }
      for (uint32_t cc = rc; cc;) {
        const int c2 = __ffs(cc) - 1;
        cc &= cc - 1;
        S.dl[pos & S.A->L.dl_mask].t = due;
        S.dl[pos & S.A->L.dl_mask].v = (r << 4) | (DL_DELIVER << 3) | (uint32_t)c2;
        pos++;
      }
      if (S.dl_head == S.dl_tail) S.dl_head_t = due;
      S.dl_tail += dl_total;
    }
    // local deliveries: join counters, components whose inputs are complete
    uint32_t join = R.join, ready = 0;
    for (uint32_t cc = lc; cc;) {
      const int c2 = __ffs(cc) - 1;
      cc &= cc - 1;
      join += 1u << (4 * c2);
      if (((join >> (4 * c2)) & 15u) == ml.npar[t][c2]) ready |= 1u << c2;
    }
    // outputs and completion
    uint32_t misc = R.misc;
    bool done = false;
    if (fin && valid) {
      if (c == ml.th_c[t]) misc |= MISC_TH_DONE;
      if ((ml.outm[t] >> c) & 1u) {
        if (ml.kind[c] == CF_GEN) S.req[r].t.tmedia = now;
        misc -= 1u;
        done = (misc & MISC_OUTS) == 0;
      }
    }
    if (valid) {
      S.req[r].r.join = join;
      S.req[r].r.misc = misc;
    }
    // running-set appends (prefill), in member order
    const uint64_t abal = __ballot(append);
    if (abal) {
      const int rn = S.si.rn[lx];
      if (append) {
        const int pos = rn + (int)lanes_below(abal);
        S.run_r[S.si.roff[lx] + pos] = r;
        S.run_k[S.si.roff[lx] + pos] = key;
        if (gated) {
          S.run_g[S.si.roff[lx] + pos] = gw;
          S.run_q[S.si.roff[lx] + pos] = gq;
        }
      }
      S.si.rn[lx] = rn + __popcll(abal);
      if (!gated) {
        const uint32_t mn = dpp_min_u32(append ? key : kNone);
        if (mn < S.si.minfin[lx]) S.si.minfin[lx] = mn;
      }
    }
    // queue appends per ready component, in member order
    if (__ballot(ready != 0)) {
      for (int c2 = 0; c2 < m.nc; c2++) {
        const uint64_t bal = __ballot((ready >> c2) & 1u);
        if (!bal) continue;
        S.events += (uint64_t)__popcll(bal);
        q_push_lanes<G>(S, stage_of(S, x, c2), bal, r);
        S.dirty |= 1ull << x;
      }
    }
    // completed requests: latencies, SLO check, per-type counts
    const uint64_t dbal = __ballot(done);
    if (dbal) {
      bool ok = false;
      int hbin = 0;
      if (done) {
        const double a = ((double)tkv * 0x1p-32) / S.lam;  // arrival_time(S, r)
        double ttft = 0.0, tpot = 0.0, media = 0.0;
        const int tc = ml.ttft_c[t];
        if (tc >= 0) {
          const double tf = S.req[r].t.tfirst;
          ttft = tf - a;
          const uint32_t n1 = nout_of(S, r, t, tc);
          if (n1 > 1) tpot = (S.req[r].t.tlast - tf) / (double)(n1 - 1);
        }
        const double e2e = now - a;
        if (ml.gen_out[t]) media = S.req[r].t.tmedia - a;
        ok = ttft <= ml.slo[t][0] && tpot <= ml.slo[t][1] && e2e <= ml.slo[t][2] && media <= ml.slo[t][3];
        if (S.hrow) hbin = target_bin(S.A->tg, S.A->nb, t, ttft, tpot, e2e, media);
        if (S.lat_slot >= 0) {
          double *Lp = S.A->lat + ((size_t)S.lat_slot * S.A->n + r) * 4;
          Lp[0] = ttft;
          Lp[1] = tpot;
          Lp[2] = e2e;
          Lp[3] = media;
        }
      }
      if (done) {
        atomicAdd(&S.sh->cnt[t], 1u);
        if (ok) atomicAdd(&S.sh->met[t], 1u);
        if (S.hrow) atomicAdd(S.hrow + t * (S.A->nb + 1) + hbin, 1u);
      }
      S.events += (uint64_t)__popcll(dbal);
      S.n_done += __popcll(dbal);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ iterations
template <bool G>
__device__ void start_iter(Sim &S, int x, int l, int si, int c, int kind, bool lazy, uint32_t bound) {
  const KModel &m = S.A->m;
  WaveShared &sh = *S.sh;
  double dur;
  int nmem = 0;
  const uint32_t fl = si_flags<G>(S.si, si);
  const int lx = (G && !(fl & SF_LLM)) ? 0 : lx_of<G>(S.si, si);
  if (kind != IT_DECODE) {
    const int qn = S.si.qn[si];
    const int beff = si_beff<G>(S.si, si);
    const int room = kind == IT_PREFILL ? beff - S.si.rn[lx] : beff;
    const int n = qn < room ? qn : room;
    const GPtr<uint32_t> dst = S.mem + (uint32_t)(x * CF_MAX_BATCH);
    q_pop<G>(S, si, n, dst);
    if (S.status & CF_ST_OVERFLOW) return;  // the triple is abandoned at the end of this instant
    uint32_t xs = 0;
    const uint32_t sel = m.xsel[c];
    for (int b = 0; b < n; b += 64) {
      const int j = b + lane_id();
      xs += (j < n) ? x_of(S, dst[j], sel) : 0u;
    }
    xs = dpp_sum_u32(xs);
    dur = (m.k0[c] + m.k1[c] * (double)xs) + m.k2[c] * (double)n;
    if (m.tp_any) dur = m.tps[c][sh.ex_tp[x]] * dur;
    if (fl & SF_ENC) {
      const bool ran = (sh.ex_st[x] >> 1) & 1u;
      if (!ran || xt_get<G, XT_LAST>(S, x) < S.now) dur = dur + m.cpu_pre;
    }
    nmem = n;
  } else if (!(fl & SF_GATED)) {
    const int rn = S.si.rn[lx];
    dur = m.d0[c] + m.d1[c] * (double)rn;
    if (m.tp_any) dur = m.tps[c][sh.ex_tp[x]] * dur;
    nmem = rn;
    // Decode run: while no input reaches this executor, its next steps are
    // decode steps of this stage with the same members, so the end of every
    // step follows by repeated addition (run_walk).  Run to the first
    // finishing step; an input reaching the executor earlier cuts the run
    // (cut_run).
    const uint32_t it0 = S.si.iter[lx];
    uint32_t itgt = it0 + 1u;
    const double t1 = S.now + dur;
    double tend = t1;
    uint32_t fin = S.si.minfin[lx];
    if constexpr (G) fin = fin < bound ? fin : bound;  // k_fine<true>: runs also stop at bound
    if (lazy && dur > 0.0 && fin > itgt) {
      const uint32_t more = fin - itgt < 65535u ? fin - itgt : 65535u;
      uint32_t taken = 0;
      tend = run_walk(t1, dur, more, __builtin_inf(), &taken);
      itgt += taken;
    }
    if constexpr (G) {
      // k_fine<true>: a thinker stage records the predicted end of every
      // step of the run in its ring, one step per lane
      if (fl & SF_THINKER) {
        const int slot = S.si.hist[lx];
        const GPtr<double> h = S.hist + (uint32_t)(slot * kRing);
        for (uint32_t i = (uint32_t)lane_id(); i <= itgt - (it0 + 1u); i += 64u) {
          uint32_t taken = 0;
          h[(it0 + 1u + i) & (kRing - 1)] = run_walk(t1, dur, i, __builtin_inf(), &taken);
        }
        S.si.sched[slot] = itgt;
      }
    }
    xt_set<G, XT_T0>(S, x, S.now);
    xt_set<G, XT_DUR>(S, x, dur);
    itgt_set<G>(S, x, itgt);
    xt_set<G, XT_END>(S, x, tend);
    sh.ex_st[x] = (sh.ex_st[x] & 2u) | 1u | ((uint32_t)kind << 2) | ((uint32_t)l << 4) | ((uint32_t)l << 8) |
                  ((uint32_t)nmem << 12) | (itgt > it0 + 1u ? EX_RUN : 0u);
    return;
  } else {
    // gated stage: mark the eligible running requests
    const int rn = S.si.rn[lx];
    const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lx];
    const SlotPtr rk = S.run_k + (uint32_t)S.si.roff[lx];
    uint32_t cntm = 0;
    if (G && S.gmark_si == si) {
      cntm = S.gmark_n;  // marked by runnable_kind in this instant
    } else {
      const double comm = m.comm;
      bool undecided = false;
      for (int b = 0; b < rn; b += 64) {
        const int j = b + lane_id();
        if (j < rn) {
          uint32_t v;
          bool el;
          if constexpr (G) {
            const Slot4 w = slot_get(rr, (uint32_t)j);
            v = w.k;
            int xth, wsi;
            el = slot_vis_g(S, w.r, w.g, w.q, v & RK_TOK, x, comm, xth, wsi, undecided) <= S.now;
          } else {
            v = rk[j];
            el = eligible<G>(S, rr[j], v & RK_TOK, c, x, undecided);
          }
          if (el != ((v & MARK) != 0)) rk[j] = v ^ MARK;  // only a changed mark is written
          cntm += el ? 1u : 0u;
        }
      }
      if (__ballot(undecided)) S.status |= CF_ST_OVERFLOW;
      cntm = dpp_sum_u32(cntm);
      __syncthreads();
    }
    S.gmark_si = -1;
    dur = m.d0[c] + m.d1[c] * (double)cntm;
    if (m.tp_any) dur = m.tps[c][sh.ex_tp[x]] * dur;
    nmem = (int)cntm;
    if constexpr (G) {
      if (fl & SF_THINKER) {  // a gated stage that is also a gate source
        const uint32_t it1 = S.si.iter[lx] + 1u;
        const int slot = S.si.hist[lx];
        if (lane_id() == 0) S.hist[(uint32_t)(slot * kRing) + (it1 & (kRing - 1))] = S.now + dur;
        S.si.sched[slot] = it1;
      }
    }
  }
  xt_set<G, XT_END>(S, x, S.now + dur);
  itgt_set<G>(S, x, S.si.iter[lx] + 1u);
  sh.ex_st[x] = (sh.ex_st[x] & 2u) | 1u | ((uint32_t)kind << 2) | ((uint32_t)l << 4) | ((uint32_t)l << 8) |
                ((uint32_t)nmem << 12);
}

template <bool G>
__device__ int runnable_kind(Sim &S, int x, int si, int c) {
  // the stage's fields are read together (one LDS latency), the LLM ones
  // before they are known to be needed
  const uint32_t fl = si_flags<G>(S.si, si);
  const int qn = S.si.qn[si];
  const int beff = si_beff<G>(S.si, si);
  const int lx = lx_of<G>(S.si, si);
  if (!(fl & SF_LLM)) return qn > 0 ? IT_BATCH : -1;
  const int rn = S.si.rn[lx];
  if (qn > 0 && rn < beff) return IT_PREFILL;
  if (rn == 0) return -1;
  if (!(fl & SF_GATED)) return IT_DECODE;
  const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lx];
  const SlotPtr rk = S.run_k + (uint32_t)S.si.roff[lx];
  bool any = false, undecided = false;
  if constexpr (G) {
    // k_fine<true>: mark every eligible slot now; a decode step started on
    // this stage in the same instant takes the marks as they are
    uint32_t cnt = 0;
    const double comm = S.A->m.comm;
    for (int b = 0; b < rn; b += 64) {
      const int j = b + lane_id();
      if (j < rn) {
        const Slot4 w = slot_get(rr, (uint32_t)j);
        const uint32_t v = w.k;
        int xth, wsi;
        const bool el = slot_vis_g(S, w.r, w.g, w.q, v & RK_TOK, x, comm, xth, wsi, undecided) <= S.now;
        if (el != ((v & MARK) != 0)) rk[j] = v ^ MARK;  // only a changed mark is written
        cnt += el ? 1u : 0u;
      }
    }
    cnt = dpp_sum_u32(cnt);
    __syncthreads();
    S.gmark_si = si;
    S.gmark_n = cnt;
    any = cnt > 0;
  } else {
    for (int b = 0; b < rn && !any; b += 64) {
      const int j = b + lane_id();
      bool el = false;
      if (j < rn) el = eligible<G>(S, rr[j], rk[j] & RK_TOK, c, x, undecided);
      any = __ballot(el) != 0;
    }
  }
  if (__ballot(undecided)) S.status |= CF_ST_OVERFLOW;
  return any ? IT_DECODE : -1;
}

// k_fine<true>: what the gated stages on executor x wait for, seen from the
// thinker stage si on x, called when none of their running requests is
// eligible.  qmin: the first step of si whose token a request whose thinker
// is si waits for.  joint: exactly one gated stage (gsi) has running
// requests, all of them wait for the next step of si; kta then receives the
// talker steps before its first request finishes.
struct GateView {
  uint32_t qmin, kta;
  int gsi;
  bool joint;
};
__device__ __forceinline__ GateView local_gate_view(const Sim &S, int x, int si) {
  const uint32_t geo = S.sh->ex_geo[x];
  const int ns = __popc((geo >> 16) & 0xFFu), first = (int)(geo & 0xFFFFu);
  const int lth = lx_of<true>(S.si, si);
  const uint32_t next = S.si.iter[lth] + 1u;
  uint32_t qmin = kNone, kta = kNone;
  int gsi = -1, nbusy = 0;
  bool other = false;  // a running request that does not wait for the next step of si
  for (int g = first; g < first + ns; g++) {
    if (!(si_flags<true>(S.si, g) & SF_GATED)) continue;
    const int lg = lx_of<true>(S.si, g);
    const int rn = S.si.rn[lg];
    if (rn == 0) continue;
    nbusy++;
    gsi = g;
    const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lg];
    for (int b = 0; b < rn; b += 64) {
      const int j = b + lane_id();
      if (j < rn) {
        const Slot4 w = slot_get(rr, (uint32_t)j);
        const uint32_t v = w.k, g = w.g;
        const uint32_t tok = v & RK_TOK;
        bool waits_next = false;
        if ((g & RG_GATED) && (int)((g >> 22) & 511u) == lth && (int)((g >> 16) & 63u) == x) {
          const uint32_t nth = g & 0xFFFFu;
          const uint32_t k = tok + 1u < nth ? tok + 1u : nth;
          const uint32_t q = w.q + k - 1u;
          // a thinker on this executor has finished once its last step is completed
          if (k > 1u && !(k == nth && q < next)) {
            qmin = q < qmin ? q : qmin;
            waits_next = q == next;
          }
        }
        other |= !waits_next;
        const uint32_t left = rk_own(v) - tok;
        kta = left < kta ? left : kta;
      }
    }
  }
  GateView v;
  v.qmin = dpp_min_u32(qmin);
  v.kta = dpp_min_u32(kta);
  v.gsi = gsi;
  v.joint = nbusy == 1 && __ballot(other) == 0;
  return v;
}

// k_fine<true>: joint run of thinker stage sth (index lth on x) and gated
// stage sta.  With no other stage runnable and every talker request waiting
// for the thinker's next token on this executor, the executor alternates a
// thinker decode step and a talker decode step over all its running
// requests, so every step end follows by alternately adding the two step
// durations.  The run stops at the first step with a finishing request of
// either stage; an input cuts it (cut_run).  Returns false (nothing started)
// for steps of zero duration.
__device__ __forceinline__ bool start_joint(Sim &S, int x, int lth, int sth, int sta, uint32_t kta) {
  const KModel &m = S.A->m;
  WaveShared &sh = *S.sh;
  const int cth = si_comp<true>(S.si, sth), cta = si_comp<true>(S.si, sta);
  const int lx = lx_of<true>(S.si, sth), lg = lx_of<true>(S.si, sta);
  double d1 = m.d0[cth] + m.d1[cth] * (double)S.si.rn[lx];
  double d2 = m.d0[cta] + m.d1[cta] * (double)S.si.rn[lg];
  if (m.tp_any) {
    d1 = m.tps[cth][sh.ex_tp[x]] * d1;
    d2 = m.tps[cta][sh.ex_tp[x]] * d2;
  }
  if (!(d1 > 0.0) || !(d2 > 0.0)) return false;
  const uint32_t it0 = S.si.iter[lx];
  const uint32_t kth = S.si.minfin[lx] - it0;  // thinker steps up to its first finisher
  uint32_t n = 2u * (kth < kThRun ? kth : kThRun) - 1u;
  if (2u * kta < n) n = 2u * kta;
  const int slot = S.si.hist[lx];
  const GPtr<double> h = S.hist + (uint32_t)(slot * kRing);
  // thinker step s, then talker step s while the run lasts; lane j keeps the
  // end of the j-th thinker step of the current block of 64, written to the
  // ring when the block is complete
  const uint32_t nth = (n + 1u) >> 1;
  double t = S.now, tl = 0.0;
  for (uint32_t s = 1; s <= nth; s++) {
    t = t + d1;
    const uint32_t j = (s - 1u) & 63u;
    tl = (uint32_t)lane_id() == j ? t : tl;
    if (j == 63u || s == nth) {
      if ((uint32_t)lane_id() <= j) h[(it0 + s - j + (uint32_t)lane_id()) & (kRing - 1)] = tl;
    }
    if (2u * s <= n) t = t + d2;
  }
  S.si.sched[slot] = it0 + nth;
  xt_set<true, XT_T0>(S, x, S.now);
  xt_set<true, XT_DUR>(S, x, d1);
  S.r_dur2 = lane_id() == x ? d2 : S.r_dur2;
  itgt_set<true>(S, x, n);  // steps of the run, thinker first
  xt_set<true, XT_END>(S, x, t);
  const uint32_t lta = (uint32_t)(sta - (int)(sh.ex_geo[x] & 0xFFFFu));
  sh.ex_st[x] = (sh.ex_st[x] & 2u) | 1u | (IT_JOINT << 2) | ((uint32_t)lth << 4) | ((uint32_t)lth << 8) | EX_RUN |
                (lta << 22);
  return true;
}

template <bool G>
__device__ __forceinline__ void try_start(Sim &S, int x) {
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[x];
  const uint32_t geo = sh.ex_geo[x];
  const int ns = __popc((geo >> 16) & 0xFFu), first = (int)(geo & 0xFFFFu);
  const int rr = (st >> 4) & 15u;
  for (int i = 0; i < ns; i++) {
    int l = (rr == 15) ? i : rr + 1 + i;  // rr < ns, i < ns
    if (l >= ns) l -= ns;
    const int si = first + l;
    const int kind = runnable_kind<G>(S, x, si, si_comp<G>(S.si, si));
    if (kind >= 0) {
      bool lazy = false;
      uint32_t bound = kNone;
      const uint32_t fl = si_flags<G>(S.si, si);
      const uint32_t no_run = G ? SF_GATED : (SF_THINKER | SF_GATED);
      if (kind == IT_DECODE && !(fl & no_run) &&
          (S.si.qn[si] == 0 || S.si.rn[lx_of<G>(S.si, si)] >= si_beff<G>(S.si, si))) {
        lazy = true;  // ... unless a stage checked after this one has work
        for (int i2 = i + 1; i2 < ns && lazy; i2++) {
          int l2 = (rr == 15) ? i2 : rr + 1 + i2;
          if (l2 >= ns) l2 -= ns;
          if (runnable_kind<G>(S, x, first + l2, si_comp<G>(S.si, first + l2)) >= 0) lazy = false;
        }
        if constexpr (G) {
          if (lazy && (fl & SF_THINKER)) {
            bound = S.si.iter[lx_of<G>(S.si, si)] + kThRun;
            if ((S.ta_exec_mask >> x) & 1ull) {
              const GateView gv = local_gate_view(S, x, si);
              if (gv.joint && start_joint(S, x, l, si, gv.gsi, gv.kta)) {
                notify(S, S.si.hist[lx_of<G>(S.si, si)]);
                return;
              }
              bound = gv.qmin < bound ? gv.qmin : bound;
            }
          }
        }
      }
      start_iter<G>(S, x, l, si, si_comp<G>(S.si, si), kind, lazy, bound);
      if constexpr (G) {
        if ((fl & SF_THINKER) && kind == IT_DECODE) notify(S, S.si.hist[lx_of<G>(S.si, si)]);
      }
      return;
    }
  }
}

// An input reached executor x, busy in a decode run: the run stops at the
// first step that ends at or after now (the steps before it are unchanged).
template <bool G>
__device__ void cut_run(Sim &S, int x) {
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[x];
  if (!(st & EX_RUN) || !(xt_get<G, XT_END>(S, x) > S.now)) return;
  const int si = (int)(sh.ex_geo[x] & 0xFFFFu) + ((st >> 8) & 15u);
  if constexpr (G) {
    if (((st >> 2) & 3u) == IT_JOINT) {
      const uint32_t n = itgt_get<true>(S, x);
      const double d1 = xt_get<true, XT_DUR>(S, x), d2 = lane_val(S.r_dur2, x);
      double t = xt_get<true, XT_T0>(S, x) + d1;
      uint32_t j = 1;
      while (t < S.now && j < n) {
        j++;
        t = t + ((j & 1u) ? d1 : d2);
      }
      xt_set<true, XT_END>(S, x, t);
      itgt_set<true>(S, x, j);
      if (j < n) {
        const int lx = lx_of<true>(S.si, si);
        const int slot = S.si.hist[lx];
        S.si.sched[slot] = S.si.iter[lx] + ((j + 1u) >> 1);
        notify(S, slot);
      }
      return;
    }
  }
  const int lx = lx_of<G>(S.si, si);
  const uint32_t it0 = S.si.iter[lx];
  const uint32_t itgt = itgt_get<G>(S, x);
  const double dur = xt_get<G, XT_DUR>(S, x);
  uint32_t taken = 0;
  const double t = run_walk(xt_get<G, XT_T0>(S, x) + dur, dur, itgt - (it0 + 1u), S.now, &taken);
  const uint32_t j = it0 + 1u + taken;
  xt_set<G, XT_END>(S, x, t);
  itgt_set<G>(S, x, j);
  if (j <= it0 + 1u) sh.ex_st[x] = st & ~EX_RUN;
  if constexpr (G) {
    if ((si_flags<G>(S.si, si) & SF_THINKER) && j < itgt) {
      const int slot = S.si.hist[lx];
      S.si.sched[slot] = j;
      notify(S, slot);
    }
  }
}

__device__ __forceinline__ void thinker_tick(Sim &S) {
  if (S.remote_gate) dl_push1(S, S.now + S.A->m.comm, (DL_TICK << 3));
}

// compacts stage si's running slots, dropping the lanes flagged in drop[]
template <bool G>
__device__ void run_compact(Sim &S, int si, const bool *drop) {
  const int lx = lx_of<G>(S.si, si);
  const int rn = S.si.rn[lx];
  const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lx];
  const SlotPtr rk = S.run_k + (uint32_t)S.si.roff[lx];
  // k_fine<true>: a slot's four words move together (one 16-byte load and store)
  uint32_t vr[CF_MAX_BATCH / 64], vk[CF_MAX_BATCH / 64], vg[CF_MAX_BATCH / 64], vq[CF_MAX_BATCH / 64];
  bool keep[CF_MAX_BATCH / 64];
#pragma unroll
  for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
    const int j = p * 64 + lane_id();
    keep[p] = false;
    vr[p] = 0;
    vk[p] = 0;
    vg[p] = 0;
    vq[p] = 0;
    if (j < rn) {
      if constexpr (G) {
        const Slot4 w = slot_get(rr, (uint32_t)j);
        vr[p] = w.r;
        vk[p] = w.k;
        vg[p] = w.g;
        vq[p] = w.q;
      } else {
        vr[p] = rr[j];
        vk[p] = rk[j];
      }
      keep[p] = !drop[p];
    }
  }
  __syncthreads();
  uint32_t w = 0, mn = kNone;
#pragma unroll
  for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
    const uint64_t bal = __ballot(keep[p]);
    if (keep[p]) {
      const uint32_t d = w + lanes_below(bal);
      if constexpr (G) {
        slot_put(rr, d, Slot4{vr[p], vk[p], vg[p], vq[p]});
      } else {
        rr[d] = vr[p];
        rk[d] = vk[p];
      }
      mn = vk[p] < mn ? vk[p] : mn;
    }
    w += (uint32_t)__popcll(bal);
  }
  __syncthreads();
  S.si.rn[lx] = (int)w;
  if (!(si_flags<G>(S.si, si) & SF_GATED)) S.si.minfin[lx] = dpp_min_u32(mn);
}

// processes the running slots flagged in fin[] as finishing members (slot
// order), and drops them from the running set.  k_fine<false> takes them
// straight from their slots; k_fine<true> first collects them into mem (the
// shorter members_done loop measures faster there).
template <bool G>
__device__ void finish_slots(Sim &S, int x, int si, int c, const bool *fin) {
  const int lx = lx_of<G>(S.si, si);
  const int rn = S.si.rn[lx];
  const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lx];
  if constexpr (G) {
    const GPtr<uint32_t> mem = S.mem + (uint32_t)(x * CF_MAX_BATCH);
    uint32_t nf = 0;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
      const int j = p * 64 + lane_id();
      const bool f = j < rn && fin[p];
      const uint64_t bal = __ballot(f);
      if (f) mem[nf + lanes_below(bal)] = rr[j];
      nf += (uint32_t)__popcll(bal);
    }
    __syncthreads();
    members_done<G>(S, x, si, c, IT_FINISH, (int)nf, mem);
  } else {
    uint32_t fbits = 0;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) fbits |= (fin[p] ? 1u : 0u) << p;
    members_done<G>(S, x, si, c, IT_FINISH, rn, S.mem, &rr, fbits);
  }
  run_compact<G>(S, si, fin);
}

// k_fine<true>: end of a joint run of n steps (thinker first): the thinker
// stage advanced (n + 1) / 2 steps and every running talker request gained
// n / 2 tokens; the stage of the last step resumes the round robin and its
// finishing requests finish.
__device__ __forceinline__ void complete_joint(Sim &S, int x, uint32_t st) {
  WaveShared &sh = *S.sh;
  const int first = (int)(sh.ex_geo[x] & 0xFFFFu);
  const int lth = (st >> 8) & 15u, lta = (st >> 22) & 15u;
  const int sth = first + lth, sta = first + lta;
  const uint32_t n = itgt_get<true>(S, x);
  const uint32_t nth_s = (n + 1u) >> 1, nta_s = n >> 1;
  const uint32_t llast = (n & 1u) ? (uint32_t)lth : (uint32_t)lta;
  sh.ex_st[x] = (st & ~(1u | EX_RUN | (15u << 4) | (15u << 22))) | 2u | (llast << 4);
  xt_set<true, XT_LAST>(S, x, S.now);
  xt_set<true, XT_END>(S, x, __builtin_inf());  // idle: no pending end
  S.dirty |= 1ull << x;
  // thinker
  const int lx = lx_of<true>(S.si, sth);
  const int cth = si_comp<true>(S.si, sth);
  const int rn = S.si.rn[lx];
  const uint32_t it = S.si.iter[lx] + nth_s;
  S.si.iter[lx] = it;
  S.events += (uint64_t)rn * (uint64_t)nth_s;
  // talker
  const int lg = lx_of<true>(S.si, sta);
  const int cta = si_comp<true>(S.si, sta);
  const int rng = S.si.rn[lg];
  const SlotPtr rkg = S.run_k + (uint32_t)S.si.roff[lg];
  bool fin[CF_MAX_BATCH / 64];
#pragma unroll
  for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
    const int j = p * 64 + lane_id();
    fin[p] = false;
    if (j < rng) {
      const uint32_t v = rkg[j];
      const uint32_t tok = (v & RK_TOK) + nta_s;
      rkg[j] = (v & (0x7FFFu << 16)) | tok;
      fin[p] = !(n & 1u) && tok == rk_own(v);
    }
  }
  S.events += (uint64_t)rng * (uint64_t)nta_s;
  __syncthreads();
  if (n & 1u) {
    if (it == S.si.minfin[lx]) {
      const SlotPtr rk = S.run_k + (uint32_t)S.si.roff[lx];
#pragma unroll
      for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
        const int j = p * 64 + lane_id();
        fin[p] = j < rn && rk[j] == it;
      }
      finish_slots<true>(S, x, sth, cth, fin);
    }
  } else {
    bool anyf = false;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) anyf |= __ballot(fin[p]) != 0;
    if (anyf) finish_slots<true>(S, x, sta, cta, fin);
  }
}

template <bool G>
__device__ __forceinline__ void complete_iter(Sim &S, int x) {
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[x];
  const int kind = (st >> 2) & 3u, l = (st >> 8) & 15u, nmem = (st >> 12) & 511u;
  if constexpr (G) {
    if (kind == (int)IT_JOINT) {
      complete_joint(S, x, st);
      return;
    }
  }
  const int si = (int)(sh.ex_geo[x] & 0xFFFFu) + l;
  const int c = si_comp<G>(S.si, si);
  const uint32_t fl = si_flags<G>(S.si, si);
  sh.ex_st[x] = (st & ~(1u | EX_RUN)) | 2u;  // idle, has run
  xt_set<G, XT_LAST>(S, x, S.now);
  xt_set<G, XT_END>(S, x, __builtin_inf());  // idle: no pending end
  S.dirty |= 1ull << x;
  if (kind == IT_BATCH || kind == IT_PREFILL) {
    S.events += (uint64_t)nmem;
    members_done<G>(S, x, si, c, kind, nmem, S.mem + (uint32_t)(x * CF_MAX_BATCH));
    if constexpr (!G) {
      if (fl & SF_THINKER) thinker_tick(S);
    }
    return;
  }
  const int lx = lx_of<G>(S.si, si);
  const int rn = S.si.rn[lx];
  const uint32_t it0 = S.si.iter[lx];
  const uint32_t it = (fl & SF_GATED) ? it0 + 1u : itgt_get<G>(S, x);
  S.si.iter[lx] = it;  // k_fine<true>: a thinker's ring already holds the end of these steps
  if constexpr (!G) {
    if ((fl & SF_THINKER) && lane_id() == 0) S.hist[(uint32_t)(S.si.hist[si] * kHist) + (it & (kHist - 1))] = S.now;
  }
  const SlotPtr rk = S.run_k + (uint32_t)S.si.roff[lx];
  if (!(fl & SF_GATED)) {
    S.events += (uint64_t)rn * (uint64_t)(it - it0);
    if (it == S.si.minfin[lx]) {
      bool fin[CF_MAX_BATCH / 64];
#pragma unroll
      for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
        const int j = p * 64 + lane_id();
        fin[p] = j < rn && rk[j] == it;
      }
      finish_slots<G>(S, x, si, c, fin);
    }
  } else {
    // gated decode step: every marked slot gains one token
    bool fin[CF_MAX_BATCH / 64];
    uint32_t part = 0;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) {
      const int j = p * 64 + lane_id();
      fin[p] = false;
      if (j < rn) {
        const uint32_t v = rk[j];
        if (v & MARK) {
          const uint32_t tok = (v & RK_TOK) + 1u;
          rk[j] = (v & (0x7FFFu << 16)) | tok;
          part++;
          fin[p] = tok == rk_own(v);
        }
      }
    }
    S.events += (uint64_t)dpp_sum_u32(part);
    __syncthreads();
    bool anyf = false;
#pragma unroll
    for (int p = 0; p < CF_MAX_BATCH / 64; p++) anyf |= __ballot(fin[p]) != 0;
    if (anyf) finish_slots<G>(S, x, si, c, fin);
  }
  if constexpr (!G) {
    if (fl & SF_THINKER) thinker_tick(S);
  }
}

// k_fine<true>: recomputes the wake time of executor y, which hosts a gated
// stage: the earliest visibility time, after now, of the token that a
// blocked request of its gated stages waits for from a thinker on another
// executor (a local thinker's steps end on y itself).  Only kept while y is
// idle or in a decode run; y registers with the thinker stages whose steps
// are not final.  Returns whether some such request is eligible already.
__device__ __forceinline__ bool gate_wake(Sim &S, int y) {
  WaveShared &sh = *S.sh;
  const uint32_t st = sh.ex_st[y];
  double w = __builtin_inf();
  bool now_el = false;
  if (!(st & 1u) || (st & EX_RUN)) {
    const uint32_t geo = sh.ex_geo[y];
    const int ns = __popc((geo >> 16) & 0xFFu), first = (int)(geo & 0xFFFFu);
    const double comm = S.A->m.comm;
    bool undecided = false;
    for (int g = first; g < first + ns; g++) {
      if (!(si_flags<true>(S.si, g) & SF_GATED)) continue;
      const int lg = lx_of<true>(S.si, g);
      const int rn = S.si.rn[lg];
      const SlotPtr rr = S.run_r + (uint32_t)S.si.roff[lg];
      for (int b = 0; b < rn; b += 64) {
        const int j = b + lane_id();
        if (j < rn) {
          const Slot4 sw = slot_get(rr, (uint32_t)j);
          int xth, wsi;
          const double tv = slot_vis_g(S, sw.r, sw.g, sw.q, sw.k & RK_TOK, y, comm, xth, wsi, undecided);
          if (xth != y) {
            if (wsi >= 0) atomicOr((unsigned long long *)&S.si.watch[wsi], 1ull << y);
            if (tv <= S.now) now_el = true;
            else w = tv < w ? tv : w;
          }
        }
      }
    }
    if (__ballot(undecided)) S.status |= CF_ST_OVERFLOW;
    w = wave_min_time(w);
    now_el = __ballot(now_el) != 0;
  }
  S.r_wake = lane_id() == y ? w : S.r_wake;  // w is wave-uniform here
  return now_el;
}

// ------------------------------------------------------------------ setup
template <bool G>
__device__ bool setup_plan(Sim &S, int p) {
  const FineArgs &A = *S.A;
  const KModel &m = A.m;
  WaveShared &sh = *S.sh;
  const size_t P = (size_t)A.P;
  const int lane = lane_id();
  const int nv = ri(A.n_nodes[p]);
  if (nv < 1 || nv > CF_MAX_NODES) return false;
  bool groups_ok = true;
  if (lane < CF_MAX_NODES) {
    const uint32_t rep = lane < nv ? A.node_rep[lane * P + p] : 0;
    const uint32_t rep2 = (lane < nv && A.node_rep2) ? A.node_rep2[lane * P + p] : 0;
    sh.vcomp[lane] = lane < nv ? A.node_comp[lane * P + p] : 0;
    sh.vrep[lane] = (uint8_t)(rep + rep2 < 255 ? rep + rep2 : 255);
    sh.vrep1[lane] = (uint8_t)rep;
    sh.vbatch[lane] = lane < nv ? A.node_batch[lane * P + p] : 0;
    sh.vbatch2[lane] = rep2 ? A.node_batch2[lane * P + p] : 0;
    const uint32_t w = rep2 ? A.node_w[lane * P + p] : 0;
    sh.vw[lane] = (uint8_t)w;
    if (rep2 && (rep < 1 || w < 1 || w > 9 || sh.vbatch2[lane] < 1 || sh.vbatch2[lane] > CF_MAX_BATCH ||
                 A.node_gpus2[lane * P + p] < 1))
      groups_ok = false;
  }
  if (__ballot(!groups_ok)) return false;
  for (int j = lane; j < CF_MAX_TYPES * 2 * CF_MAX_COMP; j += 64) (&sh.route[0][0][0])[j] = A.alt_node[j * P + p];
  if (lane < CF_MAX_TYPES) sh.nalt[lane] = lane < m.nt ? A.n_alt[lane * P + p] : 0;
  if (lane < 2 * CF_MAX_TYPES) (&sh.aw[0][0])[lane] = A.alt_w[lane * P + p];
  __syncthreads();
  int base = 0, nsi = 0;
  for (int v = 0; v < nv; v++) {
    const int cm = sh.vcomp[v], rep = sh.vrep[v], b = sh.vbatch[v];
    if (cm == 0 || (cm >> m.nc) || rep < 1 || b < 1 || b > CF_MAX_BATCH) return false;
    sh.vminc[v] = (uint8_t)(__ffs(cm) - 1);
    sh.vbase[v] = (uint8_t)(base < 255 ? base : 255);
    base += rep;
    nsi += rep * __popc(cm);
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
  if (nsi > A.nsi_cap) {
    S.status |= CF_ST_OVERFLOW;
    return true;
  }
  // capacities of the running slots and thinker rings
  int run_need = 0, ring_need = 0, llm_need = 0;
  uint64_t ta_mask = 0;
  for (int v = 0; v < nv; v++) {
    const uint32_t cm = sh.vcomp[v];
    if (cm & m.gated_mask)
      for (int j = 0; j < sh.vrep[v]; j++) ta_mask |= 1ull << (sh.vbase[v] + j);
    for (uint32_t cc = cm; cc;) {
      const int c = __ffs(cc) - 1;
      cc &= cc - 1;
      if (m.kind[c] == CF_LLM) {
        run_need += sh.vrep1[v] * (sh.vbatch[v] < m.cap[c] ? sh.vbatch[v] : m.cap[c]);
        run_need += (sh.vrep[v] - sh.vrep1[v]) * (sh.vbatch2[v] < m.cap[c] ? sh.vbatch2[v] : m.cap[c]);
      }
      if ((m.gate_src_mask >> c) & 1u) ring_need += sh.vrep[v];
      if constexpr (G) {
        if (m.kind[c] == CF_LLM) llm_need += sh.vrep[v];
      }
    }
  }
  S.ta_exec_mask = ta_mask;
  if (run_need > A.L.run_cap || ring_need > A.L.hist_slots) {
    S.status |= CF_ST_OVERFLOW;
    return true;
  }
  if constexpr (G) {
    if (llm_need > A.nl_cap || ring_need > A.nt_cap) {
      S.status |= CF_ST_OVERFLOW;
      return true;
    }
  }
  // executors, one lane each
  if constexpr (G) {
    S.r_tend = __builtin_inf();
    S.r_last = 0.0;
    S.r_t0 = 0.0;
    S.r_dur = 0.0;
    S.r_wake = __builtin_inf();
    S.r_dur2 = 0.0;
    S.r_itgt = 0;
  }
  if (lane < S.nx) {
    int v = 0;
    while (v + 1 < nv && sh.vbase[v + 1] <= lane) v++;
    int first = 0;
    for (int u = 0; u < v; u++) first += sh.vrep[u] * __popc(sh.vcomp[u]);
    first += (lane - sh.vbase[v]) * __popc(sh.vcomp[v]);
    if (m.tp_any) {
      const bool second = lane - sh.vbase[v] >= sh.vrep1[v];
      const uint32_t g = second ? A.node_gpus2[v * P + p] : A.node_gpus[v * P + p];
      sh.ex_tp[lane] = (uint8_t)(g < 1 ? 0 : (g > 8 ? 7 : g - 1));
    }
    sh.ex_geo[lane] = (uint32_t)first | ((uint32_t)sh.vcomp[v] << 16) | ((uint32_t)v << 24);
    sh.ex_st[lane] = 15u << 4;  // idle, never ran, no stage run yet
    if constexpr (!G) {
      S.xt[XT_END * CF_MAX_EXEC + lane] = __builtin_inf();
      S.xt[XT_LAST * CF_MAX_EXEC + lane] = 0.0;
      S.xt[XT_T0 * CF_MAX_EXEC + lane] = 0.0;
      S.xt[XT_DUR * CF_MAX_EXEC + lane] = 0.0;
    }
    if constexpr (!G) S.itgt[lane] = 0;
  }
  if constexpr (G) S.rewake = 0;
  // stage instances, one lane each (prefix sums give run-slot and ring offsets)
  int roff_carry = 0, hs_carry = 0, l_carry = 0;
  for (int s0 = 0; s0 < nsi; s0 += 64) {
    const int s = s0 + lane;
    int c = 0, beff = 0;
    bool llm = false, thk = false;
    if (s < nsi) {
      int v = 0, acc = 0;
      while (acc + sh.vrep[v] * __popc(sh.vcomp[v]) <= s) {
        acc += sh.vrep[v] * __popc(sh.vcomp[v]);
        v++;
      }
      const int per = __popc(sh.vcomp[v]);
      const int k = (s - acc) % per;
      uint32_t cc = sh.vcomp[v];
      for (int q = 0; q < k; q++) cc &= cc - 1;
      c = __ffs(cc) - 1;
      // the batch of the executor's configuration
      const int bn = (s - acc) / per < sh.vrep1[v] ? sh.vbatch[v] : sh.vbatch2[v];
      beff = bn < m.cap[c] ? bn : m.cap[c];
      llm = m.kind[c] == CF_LLM;
      thk = (m.gate_src_mask >> c) & 1u;
    }
    uint32_t tot_r, tot_h, tot_l = 0, lo = 0;
    const uint32_t ro = wave_excl_scan(llm ? (uint32_t)beff : 0u, tot_r);
    const uint32_t ho = wave_excl_scan(thk ? 1u : 0u, tot_h);
    if constexpr (G) lo = wave_excl_scan(llm ? 1u : 0u, tot_l);
    if (s < nsi) {
      const uint32_t fl = (llm ? SF_LLM : 0) | (((m.gated_mask >> c) & 1u) ? SF_GATED : 0) |
                          (thk ? SF_THINKER : 0) | (m.kind[c] == CF_ENC ? SF_ENC : 0) |
                          (m.kind[c] == CF_GEN ? SF_GEN : 0);
      if constexpr (!G) {
        S.si.comp[s] = (uint8_t)c;
        S.si.flags[s] = (uint8_t)fl;
        S.si.beff[s] = (uint16_t)beff;
      }
      S.si.qn[s] = 0;
      if constexpr (G) {
        S.si.qh[s] = qend(-1, 0);
        S.si.qt[s] = qend(-1, 0);
      } else {
        S.si.qhc[s] = -1;
        S.si.qtc[s] = -1;
        S.si.qhp[s] = 0;
        S.si.qtp[s] = 0;
      }
      if constexpr (G) {
        const int ls = l_carry + (int)lo, slot = hs_carry + (int)ho;
        S.si.word[s] = fl | ((uint32_t)c << 8) | ((uint32_t)beff << 12) | ((llm ? (uint32_t)ls : kNoLsi) << 21);
        if (llm) {
          S.si.rn[ls] = 0;
          S.si.iter[ls] = 0;
          S.si.minfin[ls] = kNone;
          S.si.roff[ls] = roff_carry + (int)ro;
          S.si.hist[ls] = thk ? (int16_t)slot : (int16_t)-1;
        }
        if (thk) {
          S.si.sched[slot] = 0;
          S.si.watch[slot] = 0;
        }
      } else {
        S.si.rn[s] = 0;
        S.si.iter[s] = 0;
        S.si.minfin[s] = kNone;
        S.si.roff[s] = roff_carry + (int)ro;
        S.si.hist[s] = thk ? (int16_t)(hs_carry + (int)ho) : (int16_t)-1;
      }
    }
    roff_carry += (int)tot_r;
    hs_carry += (int)tot_h;
    if constexpr (G) l_carry += (int)tot_l;
  }
  __syncthreads();
  return true;
}

extern __shared__ char dyn_lds[];

template <bool G>
// k_fine<false> is held to 72 VGPRs (7 wavefronts per SIMD); k_fine<true>,
// whose LDS table allows fewer wavefronts per CU, to 128.
__global__ void __launch_bounds__(64, G ? 4 : 7) k_fine(const FineArgs *__restrict__ Ap) {
  __shared__ WaveLds<G> wl;
  WaveShared &sh = wl.w;
  const FineArgs &A = *Ap;
  const KModel &m = A.m;
  const int lane = lane_id();
  Sim S;
  S.A = Ap;
  S.sh = &sh;
  {
    const int cap = A.nsi_cap;
    char *p = dyn_lds;
    if constexpr (G) {
      // 8-byte words first: cap, nl_cap and nt_cap are multiples of 64 and the
      // static LDS a multiple of 8 bytes, so every array is aligned
      const int lcap = A.nl_cap, tcap = A.nt_cap;
      S.si.watch = (uint64_t *)p; p += 8 * tcap;
      S.si.qh = (uint32_t *)p; p += 4 * cap;
      S.si.qt = (uint32_t *)p; p += 4 * cap;
      S.si.qn = (int *)p; p += 4 * cap;
      S.si.roff = (int *)p; p += 4 * lcap;
      S.si.rn = (int *)p; p += 4 * lcap;
      S.si.iter = (uint32_t *)p; p += 4 * lcap;
      S.si.minfin = (uint32_t *)p; p += 4 * lcap;
      S.si.sched = (uint32_t *)p; p += 4 * tcap;
      S.si.word = (uint32_t *)p; p += 4 * cap;
      S.si.hist = (int16_t *)p; p += 2 * lcap;
    } else {
      S.si.qhc = (int *)p; p += 4 * cap;
      S.si.qtc = (int *)p; p += 4 * cap;
      S.si.qn = (int *)p; p += 4 * cap;
      S.si.roff = (int *)p; p += 4 * cap;
      S.si.rn = (int *)p; p += 4 * cap;
      S.si.iter = (uint32_t *)p; p += 4 * cap;
      S.si.minfin = (uint32_t *)p; p += 4 * cap;
      S.si.beff = (uint16_t *)p; p += 2 * cap;
      S.si.hist = (int16_t *)p; p += 2 * cap;
      S.si.comp = (uint8_t *)p; p += cap;
      S.si.flags = (uint8_t *)p; p += cap;
      S.si.qhp = (uint8_t *)p; p += cap;
      S.si.qtp = (uint8_t *)p; p += cap;
    }
  }
  if constexpr (!G) {
    S.xt = wl.xt;
    S.itgt = wl.ex_itgt;
  }
  // model tables for per-lane indexing
  for (int j = lane; j < CF_MAX_TYPES * CF_MAX_COMP; j += 64) {
    (&sh.ml.child[0][0])[j] = (&m.child[0][0])[j];
    (&sh.ml.npar[0][0])[j] = (&m.npar[0][0])[j];
  }
  if (lane < CF_MAX_TYPES) {
    sh.ml.ttft_c[lane] = m.ttft_c[lane];
    sh.ml.th_c[lane] = m.th_c[lane];
    sh.ml.ta_c[lane] = m.ta_c[lane];
    sh.ml.outm[lane] = (uint8_t)m.outm[lane];
    sh.ml.pfo[lane] = (uint8_t)m.pfo[lane];
    sh.ml.gen_out[lane] = m.gen_out[lane];
    sh.ml.kind[lane] = (uint8_t)m.kind[lane];
    sh.ml.nout_attr[lane] = (uint8_t)m.nout_attr[lane];
  }
  if (lane < CF_MAX_TYPES * 4) (&sh.ml.slo[0][0])[lane] = (&m.slo[0][0])[lane];
  char *slab = A.slab + (size_t)blockIdx.x * A.L.bytes;
  const Layout &L = A.L;
  S.req = gptr_at<Req>(slab, L.req);
  {
    // running slots interleaved: 4 words per slot (k_fine<true>), 2 (k_fine<false>)
    constexpr uint32_t sh = G ? 2u : 1u;
    CF_GLOBAL uint32_t *run = (CF_GLOBAL uint32_t *)(slab + L.run);
    S.run_r = SlotPtr{run, sh};
    S.run_k = SlotPtr{run + 1, sh};
    S.run_g = SlotPtr{G ? run + 2 : run, sh};
    S.run_q = SlotPtr{G ? run + 3 : run, sh};
  }
  S.hist = gptr_at<double>(slab, L.hist);
  S.mem = gptr_at<uint32_t>(slab, L.mem);
  S.dl = gptr_at<DlEnt>(slab, L.dl);
  S.pool = gptr_at<uint32_t>(slab, L.pool);
  S.pool_next = gptr_at<int>(slab, L.pool_next);
  S.pool_free = gptr_at<int>(slab, L.pool_free);
  __syncthreads();
  const unsigned int per_seed = (unsigned int)A.n_plans * (unsigned int)A.K;
  for (;;) {
    unsigned int tk = 0;
    if (lane == 0) tk = atomicAdd(A.ticket, 1u);
    tk = ru(tk);
    if (tk >= A.total) break;
    // seed-major, then by rate: a triple costs more the lower its rate (less
    // batching, more instants per request), so the costliest triples of a
    // seed are taken first and the launch ends on cheap ones.  With an order
    // table the pairs go by ascending rate over all plans, else by rate
    // index, then plan.
    const int s = (int)(tk / per_seed);
    const unsigned int rem = tk % per_seed;
    int k, i;
    if (A.order) {
      const uint32_t e = ru(A.order[rem]);
      i = (int)(e / (unsigned)A.K);
      k = (int)(e % (unsigned)A.K);
    } else {
      k = (int)(rem / (unsigned)A.n_plans);
      i = (int)(rem % (unsigned)A.n_plans);
    }
    const int p = ri(A.plan_ids[i]);
    const size_t oidx = ((size_t)i * A.K + k) * A.S + s;
    S.soff = (size_t)s * A.n;
    S.lam = rdb(A.rates[(size_t)i * A.K + k]);
    S.events = 0;
    S.status = 0;
    S.dirty = 0;
    S.gmark_si = -1;
    S.dl_head = S.dl_tail = 0;
    S.dl_head_t = __builtin_inf();
    S.pool_top = 0;
    S.pool_fresh = 0;
    S.n_done = 0;
    S.now = 0.0;
    S.lat_slot = -1;
    S.hrow = A.hist ? A.hist + oidx * (size_t)m.nt * (size_t)(A.nb + 1) : nullptr;
    for (int j = 0; j < A.n_lat; j++)
      if (A.lat_triples[j] == (int32_t)oidx) S.lat_slot = j;
    if (lane < CF_MAX_TYPES) {
      sh.met[lane] = 0;
      sh.cnt[lane] = 0;
    }
    __syncthreads();
    const bool ok = (p >= 0 && p < A.P) && S.lam > 0.0 && S.lam < __builtin_inf() && setup_plan<G>(S, p);
    if (!ok) S.status |= CF_ST_INVALID;
    if (ok && !(S.status & CF_ST_OVERFLOW) && A.n > 0) {
      uint32_t next_arr = 0;
      S.t_arr = rdb(arrival_time(S, 0));
      uint64_t instants = 0;
      for (;;) {
        // --- next pending time
        double te = __builtin_inf();
        // an idle executor's end is +inf (so are the lanes past the plan's executors)
        if (lane < S.nx) te = xt_own<G, XT_END>(S);
        if constexpr (G) {
          if (lane < S.nx) {
            const double wk = S.r_wake;
            te = wk < te ? wk : te;
          }
        }
        te = wave_min_time(te);
        double t = te < S.dl_head_t ? te : S.dl_head_t;
        t = S.t_arr < t ? S.t_arr : t;
        if (t == __builtin_inf()) break;
        S.now = t;
        if (++instants > 2 * S.events + 16ull * (uint64_t)A.n + 4096ull || instants > A.lim_instants) {
          S.status |= CF_ST_DEADLOCK;
          break;
        }
        // --- step 1: iterations ending at t, ascending executor
        if (te == t) {
          uint64_t done = __ballot(lane < S.nx && xt_own<G, XT_END>(S) == t);
          if constexpr (G) {
            // wake times due: the executor examines its stages in step 3
            const bool wk = lane < S.nx && S.r_wake == t;
            if (wk) S.r_wake = __builtin_inf();
            S.dirty |= __ballot(wk);
          }
          while (done) {
            const int x = __ffsll((long long)done) - 1;
            done &= done - 1;
            complete_iter<G>(S, x);
          }
        }
        // --- step 2: delayed deliveries due at t (production order), then arrivals at t
        while (S.dl_head != S.dl_tail && S.dl_head_t == t) {
          const uint32_t v = ru(S.dl[S.dl_head & L.dl_mask].v);
          S.dl_head++;
          S.dl_head_t = S.dl_head != S.dl_tail ? rdb(S.dl[S.dl_head & L.dl_mask].t) : __builtin_inf();
          if (((v >> 3) & 1u) == DL_TICK) S.dirty |= S.ta_exec_mask;
          else dl_deliver<G>(S, v >> 4, (int)(v & 7u));
        }
        while (next_arr < (uint32_t)A.n && S.t_arr == t) {
          // the next arrival's time is loaded while this one is handled
          const uint64_t tk = next_arr + 1u < (uint32_t)A.n ? gload(A.ticks, S.soff + next_arr + 1u) : 0ull;
          arrive<G>(S, next_arr);
          next_arr++;
          S.t_arr = next_arr < (uint32_t)A.n ? rdb(((double)tk * 0x1p-32) / S.lam) : __builtin_inf();
        }
        // --- step 3: idle executors whose state changed may start an iteration
        uint64_t cand = S.dirty;
        S.dirty = 0;
        __syncthreads();
        if constexpr (G) {
          // Examine the dirty executors; then recompute the wake times of the
          // executors examined or notified.  An executor found with a request
          // eligible now is examined once more (at most once per instant).
          uint64_t extra = 0;
          for (;;) {
            S.rewake |= cand & S.ta_exec_mask;
            while (cand) {
              const int x = __ffsll((long long)cand) - 1;
              cand &= cand - 1;
              if (!(sh.ex_st[x] & 1u)) try_start<G>(S, x);
              else cut_run<G>(S, x);
            }
            while (S.rewake) {
              const int y = __ffsll((long long)S.rewake) - 1;
              S.rewake &= S.rewake - 1;
              if (gate_wake(S, y) && !((extra >> y) & 1ull)) cand |= 1ull << y;
            }
            if (!cand || (S.status & CF_ST_OVERFLOW)) break;
            extra |= cand;
          }
        } else {
          while (cand) {
            const int x = __ffsll((long long)cand) - 1;
            cand &= cand - 1;
            if (!(sh.ex_st[x] & 1u)) try_start<G>(S, x);
            else cut_run<G>(S, x);
          }
        }
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
__global__ void k_fine_zero(uint32_t *p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}
__global__ void k_fine_reset3(unsigned int *v) {
  v[0] = 0u;
  v[1] = 0u;
  v[2] = 0u;
}

// Position of each (plan, rate) pair when the pairs are sorted by ascending
// rate, ties and NaN (last) by pair index: order[rank] = i * K + k.  One
// thread per pair counts the pairs before it, reading them in LDS tiles.
constexpr int kRankTile = 1024;
__device__ __forceinline__ uint64_t rate_key(double r) {
  uint64_t b = __builtin_bit_cast(uint64_t, r);
  if (r != r) return ~0ull;  // NaN last
  return (b >> 63) ? ~b : (b | (1ull << 63));  // IEEE order as unsigned order
}
__global__ void __launch_bounds__(256) k_rate_order(const double *__restrict__ rates, uint32_t n,
                                                    uint32_t *__restrict__ order) {
  __shared__ uint64_t tile[kRankTile];
  const uint32_t e = blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t key = e < n ? rate_key(rates[e]) : 0ull;
  uint32_t rank = 0;
  for (uint32_t base = 0; base < n; base += kRankTile) {
    __syncthreads();
    for (uint32_t t = threadIdx.x; t < kRankTile; t += blockDim.x)
      tile[t] = base + t < n ? rate_key(rates[base + t]) : ~0ull;
    __syncthreads();
    const uint32_t lim = n - base < (uint32_t)kRankTile ? n - base : (uint32_t)kRankTile;
    for (uint32_t t = 0; t < lim; t++) {
      const uint64_t o = tile[t];
      rank += (o < key || (o == key && base + t < e)) ? 1u : 0u;
    }
  }
  if (e < n) order[rank] = e;
}

// stage instances, LLM stage instances and gate-source stage instances of
// the largest selected plans (out[0..2]; malformed plans are skipped)
__global__ void k_max_si(const uint8_t *n_nodes, const uint8_t *node_comp, const uint8_t *node_rep,
                         const uint8_t *node_rep2, int P, const int32_t *ids, int n, uint32_t llm_mask,
                         uint32_t src_mask, unsigned int *out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int p = ids[i];
  if (p < 0 || p >= P) return;
  const int nv = n_nodes[p];
  if (nv < 1 || nv > CF_MAX_NODES) return;
  unsigned int nsi = 0, nl = 0, nt = 0;
  for (int v = 0; v < nv; v++) {
    const unsigned int rep = node_rep[(size_t)v * P + p] + (node_rep2 ? node_rep2[(size_t)v * P + p] : 0u);
    const unsigned int cm = node_comp[(size_t)v * P + p];
    nsi += rep * (unsigned int)__popc(cm);
    nl += rep * (unsigned int)__popc(cm & llm_mask);
    nt += rep * (unsigned int)__popc(cm & src_mask);
  }
  atomicMax(out, nsi < (unsigned)kMaxSI ? nsi : (unsigned)kMaxSI);
  atomicMax(out + 1, nl < (unsigned)kMaxSI ? nl : (unsigned)kMaxSI);
  atomicMax(out + 2, nt < (unsigned)kMaxSI ? nt : (unsigned)kMaxSI);
}

Layout make_layout(const KModel &m, int n) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  int per_exec_run = 0, n_th = 0;
  for (int c = 0; c < m.nc; c++) {
    if (m.kind[c] == CF_LLM) per_exec_run += m.cap[c] < CF_MAX_BATCH ? m.cap[c] : CF_MAX_BATCH;
    if ((m.gate_src_mask >> c) & 1u) n_th++;
  }
  L.run_cap = CF_MAX_EXEC * per_exec_run;
  L.hist_slots = CF_MAX_EXEC * n_th;
  L.req = take(sizeof(Req) * (size_t)n);
  L.run = take((m.gated_mask ? 16 : 8) * (size_t)L.run_cap);
  L.hist = take(8 * (size_t)L.hist_slots * (m.gated_mask ? kRing : kHist) + 8);
  L.mem = take(4 * (size_t)CF_MAX_EXEC * CF_MAX_BATCH);
  size_t dl = 4096;
  while (dl < 2 * (size_t)n + 8192) dl <<= 1;
  L.dl_mask = (uint32_t)(dl - 1);
  L.dl = take(sizeof(DlEnt) * dl);
  const int maxq = m.max_path > 0 ? m.max_path : 1;
  L.n_chunks = (int)(((size_t)n * maxq + kChunk - 1) / kChunk) + 2 * kMaxSI + 16;
  L.pool = take(4 * (size_t)L.n_chunks * kChunk);
  L.pool_next = take(4 * (size_t)L.n_chunks);
  L.pool_free = take(4 * (size_t)L.n_chunks);
  L.bytes = (off + 4095) & ~(size_t)4095;
  return L;
}

// The allocation-free variant's scratch: one fixed array per device, held
// from the library's load on that device until the process ends.  Host code
// uses the device address hipGetSymbolAddress returns for the current device
// (fixed_scratch_of), never the array's name.
constexpr size_t kFixedScratch = 64ull << 20;
static __device__ __align__(256) char scratch[kFixedScratch];

constexpr int kMaxDevFixed = 64;
std::mutex g_fixed_mu;
char *g_fixed[kMaxDevFixed];

// device address of `scratch` on the current device (looked up once per device)
cf_status fixed_scratch_of(char **ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevFixed) return set_error(CF_EHIP, "no current HIP device");
  std::lock_guard<std::mutex> lock(g_fixed_mu);
  if (!g_fixed[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return set_error(CF_EHIP, "hipGetSymbolAddress of the fixed scratch failed: %s", hipGetErrorString(e));
    }
    g_fixed[dev] = (char *)p;
  }
  *ptr = g_fixed[dev];
  return CF_OK;
}

constexpr size_t kFineHdr = 8192;  // ticket, stage counts, the argument block
// launches of at most this many (plan, rate) pairs take them by ascending rate
// (k_rate_order: quadratic in the pairs, ~1 ms at the limit)
constexpr size_t kOrderMax = 1u << 17;

// cf_eval_fine and cf_eval_fine_noalloc: with fixed == nullptr the call's
// scratch comes from the library's cached allocations, else from the fixed
// region [fixed, fixed + fixed_cap), which bounds the number of wavefronts.
cf_status eval_fine(const cf_model_desc *model, const cf_plan_table *plans, const int32_t *plan_ids_dev,
                    int32_t n_plans, const double *rates_dev, int32_t K, const cf_trace *trace, uint32_t flags,
                    const cf_fine_out *out, void *stream, char *fixed, size_t fixed_cap) {
  FineArgs a;
  memset(&a, 0, sizeof a);
  cf_status st = lower_model(model, &a.m);
  if (st != CF_OK) return st;
  if (!plans || !trace || !out) return set_error(CF_EINVAL, "NULL argument");
  if (trace->n_req > 0 && (!trace->arr_ticks_dev || !trace->type_dev || !trace->patches_dev || !trace->prompt_dev ||
                           !trace->out_dev || !trace->aud_in_ms_dev || !trace->aud_out_ms_dev ||
                           !trace->rkey0_dev || !trace->rkey1_dev || !trace->akey_dev))
    return set_error(CF_EINVAL, "NULL trace array");
  if (flags & ~(CF_DUMP_LAT | CF_EARLY_EXIT)) return set_error(CF_EINVAL, "unknown flags");
  if (flags & CF_EARLY_EXIT) return set_error(CF_EUNSUPPORTED, "CF_EARLY_EXIT is not built");
  const bool dump = (flags & CF_DUMP_LAT) != 0;
  if (n_plans < 0 || K < 1 || trace->n_seeds < 1 || trace->n_req < 0 || plans->P < 0)
    return set_error(CF_EINVAL, "sizes");
  if (n_plans == 0) return CF_OK;
  if (!plan_ids_dev || !rates_dev) return set_error(CF_EINVAL, "NULL argument");
  if (!out->met_dev || !out->cnt_dev || !out->events_dev || !out->status_dev)
    return set_error(CF_EINVAL, "NULL output array");
  if (dump && (!out->lat_dev || out->n_lat < 0 || (out->n_lat > 0 && !out->lat_triples_dev)))
    return set_error(CF_EINVAL, "latency dump arguments");
  if (out->lim_chunks < 0 || out->lim_delay < 0 ||
      (out->lim_delay != 0 && (out->lim_delay < 2 || (out->lim_delay & (out->lim_delay - 1)) != 0)))
    return set_error(CF_EINVAL, "test limits: lim_chunks >= 0, lim_delay 0 or a power of two >= 2");
  if (trace->n_req > (1 << 26)) return set_error(CF_ECAPACITY, "n_req above 2^26");
  const unsigned long long total = (unsigned long long)n_plans * K * trace->n_seeds;
  if (total >= 0xFFFFFFFFull - 65536ull) return set_error(CF_ECAPACITY, "too many triples in one call");
  a.P = plans->P;
  a.n_nodes = plans->n_nodes_dev;
  a.node_comp = plans->node_comp_dev;
  a.node_rep = plans->node_rep_dev;
  a.node_gpus = plans->node_gpus_dev;
  a.node_batch = plans->node_batch_dev;
  a.n_alt = plans->n_alt_dev;
  a.alt_w = plans->alt_w_dev;
  a.alt_node = plans->alt_node_dev;
  {
    const int ng = (plans->node_rep2_dev != nullptr) + (plans->node_batch2_dev != nullptr) +
                   (plans->node_gpus2_dev != nullptr) + (plans->node_w_dev != nullptr);
    if (ng != 0 && ng != 4) return set_error(CF_EINVAL, "second-configuration arrays: all four or none");
  }
  a.node_rep2 = plans->node_rep2_dev;
  a.node_batch2 = plans->node_batch2_dev;
  a.node_gpus2 = plans->node_gpus2_dev;
  a.node_w = plans->node_w_dev;
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
  a.lat = dump ? out->lat_dev : nullptr;
  a.lat_triples = dump ? out->lat_triples_dev : nullptr;
  a.n_lat = dump ? out->n_lat : 0;
  a.hist = nullptr;
  a.tg = nullptr;
  a.nb = 0;
  a.L = make_layout(a.m, trace->n_req);
  a.total = (unsigned int)total;
  // test limits: smaller capacities inside the same slab (every index stays below the capped value)
  if (out->lim_chunks > 0 && out->lim_chunks < a.L.n_chunks) a.L.n_chunks = out->lim_chunks;
  if (out->lim_delay > 0 && (uint32_t)(out->lim_delay - 1) < a.L.dl_mask) a.L.dl_mask = (uint32_t)(out->lim_delay - 1);
  a.lim_instants = out->lim_instants ? out->lim_instants : ~0ull;
  long long waves = 8192;
  if (const char *e = getenv("CF_FINE_WAVES")) waves = atoll(e);
  if (waves < 1) waves = 1;
  if ((unsigned long long)waves > total) waves = (long long)total;
  size_t free_b = 0, tot_b = 0;
  if (hipMemGetInfo(&free_b, &tot_b) == hipSuccess && free_b > 0) {
    const size_t budget = free_b / 2;
    while (waves > 64 && (size_t)waves * a.L.bytes > budget) waves /= 2;
  }
  static_assert(sizeof(FineArgs) + 512 <= kFineHdr, "FineArgs must fit the scratch header");
  char *scr;
  size_t hdr = kFineHdr;
  const size_t npairs = (size_t)n_plans * (size_t)K;
  const size_t order_bytes = npairs <= kOrderMax ? (sizeof(uint32_t) * npairs + 255) & ~(size_t)255 : 0;
  size_t order_off = 0;
  if (fixed) {
    // the target table (if any) and the pair order follow the header; the
    // slabs of as many wavefronts as fit follow them
    if (out->n_bins > 0) {
      st = check_targets(a.m.nt, out->n_bins, out->hist_targets_host);
      if (st != CF_OK) return st;
      hdr += (sizeof(double) * (size_t)a.m.nt * (size_t)out->n_bins * 4 + 255) & ~(size_t)255;
    }
    order_off = hdr;
    hdr += order_bytes;
    if (fixed_cap < hdr + a.L.bytes)
      return set_error(CF_ECAPACITY, "one simulation of %d requests needs %zu bytes of scratch; the fixed scratch holds %zu",
                       trace->n_req, hdr + a.L.bytes, fixed_cap);
    const size_t fit = (fixed_cap - hdr) / a.L.bytes;
    if ((size_t)waves > fit) waves = (long long)fit;
    scr = fixed;
  } else {
    order_off = hdr;
    hdr += order_bytes;
    scr = (char *)scratch_get(SCR_FINE, hdr + (size_t)waves * a.L.bytes, &st);
    if (!scr) return st;
  }
  a.ticket = (unsigned int *)scr;
  unsigned int *max_si = (unsigned int *)(scr + 64);
  FineArgs *args_dev = (FineArgs *)(scr + 512);
  a.slab = scr + hdr;
  hipStream_t s = as_stream(stream);
  a.order = nullptr;
  if (order_bytes) {
    uint32_t *order = (uint32_t *)(scr + order_off);
    hipLaunchKernelGGL(k_rate_order, dim3((unsigned)((npairs + 255) / 256)), dim3(256), 0, s, rates_dev,
                       (uint32_t)npairs, order);
    a.order = order;
  }
  // size the LDS stage table from the largest selected plan
  uint32_t llm_mask = 0;
  for (int c = 0; c < a.m.nc; c++)
    if (a.m.kind[c] == CF_LLM) llm_mask |= 1u << c;
  hipLaunchKernelGGL(k_fine_reset3, dim3(1), dim3(1), 0, s, max_si);
  hipLaunchKernelGGL(k_max_si, dim3((unsigned)((n_plans + 255) / 256)), dim3(256), 0, s, a.n_nodes, a.node_comp,
                     a.node_rep, a.node_rep2, a.P, plan_ids_dev, n_plans, llm_mask, (uint32_t)a.m.gate_src_mask,
                     max_si);
  unsigned int caps[3] = {0, 0, 0};
  st = hip_check(hipMemcpyAsync(caps, max_si, sizeof caps, hipMemcpyDeviceToHost, s), "copy stage count");
  if (st != CF_OK) return st;
  st = hip_check(hipStreamSynchronize(s), "stage count sync");
  if (st != CF_OK) return st;
  auto round64 = [](unsigned int v) { return v < 64u ? 64 : (int)((v + 63u) & ~63u); };
  // k_fine<false>'s table needs 8-entry alignment only; a small table leaves room for more wavefronts per CU
  auto round16 = [](unsigned int v) { return v < 16u ? 16 : (int)((v + 15u) & ~15u); };
  a.nsi_cap = a.m.gated_mask ? round64(caps[0]) : round16(caps[0]);
  a.nl_cap = round64(caps[1]);
  a.nt_cap = round64(caps[2]);
  const size_t lds = a.m.gated_mask ? kSiBytesG * (size_t)a.nsi_cap + kLlmBytesG * (size_t)a.nl_cap +
                                          kThBytesG * (size_t)a.nt_cap
                                    : kSiBytes * (size_t)a.nsi_cap;
  st = hip_check(hipMemcpyAsync(args_dev, &a, sizeof a, hipMemcpyHostToDevice, s), "copy fine args");
  if (st != CF_OK) return st;
  if (out->n_bins > 0) {
    // optional latency histograms: target table to the device, counters cleared by a kernel
    if (!out->hist_dev) return set_error(CF_EINVAL, "n_bins > 0 without hist_dev");
    if (fixed) {
      char *tg = scr + kFineHdr;
      st = hip_check(hipMemcpyAsync(tg, out->hist_targets_host, sizeof(double) * (size_t)a.m.nt * out->n_bins * 4,
                                    hipMemcpyHostToDevice, s),
                     "target table copy");
      a.tg = (const double *)tg;
    } else {
      st = load_targets(a.m.nt, out->n_bins, out->hist_targets_host, &a.tg, s);
    }
    if (st != CF_OK) return st;
    a.hist = out->hist_dev;
    a.nb = out->n_bins;
    const size_t nh = total * (size_t)a.m.nt * (size_t)(a.nb + 1);
    hipLaunchKernelGGL(k_fine_zero, dim3((unsigned)((nh + 255) / 256)), dim3(256), 0, s, a.hist, nh);
    st = hip_check(hipMemcpyAsync(args_dev, &a, sizeof a, hipMemcpyHostToDevice, s), "copy fine args");
    if (st != CF_OK) return st;
  }
  hipLaunchKernelGGL(k_fine_reset, dim3(1), dim3(1), 0, s, a.ticket);
  if (a.m.gated_mask)
    hipLaunchKernelGGL(k_fine<true>, dim3((unsigned)waves), dim3(64), lds, s, (const FineArgs *)args_dev);
  else
    hipLaunchKernelGGL(k_fine<false>, dim3((unsigned)waves), dim3(64), lds, s, (const FineArgs *)args_dev);
  st = hip_check(hipGetLastError(), "cf_eval_fine launch");
  if (st != CF_OK) return st;
  // the argument block is copied from host memory on the stream: wait for it
  return hip_check(hipStreamSynchronize(s), "cf_eval_fine sync");
}

}  // namespace
}  // namespace cf

extern "C" cf_status cf_eval_fine(const cf_model_desc *model, const cf_plan_table *plans,
                                  const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev, int32_t K,
                                  const cf_trace *trace, uint32_t flags, const cf_fine_out *out, void *stream) {
  return cf::eval_fine(model, plans, plan_ids_dev, n_plans, rates_dev, K, trace, flags, out, stream, nullptr, 0);
}

extern "C" cf_status cf_eval_fine_noalloc(const cf_model_desc *model, const cf_plan_table *plans,
                                          const int32_t *plan_ids_dev, int32_t n_plans, const double *rates_dev,
                                          int32_t K, const cf_trace *trace, uint32_t flags, const cf_fine_out *out,
                                          void *stream) {
  char *fixed = nullptr;
  const cf_status st = cf::fixed_scratch_of(&fixed);
  if (st != CF_OK) return st;
  return cf::eval_fine(model, plans, plan_ids_dev, n_plans, rates_dev, K, trace, flags, out, stream, fixed,
                       cf::kFixedScratch);
}
