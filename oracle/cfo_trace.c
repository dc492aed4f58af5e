/*
 * cfo_trace.c -- oracle (test infrastructure only): counter-based random
 * numbers, the pinned log/exp, and synthetic Any-to-Any request traces.
 *
 * The paper drives its simulator with a workload: a set of requests with
 * per-type fractions pi_t and arrival timestamps (Sec. 3.1; Poisson
 * intervals for the text-to-image study, Sec. 6.4).  The trace here is
 * keyed only by (seed, request id), so every plan and every rate sees the
 * same requests (common random numbers).
 *
 *   Philox4x64-10: Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
 *   easy as 1, 2, 3", SC'11.  Pinned by the tests against numpy's Philox.
 *   cfo_log / cfo_exp: Cody-Waite argument reduction followed by a series
 *   (atanh series for log, Taylor for exp); pinned against mpmath.
 */
#include "cfo.h"
#include <math.h>
#include <string.h>

/* ---------------- Philox4x64-10 ---------------- */
static const uint64_t PH_M0 = 0xD2E7470EE14C6C93ull;
static const uint64_t PH_M1 = 0xCA5A826395121157ull;
static const uint64_t PH_W0 = 0x9E3779B97F4A7C15ull; /* golden ratio */
static const uint64_t PH_W1 = 0xBB67AE8584CAA73Bull; /* sqrt(3) - 1 */

void cfo_philox(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) { k0 += PH_W0; k1 += PH_W1; }
    unsigned __int128 p0 = (unsigned __int128)PH_M0 * x0;
    unsigned __int128 p1 = (unsigned __int128)PH_M1 * x2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t y0 = hi1 ^ x1 ^ k0;
    uint64_t y1 = lo1;
    uint64_t y2 = hi0 ^ x3 ^ k1;
    uint64_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* open-interval uniform: (2*(x>>12)+1) * 2^-53, exact in fp64 */
double cfo_uniform(uint64_t x) {
  return (double)(((x >> 12) << 1) | 1u) * 0x1p-53;
}

/* ---------------- pinned log / exp ---------------- */
static double bits_to_double(uint64_t b) { double d; memcpy(&d, &b, 8); return d; }
static uint64_t double_to_bits(double d) { uint64_t b; memcpy(&b, &d, 8); return b; }

/* ln 2 split: HI = ln 2 rounded to 32 significant bits, LO = fl(ln 2 - HI) */
#define CFO_LN2_HI 0x1.62e42ff000000p-1
#define CFO_LN2_LO (-0x1.718432a1b0e26p-35)
#define CFO_INV_LN2 0x1.71547652b82fep+0
#define CFO_SQRT2 0x1.6a09e667f3bcdp+0

/* log(x) for positive normal x:
 *   x = 2^e * m, m in (sqrt2/2, sqrt2], f = m - 1 (exact), s = f/(2+f), z = s^2;
 *   log m = 2 atanh s = f - s (f - R) with R = 2z/3 + 2z^2/5 + ...,
 *   arranged as f - (h - s (h + R)) with h = f^2/2 so that the large part f
 *   stays exact and only small corrections are rounded. */
double cfo_log(double x) {
  uint64_t b = double_to_bits(x);
  int e = (int)((b >> 52) & 0x7ff) - 1023;
  double m = bits_to_double((b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull);
  if (m > CFO_SQRT2) { m = m * 0.5; e = e + 1; }
  double f = m - 1.0;
  double s = f / (2.0 + f);
  double z = s * s;
  /* R = sum_{k=1..10} 2 z^k / (2k+1), coefficients correctly rounded */
  double p = 2.0 / 21.0;
  for (int k = 9; k >= 1; k--) p = p * z + 2.0 / (double)(2 * k + 1);
  double R = z * p;
  double h = 0.5 * f * f;
  double de = (double)e;
  return de * CFO_LN2_HI - ((h - (s * (h + R) + de * CFO_LN2_LO)) - f);
}

/* exp(x) for |x| <= 700:  n = rint(x / ln2), r = x - n ln2 (two steps),
 * Taylor series to degree 14, result scaled by 2^n through the exponent. */
double cfo_exp(double x) {
  static double inv_fact[15];
  static int init = 0;
  if (!init) {
    /* 1/k! as correctly rounded doubles, from exact integer factorials */
    double fact = 1.0; /* k! is exact in fp64 for k <= 18 */
    for (int k = 0; k <= 14; k++) { if (k > 0) fact = fact * (double)k; inv_fact[k] = 1.0 / fact; }
    init = 1;
  }
  double n = rint(x * CFO_INV_LN2);
  double r = (x - n * CFO_LN2_HI) - n * CFO_LN2_LO;
  double p = inv_fact[14];
  for (int k = 13; k >= 0; k--) p = p * r + inv_fact[k];
  int ni = (int)n;
  double scale = bits_to_double((uint64_t)(ni + 1023) << 52);
  return p * scale;
}

/* ---------------- samplers ---------------- */
enum { F_ARRIVAL = 0, F_PROMPT = 1, F_OUT = 2, F_PATCH = 3, F_AUDIN = 4, F_AUDOUT = 5, F_ROUTE = 6 };

static void draw_block(uint64_t seed, uint64_t req, uint64_t field, uint64_t attempt, uint64_t out[4]) {
  uint64_t ctr[4] = {req, field, attempt, 0};
  uint64_t key[2] = {seed, 0};
  cfo_philox(ctr, key, out);
}

/* uniform integer on [lo, hi] from the upper 32 bits */
static int64_t uniform_int(uint64_t x, int64_t lo, int64_t hi) {
  uint64_t span = (uint64_t)(hi - lo + 1);
  return lo + (int64_t)(((x >> 32) * span) >> 32);
}

/* standard normal by the Marsaglia polar method: attempt k uses block
 * (req, field, k); within a block the pairs (x0,x1) then (x2,x3) are tried.
 * After 32 blocks without acceptance the value is 0. */
static double normal_draw(uint64_t seed, uint64_t req, uint64_t field) {
  for (uint64_t k = 0; k < 32; k++) {
    uint64_t x[4];
    draw_block(seed, req, field, k, x);
    for (int h = 0; h < 2; h++) {
      double v1 = 2.0 * cfo_uniform(x[2 * h]) - 1.0;
      double v2 = 2.0 * cfo_uniform(x[2 * h + 1]) - 1.0;
      double w = v1 * v1 + v2 * v2;
      if (w > 0.0 && w < 1.0) {
        double q = (-2.0 * cfo_log(w)) / w;
        return v1 * sqrt(q);
      }
    }
  }
  return 0.0;
}

static int64_t clamp64(int64_t v, int64_t lo, int64_t hi) { return v < lo ? lo : (v > hi ? hi : v); }

static int64_t draw_length(const cfo_dist *d, uint64_t seed, uint64_t req, uint64_t field) {
  switch (d->kind) {
  case CFO_D_CONST:
    return (int64_t)d->p0;
  case CFO_D_LOGNORMAL: {
    double z = normal_draw(seed, req, field);
    double v = cfo_exp(d->p0 + d->p1 * z);
    return clamp64((int64_t)rint(d->scale * v), d->lo, d->hi);
  }
  case CFO_D_EXP: {
    uint64_t x[4];
    draw_block(seed, req, field, 0, x);
    double e = -cfo_log(cfo_uniform(x[0]));
    return clamp64((int64_t)rint(d->p0 * e), d->lo, d->hi);
  }
  default:
    return 0;
  }
}

static uint32_t ceil_div80(uint32_t v) { return (v + 79u) / 80u; }

int cfo_trace_gen(const cfo_model *m, const uint64_t *seeds, int32_t n_seeds, int32_t n_req,
                  cfo_trace *tr, uint64_t *moments) {
  if (n_seeds < 0 || n_req < 0 || m->n_types < 1 || m->n_types > CFO_MAXT) return -1;
  uint64_t wsum = 0;
  for (int t = 0; t < m->n_types; t++) wsum += m->weight[t];
  if (wsum == 0 || wsum > 0xFFFFFFFFull) return -1;
  memset(moments, 0, sizeof(uint64_t) * (size_t)n_seeds * m->n_types * 8);
  for (int s = 0; s < n_seeds; s++) {
    uint64_t seed = seeds[s];
    uint64_t acc = 0;
    for (int i = 0; i < n_req; i++) {
      size_t o = (size_t)s * n_req + i;
      uint64_t x[4];
      draw_block(seed, (uint64_t)i, F_ARRIVAL, 0, x);
      /* exponential gap in units of 2^-32 of the mean inter-arrival time */
      double g = -cfo_log(cfo_uniform(x[0])) * 0x1p32;
      acc += (uint64_t)rint(g);
      tr->arr_ticks[o] = acc;
      /* request type: weighted choice on the upper 32 bits */
      uint64_t v = ((x[1] >> 32) * wsum) >> 32;
      int t = 0;
      uint64_t cum = m->weight[0];
      while (cum <= v) { t++; cum += m->weight[t]; }
      tr->type[o] = (uint8_t)t;
      int nimg = 0;
      if (m->img_kind[t] == CFO_I_CONST) nimg = m->img_lo[t];
      else if (m->img_kind[t] == CFO_I_UNIFORM) nimg = (int)uniform_int(x[2], m->img_lo[t], m->img_hi[t]);
      tr->n_img[o] = (uint8_t)nimg;
      uint32_t patches = 0;
      if (nimg > 0) {
        uint64_t y[4];
        draw_block(seed, (uint64_t)i, F_PATCH, 0, y);
        for (int k = 0; k < nimg; k++) patches += (uint32_t)uniform_int(y[k], m->patch_lo, m->patch_hi);
      }
      tr->patches[o] = (uint16_t)patches;
      tr->prompt[o] = (uint16_t)draw_length(&m->len[t][0], seed, (uint64_t)i, F_PROMPT);
      tr->out[o] = (uint16_t)draw_length(&m->len[t][1], seed, (uint64_t)i, F_OUT);
      tr->aud_in_ms[o] = (uint32_t)draw_length(&m->len[t][2], seed, (uint64_t)i, F_AUDIN);
      tr->aud_out_ms[o] = (uint32_t)draw_length(&m->len[t][3], seed, (uint64_t)i, F_AUDOUT);
      uint64_t y[4];
      draw_block(seed, (uint64_t)i, F_ROUTE, 0, y);
      tr->rkey0[o] = y[0];
      tr->rkey1[o] = y[1];
      tr->akey[o] = (uint32_t)(y[2] >> 32);
      /* per-type moments: count, then the sum of every attribute */
      uint64_t *mo = moments + ((size_t)s * m->n_types + t) * 8;
      mo[0] += 1;
      mo[1 + CFO_A_PROMPT] += tr->prompt[o];
      mo[1 + CFO_A_OUT] += tr->out[o];
      mo[1 + CFO_A_PATCHES] += tr->patches[o];
      mo[1 + CFO_A_AUDIN_MS] += tr->aud_in_ms[o];
      mo[1 + CFO_A_AUDOUT_MS] += tr->aud_out_ms[o];
      mo[1 + CFO_A_AUDIN_TOK] += ceil_div80(tr->aud_in_ms[o]);
      mo[1 + CFO_A_AUDOUT_TOK] += ceil_div80(tr->aud_out_ms[o]);
    }
  }
  return 0;
}

/* ---------------- element-wise helpers for the tests ---------------- */
void cfo_math_n(int32_t op, const double *x, const double *y, double *out, int64_t n) {
  for (int64_t i = 0; i < n; i++) {
    double a = x[i], r = 0.0;
    switch (op) {
    case 0: r = cfo_log(a); break;
    case 1: r = cfo_exp(a); break;
    case 2: r = sqrt(a); break;
    case 3: r = a / y[i]; break;
    case 4: { uint64_t b; memcpy(&b, &a, 8); r = cfo_uniform(b); } break;
    default: break;
    }
    out[i] = r;
  }
}

void cfo_philox_n(const uint64_t *ctr, const uint64_t *key, uint64_t *out, int64_t n) {
  for (int64_t i = 0; i < n; i++) cfo_philox(ctr + 4 * i, key + 2 * i, out + 4 * i);
}
