// cf_abi.hip -- host side of libcf: error reporting, descriptor validation
// and lowering, version.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "cf_internal.h"

namespace cf {

static thread_local char g_err[512];

cf_status set_error(cf_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

cf_status hip_check(hipError_t e, const char *what) {
  if (e == hipSuccess) return CF_OK;
  return set_error(CF_EHIP, "%s: %s", what, hipGetErrorString(e));
}

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

static bool finite_nonneg(double v) { return isfinite(v) && v >= 0.0; }

// largest value attribute a (CF_ATTR_*) of a type-t request can take
static uint64_t attr_hi(const cf_model_desc *d, int t, int a) {
  auto len_hi = [&](int j) -> uint64_t {
    const cf_dist &L = d->len[t][j];
    if (L.kind == CF_DIST_NONE) return 0;
    if (L.kind == CF_DIST_CONST) return (uint64_t)ceil(L.p0);
    return (uint64_t)L.hi;
  };
  switch (a) {
    case CF_ATTR_PROMPT: return len_hi(0);
    case CF_ATTR_OUT: return len_hi(1);
    case CF_ATTR_PATCHES: {
      if (d->img_kind[t] == CF_IMG_NONE) return 0;
      const uint64_t n = (uint64_t)(d->img_lo[t] > d->img_hi[t] ? d->img_lo[t] : d->img_hi[t]);
      return n * (uint64_t)d->patch_hi;
    }
    case CF_ATTR_AUDIN_MS: return len_hi(2);
    case CF_ATTR_AUDOUT_MS: return len_hi(3);
    case CF_ATTR_AUDIN_TOK: return (len_hi(2) + 79u) / 80u;
    case CF_ATTR_AUDOUT_TOK: return (len_hi(3) + 79u) / 80u;
    default: return 0;
  }
}

cf_status lower_model(const cf_model_desc *d, KModel *k) {
  if (!d) return set_error(CF_EINVAL, "model descriptor is NULL");
  memset(k, 0, sizeof *k);
  const int nc = d->n_comp, nt = d->n_types;
  if (nc < 1 || nc > CF_MAX_COMP) return set_error(CF_EINVAL, "n_comp %d out of 1..8", nc);
  if (nt < 1 || nt > CF_MAX_TYPES) return set_error(CF_EINVAL, "n_types %d out of 1..8", nt);
  k->nc = nc;
  k->nt = nt;
  const uint32_t all = (1u << nc) - 1u;
  for (int c = 0; c < nc; c++) {
    if (d->kind[c] < CF_ENC || d->kind[c] > CF_GEN) return set_error(CF_EINVAL, "kind[%d]", c);
    if (!finite_nonneg(d->k0[c]) || !finite_nonneg(d->k1[c]) || !finite_nonneg(d->k2[c]) ||
        !finite_nonneg(d->d0[c]) || !finite_nonneg(d->d1[c]))
      return set_error(CF_EINVAL, "latency coefficients of component %d must be finite and >= 0", c);
    if (d->x_sel[c] >> 7) return set_error(CF_EINVAL, "x_sel[%d]", c);
    if (d->kind[c] == CF_LLM && (d->nout_attr[c] < 0 || d->nout_attr[c] > 6))
      return set_error(CF_EINVAL, "nout_attr[%d]", c);
    if (d->batch_cap[c] < 1 || d->batch_cap[c] > CF_MAX_BATCH)
      return set_error(CF_EINVAL, "batch_cap[%d] out of 1..256", c);
    int g = d->gate_src[c];
    if (g != -1) {
      if (g < 0 || g >= c || d->kind[c] != CF_LLM || d->kind[g] != CF_LLM)
        return set_error(CF_EINVAL, "gate_src[%d] must name an earlier LLM of an LLM", c);
      k->gate_src_mask |= 1u << g;
      k->gated_mask |= 1u << c;
    }
    k->kind[c] = d->kind[c];
    k->k0[c] = d->k0[c]; k->k1[c] = d->k1[c]; k->k2[c] = d->k2[c];
    k->d0[c] = d->d0[c]; k->d1[c] = d->d1[c];
    k->xsel[c] = d->x_sel[c];
    k->nout_attr[c] = d->nout_attr[c];
    k->cap[c] = d->batch_cap[c];
  }
  if (!finite_nonneg(d->comm_s) || !finite_nonneg(d->cpu_pre_s))
    return set_error(CF_EINVAL, "comm_s and cpu_pre_s must be finite and >= 0");
  k->comm = d->comm_s;
  k->cpu_pre = d->cpu_pre_s;
  k->tp_any = 0;
  for (int c = 0; c < CF_MAX_COMP; c++)
    for (int g = 0; g < 8; g++) {
      const double v = c < nc ? d->tp_scale[c][g] : 0.0;
      if (!(v >= 0.0) || v > 1e300) return set_error(CF_EINVAL, "tp_scale[%d][%d] must be finite and >= 0", c, g);
      k->tps[c][g] = v == 0.0 ? 1.0 : v;
      if (k->tps[c][g] != 1.0) k->tp_any = 1;
    }
  if (d->patch_lo < 0 || d->patch_hi < d->patch_lo || d->patch_hi > 16383)
    return set_error(CF_EINVAL, "patch range");
  k->patch_lo = d->patch_lo;
  k->patch_hi = d->patch_hi;
  uint64_t wsum = 0;
  for (int t = 0; t < nt; t++) {
    const uint32_t path = d->path_mask[t];
    if (path == 0 || (path & ~all)) return set_error(CF_EINVAL, "path_mask[%d]", t);
    if (d->out_mask[t] == 0 || (d->out_mask[t] & ~path)) return set_error(CF_EINVAL, "out_mask[%d]", t);
    if (d->prefill_only[t] & ~path) return set_error(CF_EINVAL, "prefill_only[%d]", t);
    k->weight[t] = d->weight[t];
    wsum += d->weight[t];
    k->path[t] = path;
    k->outm[t] = d->out_mask[t];
    k->pfo[t] = d->prefill_only[t];
    k->ttft_c[t] = -1;
    k->th_c[t] = -1;
    k->ta_c[t] = -1;
    int npath = 0;
    for (int c = 0; c < nc; c++) {
      const uint32_t par = d->parents[t][c];
      if (!((path >> c) & 1u)) {
        if (par) return set_error(CF_EINVAL, "parents of component %d off the path of type %d", c, t);
        continue;
      }
      npath++;
      if (par & ~path) return set_error(CF_EINVAL, "parent off the path (type %d)", t);
      if (par >> c) return set_error(CF_EINVAL, "edges must go from lower to higher index (type %d)", t);
      if (par == 0) k->srcm[t] |= 1u << c;
      k->npar[t][c] = (uint8_t)__builtin_popcount(par);
      if (d->kind[c] == CF_LLM && k->ttft_c[t] < 0) k->ttft_c[t] = (int8_t)c;
      if (d->kind[c] == CF_GEN && ((d->out_mask[t] >> c) & 1u)) k->gen_out[t] = 1;
    }
    k->max_path = npath > k->max_path ? npath : k->max_path;
    for (int c2 = 0; c2 < nc; c2++) {
      if (!((path >> c2) & 1u)) continue;
      const int g = d->gate_src[c2];
      const bool stream = g >= 0 && ((d->parents[t][c2] >> g) & 1u);
      if (stream) {
        if (k->ta_c[t] >= 0) return set_error(CF_EUNSUPPORTED, "more than one gated component (type %d)", t);
        if (g != k->ttft_c[t])
          return set_error(CF_EUNSUPPORTED, "the gate source must be the first LLM of the path (type %d)", t);
        if ((d->prefill_only[t] >> g) & 1u)
          return set_error(CF_EUNSUPPORTED, "a gate source cannot be prefill-only (type %d)", t);
        k->th_c[t] = (int8_t)g;
        k->ta_c[t] = (int8_t)c2;
      }
      for (int c = 0; c < nc; c++)
        if (((d->parents[t][c2] >> c) & 1u) && !(stream && c == g)) k->child[t][c] |= (uint8_t)(1u << c2);
    }
    if (d->img_kind[t] < CF_IMG_NONE || d->img_kind[t] > CF_IMG_UNIFORM) return set_error(CF_EINVAL, "img_kind[%d]", t);
    if (d->img_kind[t] != CF_IMG_NONE &&
        (d->img_lo[t] < 0 || d->img_hi[t] < d->img_lo[t] || d->img_hi[t] > 4))
      return set_error(CF_EINVAL, "images of type %d out of 0..4", t);
    k->img_kind[t] = d->img_kind[t];
    k->img_lo[t] = d->img_lo[t];
    k->img_hi[t] = d->img_hi[t];
    for (int j = 0; j < 4; j++) {
      const cf_dist &L = d->len[t][j];
      const int64_t cap = j < 2 ? 65535 : 0xFFFFFFFFll;
      if (L.kind < CF_DIST_NONE || L.kind > CF_DIST_EXP) return set_error(CF_EINVAL, "dist kind");
      if (L.kind != CF_DIST_NONE) {
        if (L.lo < 0 || L.hi < L.lo || L.hi > cap || !isfinite(L.p0) || !isfinite(L.p1) || !isfinite(L.scale))
          return set_error(CF_EINVAL, "length distribution %d of type %d", j, t);
        if (L.kind == CF_DIST_CONST && (L.p0 < 0 || L.p0 > (double)cap))
          return set_error(CF_EINVAL, "constant length out of range");
      }
      k->len[t][j] = L;
    }
    for (int j = 0; j < 4; j++) {
      if (isnan(d->slo[t][j])) return set_error(CF_EINVAL, "slo[%d][%d] is NaN", t, j);
      k->slo[t][j] = d->slo[t][j];
    }
  }
  // the simulator of models with a gated stage keeps that stage's own output
  // length of a running request in 15 bits
  for (int c = 0; c < nc; c++) {
    if (!((k->gated_mask >> c) & 1u)) continue;
    for (int t = 0; t < nt; t++) {
      if (!((d->path_mask[t] >> c) & 1u) || ((d->prefill_only[t] >> c) & 1u)) continue;
      if (attr_hi(d, t, d->nout_attr[c]) > 32767u)
        return set_error(CF_EUNSUPPORTED, "gated component %d: output length of type %d can exceed 32767 tokens", c, t);
    }
  }
  if (wsum == 0 || wsum > 0xFFFFFFFFull) return set_error(CF_EINVAL, "type weights must sum to 1..2^32-1");
  k->wsum = wsum;
  if (d->theta_den == 0) return set_error(CF_EINVAL, "theta_den is 0");
  k->theta_num = d->theta_num;
  k->theta_den = d->theta_den;
  return CF_OK;
}

}  // namespace cf

extern "C" {

size_t cf_last_error(char *buf, size_t n) {
  size_t len = strlen(cf::g_err);
  if (buf && n) {
    size_t m = len < n - 1 ? len : n - 1;
    memcpy(buf, cf::g_err, m);
    buf[m] = 0;
  }
  return len;
}

const char *cf_status_str(cf_status s) {
  switch (s) {
    case CF_OK: return "ok";
    case CF_EINVAL: return "invalid argument";
    case CF_ENOMEM: return "out of device memory";
    case CF_EHIP: return "HIP runtime error";
    case CF_ECAPACITY: return "capacity limit exceeded";
    case CF_EUNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

const char *cf_version(void) { return "libcf 0.1 gfx950"; }

}  // extern "C"

namespace cf {
namespace {
struct ScratchRegion { void *p = nullptr; size_t cap = 0; };
constexpr int kMaxDev = 64;
ScratchRegion g_scr[kMaxDev][SCR_NSLOTS];
}  // namespace

void *scratch_get(int slot, size_t bytes, cf_status *st) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
    *st = set_error(CF_EHIP, "no current HIP device");
    return nullptr;
  }
  ScratchRegion &r = g_scr[dev][slot];
  if (bytes <= r.cap && r.p) return r.p;
  if (r.p) {
    (void)hipDeviceSynchronize();
    (void)hipFree(r.p);
    r.p = nullptr;
    r.cap = 0;
  }
  size_t want = bytes < 4096 ? 4096 : bytes;
  if (hipMalloc(&r.p, want) != hipSuccess) {
    (void)hipGetLastError();
    r.p = nullptr;
    *st = set_error(CF_ENOMEM, "hipMalloc of %zu bytes of scratch failed", want);
    return nullptr;
  }
  r.cap = want;
  return r.p;
}
}  // namespace cf

namespace cf {
cf_status check_targets(int T, int n_bins, const double *host) {
  if (n_bins < 1 || n_bins > 64) return set_error(CF_EINVAL, "n_bins must be in 1..64");
  if (!host) return set_error(CF_EINVAL, "NULL target table");
  for (int t = 0; t < T; t++)
    for (int b = 0; b < n_bins; b++)
      for (int j = 0; j < 4; j++) {
        const double v = host[((size_t)t * n_bins + b) * 4 + j];
        if (v != v) return set_error(CF_EINVAL, "NaN target [%d][%d][%d]", t, b, j);
        if (b > 0 && v < host[((size_t)t * n_bins + b - 1) * 4 + j])
          return set_error(CF_EINVAL, "targets decrease at [%d][%d][%d]", t, b, j);
      }
  return CF_OK;
}

cf_status load_targets(int T, int n_bins, const double *host, const double **dev, hipStream_t s) {
  cf_status st = check_targets(T, n_bins, host);
  if (st != CF_OK) return st;
  const size_t bytes = sizeof(double) * (size_t)T * n_bins * 4;
  void *d = scratch_get(SCR_TARGETS, bytes, &st);
  if (!d) return st;
  st = hip_check(hipMemcpyAsync(d, host, bytes, hipMemcpyHostToDevice, s), "target table copy");
  *dev = (const double *)d;
  return st;
}
}  // namespace cf

extern "C" cf_status cf_release_scratch(void) {
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (int d = 0; d < cf::kMaxDev; d++)
    for (int s = 0; s < cf::SCR_NSLOTS; s++)
      if (cf::g_scr[d][s].p) {
        (void)hipSetDevice(d);
        (void)hipDeviceSynchronize();
        (void)hipFree(cf::g_scr[d][s].p);
        cf::g_scr[d][s].p = nullptr;
        cf::g_scr[d][s].cap = 0;
      }
  (void)hipSetDevice(cur);
  return CF_OK;
}
