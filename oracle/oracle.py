"""ctypes wrapper of the oracle (test infrastructure only).

Only tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  It marshals a workload configuration into the oracle's
own model structure (``cfo.h``) with its own reading of the JSON, and calls
the single-threaded C oracle on host arrays.
"""
import ctypes as C
import math
import os

import numpy as np

from . import build as _build

MAXC, MAXT, MAXV = 8, 8, 16
KIND = {"ENC": 0, "LLM": 1, "GEN": 2}
ATTR = {"prompt": 0, "out": 1, "patches": 2, "aud_in_ms": 3, "aud_out_ms": 4, "aud_in_tok": 5,
        "aud_out_tok": 6}
ST_INVALID, ST_DEADLOCK = 1, 2


class Dist(C.Structure):
    _fields_ = [("kind", C.c_int32), ("pad", C.c_int32), ("p0", C.c_double), ("p1", C.c_double),
                ("scale", C.c_double), ("lo", C.c_int64), ("hi", C.c_int64)]


class Model(C.Structure):
    _fields_ = [
        ("n_comp", C.c_int32), ("n_types", C.c_int32),
        ("kind", C.c_int32 * MAXC),
        ("k0", C.c_double * MAXC), ("k1", C.c_double * MAXC), ("k2", C.c_double * MAXC),
        ("d0", C.c_double * MAXC), ("d1", C.c_double * MAXC),
        ("x_sel", C.c_uint32 * MAXC), ("nout_attr", C.c_int32 * MAXC),
        ("gate_src", C.c_int32 * MAXC), ("batch_cap", C.c_int32 * MAXC),
        ("comm_s", C.c_double), ("cpu_pre_s", C.c_double),
        ("weight", C.c_uint32 * MAXT),
        ("path_mask", C.c_uint32 * MAXT), ("out_mask", C.c_uint32 * MAXT),
        ("prefill_only", C.c_uint32 * MAXT),
        ("parents", (C.c_uint32 * MAXC) * MAXT),
        ("img_kind", C.c_int32 * MAXT), ("img_lo", C.c_int32 * MAXT), ("img_hi", C.c_int32 * MAXT),
        ("patch_lo", C.c_int32), ("patch_hi", C.c_int32),
        ("len", (Dist * 4) * MAXT),
        ("slo", (C.c_double * 4) * MAXT),
        ("theta_num", C.c_uint32), ("theta_den", C.c_uint32),
        ("tp_scale", (C.c_double * 8) * 8),
    ]


class Trace(C.Structure):
    _fields_ = [("n_seeds", C.c_int32), ("n_req", C.c_int32),
                ("arr_ticks", C.c_void_p), ("type", C.c_void_p), ("n_img", C.c_void_p),
                ("patches", C.c_void_p), ("prompt", C.c_void_p), ("out", C.c_void_p),
                ("aud_in_ms", C.c_void_p), ("aud_out_ms", C.c_void_p),
                ("rkey0", C.c_void_p), ("rkey1", C.c_void_p), ("akey", C.c_void_p)]


class Plans(C.Structure):
    _fields_ = [("P", C.c_int32), ("n_nodes", C.c_void_p), ("node_comp", C.c_void_p),
                ("node_rep", C.c_void_p), ("node_batch", C.c_void_p), ("node_gpus", C.c_void_p),
                ("n_alt", C.c_void_p), ("alt_w", C.c_void_p), ("alt_node", C.c_void_p),
                ("node_rep2", C.c_void_p), ("node_batch2", C.c_void_p), ("node_gpus2", C.c_void_p),
                ("node_w", C.c_void_p)]


class EnumOpts(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("k_s", C.c_int32), ("share", C.c_int32),
                ("colocatable", C.c_uint32 * 8), ("n_batch", C.c_int32 * 8),
                ("batch", (C.c_uint16 * 8) * 8), ("n_gpu_opt", C.c_int32 * 8),
                ("gpu_opt", (C.c_uint8 * 4) * 8), ("het", C.c_int32)]


class Logical(C.Structure):
    _fields_ = [("n_nodes", C.c_uint8), ("node_comp", C.c_uint8 * 16), ("n_alt", C.c_uint8 * 8),
                ("alt_node", ((C.c_uint8 * 8) * 2) * 8)]


TRACE_FIELDS = [("arr_ticks", np.uint64), ("type", np.uint8), ("n_img", np.uint8),
                ("patches", np.uint16), ("prompt", np.uint16), ("out", np.uint16),
                ("aud_in_ms", np.uint32), ("aud_out_ms", np.uint32), ("rkey0", np.uint64),
                ("rkey1", np.uint64), ("akey", np.uint32)]

_lib = None


def lib():
    global _lib
    if _lib is None:
        _build.ensure_built()
        L = C.CDLL(_build.LIB)
        vp, i32, dbl = C.c_void_p, C.c_int32, C.c_double
        L.cfo_philox.argtypes = [vp, vp, vp]
        L.cfo_log.argtypes = [dbl]
        L.cfo_log.restype = dbl
        L.cfo_exp.argtypes = [dbl]
        L.cfo_exp.restype = dbl
        L.cfo_uniform.argtypes = [C.c_uint64]
        L.cfo_uniform.restype = dbl
        L.cfo_trace_gen.argtypes = [vp, vp, i32, i32, vp, vp]
        L.cfo_eval_coarse.argtypes = [vp, vp, vp, i32, vp, vp, vp]
        L.cfo_select_topk.argtypes = [vp, vp, i32, i32, vp, vp]
        L.cfo_rate_grid.argtypes = [vp, vp, i32, i32, dbl, vp]
        L.cfo_sim_triple.argtypes = [vp, vp, i32, dbl, vp, i32, vp, vp, vp, vp, vp, vp]
        L.cfo_goodput_reduce.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp, C.c_uint32, C.c_uint32,
                                         i32, vp, vp, vp]
        L.cfo_bisect.argtypes = [vp, vp, vp, i32, vp, i32, vp, C.c_uint32, C.c_uint32, vp, vp, vp, vp, vp]
        L.cfo_latency_hist.argtypes = [vp, vp, i32, i32, i32, vp, vp]
        L.cfo_mc_curve.argtypes = [vp, vp, vp, i32, vp, vp, dbl, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.cfo_enum_logical.argtypes = [vp, vp, vp, i32, vp]
        L.cfo_enum_count.argtypes = [vp, vp, vp]
        L.cfo_enum_count.restype = C.c_uint64
        L.cfo_enum_plans.argtypes = [vp, vp, vp, i32, C.c_uint64, i32] + [vp] * 8
        L.cfo_argmax.argtypes = [vp, i32]
        L.cfo_argmax.restype = i32
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p)


# ---------------------------------------------------------------- model
def _dist(spec, audio):
    d = Dist()
    d.scale, d.lo, d.hi = 1.0, 1, (600000 if audio else 32767)
    if not spec:
        d.kind = 0
        return d
    (k, v), = spec.items()
    if k == "const":
        d.kind, d.p0 = 1, float(v)
    elif k in ("lognormal", "lognormal_s"):
        d.kind, d.p0, d.p1 = 2, float(v[0]), float(v[1])
        d.scale = 1000.0 if k == "lognormal_s" else 1.0
    elif k == "exp":
        d.kind, d.p0 = 3, float(v)
    else:
        raise ValueError(k)
    return d


def make_model(mcfg):
    """The oracle's own reading of a model description (JSON dict)."""
    m = Model()
    comps = mcfg["components"]
    names = {c["name"]: i for i, c in enumerate(comps)}
    m.n_comp, m.n_types = len(comps), len(mcfg["types"])
    for i, c in enumerate(comps):
        m.kind[i] = KIND[c["kind"]]
        m.k0[i], m.k1[i], m.k2[i] = (float(v) for v in c["k"])
        dec = c.get("decode", [0.0, 0.0])
        m.d0[i], m.d1[i] = float(dec[0]), float(dec[1])
        m.x_sel[i] = sum(1 << ATTR[a] for a in c.get("x", []))
        m.nout_attr[i] = ATTR[c.get("n_out", "out")]
        m.gate_src[i] = names[c["gate"]] if c.get("gate") else -1
        m.batch_cap[i] = int(c.get("batch_cap", 256))
        tps = {int(g): float(v) for g, v in c.get("tp_scale", {}).items()}
        for g in range(1, 9):
            m.tp_scale[i][g - 1] = tps.get(g, 1.0)
    m.comm_s = float(mcfg["comm_s"])
    m.cpu_pre_s = float(mcfg.get("cpu_pre_s", 0.0))
    for t, ty in enumerate(mcfg["types"]):
        m.weight[t] = int(ty["weight"])
        m.path_mask[t] = sum(1 << names[c] for c in ty["comps"])
        m.out_mask[t] = sum(1 << names[c] for c in ty["outputs"])
        m.prefill_only[t] = sum(1 << names[c] for c in ty.get("prefill_only", []))
        for a, b in ty.get("edges", []):
            m.parents[t][names[b]] |= 1 << names[a]
        img = ty.get("images")
        if not img:
            m.img_kind[t] = 0
        elif "const" in img:
            m.img_kind[t], m.img_lo[t], m.img_hi[t] = 1, int(img["const"]), int(img["const"])
        else:
            m.img_kind[t], m.img_lo[t], m.img_hi[t] = 2, int(img["uniform"][0]), int(img["uniform"][1])
        m.len[t][0] = _dist(ty.get("prompt"), False)
        m.len[t][1] = _dist(ty.get("out"), False)
        m.len[t][2] = _dist(ty.get("aud_in"), True)
        m.len[t][3] = _dist(ty.get("aud_out"), True)
        slo = ty.get("slo", {})
        for j, key in enumerate(("ttft", "tpot", "e2e", "media")):
            m.slo[t][j] = float(slo[key]) if key in slo else math.inf
    m.patch_lo, m.patch_hi = (int(v) for v in mcfg.get("patches_per_image", [256, 1024]))
    th = mcfg.get("theta", [9, 10])
    m.theta_num, m.theta_den = int(th[0]), int(th[1])
    return m


# ---------------------------------------------------------------- primitives
def philox(ctr, key):
    c = np.asarray(ctr, np.uint64)
    k = np.asarray(key, np.uint64)
    out = np.zeros(4, np.uint64)
    lib().cfo_philox(_ptr(c), _ptr(k), _ptr(out))
    return out


def cf_log(x):
    return lib().cfo_log(float(x))


def cf_exp(x):
    return lib().cfo_exp(float(x))


def uniform(x):
    return lib().cfo_uniform(int(x))


# ---------------------------------------------------------------- trace
def trace_gen(model, seeds, n_req):
    S = len(seeds)
    tr = {f: np.zeros(S * n_req, dt) for f, dt in TRACE_FIELDS}
    moments = np.zeros((S, model.n_types, 8), np.uint64)
    seeds_a = np.asarray(seeds, np.uint64)
    st = _trace_struct(tr, S, n_req)
    rc = lib().cfo_trace_gen(C.byref(model), _ptr(seeds_a), S, n_req, C.byref(st), _ptr(moments))
    if rc != 0:
        raise ValueError("cfo_trace_gen failed")
    tr["n_seeds"], tr["n_req"] = S, n_req
    tr["moments"] = moments
    return tr


def _trace_struct(tr, S, n_req):
    st = Trace()
    st.n_seeds, st.n_req = S, n_req
    for f, _ in TRACE_FIELDS:
        setattr(st, f, tr[f].ctypes.data)
    return st


def trace_struct(tr):
    return _trace_struct(tr, tr["n_seeds"], tr["n_req"])


# ---------------------------------------------------------------- plans
def plans_struct(tab):
    st = Plans()
    st.P = tab.P
    keep = []
    for f in ("n_nodes", "node_comp", "node_rep", "node_batch", "node_gpus", "n_alt", "alt_w",
              "alt_node", "node_rep2", "node_batch2", "node_gpus2", "node_w"):
        if getattr(tab, f, None) is None:  # a table without second executor groups
            continue
        a = np.ascontiguousarray(getattr(tab, f))
        keep.append(a)
        setattr(st, f, a.ctypes.data)
    st._keep = keep
    return st


def eval_coarse(model, tab, moments0, n_gpus):
    P = tab.P
    rd = np.zeros(P, np.float64)
    bn = np.zeros(P, np.int32)
    fl = np.zeros(P, np.uint8)
    mo = np.ascontiguousarray(moments0, dtype=np.uint64)
    pst = plans_struct(tab)
    lib().cfo_eval_coarse(C.byref(model), C.byref(pst), _ptr(mo), int(n_gpus), _ptr(rd), _ptr(bn),
                          _ptr(fl))
    return rd, bn, fl


def select_topk(rd, flags, k):
    P = len(rd)
    ids = np.zeros(max(k, 1), np.int32)
    nsel = C.c_int32(0)
    lib().cfo_select_topk(_ptr(np.ascontiguousarray(rd)), _ptr(np.ascontiguousarray(flags)), P,
                          int(k), _ptr(ids), C.byref(nsel))
    return ids[:nsel.value].copy()


def rate_grid(rd, ids, K, alpha_max=1.0):
    ids = np.ascontiguousarray(ids, np.int32)
    rates = np.zeros((len(ids), K), np.float64)
    lib().cfo_rate_grid(_ptr(np.ascontiguousarray(rd)), _ptr(ids), len(ids), int(K),
                        float(alpha_max), _ptr(rates))
    return rates


def sim_triple(model, tab, plan_id, rate, tr, seed_idx, want_lat=False, want_diag=False,
               _pst=None, _tst=None):
    T = model.n_types
    met = np.zeros(T, np.uint32)
    cnt = np.zeros(T, np.uint32)
    ev = C.c_uint64(0)
    st = C.c_uint32(0)
    lat = np.zeros((tr["n_req"], 4), np.float64) if want_lat else None
    diag = np.zeros(4, np.float64) if want_diag else None
    pst = _pst if _pst is not None else plans_struct(tab)
    tst = _tst if _tst is not None else trace_struct(tr)
    lib().cfo_sim_triple(C.byref(model), C.byref(pst), int(plan_id), float(rate), C.byref(tst),
                         int(seed_idx), _ptr(met), _ptr(cnt), C.byref(ev), C.byref(st),
                         _ptr(lat) if lat is not None else None,
                         _ptr(diag) if diag is not None else None)
    out = dict(met=met, cnt=cnt, events=ev.value, status=st.value)
    if want_lat:
        out["lat"] = lat
    if want_diag:
        out["diag"] = diag
    return out


def eval_fine(model, tab, plan_ids, rates, tr, triples=None):
    """Every (plan, rate, seed) triple, or only the listed (i, k, s) triples.

    Returns met, cnt [n_plans, K, S, T], events and status [n_plans, K, S];
    entries of triples not simulated stay zero."""
    n_plans, K = rates.shape
    S, T = tr["n_seeds"], model.n_types
    met = np.zeros((n_plans, K, S, T), np.uint32)
    cnt = np.zeros((n_plans, K, S, T), np.uint32)
    events = np.zeros((n_plans, K, S), np.uint64)
    status = np.zeros((n_plans, K, S), np.uint32)
    pst, tst = plans_struct(tab), trace_struct(tr)
    if triples is None:
        triples = [(i, k, s) for i in range(n_plans) for k in range(K) for s in range(S)]
    for (i, k, s) in triples:
        o = sim_triple(model, tab, int(plan_ids[i]), float(rates[i, k]), tr, s, _pst=pst, _tst=tst)
        met[i, k, s], cnt[i, k, s] = o["met"], o["cnt"]
        events[i, k, s], status[i, k, s] = o["events"], o["status"]
    return met, cnt, events, status


def eval_mc(model, tab, plan_ids, rd, moments0, alpha, tr, seed_idx, n_sample, want_lat=False):
    """Phase 2 (Monte Carlo latency) of plans plan_ids: met, cnt [n, T] u32, goodput G [n, T]
    and, with want_lat, the latencies [n, n_sample, 4] of every sampled request."""
    ids = np.ascontiguousarray(plan_ids, np.int32)
    n, T = len(ids), model.n_types
    met = np.zeros((n, T), np.uint32)
    cnt = np.zeros((n, T), np.uint32)
    gt = np.zeros((n, T), np.float64)
    lat = np.zeros((n, n_sample, 4), np.float64) if want_lat else None
    L = lib()
    L.cfo_eval_mc.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                              C.c_double, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                              C.c_void_p, C.c_void_p]
    pst, tst = plans_struct(tab), trace_struct(tr)
    L.cfo_eval_mc(C.byref(model), C.byref(pst), _ptr(ids), n, _ptr(np.ascontiguousarray(rd, np.float64)),
                  _ptr(np.ascontiguousarray(moments0, np.uint64)), float(alpha), C.byref(tst),
                  int(seed_idx), int(n_sample), _ptr(met), _ptr(cnt), _ptr(gt),
                  _ptr(lat) if lat is not None else None)
    return (met, cnt, gt, lat) if want_lat else (met, cnt, gt)


def pareto(g):
    """keep[i] = 0 iff another row of g is >= everywhere and > somewhere."""
    g = np.ascontiguousarray(g, np.float64)
    n, T = g.shape
    keep = np.zeros(n, np.uint8)
    L = lib()
    L.cfo_pareto.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]
    L.cfo_pareto(_ptr(g), n, T, _ptr(keep))
    return keep


def goodput_reduce(met, cnt, rates, theta, n_req, status=None):
    """Highest feasible rate and goodput per plan; status [n_plans, K, S] (None: every
    simulation ended normally) makes a rate with a failed simulation infeasible."""
    n_plans, K, S, T = met.shape
    if status is None:
        status = np.zeros((n_plans, K, S), np.uint32)
    status = np.ascontiguousarray(status, np.uint32)
    assert status.shape == (n_plans, K, S)
    kstar = np.zeros(n_plans, np.int32)
    gt = np.zeros((n_plans, T), np.float64)
    g = np.zeros(n_plans, np.float64)
    if np.asarray(met).max(initial=0) > 0xFFFFFFFF or np.asarray(cnt).max(initial=0) > 0xFFFFFFFF:
        raise ValueError("counts above 32 bits")
    lib().cfo_goodput_reduce(_ptr(np.ascontiguousarray(met, np.uint32)), _ptr(np.ascontiguousarray(cnt, np.uint32)),
                             _ptr(status), n_plans, K, S, T, _ptr(np.ascontiguousarray(rates, np.float64)), int(theta[0]),
                             int(theta[1]), int(n_req), _ptr(kstar), _ptr(gt), _ptr(g))
    return kstar, gt, g


def argmax(goodput):
    g = np.ascontiguousarray(goodput, np.float64)
    return int(lib().cfo_argmax(_ptr(g), len(g)))


def math_n(op, x, y=None):
    L = lib()
    L.cfo_math_n.argtypes = [C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64]
    x = np.ascontiguousarray(x, np.float64)
    yy = np.ascontiguousarray(y, np.float64) if y is not None else None
    out = np.zeros_like(x)
    L.cfo_math_n(int(op), _ptr(x), _ptr(yy) if yy is not None else None, _ptr(out), x.size)
    return out


def philox_n(ctr, key):
    L = lib()
    L.cfo_philox_n.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64]
    ctr = np.ascontiguousarray(ctr, np.uint64)
    key = np.ascontiguousarray(key, np.uint64)
    out = np.zeros_like(ctr)
    L.cfo_philox_n(_ptr(ctr), _ptr(key), _ptr(out), ctr.shape[0])
    return out


# ---------------------------------------------------------------- plan enumeration
def enum_opts(mcfg, spec, n_gpus):
    """Enumeration options from a model description and an ``enumerate`` spec:
    k_s, share, colocatable edges (default: every edge of every type), per-component
    batch knobs and GPUs-per-executor options (default [1])."""
    o = EnumOpts()
    names = {c["name"]: i for i, c in enumerate(mcfg["components"])}
    o.n_gpus, o.k_s, o.share = int(n_gpus), int(spec.get("k_s", 2)), int(bool(spec.get("share", True)))
    o.het = int(bool(spec.get("het", False)))
    edges = spec.get("colocatable")
    if edges is None:
        edges = [e for t in mcfg["types"] for e in t.get("edges", [])]
    for a, b in edges:
        o.colocatable[names[a]] |= 1 << names[b]
    for c in mcfg["components"]:
        i = names[c["name"]]
        knobs = spec["batch"][c["name"]]
        o.n_batch[i] = len(knobs)
        for k, v in enumerate(knobs):
            o.batch[i][k] = int(v)
        g = spec.get("gpus", {}).get(c["name"], [1])
        o.n_gpu_opt[i] = len(g)
        for k, v in enumerate(g):
            o.gpu_opt[i][k] = int(v)
    return o


def enum_logical(model, opts, cap=200000):
    out = (Logical * cap)()
    n = C.c_int32(0)
    rc = lib().cfo_enum_logical(C.byref(model), C.byref(opts), out, int(cap), C.byref(n))
    if rc != 0:
        raise RuntimeError("cfo_enum_logical failed (%d)" % rc)
    return out[: n.value]


def logical_array(logical):
    arr = (Logical * max(len(logical), 1))()
    for i, L in enumerate(logical):
        arr[i] = L
    return arr


def enum_count(model, opts, L):
    return int(lib().cfo_enum_count(C.byref(model), C.byref(opts), C.byref(L)))


def enum_plans(model, opts, logical, first, count):
    """Physical plans first..first+count-1 as a plan table (inputs.PlanTable layout)."""
    from paper_2512_14098_amd.inputs.plans import PlanTable
    tab = PlanTable(int(count))
    arr = logical_array(logical)
    rc = lib().cfo_enum_plans(C.byref(model), C.byref(opts), arr, len(logical), C.c_uint64(int(first)),
                              int(count), *[_ptr(getattr(tab, f)) for f in PlanTable.FIELDS])
    if rc != 0:
        raise RuntimeError("cfo_enum_plans failed (%d)" % rc)
    return tab


# ---------------------------------------------------------------- latency CDFs over target tables
def latency_hist(lat, types, T, targets):
    """hist[T][n_bins + 1] of requests by the first target bin they meet (targets [T][n_bins][4])."""
    targets = np.ascontiguousarray(targets, np.float64)
    nb = targets.shape[1]
    lat = np.ascontiguousarray(lat, np.float64)
    types = np.ascontiguousarray(types, np.uint8)
    h = np.zeros((T, nb + 1), np.uint32)
    lib().cfo_latency_hist(_ptr(lat), _ptr(types), len(types), int(T), int(nb), _ptr(targets), _ptr(h))
    return h


def mc_curve(model, tab, plan_ids, rd, moments0, alpha, tr, seed_idx, n_sample, targets):
    """Phase 2 with its latency CDF over a target table: (met, cnt, gt, hist, curve)."""
    ids = np.ascontiguousarray(plan_ids, np.int32)
    n, T = len(ids), model.n_types
    targets = np.ascontiguousarray(targets, np.float64)
    nb = targets.shape[1]
    met = np.zeros((n, T), np.uint32)
    cnt = np.zeros((n, T), np.uint32)
    gt = np.zeros((n, T), np.float64)
    hist = np.zeros((n, T, nb + 1), np.uint32)
    curve = np.zeros((n, nb, T), np.float64)
    pst, tst = plans_struct(tab), trace_struct(tr)
    lib().cfo_mc_curve(C.byref(model), C.byref(pst), _ptr(ids), n, _ptr(np.ascontiguousarray(rd, np.float64)),
                       _ptr(np.ascontiguousarray(moments0, np.uint64)), float(alpha), C.byref(tst), int(seed_idx),
                       int(n_sample), int(nb), _ptr(targets), _ptr(met), _ptr(cnt), _ptr(gt), _ptr(hist),
                       _ptr(curve))
    return met, cnt, gt, hist, curve


def scaled_targets(model, scales):
    """A target table: the type's own bounds times each scale (inf stays inf)."""
    T = model.n_types
    out = np.zeros((T, len(scales), 4), np.float64)
    for t in range(T):
        for b, sc in enumerate(scales):
            for j in range(4):
                out[t, b, j] = model.slo[t][j] * float(sc)
    return out


def bisect(model, tab, plan_ids, rates, tr, theta):
    """Rate bisection per plan over its grid: (kstar, goodput_t, goodput, n_eval, events)."""
    ids = np.ascontiguousarray(plan_ids, np.int32)
    rates = np.ascontiguousarray(rates, np.float64)
    n, K, T = len(ids), rates.shape[1], model.n_types
    ks = np.zeros(n, np.int32)
    gt = np.zeros((n, T), np.float64)
    g = np.zeros(n, np.float64)
    ne = np.zeros(n, np.int32)
    ev = np.zeros(n, np.uint64)
    lib().cfo_bisect(C.byref(model), C.byref(plans_struct(tab)), _ptr(ids), n, _ptr(rates), int(K),
                     C.byref(trace_struct(tr)), int(theta[0]), int(theta[1]), _ptr(ks), _ptr(gt), _ptr(g),
                     _ptr(ne), _ptr(ev))
    return ks, gt, g, ne, ev
