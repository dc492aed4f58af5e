"""Python binding of libcf (``include/cf.h``): argument marshalling only.

Every function has the name of the C entry point it calls.  Device arrays
are torch tensors on the current HIP device; each call runs on torch's
current stream.  Nothing is computed here: the library runs every step in
its HIP kernels, and a missing library raises at import.
"""
import ctypes as C
import math
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcf.so")

MAX_COMP, MAX_TYPES, MAX_NODES = 8, 8, 16
KIND = {"ENC": 0, "LLM": 1, "GEN": 2}
ATTR = {"prompt": 0, "out": 1, "patches": 2, "aud_in_ms": 3, "aud_out_ms": 4, "aud_in_tok": 5,
        "aud_out_tok": 6}
FLAG_KEEP, FLAG_OVER_BUDGET, FLAG_INVALID, FLAG_REDUNDANT = 1, 2, 4, 8
ST_INVALID, ST_DEADLOCK, ST_OVERFLOW = 1, 2, 4
CF_FULL, CF_DUMP_LAT, CF_EARLY_EXIT = 0, 1, 2  # cf_eval_fine flags


class CfError(RuntimeError):
    pass


class cf_dist(C.Structure):
    _fields_ = [("kind", C.c_int32), ("reserved", C.c_int32), ("p0", C.c_double), ("p1", C.c_double),
                ("scale", C.c_double), ("lo", C.c_int64), ("hi", C.c_int64)]


class cf_model_desc(C.Structure):
    _fields_ = [
        ("n_comp", C.c_int32), ("n_types", C.c_int32), ("kind", C.c_int32 * MAX_COMP),
        ("k0", C.c_double * MAX_COMP), ("k1", C.c_double * MAX_COMP), ("k2", C.c_double * MAX_COMP),
        ("d0", C.c_double * MAX_COMP), ("d1", C.c_double * MAX_COMP),
        ("x_sel", C.c_uint32 * MAX_COMP), ("nout_attr", C.c_int32 * MAX_COMP),
        ("gate_src", C.c_int32 * MAX_COMP), ("batch_cap", C.c_int32 * MAX_COMP),
        ("comm_s", C.c_double), ("cpu_pre_s", C.c_double),
        ("weight", C.c_uint32 * MAX_TYPES), ("path_mask", C.c_uint32 * MAX_TYPES),
        ("out_mask", C.c_uint32 * MAX_TYPES), ("prefill_only", C.c_uint32 * MAX_TYPES),
        ("parents", (C.c_uint32 * MAX_COMP) * MAX_TYPES),
        ("img_kind", C.c_int32 * MAX_TYPES), ("img_lo", C.c_int32 * MAX_TYPES),
        ("img_hi", C.c_int32 * MAX_TYPES), ("patch_lo", C.c_int32), ("patch_hi", C.c_int32),
        ("len", (cf_dist * 4) * MAX_TYPES), ("slo", (C.c_double * 4) * MAX_TYPES),
        ("theta_num", C.c_uint32), ("theta_den", C.c_uint32),
        ("tp_scale", (C.c_double * 8) * MAX_COMP),
    ]


class cf_trace(C.Structure):
    _fields_ = [("n_seeds", C.c_int32), ("n_req", C.c_int32)] + [
        (f + "_dev", C.c_void_p) for f in ("arr_ticks", "type", "n_img", "patches", "prompt", "out",
                                           "aud_in_ms", "aud_out_ms", "rkey0", "rkey1", "akey")]


class cf_plan_table(C.Structure):
    _fields_ = [("P", C.c_int32)] + [
        (f + "_dev", C.c_void_p) for f in ("n_nodes", "node_comp", "node_rep", "node_batch",
                                           "node_gpus", "n_alt", "alt_w", "alt_node",
                                           "node_rep2", "node_batch2", "node_gpus2", "node_w")]


class cf_enum_opts(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("k_s", C.c_int32), ("share", C.c_int32),
                ("colocatable", C.c_uint32 * MAX_COMP), ("n_batch", C.c_int32 * MAX_COMP),
                ("batch", (C.c_uint16 * 8) * MAX_COMP), ("n_gpu_opt", C.c_int32 * MAX_COMP),
                ("gpu_opt", (C.c_uint8 * 4) * MAX_COMP), ("het", C.c_int32)]


LOGICAL_BYTES = 1 + 16 + 8 + 8 * 2 * 8  # sizeof(cf_logical)


class cf_fine_out(C.Structure):
    _fields_ = [("met_dev", C.c_void_p), ("cnt_dev", C.c_void_p), ("events_dev", C.c_void_p),
                ("status_dev", C.c_void_p), ("lat_dev", C.c_void_p), ("lat_triples_dev", C.c_void_p),
                ("n_lat", C.c_int32), ("hist_dev", C.c_void_p), ("hist_targets_host", C.c_void_p),
                ("n_bins", C.c_int32), ("lim_chunks", C.c_int32), ("lim_delay", C.c_int32),
                ("lim_instants", C.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise CfError("libcf.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, u32, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_double
    sigs = {
        "cf_last_error": ([vp, C.c_size_t], C.c_size_t),
        "cf_status_str": ([i32], C.c_char_p),
        "cf_version": ([], C.c_char_p),
        "cf_trace_gen": ([vp, vp, i32, i32, vp, vp, vp], i32),
        "cf_eval_coarse": ([vp, vp, vp, i32, vp, vp, vp, vp], i32),
        "cf_select_topk": ([vp, vp, i32, i32, vp, vp, vp], i32),
        "cf_rate_grid": ([vp, vp, i32, i32, dbl, vp, vp], i32),
        "cf_topk_merge": ([vp, vp, i32, vp, vp, i32, C.c_uint64, i32, vp, vp, vp], i32),
        "cf_eval_fine": ([vp, vp, vp, i32, vp, i32, vp, u32, vp, vp], i32),
        "cf_eval_fine_noalloc": ([vp, vp, vp, i32, vp, i32, vp, u32, vp, vp], i32),
        "cf_goodput_reduce": ([vp, i32, i32, i32, i32, vp, u32, u32, i32, vp, vp, vp, vp], i32),
        "cf_eval_mc": ([vp, vp, vp, i32, vp, vp, dbl, vp, i32, i32, vp, vp, vp, vp, vp], i32),
        "cf_pareto": ([vp, i32, i32, vp, vp, vp, i32, vp], i32),
        "cf_eval_mc_curve": ([vp, vp, vp, i32, vp, vp, dbl, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp], i32),
        "cf_goodput_curve": ([vp, i32, i32, i32, i32, vp, C.c_uint32, C.c_uint32, i32, vp, vp, vp, vp], i32),
        "cf_eval_bisect": ([vp, vp, vp, i32, vp, i32, vp, C.c_uint32, C.c_uint32, vp, vp, vp, vp, vp, vp, vp], i32),
        "cf_enum_screen": ([vp, vp, vp, i32, vp, C.c_uint64, C.c_uint64, i32, vp, i32, vp, vp, vp, vp], i32),
        "cf_enum_logical": ([vp, vp, vp, i32, vp], i32),
        "cf_enum_count": ([vp, vp, vp, i32, vp, vp, vp], i32),
        "cf_enum_plans": ([vp, vp, vp, i32, vp, C.c_uint64, C.c_uint64, i32, vp, vp], i32),
        "cf_select_best": ([vp, i32, vp, vp], i32),
        "cf_math_eval": ([i32, vp, vp, vp, i64, vp], i32),
        "cf_philox_eval": ([vp, vp, vp, i64, vp], i32),
        "cf_release_scratch": ([], i32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


_lib = _load()
EXPORTED = ("cf_last_error", "cf_status_str", "cf_version", "cf_trace_gen", "cf_eval_coarse",
            "cf_select_topk", "cf_topk_merge", "cf_rate_grid", "cf_eval_fine", "cf_eval_fine_noalloc", "cf_eval_bisect", "cf_eval_mc",
            "cf_eval_mc_curve", "cf_goodput_curve", "cf_pareto",
            "cf_enum_logical", "cf_enum_count", "cf_enum_plans", "cf_enum_screen",
            "cf_goodput_reduce", "cf_select_best", "cf_math_eval", "cf_philox_eval", "cf_release_scratch")


def lib():
    return _lib


def _check(rc, what):
    if rc != 0:
        buf = C.create_string_buffer(512)
        _lib.cf_last_error(buf, 512)
        raise CfError("%s: %s (%s)" % (what, _lib.cf_status_str(rc).decode(), buf.value.decode()))


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _p(t):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise CfError("expected a contiguous device tensor")
    return C.c_void_p(t.data_ptr())


def _in(t, dtype, what, numel=None, ndim=None):
    """A caller's device tensor checked for the element type (and size) the C ABI reads."""
    if t.dtype != dtype:
        raise CfError("%s: expected %s, got %s" % (what, dtype, t.dtype))
    if numel is not None and t.numel() != numel:
        raise CfError("%s: expected %d elements, got %d" % (what, numel, t.numel()))
    if ndim is not None and t.dim() != ndim:
        raise CfError("%s: expected %d dimensions, got %d" % (what, ndim, t.dim()))
    return _p(t.contiguous())


# ------------------------------------------------------------------ model
def _dist(spec, audio):
    d = cf_dist()
    d.scale, d.lo, d.hi = 1.0, 1, (600000 if audio else 32767)
    if not spec:
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
        raise CfError("unknown length distribution " + k)
    return d


def model_desc(mcfg):
    """cf_model_desc from a model description (JSON dict)."""
    d = cf_model_desc()
    comps = mcfg["components"]
    idx = {c["name"]: i for i, c in enumerate(comps)}
    d.n_comp, d.n_types = len(comps), len(mcfg["types"])
    for i, c in enumerate(comps):
        d.kind[i] = KIND[c["kind"]]
        d.k0[i], d.k1[i], d.k2[i] = (float(v) for v in c["k"])
        dec = c.get("decode", [0.0, 0.0])
        d.d0[i], d.d1[i] = float(dec[0]), float(dec[1])
        d.x_sel[i] = sum(1 << ATTR[a] for a in c.get("x", []))
        d.nout_attr[i] = ATTR[c.get("n_out", "out")]
        d.gate_src[i] = idx[c["gate"]] if c.get("gate") else -1
        d.batch_cap[i] = int(c.get("batch_cap", 256))
        for g, v in c.get("tp_scale", {}).items():  # GPUs per executor -> latency multiplier
            if not 1 <= int(g) <= 8:
                raise CfError("tp_scale keys are GPUs per executor, 1..8")
            d.tp_scale[i][int(g) - 1] = float(v)
    d.comm_s = float(mcfg["comm_s"])
    d.cpu_pre_s = float(mcfg.get("cpu_pre_s", 0.0))
    for t, ty in enumerate(mcfg["types"]):
        d.weight[t] = int(ty["weight"])
        d.path_mask[t] = sum(1 << idx[c] for c in ty["comps"])
        d.out_mask[t] = sum(1 << idx[c] for c in ty["outputs"])
        d.prefill_only[t] = sum(1 << idx[c] for c in ty.get("prefill_only", []))
        for a, b in ty.get("edges", []):
            d.parents[t][idx[b]] |= 1 << idx[a]
        img = ty.get("images")
        if img and "const" in img:
            d.img_kind[t], d.img_lo[t], d.img_hi[t] = 1, int(img["const"]), int(img["const"])
        elif img:
            d.img_kind[t], d.img_lo[t], d.img_hi[t] = 2, int(img["uniform"][0]), int(img["uniform"][1])
        for j, (key, audio) in enumerate((("prompt", False), ("out", False), ("aud_in", True),
                                          ("aud_out", True))):
            d.len[t][j] = _dist(ty.get(key), audio)
        slo = ty.get("slo", {})
        for j, key in enumerate(("ttft", "tpot", "e2e", "media")):
            d.slo[t][j] = float(slo[key]) if key in slo else math.inf
    d.patch_lo, d.patch_hi = (int(v) for v in mcfg.get("patches_per_image", [256, 1024]))
    th = mcfg.get("theta", [9, 10])
    d.theta_num, d.theta_den = int(th[0]), int(th[1])
    return d


# ------------------------------------------------------------------ device containers
TRACE_FIELDS = [("arr_ticks", torch.int64), ("type", torch.uint8), ("n_img", torch.uint8),
                ("patches", torch.int16), ("prompt", torch.int16), ("out", torch.int16),
                ("aud_in_ms", torch.int32), ("aud_out_ms", torch.int32), ("rkey0", torch.int64),
                ("rkey1", torch.int64), ("akey", torch.int32)]


class DeviceTrace:
    """Trace arrays in HBM (seed-major [S * n]) and their cf_trace view."""

    def __init__(self, n_seeds, n_req, device="cuda"):
        self.n_seeds, self.n_req = int(n_seeds), int(n_req)
        self.t = {f: torch.empty(self.n_seeds * self.n_req, dtype=dt, device=device)
                  for f, dt in TRACE_FIELDS}
        self.c = cf_trace()
        self.c.n_seeds, self.c.n_req = self.n_seeds, self.n_req
        for f, _ in TRACE_FIELDS:
            setattr(self.c, f + "_dev", self.t[f].data_ptr())

    def seed_view(self, s):
        """The trace of seed index s alone (a one-seed view of the same device arrays)."""
        if not 0 <= s < self.n_seeds:
            raise CfError("seed index %d outside 0..%d" % (s, self.n_seeds - 1))
        v = DeviceTrace.__new__(DeviceTrace)
        v.n_seeds, v.n_req = 1, self.n_req
        v.t = {f: self.t[f][s * self.n_req:(s + 1) * self.n_req] for f, _ in TRACE_FIELDS}
        v.c = cf_trace()
        v.c.n_seeds, v.c.n_req = 1, self.n_req
        for f, _ in TRACE_FIELDS:
            setattr(v.c, f + "_dev", v.t[f].data_ptr())
        return v

    def to_numpy(self):
        """Host copy with the unsigned dtypes of the C layout."""
        unsigned = {"arr_ticks": np.uint64, "type": np.uint8, "n_img": np.uint8, "patches": np.uint16,
                    "prompt": np.uint16, "out": np.uint16, "aud_in_ms": np.uint32,
                    "aud_out_ms": np.uint32, "rkey0": np.uint64, "rkey1": np.uint64, "akey": np.uint32}
        out = {f: self.t[f].cpu().numpy().view(unsigned[f]) for f, _ in TRACE_FIELDS}
        out["n_seeds"], out["n_req"] = self.n_seeds, self.n_req
        return out

    @staticmethod
    def from_numpy(tr, device="cuda"):
        d = DeviceTrace(tr["n_seeds"], tr["n_req"], device)
        for f, dt in TRACE_FIELDS:
            a = np.ascontiguousarray(tr[f])
            d.t[f].copy_(torch.from_numpy(a.view({torch.int64: np.int64, torch.uint8: np.uint8,
                                                  torch.int16: np.int16,
                                                  torch.int32: np.int32}[dt])))
        return d


class DevicePlans:
    """Plan table (paper_2512_14098_amd.inputs.PlanTable) copied to HBM."""

    FIELDS = ("n_nodes", "node_comp", "node_rep", "node_batch", "node_gpus", "n_alt", "alt_w",
              "alt_node")
    # a node's second executor configuration: copied only when some node of the table has one
    GROUP_FIELDS = ("node_rep2", "node_batch2", "node_gpus2", "node_w")

    def __init__(self, tab, device="cuda"):
        self.P = tab.P
        self.t = {}
        self.c = cf_plan_table()
        self.c.P = tab.P
        split = getattr(tab, "node_rep2", None) is not None and bool(np.any(tab.node_rep2))
        for f in self.FIELDS + (self.GROUP_FIELDS if split else ()):
            a = np.ascontiguousarray(getattr(tab, f))
            if a.dtype == np.uint16:
                a = a.view(np.int16)
            self.t[f] = torch.from_numpy(a).to(device)
            setattr(self.c, f + "_dev", self.t[f].data_ptr())

    SHAPES = {"n_nodes": (None, torch.uint8), "node_comp": (16, torch.uint8), "node_rep": (16, torch.uint8),
              "node_batch": (16, torch.int16), "node_gpus": (16, torch.uint8), "n_alt": (8, torch.uint8),
              "alt_w": (16, torch.uint8), "alt_node": (128, torch.uint8), "node_rep2": (16, torch.uint8),
              "node_batch2": (16, torch.int16), "node_gpus2": (16, torch.uint8), "node_w": (16, torch.uint8)}

    @classmethod
    def empty(cls, P, device="cuda", groups=False):
        """An unfilled device plan table of P columns (written by cf_enum_plans); groups: with
        the second-configuration arrays (needed for plans of an enumeration with het)."""
        self = cls.__new__(cls)
        self.P, self.t, self.c = int(P), {}, cf_plan_table()
        self.c.P = self.P
        for f in cls.FIELDS + (cls.GROUP_FIELDS if groups else ()):
            rows, dt = cls.SHAPES[f]
            shape = (self.P,) if rows is None else (rows, self.P)
            self.t[f] = torch.empty(shape, dtype=dt, device=device)
            setattr(self.c, f + "_dev", self.t[f].data_ptr())
        return self

    def to_host(self):
        """The table as an inputs.PlanTable (host copy)."""
        from .inputs.plans import PlanTable
        tab = PlanTable(self.P)
        for f in self.FIELDS + tuple(g for g in self.GROUP_FIELDS if g in self.t):
            a = self.t[f].cpu().numpy()
            setattr(tab, f, a.view(np.uint16) if f in ("node_batch", "node_batch2") else a)
        return tab


# ------------------------------------------------------------------ entry points
def cf_trace_gen(desc, seeds, n_req, device="cuda"):
    tr = DeviceTrace(len(seeds), n_req, device)
    moments = torch.empty((len(seeds), desc.n_types, 8), dtype=torch.int64, device=device)
    s = (C.c_uint64 * len(seeds))(*[int(v) for v in seeds])
    _check(_lib.cf_trace_gen(C.byref(desc), s, len(seeds), int(n_req), C.byref(tr.c), _p(moments),
                             _stream()), "cf_trace_gen")
    return tr, moments


def cf_eval_coarse(desc, plans, moments_seed, n_gpus):
    P = plans.P
    dev = moments_seed.device
    rd = torch.empty(P, dtype=torch.float64, device=dev)
    bott = torch.empty(P, dtype=torch.int32, device=dev)
    flags = torch.empty(P, dtype=torch.uint8, device=dev)
    mom = _in(moments_seed, torch.int64, "moments", desc.n_types * 8)
    _check(_lib.cf_eval_coarse(C.byref(desc), C.byref(plans.c), mom,
                               int(n_gpus), _p(rd), _p(bott), _p(flags), _stream()), "cf_eval_coarse")
    return rd, bott, flags


def cf_select_topk(rd, flags, k):
    ids = torch.empty(max(int(k), 1), dtype=torch.int32, device=rd.device)
    n = C.c_int32(0)
    _check(_lib.cf_select_topk(_in(rd, torch.float64, "rd"), _in(flags, torch.uint8, "flags", rd.numel()),
                               int(rd.numel()), int(k), _p(ids), C.byref(n),
                               _stream()), "cf_select_topk")
    return ids[:n.value]


def cf_topk_merge(rd_run, gid_run, rd_win, ids_win, win_first, k):
    """Running top-k of a space screened window by window: the first min(k, n_run + n_win)
    plans of the merged order, as (rd float64, plan number int64) device tensors."""
    dev = rd_win.device
    n = min(int(k), int(rd_run.numel()) + int(ids_win.numel()))
    rd = torch.empty(max(int(k), 1), dtype=torch.float64, device=dev)
    gid = torch.empty(max(int(k), 1), dtype=torch.int64, device=dev)
    run_rd = _in(rd_run, torch.float64, "rd_run")
    run_gid = _in(gid_run, torch.int64, "gid_run", rd_run.numel())
    win_ids = _in(ids_win, torch.int32, "ids_win")
    _check(_lib.cf_topk_merge(run_rd, run_gid, int(rd_run.numel()), _in(rd_win, torch.float64, "rd_win"),
                              win_ids, int(ids_win.numel()), C.c_uint64(int(win_first)), int(k),
                              _p(rd), _p(gid), _stream()), "cf_topk_merge")
    return rd[:n], gid[:n]


def cf_rate_grid(rd, ids, K, alpha_max=1.0):
    rates = torch.empty((ids.numel(), int(K)), dtype=torch.float64, device=rd.device)
    _check(_lib.cf_rate_grid(_in(rd, torch.float64, "rd"), _in(ids, torch.int32, "ids"), int(ids.numel()), int(K),
                             float(alpha_max), _p(rates), _stream()), "cf_rate_grid")
    return rates


def _targets(targets, T):
    tg = np.ascontiguousarray(targets, np.float64)
    if tg.ndim != 3 or tg.shape[0] != T or tg.shape[2] != 4:
        raise CfError("targets must be [T][n_bins][4]")
    return tg


def cf_eval_fine(desc, plans, plan_ids, rates, trace, lat_triples=None, targets=None, limits=None, _entry="cf_eval_fine"):
    """Phase 3 of every (plan, rate, seed); with targets ([T][n_bins][4], bounds not
    decreasing with the bin) also the latency histograms hist [n_plans][K][S][T][n_bins+1];
    with lat_triples the per-request latencies of those triples (CF_DUMP_LAT); limits: a
    dict of the test capacity limits (chunks, delay, instants) of cf_fine_out."""
    n_plans, K = rates.shape
    S, T, dev = trace.n_seeds, desc.n_types, rates.device
    met = torch.empty((n_plans, K, S, T), dtype=torch.int32, device=dev)
    cnt = torch.empty((n_plans, K, S, T), dtype=torch.int32, device=dev)
    events = torch.empty((n_plans, K, S), dtype=torch.int64, device=dev)
    status = torch.empty((n_plans, K, S), dtype=torch.int32, device=dev)
    out = cf_fine_out()
    out.met_dev, out.cnt_dev = met.data_ptr(), cnt.data_ptr()
    out.events_dev, out.status_dev = events.data_ptr(), status.data_ptr()
    lat, flags = None, CF_FULL
    if lat_triples is not None and len(lat_triples) > 0:
        lt = torch.as_tensor(np.asarray(lat_triples, np.int32), device=dev)
        lat = torch.zeros((len(lat_triples), trace.n_req, 4), dtype=torch.float64, device=dev)
        out.lat_dev, out.lat_triples_dev, out.n_lat = lat.data_ptr(), lt.data_ptr(), len(lat_triples)
        flags |= CF_DUMP_LAT
    if limits:
        out.lim_chunks = int(limits.get("chunks", 0))
        out.lim_delay = int(limits.get("delay", 0))
        out.lim_instants = int(limits.get("instants", 0))
    hist = None
    if targets is not None:
        tg = _targets(targets, T)
        hist = torch.empty((n_plans, K, S, T, tg.shape[1] + 1), dtype=torch.int32, device=dev)
        out.hist_dev, out.hist_targets_host, out.n_bins = hist.data_ptr(), tg.ctypes.data, tg.shape[1]
    _check(getattr(_lib, _entry)(C.byref(desc), C.byref(plans.c), _in(plan_ids, torch.int32, "plan_ids", n_plans),
                                 int(n_plans), _in(rates, torch.float64, "rates", ndim=2), int(K), C.byref(trace.c),
                                 flags, C.byref(out), _stream()), _entry)
    return dict(met=met, cnt=cnt, events=events, status=status, lat=lat, hist=hist)


def cf_eval_fine_noalloc(desc, plans, plan_ids, rates, trace, lat_triples=None, targets=None, limits=None):
    """cf_eval_fine through the entry point that allocates no device memory of its own
    (its simulation state lives in the library's fixed per-device array; the output
    tensors are the caller's, as for every call)."""
    return cf_eval_fine(desc, plans, plan_ids, rates, trace, lat_triples, targets, limits,
                        _entry="cf_eval_fine_noalloc")


def cf_eval_bisect(desc, plans, plan_ids, rates, trace, theta):
    """Phase 3 with each plan's rate bisected over its grid: dict(kstar, goodput_t, goodput,
    n_eval, events, status)."""
    n, K = rates.shape
    T, dev = desc.n_types, rates.device
    ks = torch.empty(n, dtype=torch.int32, device=dev)
    gt = torch.empty((n, T), dtype=torch.float64, device=dev)
    g = torch.empty(n, dtype=torch.float64, device=dev)
    ne = torch.empty(n, dtype=torch.int32, device=dev)
    ev = torch.empty(n, dtype=torch.int64, device=dev)
    st = torch.empty(n, dtype=torch.int32, device=dev)
    _check(_lib.cf_eval_bisect(C.byref(desc), C.byref(plans.c), _in(plan_ids, torch.int32, "plan_ids", n), int(n),
                               _in(rates, torch.float64, "rates", ndim=2), int(K), C.byref(trace.c),
                               int(theta[0]), int(theta[1]),
                               _p(ks), _p(gt), _p(g), _p(ne), _p(ev), _p(st), _stream()), "cf_eval_bisect")
    return dict(kstar=ks, goodput_t=gt, goodput=g, n_eval=ne, events=ev, status=st)


def cf_eval_mc(desc, plans, plan_ids, rd, moments_seed, alpha, trace, seed_idx, n_sample,
               want_lat=False):
    n = int(plan_ids.numel())
    T, dev = desc.n_types, rd.device
    met = torch.empty((n, T), dtype=torch.int32, device=dev)
    cnt = torch.empty((n, T), dtype=torch.int32, device=dev)
    gt = torch.empty((n, T), dtype=torch.float64, device=dev)
    lat = torch.empty((n, int(n_sample), 4), dtype=torch.float64, device=dev) if want_lat else None
    mom = _in(moments_seed, torch.int64, "moments", T * 8)
    _check(_lib.cf_eval_mc(C.byref(desc), C.byref(plans.c), _in(plan_ids, torch.int32, "plan_ids"), n,
                           _in(rd, torch.float64, "rd"), mom, float(alpha), C.byref(trace.c), int(seed_idx),
                           int(n_sample), _p(met), _p(cnt), _p(gt), _p(lat), _stream()), "cf_eval_mc")
    return dict(met=met, cnt=cnt, goodput_t=gt, lat=lat)


def cf_eval_mc_curve(desc, plans, plan_ids, rd, moments_seed, alpha, trace, seed_idx, n_sample, targets):
    """Phase 2 with its latency CDF over a target table ([T][n_bins][4]): dict(met, cnt,
    goodput_t, hist [n][T][n_bins+1], curve [n][n_bins][T])."""
    n = int(plan_ids.numel())
    T, dev = desc.n_types, rd.device
    tg = _targets(targets, T)
    nb = tg.shape[1]
    met = torch.empty((n, T), dtype=torch.int32, device=dev)
    cnt = torch.empty((n, T), dtype=torch.int32, device=dev)
    gt = torch.empty((n, T), dtype=torch.float64, device=dev)
    hist = torch.empty((n, T, nb + 1), dtype=torch.int32, device=dev)
    curve = torch.empty((n, nb, T), dtype=torch.float64, device=dev)
    _check(_lib.cf_eval_mc_curve(C.byref(desc), C.byref(plans.c), _in(plan_ids, torch.int32, "plan_ids"), n,
                                 _in(rd, torch.float64, "rd"), _in(moments_seed, torch.int64, "moments", T * 8),
                                 float(alpha), C.byref(trace.c),
                                 int(seed_idx), int(n_sample), int(nb), tg.ctypes.data_as(C.c_void_p), _p(met),
                                 _p(cnt), _p(gt), _p(hist), _p(curve), _stream()), "cf_eval_mc_curve")
    return dict(met=met, cnt=cnt, goodput_t=gt, hist=hist, curve=curve)


def _fine_view(fine, with_hist):
    """cf_fine_out over the arrays of a cf_eval_fine result (met, cnt, status[, hist])."""
    n_plans, K, S, T = fine["met"].shape
    o = cf_fine_out()
    o.met_dev = _in(fine["met"], torch.int32, "met")
    o.cnt_dev = _in(fine["cnt"], torch.int32, "cnt", n_plans * K * S * T)
    o.status_dev = _in(fine["status"], torch.int32, "status", n_plans * K * S)
    if with_hist:
        hist = fine["hist"]
        if hist is None or hist.dim() != 5 or tuple(hist.shape[:4]) != (n_plans, K, S, T):
            raise CfError("hist must be [n_plans][K][S][T][n_bins + 1]")
        o.hist_dev = _in(hist, torch.int32, "hist")
        o.n_bins = int(hist.shape[4]) - 1
    return o, (n_plans, K, S, T)


def cf_goodput_curve(fine, rates, theta, n_req):
    """Goodput against every target bin of a phase-3 histogram (fine: a cf_eval_fine
    result with hist): kstar [n][nb], goodput_t [n][nb][T], goodput [n][nb]."""
    o, (n_plans, K, S, T) = _fine_view(fine, True)
    nb, dev = o.n_bins, fine["met"].device
    kstar = torch.empty((n_plans, nb), dtype=torch.int32, device=dev)
    gt = torch.empty((n_plans, nb, T), dtype=torch.float64, device=dev)
    g = torch.empty((n_plans, nb), dtype=torch.float64, device=dev)
    _check(_lib.cf_goodput_curve(C.byref(o), n_plans, K, S, T, _in(rates, torch.float64, "rates", n_plans * K),
                                 int(theta[0]), int(theta[1]), int(n_req), _p(kstar), _p(gt), _p(g), _stream()),
           "cf_goodput_curve")
    return kstar, gt, g


def cf_pareto(goodput_t, plan_ids=None, flags=None):
    """keep[i] (uint8) = row i not dominated; with plan_ids and flags, also clears
    CF_FLAG_KEEP in flags for the plans of dominated rows (in place)."""
    n, T = goodput_t.shape
    keep = torch.empty(n, dtype=torch.uint8, device=goodput_t.device)
    if (plan_ids is None) != (flags is None):
        raise CfError("cf_pareto: plan_ids and flags go together")
    if flags is not None and (flags.dtype != torch.uint8 or not flags.is_contiguous()):
        raise CfError("cf_pareto: flags must be a contiguous uint8 tensor (updated in place)")
    nf = int(flags.numel()) if flags is not None else 0
    _check(_lib.cf_pareto(_in(goodput_t, torch.float64, "goodput_t", ndim=2), int(n), int(T), _p(keep),
                          _in(plan_ids, torch.int32, "plan_ids", n) if plan_ids is not None else None,
                          _in(flags, torch.uint8, "flags") if flags is not None else None, nf, _stream()),
           "cf_pareto")
    return keep


def enum_opts(mcfg, spec, n_gpus):
    """cf_enum_opts from a model description and an enumeration spec (keys k_s,
    share, colocatable (edge list; default every edge of every type), batch
    {component: knobs}, gpus {component: options}, default [1])."""
    o = cf_enum_opts()
    idx = {c["name"]: i for i, c in enumerate(mcfg["components"])}
    o.n_gpus = int(n_gpus)
    o.k_s = int(spec.get("k_s", 2))
    o.share = 1 if spec.get("share", True) else 0
    o.het = 1 if spec.get("het", False) else 0
    edges = spec.get("colocatable")
    if edges is None:
        edges = [e for ty in mcfg["types"] for e in ty.get("edges", [])]
    for a, b in edges:
        o.colocatable[idx[a]] |= 1 << idx[b]
    for name, i in idx.items():
        knobs = list(spec["batch"][name])
        o.n_batch[i] = len(knobs)
        for k, v in enumerate(knobs):
            o.batch[i][k] = int(v)
        gl = list(spec.get("gpus", {}).get(name, [1]))
        o.n_gpu_opt[i] = len(gl)
        for k, v in enumerate(gl):
            o.gpu_opt[i][k] = int(v)
    return o


def cf_enum_logical(desc, opts, cap=65536):
    """Logical plans (host): uint8 array [n, LOGICAL_BYTES] in cf_logical layout."""
    buf = np.zeros((cap, LOGICAL_BYTES), np.uint8)
    n = C.c_int32(0)
    _check(_lib.cf_enum_logical(C.byref(desc), C.byref(opts), buf.ctypes.data_as(C.c_void_p), int(cap),
                                C.byref(n)), "cf_enum_logical")
    return buf[: n.value].copy()


def cf_enum_count(desc, opts, logical_dev):
    """(offsets [n+1] uint64 on the device, total physical plans)."""
    n = int(logical_dev.shape[0])
    offsets = torch.empty(n + 1, dtype=torch.int64, device=logical_dev.device)
    total = C.c_uint64(0)
    _check(_lib.cf_enum_count(C.byref(desc), C.byref(opts), _p(logical_dev.contiguous()), n, _p(offsets),
                              C.byref(total), _stream()), "cf_enum_count")
    return offsets, int(total.value)


def cf_enum_plans(desc, opts, logical_dev, offsets, total, first, count, out=None):
    """Physical plans first..first+count-1 into a device plan table (new, or out)."""
    if out is None:
        out = DevicePlans.empty(count, logical_dev.device, groups=bool(opts.het))
    _check(_lib.cf_enum_plans(C.byref(desc), C.byref(opts), _p(logical_dev.contiguous()),
                              int(logical_dev.shape[0]), _p(offsets), C.c_uint64(int(total)),
                              C.c_uint64(int(first)), int(count), C.byref(out.c), _stream()), "cf_enum_plans")
    return out


def cf_enum_screen(desc, opts, logical_dev, offsets, total, first, count, moments_seed, n_gpus):
    """Phase 1 of physical plans first..first+count-1 without their table: (rd, bottleneck, flags)."""
    dev = logical_dev.device
    rd = torch.empty(int(count), dtype=torch.float64, device=dev)
    bott = torch.empty(int(count), dtype=torch.int32, device=dev)
    flags = torch.empty(int(count), dtype=torch.uint8, device=dev)
    _check(_lib.cf_enum_screen(C.byref(desc), C.byref(opts), _p(logical_dev.contiguous()), int(logical_dev.shape[0]),
                               _p(offsets), C.c_uint64(int(total)), C.c_uint64(int(first)), int(count),
                               _in(moments_seed, torch.int64, "moments", desc.n_types * 8), int(n_gpus), _p(rd),
                               _p(bott), _p(flags), _stream()),
           "cf_enum_screen")
    return rd, bott, flags


def cf_goodput_reduce(fine, rates, theta, n_req):
    """Highest feasible rate and goodput per plan from a cf_eval_fine result (met, cnt,
    status): kstar [n], goodput_t [n][T], goodput [n]."""
    o, (n_plans, K, S, T) = _fine_view(fine, False)
    dev = fine["met"].device
    kstar = torch.empty(n_plans, dtype=torch.int32, device=dev)
    gt = torch.empty((n_plans, T), dtype=torch.float64, device=dev)
    g = torch.empty(n_plans, dtype=torch.float64, device=dev)
    _check(_lib.cf_goodput_reduce(C.byref(o), n_plans, K, S, T, _in(rates, torch.float64, "rates", n_plans * K),
                                  int(theta[0]), int(theta[1]), int(n_req), _p(kstar), _p(gt), _p(g),
                                  _stream()), "cf_goodput_reduce")
    return kstar, gt, g


def cf_select_best(goodput):
    best = torch.empty(1, dtype=torch.int32, device=goodput.device)
    _check(_lib.cf_select_best(_in(goodput, torch.float64, "goodput"), int(goodput.numel()), _p(best), _stream()),
           "cf_select_best")
    return best


def cf_math_eval(op, x, y=None):
    out = torch.empty_like(x)
    _check(_lib.cf_math_eval(int(op), _p(x), _p(y), _p(out), int(x.numel()), _stream()), "cf_math_eval")
    return out


def cf_philox_eval(ctr, key):
    out = torch.empty_like(ctr)
    _check(_lib.cf_philox_eval(_p(ctr), _p(key), _p(out), int(ctr.shape[0]), _stream()),
           "cf_philox_eval")
    return out


def cf_release_scratch():
    _check(_lib.cf_release_scratch(), "cf_release_scratch")
