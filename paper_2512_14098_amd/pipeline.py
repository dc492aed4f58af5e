"""One pass of the evaluated path on the GPU for a workload configuration.

trace generation -> phase 1 screening (Alg. 2) -> [phase 2: Monte Carlo
latency of every kept plan and Pareto pruning] -> top-K by R_d -> rate grid
-> phase 3 simulation of every (plan, rate, seed) -> goodput reduction ->
selection.  Every step is a libcf call on torch's current stream; this
module only allocates device tensors and sequences the calls.
"""
import numpy as np
import torch

from . import cf
from .inputs import load_config, make_plans, seeds_of

MAX_PHASE2 = 65536  # plans per phase-2 pass (the selection's capacity)


class Workload:
    """Device-resident inputs of one configuration (plans, model, seeds)."""

    def __init__(self, cfg, n_req=None, seeds=None, device="cuda", phase2=None):
        if isinstance(cfg, str):
            cfg = load_config(cfg)
        self.cfg = cfg
        self.desc = cf.model_desc(cfg["model"])
        self.tab = make_plans(cfg)
        self.plans = cf.DevicePlans(self.tab, device)
        self.seeds = seeds if seeds is not None else seeds_of(cfg)
        self.n_req = int(cfg["n_req"] if n_req is None else n_req)
        self.n_gpus = int(cfg["gpus"])
        self.theta = cfg["model"].get("theta", [9, 10])
        r = cfg["rates"]
        self.explicit_rates = r.get("explicit")
        self.K = len(self.explicit_rates) if self.explicit_rates else int(r["grid"])
        self.alpha_max = float(r.get("alpha_max", 1.0))
        top = cfg.get("top_k")
        self.top_k = int(top) if top else self.tab.P
        self.device = device
        # phase 2 (optional): dict(K=sampled requests, alpha=headroom), or None to go
        # from phase 1 straight to phase 3 over the top_k plans
        self.phase2 = phase2 if phase2 is not None else cfg.get("phase2")
        # optional latency-target table [T][n_bins][4]: phase 3 then also emits latency
        # histograms, and the reduction goodput at every target
        self.targets = None
        # phase 3 by rate bisection over each plan's grid instead of every grid rate
        self.bisect = False
        # phase 3 of one slice of the stage: (part, parts, seed index) simulates the selected
        # plans part, part + parts, part + 2 parts, ... at every grid rate on that one seed, and
        # reduces them over it; None simulates every plan on every seed
        self.slice = None

    def set_target_scales(self, scales):
        """Targets = each type's own bounds times each scale (ascending)."""
        T = len(self.cfg["model"]["types"])
        tg = np.empty((T, len(scales), 4), np.float64)
        for t, ty in enumerate(self.cfg["model"]["types"]):
            slo = ty.get("slo", {})
            for j, key in enumerate(("ttft", "tpot", "e2e", "media")):
                bound = float(slo[key]) if key in slo else np.inf
                tg[t, :, j] = [bound * float(sc) for sc in scales]
        self.targets = tg


def run_step(w, timers=None):
    """One pass over the whole path; returns every intermediate on the device.

    ``timers`` (optional dict) receives (start, end) torch.cuda.Event pairs
    recorded around each step on the current stream."""
    ev = {}

    def mark(name):
        if timers is None:
            return None
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        ev.setdefault(name, []).append(e)
        return e

    mark("trace")
    trace, moments = cf.cf_trace_gen(w.desc, w.seeds, w.n_req, w.device)
    mark("trace")
    mark("coarse")
    rd, bott, flags = cf.cf_eval_coarse(w.desc, w.plans, moments[0], w.n_gpus)
    mark("coarse")
    mc = None
    if w.phase2:
        mark("phase2")
        cand = cf.cf_select_topk(rd, flags, MAX_PHASE2)
        if cand.numel() >= MAX_PHASE2:
            # plans past the selection's capacity would keep their flag unevaluated
            raise cf.CfError("phase 2 takes fewer than %d kept plans" % MAX_PHASE2)
        K = min(int(w.phase2["K"]), w.n_req)
        mc = cf.cf_eval_mc(w.desc, w.plans, cand, rd, moments[0], float(w.phase2["alpha"]), trace, 0, K)
        mc["ids"] = cand
        mc["keep"] = cf.cf_pareto(mc["goodput_t"], cand, flags)
        mark("phase2")
    mark("select")
    ids = cf.cf_select_topk(rd, flags, w.top_k)
    if w.explicit_rates:
        rates = torch.tensor(w.explicit_rates, dtype=torch.float64, device=w.device).repeat(ids.numel(), 1)
    else:
        rates = cf.cf_rate_grid(rd, ids, w.K, w.alpha_max)
    mark("select")
    f_ids, f_rates, f_trace = ids, rates, trace
    if w.slice is not None:
        part, parts, s = w.slice
        f_ids, f_rates, f_trace = ids[part::parts].contiguous(), rates[part::parts].contiguous(), trace.seed_view(s)
    mark("fine")
    if w.bisect:
        fine = cf.cf_eval_bisect(w.desc, w.plans, f_ids, f_rates, f_trace, w.theta)
    else:
        fine = cf.cf_eval_fine(w.desc, w.plans, f_ids, f_rates, f_trace, targets=w.targets)
    mark("fine")
    mark("reduce")
    if w.bisect:
        kstar, gt, g = fine["kstar"], fine["goodput_t"], fine["goodput"]
    else:
        kstar, gt, g = cf.cf_goodput_reduce(fine, f_rates, w.theta, w.n_req)
    best = cf.cf_select_best(g) if f_ids.numel() > 0 else None
    curve = None
    if w.targets is not None and f_ids.numel() > 0 and not w.bisect:
        curve = dict(zip(("kstar", "goodput_t", "goodput"),
                         cf.cf_goodput_curve(fine, f_rates, w.theta, w.n_req)))
    mark("reduce")
    if timers is not None:
        timers.update(ev)
    return dict(trace=trace, moments=moments, rd=rd, bottleneck=bott, flags=flags, ids=ids,
                rates=rates, fine_ids=f_ids, fine_rates=f_rates, fine=fine, kstar=kstar, goodput_t=gt, goodput=g,
                best=best, phase2=mc, curve=curve)


def reweight(w, out, weights, K=1024, alpha=0.8):
    """Phases 1 and 2 again under new request-type weights, on the samples already drawn
    (Sec. 4.4: a change of the type fractions pi_t re-weights existing samples).  Only the
    weights change: the trace, its per-type moments and the sampled requests of ``out``
    (a run_step result) are kept; phase 1 recomputes R_d and the flags, phase 2 re-walks the
    same sampled requests at the new effective batches, and Pareto pruning clears the keep
    flag of dominated plans.  Phase 3 is not re-weighted: a different mix changes queueing,
    so it needs a new simulation."""
    mcfg = dict(w.cfg["model"])
    if len(weights) != len(mcfg["types"]):
        raise cf.CfError("one weight per request type")
    mcfg["types"] = [dict(t, weight=int(wt)) for t, wt in zip(mcfg["types"], weights)]
    desc = cf.model_desc(mcfg)
    rd, bott, flags = cf.cf_eval_coarse(desc, w.plans, out["moments"][0], w.n_gpus)
    cand = cf.cf_select_topk(rd, flags, MAX_PHASE2)
    if cand.numel() >= MAX_PHASE2:
        raise cf.CfError("phase 2 takes fewer than %d kept plans" % MAX_PHASE2)
    K = min(int(K), w.n_req)
    mc = cf.cf_eval_mc(desc, w.plans, cand, rd, out["moments"][0], float(alpha), out["trace"], 0, K)
    mc["ids"] = cand
    mc["keep"] = cf.cf_pareto(mc["goodput_t"], cand, flags)
    return dict(desc=desc, rd=rd, bottleneck=bott, flags=flags, phase2=mc)


def screen_space(desc, opts, logical_dev, offsets, total, moments_seed, n_gpus, k, first=0, count=None,
                 window=1 << 24):
    """Phase 1 (Alg. 2) over plans first .. first+count-1 of an enumerated space (Alg. 1),
    one window of at most ``window`` plans at a time without writing their table
    (cf_enum_screen), keeping the k plans with the largest R_d among those phase 1 keeps
    (cf_select_topk per window, cf_topk_merge across windows).  Returns (rd, plan numbers)
    as device tensors in the order of cf_select_topk: R_d descending, ties by plan number."""
    count = int(total) - int(first) if count is None else int(count)
    if not 1 <= window <= 1 << 24:
        raise cf.CfError("window must be in 1..2^24 plans")
    dev = logical_dev.device
    rd_run = torch.empty(0, dtype=torch.float64, device=dev)
    gid_run = torch.empty(0, dtype=torch.int64, device=dev)
    w0, end = int(first), int(first) + count
    while w0 < end:
        c = min(int(window), end - w0)
        rd, _, flags = cf.cf_enum_screen(desc, opts, logical_dev, offsets, total, w0, c, moments_seed, n_gpus)
        ids = cf.cf_select_topk(rd, flags, k)
        if ids.numel():
            rd_run, gid_run = cf.cf_topk_merge(rd_run, gid_run, rd, ids, w0, k)
        w0 += c
    return rd_run, gid_run


def best_plan(out):
    """Host-side summary of a step's selection."""
    if out["best"] is None:
        return None
    b = int(out["best"].item())
    return dict(index=b, plan_id=int(out["fine_ids"][b].item()), goodput=float(out["goodput"][b].item()),
                kstar=int(out["kstar"][b].item()))


def events_total(out):
    return int(out["fine"]["events"].sum().item())


def status_summary(out):
    st = out["fine"]["status"].cpu().numpy()
    return {int(k): int(v) for k, v in zip(*np.unique(st, return_counts=True))}
