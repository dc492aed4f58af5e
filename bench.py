"""Benchmark: simulated request-events/s and plans fully evaluated/s on one GPU.

A step is one pass of the whole evaluated path over one synthetic workload:
trace generation, phase-1 screening of every plan, top-K selection, rate
grid, phase-3 simulation of every (plan, rate, seed) triple, goodput
reduction and selection.  Default workload: c1 (E->L on 8 simulated GPUs,
1000 plans screened, the kept ones simulated at 16 rates x 32 seeds x 10^4
requests).  Prints one JSON line.

Other modes (each prints its own JSON line and exits): --enum times plan
enumeration on the device, phase-1 screening of its output, the fused
enumeration-and-screening kernel and a windowed screening with a running top-k;
--phase2 times phase 2 (Monte Carlo latency of every plan phase 1 keeps, default
workload c4) and Pareto pruning; --stress times the HBM-bound steps at full c4
size; --copy-probe runs the plain copy the HBM byte counters are calibrated on.
Variants of the default step: --curve N adds goodput curves over N latency-target
scales, --bisect bisects each plan's rate instead of simulating every grid rate,
--config/--seeds/--plans pick another workload or a sample of one.  The default
run also times the oracle on the host (single core, then one process per core).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "simulated request-events/sec and candidate plans fully evaluated/sec, 1 GPU"
PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9 / 1e12  # T lane-ops/s: CUs x SIMDs x lanes x clock
OPS_PER_EVENT = 4.0  # algorithmic lane-ops per request-event
KERNEL_SOURCES = ("paper_2512_14098_amd/csrc/k_fine.hip", "paper_2512_14098_amd/csrc/cf_internal.h",
                  "paper_2512_14098_amd/csrc/cf_run.h")
MC_KERNEL_SOURCES = ("paper_2512_14098_amd/csrc/k_mc.hip", "paper_2512_14098_amd/csrc/cf_internal.h",
                     "paper_2512_14098_amd/csrc/cf_run.h")
# HBM bytes per launch of the dominant kernel from rocprofv3 counters (FETCH_SIZE x 2.0 +
# WRITE_SIZE x 1.0, the scale factors a plain 1 GiB device copy gives), keyed by the kernel
# source the counters were taken on and the workload (with its sample); any other source or
# workload reports null
_W_C1 = ("c1: MLLM graph E->L on 8 simulated GPUs (7B LLM, 600M ViT); ~1000 plans; 16-point rate grid; "
         "32 seeds x 10000 requests")
_W_C2_SEEDS2 = ("c2: Omni graph (E_img, E_aud) -> thinker -> gated talker -> audio generator on 16 simulated GPUs; "
                "~10000 sampled plans; 16 rates; 32 seeds x 20000 requests (sample: first 2 of its 32 seeds)")
_W_C3_SEED0 = ("c3: Text-to-image graph L -> 50-step diffusion G (1024^2) mixed 50/50 with text-only LLM requests "
               "on 32 simulated GPUs; ~50000 sampled plans; 16 rates; 64 seeds x 50000 requests "
               "(sample: first 1 of its 64 seeds)")
_W_C4_STEP = ("c4: Full coarse-to-fine sweep of the omni graph on 64 simulated GPUs: coarse screening of 10^6 "
              "sampled plans, the top 1000 by R_d simulated at 32 rates x 64 seeds x 100000 requests; each step: "
              "the trace of all 64 seeds, phase 1 over all 1000000 plans, the top 1000 and their 32-rate grid, "
              "phase 3 of every selected plan at every rate on one seed (seed g at step g), their goodput reduction")
MEASURED_TRAFFIC = {
    ("7ed4a4b598700ba3", _W_C4_STEP): 1.4861e13,
    ("7ed4a4b598700ba3", _W_C1): 8.4908e11,
    ("7ed4a4b598700ba3", _W_C2_SEEDS2): 7.9068e11,
    ("7ed4a4b598700ba3", _W_C3_SEED0): 1.8009e12,
}
# VALU lane rate of the k_fine launch by rocprofv3 counters (SQ_INSTS_VALU x SQ_THREAD_CYCLES_VALU /
# SQ_ACTIVE_INST_VALU / kernel time / PEAK_LANE_OPS), keyed like MEASURED_TRAFFIC
MEASURED_LANE_FRAC = {
    ("7ed4a4b598700ba3", _W_C4_STEP): 0.3829,
    ("7ed4a4b598700ba3", _W_C1): 0.4314,
    ("7ed4a4b598700ba3", _W_C2_SEEDS2): 0.4059,
    ("7ed4a4b598700ba3", _W_C3_SEED0): 0.3950,
}
ENUM_KERNEL_SOURCES = ("paper_2512_14098_amd/csrc/k_enum.hip", "paper_2512_14098_amd/csrc/cf_internal.h",
                       "paper_2512_14098_amd/csrc/cf_phase1.h")
# bytes per k_enum_unrank launch of 2^25 plans (the write counter reads exactly the table bytes)
ENUM_MEASURED_TRAFFIC = {("b9ac6efd2fcc5a5b", 1 << 25): 7.8191e9}
MC_MEASURED_TRAFFIC = {
    ("7c84b8868934b26b", "c4 phase 2: the 17471 plans phase 1 keeps of 1000000, 1024 sampled requests (seed 0), "
     "alpha 0.8, then Pareto pruning"): 3.7331e8,
}


def kernel_source_id(files=KERNEL_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _oracle_triples(cfg, seeds, n_req, triples, budget_s):
    """One worker of the all-cores CPU baseline: the oracle on its share of the triples
    (plan id, rate, index into seeds) until the budget is spent."""
    from oracle import oracle as O
    from paper_2512_14098_amd.inputs import make_plans
    tab = make_plans(cfg)
    m = O.make_model(cfg["model"])
    otr = O.trace_gen(m, seeds, n_req)
    pst, tst = O.plans_struct(tab), O.trace_struct(otr)
    ev, n, t0 = 0, 0, time.perf_counter()
    for (p, rate, s) in triples:
        ev += O.sim_triple(m, tab, p, rate, otr, s, _pst=pst, _tst=tst)["events"]
        n += 1
        if time.perf_counter() - t0 > budget_s:
            break
    return ev, n, time.perf_counter() - t0


def cpu_baseline_all_cores(w, ids, rates, order, seeds_needed, budget_s, workers):
    """The same oracle in one process per host core (processes started fresh, no GPU in
    them), the sampled triples dealt round-robin; value = total request-events / the
    longest worker's timed loop."""
    import multiprocessing as mp
    jobs = [[] for _ in range(workers)]
    j = 0
    for (i, k, s) in order:
        if s in seeds_needed:
            jobs[j % workers].append((int(ids[i]), float(rates[i, k]), seeds_needed.index(s)))
            j += 1
    seeds = [w.seeds[s] for s in seeds_needed]
    with mp.get_context("spawn").Pool(workers) as pool:
        res = pool.starmap(_oracle_triples, [(w.cfg, seeds, w.n_req, jb, budget_s) for jb in jobs])
    ev, n, dt = sum(r[0] for r in res), sum(r[1] for r in res), max(r[2] for r in res)
    return {"value": ev / dt, "unit": "request-events/s", "cores": workers, "kind": "oracle",
            "sample": "%d triples of this workload drawn uniformly over its selected plans, its rates and "
                      "its first %d seeds, in %d processes (%d request-events, longest worker %.1f s)"
                      % (n, len(seeds_needed), workers, ev, dt)}


def host_info():
    """CPU model and core count of this host, for the CPU-baseline record."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(),
            "affinity": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}


def cpu_baseline(w, budget_s, all_cores=0, events_per_step=None):
    """The oracle, single-threaded on this host (pinned to one core), on a
    bounded sample of the same workload's triples (spread over plans, rates and
    seeds); the oracle's own phase 1, selection and rate grid choose the plans
    and rates.  With events_per_step, also the time one full step would take at
    the measured rate (extrapolated linearly in request-events)."""
    import numpy as np

    from oracle import oracle as O
    m = O.make_model(w.cfg["model"])
    mom0 = O.trace_gen(m, [w.seeds[0]], w.n_req)["moments"][0]
    pst = O.plans_struct(w.tab)
    # the oracle's phase 1 over the whole plan table, on one core
    saved_aff = None
    try:
        saved_aff = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(saved_aff)})
    except (AttributeError, OSError):
        saved_aff = None
    t0 = time.perf_counter()
    rd, _, fl = O.eval_coarse(m, w.tab, mom0, w.n_gpus)
    coarse_s = time.perf_counter() - t0
    if saved_aff is not None:
        try:
            os.sched_setaffinity(0, saved_aff)
        except OSError:
            pass
    ids = O.select_topk(rd, fl, w.top_k)
    if w.explicit_rates:
        rates = np.tile(np.asarray(w.explicit_rates, np.float64), (len(ids), 1))
    else:
        rates = O.rate_grid(rd, ids, w.K, w.alpha_max)
    # seeds drawn from the first few only: the oracle generates the trace of every seed it
    # samples, which for 64 seeds of 10^5 requests would cost more than the timed budget
    S = min(len(w.seeds), 4)
    order = []
    rng = np.random.default_rng(0)
    for _ in range(32768):  # enough for every core's budget
        order.append((int(rng.integers(len(ids))), int(rng.integers(rates.shape[1])), int(rng.integers(S))))
    seeds_needed = sorted({s for _, _, s in order[:256]})
    otr = O.trace_gen(m, [w.seeds[s] for s in seeds_needed], w.n_req)
    tst = O.trace_struct(otr)
    host = host_info()
    pinned = None
    try:
        saved = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(saved)})
        pinned = min(saved)
    except (AttributeError, OSError):
        pass
    ev, n, t0 = 0, 0, time.perf_counter()
    for (i, k, s) in order:
        if s not in seeds_needed:
            continue
        o = O.sim_triple(m, w.tab, int(ids[i]), float(rates[i, k]), otr, seeds_needed.index(s),
                         _pst=pst, _tst=tst)
        ev += o["events"]
        n += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    if pinned is not None:
        try:
            os.sched_setaffinity(0, saved)
        except OSError:
            pass
    res = {"value": ev / dt, "unit": "request-events/s", "cores": 1, "kind": "oracle",
           "sample": "%d triples of this workload drawn uniformly over its selected plans, its rates and "
                     "its first %d seeds (%d request-events in %.1f s, single thread%s)"
                     % (n, S, ev, dt, "" if pinned is None else ", pinned to core %d" % pinned),
           "host": host,
           "coarse": {"value": w.tab.P / coarse_s, "unit": "plans/s", "cores": 1, "kind": "oracle",
                      "sample": "phase 1 over all %d plans of the workload in %.2f s, single thread"
                                % (w.tab.P, coarse_s)}}
    if events_per_step:
        res["full_step_s_extrapolated"] = events_per_step / res["value"]
    if all_cores > 1:
        res["all_cores"] = cpu_baseline_all_cores(w, ids, rates, order, seeds_needed, budget_s, all_cores)
        if events_per_step:
            res["all_cores"]["full_step_s_extrapolated"] = events_per_step / res["all_cores"]["value"]
    return res


def stress(reps, steps):
    """HBM-bound steps at full size on the c4 inputs, each timed with HIP events on the stream it
    runs on: trace generation of all 64 seeds x 10^5 requests (write-bound), and phase-1
    screening of the 10^6 c4 plans tiled reps times (read-bound).  Algorithmic bytes: the trace
    fields written (44 B per request); per plan, the table bytes the screening must read (plan
    node count, 5 B per node, per type its alternative count and, per alternative, the weight and
    one node byte per path component) plus the 13 B written (R_d, bottleneck, flags)."""
    import numpy as np
    import torch

    from paper_2512_14098_amd import cf
    from paper_2512_14098_amd.inputs import load_config, make_plans, seeds_of
    cfg = load_config("c4")
    desc = cf.model_desc(cfg["model"])
    seeds, n = seeds_of(cfg), int(cfg["n_req"])
    peak = 8.0e12

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            out = fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps / 1e3, out

    t_tr, (tr, mom) = timed(lambda: cf.cf_trace_gen(desc, seeds, n))
    tr_bytes = 44.0 * len(seeds) * n
    print(json.dumps({"stress": "cf_trace_gen", "workload": "c4 trace: %d seeds x %d requests" % (len(seeds), n),
                      "ms": t_tr * 1e3, "requests_per_s": len(seeds) * n / t_tr,
                      "roofline": {"bound": "hbm", "achieved": tr_bytes / t_tr / 1e9, "peak": peak / 1e9,
                                   "unit": "GB/s", "frac": tr_bytes / t_tr / peak,
                                   "alg_bytes_per_request": 44}}), flush=True)
    tab = make_plans(cfg)
    base = cf.DevicePlans(tab)
    big = cf.DevicePlans.__new__(cf.DevicePlans)
    big.P, big.t, big.c = base.P * reps, {}, cf.cf_plan_table()
    big.c.P = big.P
    for f, t in base.t.items():
        big.t[f] = t.repeat(reps) if t.dim() == 1 else t.repeat(1, reps)
        setattr(big.c, f + "_dev", big.t[f].data_ptr())
    del base
    nt = desc.n_types
    path_len = np.array([bin(int(desc.path_mask[t])).count("1") for t in range(nt)])
    na = tab.n_alt[:nt].astype(np.int64)
    per_plan = 1 + 5 * tab.n_nodes.astype(np.int64) + (na * (1 + path_len[:, None])).sum(axis=0) + nt + 13
    plan_bytes = float(per_plan.sum()) * reps
    t_co, _ = timed(lambda: cf.cf_eval_coarse(desc, big, mom[0], int(cfg["gpus"])))
    print(json.dumps({"stress": "cf_eval_coarse", "workload": "c4 plans: %d sampled plans tiled %d times" % (tab.P, reps),
                      "plans": big.P, "ms": t_co * 1e3, "plans_per_s": big.P / t_co,
                      "roofline": {"bound": "hbm", "achieved": plan_bytes / t_co / 1e9, "peak": peak / 1e9,
                                   "unit": "GB/s", "frac": plan_bytes / t_co / peak,
                                   "alg_bytes_per_plan": plan_bytes / big.P,
                                   "table_bytes_per_plan": 233 + 13}}), flush=True)


PHASE2_OPS = {"component": 6.0, "llm_component": 8.0, "gated_token": 4.0, "slo": 5.0}


def phase2_ops_per_plan(cfg, tr_np, K):
    """Algorithmic lane-ops of one plan's phase 2 over the first K requests of seed 0: per
    request, 6 per encoder/generator visited (latest input, (k0 + k1 (b x)) + k2 b, finish),
    8 per LLM visited (latest input, prefill, decode step time, closed-form end of the decode
    run), 4 per gated decode token after the first (source token, its arrival, wait, step),
    5 for the SLO test and count.  The same for every plan (paths depend on the type only)."""
    import numpy as np
    mc = cfg["model"]
    comps = mc["components"]
    ttype = tr_np["type"][:K].astype(np.int64)
    attrs = {"prompt": tr_np["prompt"][:K].astype(np.int64), "out": tr_np["out"][:K].astype(np.int64),
             "patches": tr_np["patches"][:K].astype(np.int64),
             "aud_in_ms": tr_np["aud_in_ms"][:K].astype(np.int64),
             "aud_out_ms": tr_np["aud_out_ms"][:K].astype(np.int64)}
    attrs["aud_in_tok"] = (attrs["aud_in_ms"] + 79) // 80
    attrs["aud_out_tok"] = (attrs["aud_out_ms"] + 79) // 80
    total = 0.0
    for t, ty in enumerate(mc["types"]):
        sel = ttype == t
        nreq = int(sel.sum())
        if nreq == 0:
            continue
        ops = PHASE2_OPS["slo"]
        for cn in ty["comps"]:
            c = next(x for x in comps if x["name"] == cn)
            ops += PHASE2_OPS["llm_component"] if c["kind"] == "LLM" else PHASE2_OPS["component"]
        total += ops * nreq
        for cn in ty["comps"]:
            c = next(x for x in comps if x["name"] == cn)
            if c.get("gate") in ty["comps"] and [c["gate"], cn] in [list(e) for e in ty.get("edges", [])]:
                tok = np.maximum(attrs[c.get("n_out", "out")][sel], 1)
                total += PHASE2_OPS["gated_token"] * float((tok - 1).sum())
    return total


def phase2_bench(args):
    """Phase 2 (Monte Carlo latency with occupancy-aware batches) of every plan phase 1 keeps,
    then Pareto pruning, timed with HIP events on the stream they run on."""
    import numpy as np
    import torch

    from paper_2512_14098_amd import cf
    from paper_2512_14098_amd.inputs import load_config, make_plans, seeds_of
    cfg = load_config(args.config)
    K, alpha = int(args.mc_samples), float(args.mc_alpha)
    desc = cf.model_desc(cfg["model"])
    seed = seeds_of(cfg)[0]
    print("bench: phase 2 on %s, plans" % args.config, file=sys.stderr, flush=True)
    tab = make_plans(cfg)
    plans = cf.DevicePlans(tab)
    tr, mom = cf.cf_trace_gen(desc, [seed], max(K, 1))
    rd, _, flags = cf.cf_eval_coarse(desc, plans, mom[0], int(cfg["gpus"]))
    cand = cf.cf_select_topk(rd, flags, 65536)
    n = int(cand.numel())
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]

    def step():
        ev[0].record()
        out = cf.cf_eval_mc(desc, plans, cand, rd, mom[0], alpha, tr, 0, K)
        ev[1].record()
        keep = cf.cf_pareto(out["goodput_t"], cand, flags)
        ev[2].record()
        return out, keep

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mc_ms, par_ms = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out, keep = step()
        torch.cuda.synchronize()
        mc_ms.append(ev[0].elapsed_time(ev[1]))
        par_ms.append(ev[1].elapsed_time(ev[2]))
    elapsed = time.perf_counter() - t0
    kept = int(keep.sum().item())
    ops = phase2_ops_per_plan(cfg, tr.to_numpy(), K) * n
    mc_s = sum(mc_ms) / len(mc_ms) / 1e3
    achieved = ops / mc_s / 1e12
    workload = ("%s phase 2: the %d plans phase 1 keeps of %d, %d sampled requests (seed %d), alpha %g, "
                "then Pareto pruning" % (args.config, n, tab.P, K, seed, alpha))
    res = {"metric": "candidate plans through phase 2 (Monte Carlo latency + Pareto pruning)/sec, 1 GPU",
           "value": n * args.steps / elapsed, "unit": "plans/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": elapsed * 1e3 / args.steps, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
           "config": {"workload": workload, "plans": n, "kept_after_pareto": kept, "mc_ms": mc_ms,
                      "pareto_ms": par_ms},
           "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_LANE_OPS, "unit": "TOP/s",
                        "frac": achieved / PEAK_LANE_OPS,
                        "traffic": MC_MEASURED_TRAFFIC.get((kernel_source_id(MC_KERNEL_SOURCES), workload)),
                        "kernel": "k_mc",
                        "ops_per_plan": ops / max(n, 1), "kernel_ms": sum(mc_ms) / len(mc_ms)}}
    if not args.no_cpu_baseline and n > 0:
        from oracle import oracle as O
        m = O.make_model(cfg["model"])
        otr = O.trace_gen(m, [seed], max(K, 1))
        # the oracle's own phase 1 and selection give the plans it walks
        rd_h, _, fl_h = O.eval_coarse(m, tab, otr["moments"][0], int(cfg["gpus"]))
        ids = O.select_topk(rd_h, fl_h, n)
        done, t0 = 0, time.perf_counter()
        while done < n and time.perf_counter() - t0 < args.cpu_budget:
            chunk = ids[done:done + 16]
            O.eval_mc(m, tab, chunk, rd_h, otr["moments"][0], alpha, otr, 0, K)
            done += len(chunk)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": done / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
                               "sample": "the first %d of the %d plans (highest R_d), %d requests each, "
                                         "single thread, %.1f s" % (done, n, K, dt)}
    print(json.dumps(res), flush=True)


ENUM_PLAN_BYTES = 233  # plan-table bytes written per plan: 1 + 16 x (1 + 1 + 2 + 1) + 8 + 16 + 128


def enum_bench(args):
    """Plan enumeration on the device: the omni graph's space on 16 GPUs (c2's model, two
    subplans, shared nodes, batch knobs {16, 64, 256}), CHUNK plans per launch at evenly spaced
    starting points, then phase-1 screening of the same table.  HBM-bound: the table is written
    once (233 B per plan); the count tables and logical plans stay in cache."""
    import torch

    from paper_2512_14098_amd import cf
    from paper_2512_14098_amd.inputs import load_config
    cfg = load_config(args.config)
    mc = cfg["model"]
    N = int(cfg["gpus"])
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: [16, 64, 256] for c in mc["components"]}}
    desc, opts = cf.model_desc(mc), cf.enum_opts(mc, spec, N)
    t0 = time.perf_counter()
    logical = cf.cf_enum_logical(desc, opts)
    t_logical = time.perf_counter() - t0
    ldev = torch.from_numpy(logical).cuda()
    offsets, total = cf.cf_enum_count(desc, opts, ldev)
    chunk = int(args.enum_chunk)
    out = cf.DevicePlans.empty(chunk)
    tr, mom = cf.cf_trace_gen(desc, [0], 4096)
    starts = [(total - chunk) * i // max(args.steps - 1, 1) for i in range(args.steps)]
    for _ in range(args.warmup):
        cf.cf_enum_plans(desc, opts, ldev, offsets, total, 0, chunk, out)
        cf.cf_eval_coarse(desc, out, mom[0], N)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    enum_ms, coarse_ms, fused_ms = [], [], []
    t0 = time.perf_counter()
    for s0 in starts:
        ev[0].record()
        cf.cf_enum_plans(desc, opts, ldev, offsets, total, s0, chunk, out)
        ev[1].record()
        cf.cf_eval_coarse(desc, out, mom[0], N)
        ev[2].record()
        torch.cuda.synchronize()
        enum_ms.append(ev[0].elapsed_time(ev[1]))
        coarse_ms.append(ev[1].elapsed_time(ev[2]))
    elapsed = time.perf_counter() - t0
    # the fused path: phase 1 of the same plans without writing their table
    for s0 in starts:
        ev[0].record()
        cf.cf_enum_screen(desc, opts, ldev, offsets, total, s0, chunk, mom[0], N)
        ev[1].record()
        torch.cuda.synchronize()
        fused_ms.append(ev[0].elapsed_time(ev[1]))
    # a range screened window by window keeping the best 1000 (cf_enum_screen, cf_select_topk,
    # cf_topk_merge), host synchronisation of the selection included
    from paper_2512_14098_amd import pipeline
    win = min(chunk, 1 << 24)
    span = min(4 * win, total)  # the first plans of the space: small replica counts, many of them kept
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    top_rd, top_gid = pipeline.screen_space(desc, opts, ldev, offsets, total, mom[0], N, 1000, 0, span, win)
    torch.cuda.synchronize()
    topk_s = time.perf_counter() - t1
    e_s = sum(enum_ms) / len(enum_ms) / 1e3
    achieved = ENUM_PLAN_BYTES * chunk / e_s
    res = {"metric": "physical plans enumerated (Alg. 1, Eq. 1) and screened (phase 1)/sec, 1 GPU",
           "value": chunk * len(starts) / elapsed, "unit": "plans/s", "n_gpus": 1, "steps": len(starts),
           "warmup": args.warmup, "ms_per_step": elapsed * 1e3 / len(starts), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic",
           "config": {"workload": "%s plan space: %d logical plans, %d physical plans on %d GPUs; %d plans per "
                                  "launch at %d evenly spaced starts" % (args.config, len(logical), total, N,
                                                                         chunk, len(starts)),
                      "logical_plans": int(len(logical)), "physical_plans": total, "logical_host_s": t_logical,
                      "enum_ms": enum_ms, "coarse_ms": coarse_ms, "enum_plans_per_s": chunk / e_s,
                      "enum_coarse_plans_per_s": chunk / ((sum(enum_ms) + sum(coarse_ms)) / len(enum_ms) / 1e3),
                      "fused_ms": fused_ms, "fused_plans_per_s": chunk / (sum(fused_ms) / len(fused_ms) / 1e3),
                      "screen_topk": {"first": 0, "plans": span, "window": win, "k": 1000,
                                      "kept_in_top": int(top_gid.numel()),
                                      "ms": topk_s * 1e3, "plans_per_s": span / topk_s}},
           "roofline": {"bound": "hbm", "achieved": achieved / 1e9, "peak": 8000.0, "unit": "GB/s",
                        "frac": achieved / 8.0e12,
                        "traffic": ENUM_MEASURED_TRAFFIC.get((kernel_source_id(ENUM_KERNEL_SOURCES), chunk)),
                        "kernel": "k_enum_unrank",
                        "alg_bytes_per_plan": ENUM_PLAN_BYTES, "kernel_ms": sum(enum_ms) / len(enum_ms)}}
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        m, oo = O.make_model(mc), O.enum_opts(mc, spec, N)
        Ls = O.enum_logical(m, oo)
        done, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_budget and done < 4 * chunk:
            O.enum_plans(m, oo, Ls, starts[0] + done, 200000)
            done += 200000
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": done / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
                               "sample": "%d consecutive plans from the first start, single thread, %.1f s "
                                         "(enumeration only)" % (done, dt)}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=-1,
                    help="timed steps (default: 1 for the whole c4 workload, whose step is one seed of the fine "
                         "stage, ~40 s; else 2)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="c4")
    ap.add_argument("--slices", type=int, default=-1, metavar="F",
                    help="each step simulates one slice of the fine stage: every F-th selected plan (all "
                         "grid rates) on one seed, step g taking plan slice g %% F of seed g // F (default: 1 "
                         "for the whole c4 workload, i.e. every selected plan on one seed per step, else none: "
                         "every plan on every seed per step)")
    ap.add_argument("--seeds", type=int, default=0, metavar="N",
                    help="simulate only the first N seeds of the workload (a sample of a workload "
                         "too large to run whole; stated in the output)")
    ap.add_argument("--plans", type=int, default=0, metavar="N",
                    help="simulate only the first N plans phase 1 selects (a sample of a workload too "
                         "large to run whole; stated in the output)")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-workers", type=int, default=min(16, os.cpu_count() or 1), metavar="N",
                    help="processes for the all-cores oracle line of the CPU baseline (<= 1: none)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (the reference "
                         "reading for the HBM byte counters), then exit")
    ap.add_argument("--stress", type=int, default=0, metavar="REPS",
                    help="only time the HBM-bound steps at full size: trace generation of the c4 trace "
                         "and screening of the c4 plans tiled REPS times, then exit")
    ap.add_argument("--phase2", action="store_true",
                    help="only time phase 2 (Monte Carlo latency) and Pareto pruning over the plans "
                         "phase 1 keeps (default workload c4), then exit")
    ap.add_argument("--curve", type=int, default=0, metavar="BINS",
                    help="also emit phase-3 latency histograms over BINS latency-target scales (0.25x to 4x "
                         "each type's bounds, log-spaced) and reduce them to goodput at every target")
    ap.add_argument("--bisect", action="store_true",
                    help="phase 3 bisects each plan's rate over its grid (ceil(log2(K+1)) rates simulated per "
                         "plan and seed) instead of simulating every grid rate")
    ap.add_argument("--enum", action="store_true",
                    help="only time plan enumeration on the device and phase-1 screening of the enumerated "
                         "table (default model: c2's omni graph on 16 GPUs), then exit")
    ap.add_argument("--enum-chunk", type=int, default=1 << 25, metavar="PLANS")
    ap.add_argument("--mc-samples", type=int, default=1024, metavar="K")
    ap.add_argument("--mc-alpha", type=float, default=0.8)
    args = ap.parse_args()
    if args.steps < 0 and (args.enum or args.phase2 or args.stress > 0):
        args.steps = 2
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (triples are "
              "independent; they would shard by contiguous blocks of the selected plans)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_probe > 0:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "launches": 3}), flush=True)
        return

    if args.enum:
        torch.cuda.set_device(0)
        if "--config" not in sys.argv:
            args.config = "c2"
        enum_bench(args)
        return

    if args.phase2:
        torch.cuda.set_device(0)
        if args.config == "c1" and "--config" not in sys.argv:
            args.config = "c4"
        phase2_bench(args)
        return

    if args.stress > 0:
        torch.cuda.set_device(0)
        stress(args.stress, max(1, args.steps))
        return

    from paper_2512_14098_amd import cf, pipeline

    torch.cuda.set_device(0)
    print("bench: loading workload %s" % args.config, file=sys.stderr, flush=True)
    from paper_2512_14098_amd.inputs import load_config, seeds_of
    cfg = load_config(args.config)
    all_seeds = seeds_of(cfg)
    seeds = all_seeds[: args.seeds] if args.seeds > 0 else all_seeds
    w = pipeline.Workload(cfg, seeds=seeds)
    full_top = w.top_k
    w.bisect = bool(args.bisect)
    if args.curve > 0:
        w.set_target_scales([0.25 * 16.0 ** (b / max(args.curve - 1, 1)) for b in range(args.curve)])
    if args.plans > 0:
        w.top_k = min(w.top_k, args.plans)
    F = args.slices
    if F < 0:
        # c4 whole: one seed per step.  A launch of one seed's 32,000 triples keeps ~8 triples in turn on
        # each resident wavefront; thinner slices end on their longest triple (~17 s) while the rest idle
        F = 1 if (args.config == "c4" and args.seeds == 0 and args.plans == 0 and not args.bisect) else 0
    if args.steps < 0:
        args.steps = 1 if F > 0 else 2
    S = len(w.seeds)

    def set_slice(g):
        if F > 0:
            w.slice = (g % F, F, (g // F) % S)
    for i in range(args.warmup):
        set_slice(i)
        out = pipeline.run_step(w)
        torch.cuda.synchronize()
        print("bench: warmup %d done, %d request-events" % (i, pipeline.events_total(out)),
              file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    events, plans, fine_ms, timers_all, ev_tensors, st_tensors = 0, 0, [], [], [], []
    fine_plans = []
    t0 = time.perf_counter()
    for i in range(args.steps):
        set_slice(args.warmup + i)
        timers = {}
        out = pipeline.run_step(w, timers=timers)
        timers_all.append(timers)
        ev_tensors.append(out["fine"]["events"])
        st_tensors.append(out["fine"]["status"])
        fine_plans.append(int(out["fine_ids"].numel()))
        if i == 0 or (i + 1) % 5 == 0:
            print("bench: step %d launched" % i, file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stage_ms = {}
    for i, timers in enumerate(timers_all):
        s, e = timers["fine"]
        fine_ms.append(s.elapsed_time(e))
        for k, (s, e) in timers.items():
            stage_ms.setdefault(k, []).append(s.elapsed_time(e))
    events = sum(int(e.sum().item()) for e in ev_tensors)
    st = {}
    for t in st_tensors:
        for k, v in pipeline.status_summary({"fine": {"status": t}}).items():
            st[k] = st.get(k, 0) + v
    # plans fully evaluated (every rate on every seed): a sliced step does 1/S of that for its plans
    plans = sum(fine_plans) / (S if F > 0 else 1)
    elapsed = t1 - t0
    ms_per_step = elapsed * 1e3 / args.steps
    ev_step = events / args.steps
    fine_avg_s = sum(fine_ms) / len(fine_ms) / 1e3
    achieved = OPS_PER_EVENT * ev_step / fine_avg_s / 1e12
    n_sel = int(out["ids"].numel())
    workload = "%s: %s" % (args.config, w.cfg["summary"])
    if F == 1:
        workload += ("; each step: the trace of all %d seeds, phase 1 over all %d plans, the top %d and their "
                     "%d-rate grid, phase 3 of every selected plan at every rate on one seed (seed g at step g), "
                     "their goodput reduction" % (S, w.tab.P, n_sel, w.K))
    elif F > 0:
        workload += ("; each step: the trace of all %d seeds, phase 1 over all %d plans, the top %d and their "
                     "%d-rate grid, phase 3 of every %d-th selected plan at every rate on one seed (plan slice "
                     "g mod %d of seed g div %d at step g), their goodput reduction"
                     % (S, w.tab.P, n_sel, w.K, F, F, F))
    sample = []
    if args.plans > 0 and w.top_k < full_top:
        sample.append("first %d of its %d selected plans" % (w.top_k, full_top))
    if len(seeds) < len(all_seeds):
        sample.append("first %d of its %d seeds" % (len(seeds), len(all_seeds)))
    if sample:
        workload += " (sample: %s)" % ", ".join(sample)
    if args.curve > 0:
        workload += "; goodput curves over %d latency-target scales" % args.curve
    if args.bisect:
        workload += "; rates bisected over the grid"
    res = {
        "metric": METRIC,
        "value": events / elapsed,
        "unit": "request-events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "plans_per_s": plans / elapsed,
        "config": {"workload": workload, "plans_screened": w.tab.P,
                   "plans_simulated": n_sel, "rates": w.K, "seeds": len(w.seeds), "requests": w.n_req,
                   "triples": (int(out["fine"]["n_eval"].sum().item()) * len(w.seeds) if w.bisect
                               else n_sel * w.K * len(w.seeds)) if F <= 0 else None,
                   "triples_per_step": (sum(fine_plans) * w.K // args.steps) if F > 0 else None,
                   "request_events_per_step": ev_step,
                   "status_counts": st, "fine_ms": fine_ms,
                   "stage_ms": {k: sum(v) / len(v) for k, v in stage_ms.items()},
                   # the whole fine stage (every selected plan, rate and seed) at this step's rate
                   "fine_stage_s_extrapolated": (fine_avg_s * F * S) if F > 0 else fine_avg_s},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_LANE_OPS, "unit": "TOP/s",
                     "frac": achieved / PEAK_LANE_OPS,
                     "traffic": MEASURED_TRAFFIC.get((kernel_source_id(), workload)),
                     # the same kernel's VALU lane rate by the counters (instructions x active
                     # lanes / time) as a fraction of the same peak, for this source and workload
                     "counter_valu_lane_frac": MEASURED_LANE_FRAC.get((kernel_source_id(), workload)),
                     "kernel": "k_fine", "ops_per_event": OPS_PER_EVENT,
                     "kernel_ms": sum(fine_ms) / len(fine_ms)},
    }
    if not args.no_cpu_baseline:
        print("bench: cpu baseline (oracle, %.0f s budget)" % args.cpu_budget, file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget, args.cpu_workers,
                                           res["config"]["request_events_per_step"])
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
