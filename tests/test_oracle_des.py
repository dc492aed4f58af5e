"""Pins of the oracle's request-level simulator (Sec. 4.3, Alg. 2 phase 3).

Every expected value here comes from somewhere other than the oracle:

* micro-scenarios whose timelines are worked out by hand from the stated
  scheduling rules, in exact rational arithmetic on the double-valued
  coefficients (prefill priority and iteration-level batching, a prefill
  interrupting a decode run, CPU-GPU overlap of an encoder that starts idle
  or busy (Sec. 5.2), the communication delay on a disaggregated edge
  (Sec. 5.2), fork-join of two encoders, and thinker -> talker gating);
* queueing closed forms: Pollaczek-Khinchine mean sojourn of an M/G/1
  queue, with M/M/1 and M/D/1 as special cases, for a batch-1 encoder and
  for a batch-1 prefill-only LLM;
* the sample-path Little identity (time integral of the number in system
  equals the sum of sojourn times);
* zero-load latencies computed by a separate walk of the request's path;
* conservation: every request completes and the request-event count equals
  its closed form over the trace (it cannot depend on timing);
* exact invariance of all outcomes under scaling of time by a power of two
  (with compute-proportional targets this is Theorem 1 of Appendix A).
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans

from .helpers import F, comp, make_trace, model, one_plan, rtype, ticks_of

REL = 1e-12


def run(mcfg, plan, reqs, rate=1.0):
    m = O.make_model(mcfg)
    tr = make_trace(reqs)
    return O.sim_triple(m, plan, 0, rate, tr, 0, want_lat=True, want_diag=True)


def close(got, exact):
    exact = float(exact)
    assert got == pytest.approx(exact, rel=REL, abs=1e-15), (got, exact)


LLM_A = dict(k=[0.005, 2e-5, 0.0], decode=(0.008, 5e-5))


def llm_model(batch_cap=256):
    return model([comp("L", "LLM", LLM_A["k"], x=["prompt"], decode=LLM_A["decode"],
                       batch_cap=batch_cap)],
                 [rtype("t", ["L"], slo={"ttft": 10.0})])


def test_ms1_prefill_priority_and_continuous_batching():
    p0, p1, d0, d1 = F(0.005), F(2e-5), F(0.008), F(5e-5)
    plan = one_plan([(1, 1, 2)], [[(10, {0: 0})]])
    reqs = [dict(t=0.0, prompt=100, out=3), dict(t=0.001, prompt=100, out=2)]
    o = run(llm_model(), plan, reqs)
    aB = ticks_of(0.001)[1]
    e1 = p0 + p1 * 100                # prefill A
    e2 = e1 + (p0 + p1 * 100)         # B waits; prefill B (|Run| = 1 < 2)
    e3 = e2 + (d0 + d1 * 2)           # decode {A, B}; B reaches 2 tokens
    e4 = e3 + (d0 + d1 * 1)           # decode {A}; A reaches 3 tokens
    lat = o["lat"]
    close(lat[0, 0], e1); close(lat[0, 1], (e4 - e1) / 2); close(lat[0, 2], e4)
    close(lat[1, 0], e2 - aB); close(lat[1, 1], e3 - e2); close(lat[1, 2], e3 - aB)
    assert o["events"] == 6 + 5
    assert o["status"] == 0 and o["cnt"][0] == 2


def test_ms2_prefill_interrupts_decode():
    p0, p1, d0, d1 = F(0.005), F(2e-5), F(0.008), F(5e-5)
    plan = one_plan([(1, 1, 4)], [[(10, {0: 0})]])
    reqs = [dict(t=0.0, prompt=100, out=3), dict(t=0.010, prompt=50, out=2)]
    o = run(llm_model(), plan, reqs)
    aB = ticks_of(0.010)[1]
    e1 = p0 + p1 * 100            # prefill A
    e2 = e1 + (d0 + d1)           # decode {A}; B arrived meanwhile
    e3 = e2 + (p0 + p1 * 50)      # prefill B before A's next decode
    e4 = e3 + (d0 + d1 * 2)       # decode {A, B}: both finish
    lat = o["lat"]
    close(lat[0, 1], (e4 - e1) / 2)   # A's TPOT includes B's prefill
    close(lat[0, 2], e4)
    close(lat[1, 0], e3 - aB); close(lat[1, 1], e4 - e3)
    assert o["events"] == 6 + 5


def test_ms3_cpu_preprocessing_only_when_idle():
    mc = model([comp("E", "ENC", [0.002, 1e-5, 0.0], x=["patches"])],
               [rtype("i", ["E"], images={"const": 1})], cpu_pre=0.003)
    plan = one_plan([(1, 1, 1)], [[(10, {0: 0})]])
    reqs = [dict(t=0.0, patches=300), dict(t=0.001, patches=500), dict(t=0.1, patches=400)]
    o = run(mc, plan, reqs)
    a, b, cpu = F(0.002), F(1e-5), F(0.003)
    eA = ((a + b * 300) + 0) + cpu       # idle start: CPU + GPU time
    eB = eA + ((a + b * 500) + 0)        # queued while busy: GPU time only
    aC = ticks_of(0.1)[1]
    eC = aC + (((a + b * 400) + 0) + cpu)
    lat = o["lat"]
    close(lat[0, 2], eA); close(lat[1, 2], eB - ticks_of(0.001)[1]); close(lat[2, 2], eC - aC)
    assert o["events"] == 3 * 4


def _enc_llm_model():
    return model([comp("E", "ENC", [0.002, 1e-5, 0.0], x=["patches"]),
                  comp("L", "LLM", [0.005, 2e-5, 0.0], x=["prompt", "patches", "aud_in_tok"],
                       decode=(0.008, 5e-5))],
                 [rtype("img", ["E", "L"], edges=[("E", "L")], images={"const": 1})])


def test_ms4_comm_delay_on_disaggregated_edge():
    reqs = [dict(t=0.0, patches=400, prompt=100, out=2)]
    a, b, p0, p1, d0, d1, comm = F(0.002), F(1e-5), F(0.005), F(2e-5), F(0.008), F(5e-5), F(0.010)
    eE = (a + b * 400) + 0
    # disaggregated: E and L on separate executors
    o = run(_enc_llm_model(), one_plan([(1, 1, 8), (2, 1, 8)], [[(10, {0: 0, 1: 1})]]), reqs)
    eP = (eE + comm) + (p0 + p1 * 500)
    eD = eP + (d0 + d1)
    close(o["lat"][0, 0], eP); close(o["lat"][0, 1], eD - eP); close(o["lat"][0, 2], eD)
    assert o["events"] == 7
    # colocated: no communication delay
    o = run(_enc_llm_model(), one_plan([(3, 1, 8)], [[(10, {0: 0, 1: 0})]]), reqs)
    close(o["lat"][0, 0], eE + (p0 + p1 * 500))


def _fork_model():
    return model([comp("Ei", "ENC", [0.002, 1e-5, 0.0], x=["patches"]),
                  comp("Ea", "ENC", [0.002, 1e-6, 0.0], x=["aud_in_ms"]),
                  comp("L", "LLM", [0.005, 2e-5, 0.0], x=["prompt", "patches", "aud_in_tok"],
                       decode=(0.008, 5e-5))],
                 [rtype("ia", ["Ei", "Ea", "L"], edges=[("Ei", "L"), ("Ea", "L")],
                        images={"const": 1}, aud_in={"const": 2000})])


def test_ms5_fork_join():
    reqs = [dict(t=0.0, patches=300, aud_in_ms=2000, prompt=100, out=2)]
    comm, p0, p1 = F(0.010), F(0.005), F(2e-5)
    eI = (F(0.002) + F(1e-5) * 300) + 0
    eA = (F(0.002) + F(1e-6) * 2000) + 0
    X = 100 + 300 + 25  # prompt + patches + ceil(2000 / 80) audio tokens
    # three executors: L starts after the later of the two deliveries
    o = run(_fork_model(), one_plan([(1, 1, 8), (2, 1, 8), (4, 1, 8)], [[(10, {0: 0, 1: 1, 2: 2})]]),
            reqs)
    close(o["lat"][0, 0], max(eI + comm, eA + comm) + (p0 + p1 * X))
    assert o["events"] == 1 + 2 + 2 + 3 + 1
    # both encoders on one executor run one after the other (stage order)
    o = run(_fork_model(), one_plan([(3, 1, 8), (4, 1, 8)], [[(10, {0: 0, 1: 0, 2: 1})]]), reqs)
    eA2 = eI + ((F(0.002) + F(1e-6) * 2000) + 0)
    close(o["lat"][0, 0], (eA2 + comm) + (p0 + p1 * X))


def _gate_model():
    return model([comp("Th", "LLM", [0.005, 2e-5, 0.0], x=["prompt"], decode=(0.020, 0.0)),
                  comp("Ta", "LLM", [0.003, 1e-5, 0.0], x=["prompt"], decode=(0.006, 0.0),
                       n_out="aud_out_tok", gate="Th")],
                 [rtype("a", ["Th", "Ta"], edges=[("Th", "Ta")], outputs=["Th", "Ta"],
                        aud_out={"const": 240})])


def test_ms6_talker_gated_by_thinker_tokens():
    reqs = [dict(t=0.0, prompt=100, out=4, aud_out_ms=240)]  # 3 talker tokens
    comm = F(0.010)
    thp = (F(0.005) + F(2e-5) * 100) + 0
    tap = (F(0.003) + F(1e-5) * 100) + 0
    thd, tad = F(0.020) + 0, F(0.006) + 0
    # disaggregated: the talker waits for thinker tokens to become visible
    o = run(_gate_model(), one_plan([(1, 1, 8), (2, 1, 8)], [[(10, {0: 0, 1: 1})]]), reqs)
    e1 = thp
    e2, e3, e4 = e1 + thd, e1 + thd + thd, e1 + thd + thd + thd
    ta1 = (e1 + comm) + tap              # delivered when token 1 is visible
    ta2 = (e2 + comm) + tad              # token 2 visible at e2 + comm
    ta3 = (e3 + comm) + tad              # token 3 visible at e3 + comm
    assert ta1 < e2 + comm and ta3 < e4
    close(o["lat"][0, 0], e1); close(o["lat"][0, 2], e4); close(o["lat"][0, 1], (e4 - e1) / 3)
    assert o["events"] == 1 + (1 + 1 + 3) + (1 + 1 + 2) + 1
    # colocated: one executor alternates thinker and talker iterations
    o = run(_gate_model(), one_plan([(3, 1, 8)], [[(10, {0: 0, 1: 0})]]), reqs)
    t1 = thp
    t2 = t1 + tap      # talker prefill
    t3 = t2 + thd      # thinker token 2
    t4 = t3 + tad      # talker token 2 (thinker token 2 visible at once)
    t5 = t4 + thd      # thinker token 3
    t6 = t5 + tad      # talker token 3: talker done
    t7 = t6 + thd      # thinker token 4: done
    close(o["lat"][0, 2], t7); close(o["lat"][0, 1], (t7 - t1) / 3)


# ------------------------------------------------------------------ closed forms
def _mg1(mc, plan, rate, seeds, n):
    m = O.make_model(mc)
    tr = O.trace_gen(m, seeds, n)
    means, s1, s2 = [], [], []
    for s in range(len(seeds)):
        o = O.sim_triple(m, plan, 0, rate, tr, s, want_lat=True)
        assert o["status"] == 0
        means.append(o["lat"][:, 2].mean())
    return np.array(means), tr


def _enc_queue(dist):
    return model([comp("S", "ENC", [0.0, 1e-3, 0.0], x=["aud_in_ms"])],
                 [rtype("a", ["S"], aud_in=dist)])


@pytest.mark.parametrize("rho,dist", [(0.3, {"exp": 1000}), (0.6, {"exp": 1000}), (0.9, {"exp": 1000}),
                                      (0.6, {"const": 1000}), (0.9, {"const": 1000}),
                                      (0.5, {"lognormal_s": [0.0, 0.5]})])
def test_mg1_pollaczek_khinchine(rho, dist):
    plan = one_plan([(1, 1, 1)], [[(10, {0: 0})]])
    # near saturation the sample mean converges slowly: more and longer seeds
    seeds, n = (list(range(32)), 50000) if rho > 0.8 else (list(range(16)), 20000)
    mc = _enc_queue(dist)
    m = O.make_model(mc)
    tr = O.trace_gen(m, seeds, n)
    S = tr["aud_in_ms"].astype(np.float64) * 1e-3
    ES, ES2 = S.mean(), (S * S).mean()
    lam = rho / ES
    W = ES + lam * ES2 / (2 * (1 - lam * ES))
    per_seed = np.array([O.sim_triple(m, plan, 0, lam, tr, s, want_lat=True)["lat"][:, 2].mean()
                         for s in range(len(seeds))])
    se = per_seed.std(ddof=1) / np.sqrt(len(seeds))
    assert abs(per_seed.mean() - W) < 4 * se + 0.01 * W, (per_seed.mean(), W, se)


def test_mm1_sojourn_is_exponential():
    """M/M/1 sojourn time is Exp(mu - lambda): check a few quantiles."""
    plan = one_plan([(1, 1, 1)], [[(10, {0: 0})]])
    m = O.make_model(_enc_queue({"exp": 1000}))
    tr = O.trace_gen(m, list(range(8)), 20000)
    lam = 0.5
    soj = np.concatenate([O.sim_triple(m, plan, 0, lam, tr, s, want_lat=True)["lat"][:, 2]
                          for s in range(8)])
    for q in (0.25, 0.5, 0.9):
        x = -np.log(1 - q) / (1.0 - lam)
        assert abs((soj <= x).mean() - q) < 0.02


def test_llm_batch1_prefill_only_is_mg1():
    mc = model([comp("L", "LLM", [0.1, 1e-3, 0.0], x=["prompt"], decode=(0.0, 0.0))],
               [rtype("t", ["L"], prefill_only=["L"], prompt={"lognormal": [6.0, 0.5]})])
    plan = one_plan([(1, 1, 1)], [[(10, {0: 0})]])
    m = O.make_model(mc)
    seeds, n = list(range(12)), 20000
    tr = O.trace_gen(m, seeds, n)
    S = 0.1 + 1e-3 * tr["prompt"].astype(np.float64)
    ES, ES2 = S.mean(), (S * S).mean()
    lam = 0.5 / ES
    W = ES + lam * ES2 / (2 * (1 - lam * ES))
    per_seed = np.array([O.sim_triple(m, plan, 0, lam, tr, s, want_lat=True)["lat"][:, 2].mean()
                         for s in range(len(seeds))])
    se = per_seed.std(ddof=1) / np.sqrt(len(seeds))
    assert abs(per_seed.mean() - W) < 4 * se + 0.01 * W


# ------------------------------------------------------------------ invariants
@pytest.fixture(scope="module")
def c2_setup():
    cfg = load_config("c2")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [0, 1], 2000)
    return cfg, m, tab, tr


def _event_formula(cfg, m, tr, s):
    """Request-event count from the trace alone: 1 arrival, per component 1 enqueue
    plus 1 (ENC/GEN batch) or n_out (LLM prefill + decodes), 1 completion."""
    comps = cfg["model"]["components"]
    names = [c["name"] for c in comps]
    attr = {"out": tr["out"], "aud_out_tok": (tr["aud_out_ms"].astype(np.int64) + 79) // 80}
    n = tr["n_req"]
    total = 0
    for i in range(s * n, (s + 1) * n):
        ty = cfg["model"]["types"][tr["type"][i]]
        total += 2
        for cname in ty["comps"]:
            c = comps[names.index(cname)]
            if c["kind"] == "LLM":
                if cname in ty.get("prefill_only", []):
                    k = 1
                else:
                    k = max(1, int(attr[c.get("n_out", "out")][i]))
                total += 1 + k
            else:
                total += 2
    return total


def test_conservation_and_event_count(c2_setup):
    cfg, m, tab, tr = c2_setup
    rng = np.random.default_rng(3)
    for p in rng.choice(tab.P, 12, replace=False):
        for rate in (2.0, 20.0, 200.0):
            for s in (0, 1):
                o = O.sim_triple(m, tab, int(p), rate, tr, s)
                assert o["status"] == 0
                assert o["cnt"].sum() == tr["n_req"]
                assert o["events"] == _event_formula(cfg, m, tr, s)
                assert np.all(o["met"] <= o["cnt"])


def test_little_identity(c2_setup):
    cfg, m, tab, tr = c2_setup
    for p in (0, 1, 2, 3):
        o = O.sim_triple(m, tab, p, 50.0, tr, 0, want_lat=True, want_diag=True)
        area = o["diag"][0]
        assert area == pytest.approx(o["lat"][:, 2].sum(), rel=1e-9)


def _scaled_model(mcfg, f):
    import copy
    mc = copy.deepcopy(mcfg)
    for c in mc["components"]:
        c["k"] = [v * f for v in c["k"]]
        if "decode" in c:
            c["decode"] = [v * f for v in c["decode"]]
    mc["comm_s"] *= f
    mc["cpu_pre_s"] = mc.get("cpu_pre_s", 0.0) * f
    for t in mc["types"]:
        t["slo"] = {k: v * f for k, v in t.get("slo", {}).items()}
    return mc


@pytest.mark.parametrize("cfgname", ["c1", "c2", "c3"])
def test_time_scaling_by_power_of_two(cfgname):
    """Scaling every duration, delay and target by 2^k and every rate by 2^-k
    maps each sample path onto itself: counts are identical and latencies
    scale exactly (Theorem 1's scale invariance, with exact arithmetic)."""
    cfg = load_config(cfgname)
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.003
    m1 = O.make_model(mc)
    m8 = O.make_model(_scaled_model(mc, 8.0))
    tab = make_plans(cfg)
    tr = O.trace_gen(m1, [4], 1500)
    for p in (0, tab.P // 2, tab.P - 1):
        for rate in (5.0, 40.0):
            a = O.sim_triple(m1, tab, p, rate, tr, 0, want_lat=True)
            b = O.sim_triple(m8, tab, p, rate / 8.0, tr, 0, want_lat=True)
            assert np.array_equal(a["met"], b["met"]) and a["events"] == b["events"]
            assert np.array_equal(a["lat"] * 8.0, b["lat"])


def _walk_zero_load(mcfg, tab, p, tr, i, rate):
    """Latency of request i alone in the system, by walking its path."""
    comps = mcfg["components"]
    ty = mcfg["types"][tr["type"][i]]
    names = [c["name"] for c in comps]
    comm, cpu = mcfg["comm_s"], mcfg.get("cpu_pre_s", 0.0)
    t_idx = int(tr["type"][i])
    node = {names.index(c): int(tab.alt_node[(2 * t_idx) * 8 + names.index(c), p]) for c in ty["comps"]}
    parents = {names.index(b): [] for b in ty["comps"]}
    for a, b in ty.get("edges", []):
        parents[names.index(b)].append(names.index(a))
    a_r = (float(tr["arr_ticks"][i]) * 2.0 ** -32) / rate
    vals = {"prompt": int(tr["prompt"][i]), "out": int(tr["out"][i]), "patches": int(tr["patches"][i]),
            "aud_in_ms": int(tr["aud_in_ms"][i]), "aud_out_ms": int(tr["aud_out_ms"][i]),
            "aud_in_tok": (int(tr["aud_in_ms"][i]) + 79) // 80,
            "aud_out_tok": (int(tr["aud_out_ms"][i]) + 79) // 80}
    done, free = {}, {}
    t_first = t_last = None
    nfirst = None
    for c in sorted(node):
        cd = comps[c]
        ready = a_r if not parents[c] else max(
            done[q] + (comm if node[q] != node[c] else 0.0) for q in parents[c])
        start = max(ready, free.get(node[c], -1.0))
        X = float(sum(vals[k] for k in cd.get("x", [])))
        k0, k1, k2 = cd["k"]
        dur = (k0 + k1 * X) + k2 * 1.0
        if cd["kind"] == "ENC" and free.get(node[c], -1.0) < start:
            dur = dur + cpu
        t = start + dur
        if cd["kind"] == "LLM":
            nout = 1 if cd["name"] in ty.get("prefill_only", []) else max(1, vals[cd.get("n_out", "out")])
            if t_first is None:
                t_first, nfirst = t, nout
            d0, d1 = cd.get("decode", [0.0, 0.0])
            for _ in range(nout - 1):
                t = t + (d0 + d1 * 1.0)
            if nfirst is not None and t_last is None:
                t_last = t
        done[c] = t
        free[node[c]] = t
    outs = [names.index(c) for c in ty["outputs"]]
    e2e = max(done[c] for c in outs) - a_r
    ttft = t_first - a_r if t_first is not None else 0.0
    tpot = (t_last - t_first) / (nfirst - 1) if nfirst and nfirst > 1 else 0.0
    return ttft, tpot, e2e


@pytest.mark.parametrize("cfgname", ["c0", "c1", "c3"])
def test_zero_load_latency_is_sum_along_path(cfgname):
    cfg = load_config(cfgname)
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.003
    m = O.make_model(mc)
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [2], 60)
    rate = 1e-6
    single = [p for p in range(tab.P) if all(tab.n_alt[t, p] == 1 for t in range(m.n_types))]
    for p in single[:: max(1, len(single) // 6)]:
        o = O.sim_triple(m, tab, p, rate, tr, 0, want_lat=True)
        for i in range(tr["n_req"]):
            exp = _walk_zero_load(mc, tab, p, tr, i, rate)
            for j in range(3):
                assert o["lat"][i, j] == pytest.approx(exp[j], rel=1e-12, abs=1e-12), (p, i, j)


def test_invalid_route_is_reported():
    plan = one_plan([(1, 1, 8)], [[(10, {0: 0, 1: 0})]])  # node 0 does not host L
    mc = _enc_llm_model()
    o = run(mc, plan, [dict(t=0.0, patches=300, prompt=10, out=2)])
    assert o["status"] & O.ST_INVALID


def test_golden_fixtures():
    """Fixtures under tests/golden: scenarios worked by hand, stored as decimals."""
    import glob
    import json
    import os
    files = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.json")))
    assert files
    for fn in files:
        with open(fn) as f:
            g = json.load(f)
        md = g["model"]
        mcfg = model([comp("L", "LLM", [md["p0"], md["p1"], 0.0], x=["prompt"], decode=(md["d0"], md["d1"]),
                           batch_cap=256)], [rtype("t", ["L"], slo={"ttft": 10.0})])
        plan = one_plan([(1, 1, md["batch"])], [[(10, {0: 0})]])
        o = run(mcfg, plan, g["requests"])
        lat = o["lat"]
        for j, key in enumerate(("ttft", "tpot", "e2e")):
            np.testing.assert_allclose(lat[:, j], g["expect"][key], rtol=g["rel_tol"], atol=0, err_msg=fn)
        assert o["events"] == g["expect"]["request_events"], fn
