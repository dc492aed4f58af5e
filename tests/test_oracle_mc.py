"""Pins of the oracle's phase 2 (Monte Carlo latency with occupancy-aware
scaling, Sec. 4.3 Alg. 2 phase 2 and Sec. 5.2) and of its Pareto pruning.

Expected values come from outside the Monte Carlo code:

* the request-level simulator at zero load: with every node at batch 1 (so
  every effective batch is 1) and requests so far apart that each one is
  alone in the system, a request's latencies in the simulator are exactly
  its no-queueing latencies, so phase 2 must reproduce them (up to the
  rounding of absolute versus relative times), on plans whose parallel or
  gated work never shares an executor;
* effective batches worked out by hand from phase 1's capacities on a
  two-node plan, read back through an encoder and a generator whose
  iteration time is proportional to the batch size;
* a gated talker timeline worked out by hand;
* G_t = alpha R_d pi_t met_t / cnt_t recomputed from the counts;
* Pareto pruning against a brute-force dominance check written here.
"""
import itertools

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, plan_table_from_list

from .helpers import comp, make_trace, model, rtype


def _plan_one_node_per_comp(n_comp, types_comps, reps=None, colocate=()):
    """Nodes: one per component (batch 1), except groups in colocate that share a node."""
    groups = [list(g) for g in colocate]
    grouped = {c for g in groups for c in g}
    for c in range(n_comp):
        if c not in grouped:
            groups.append([c])
    groups.sort(key=min)
    node_of = {c: v for v, g in enumerate(groups) for c in g}
    reps = reps or {}
    nodes = [(sum(1 << c for c in g), reps.get(v, 1), 1, 1) for v, g in enumerate(groups)]
    routes = [[(10, {c: node_of[c] for c in comps})] for comps in types_comps]
    return dict(nodes=nodes, routes=routes)


@pytest.mark.parametrize("cfgname,colocate,reps", [
    ("c0", (), {}),
    ("c0", ((0, 1),), {}),
    ("c1", (), {0: 2, 1: 3}),
    ("c2", (), {}),
    ("c2", ((0, 2), (3, 4)), {1: 2}),
    ("c3", (), {1: 2}),
])
def test_zero_load_simulator_equals_monte_carlo(cfgname, colocate, reps):
    cfg = load_config(cfgname)
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.0
    m = O.make_model(mc)
    names = [c["name"] for c in mc["components"]]
    tcomps = [[names.index(c) for c in t["comps"]] for t in mc["types"]]
    tab = plan_table_from_list([_plan_one_node_per_comp(len(names), tcomps, reps, colocate)])
    n = 300
    tr = O.trace_gen(m, [5], n)
    # arrivals every 100 s (exact in binary), far apart and of small magnitude: the simulator's
    # absolute times then differ from phase 2's relative ones by at most a few thousand
    # roundings at 2^-38 s
    tr["arr_ticks"] = np.ascontiguousarray(np.arange(n, dtype=np.uint64) * np.uint64(100 << 32))
    des = O.sim_triple(m, tab, 0, 1.0, tr, 0, want_lat=True)
    assert des["status"] == 0
    arr = np.arange(n) * 100.0
    assert np.all(arr[1:] > arr[:-1] + des["lat"][:-1, 2]), "requests overlap: not zero load"
    rd, _, fl = O.eval_coarse(m, tab, tr["moments"][0], 64)
    met, cnt, gt, lat = O.eval_mc(m, tab, [0], rd, tr["moments"][0], 0.8, tr, 0, n, want_lat=True)
    np.testing.assert_allclose(lat[0], des["lat"], rtol=0, atol=1e-7)
    assert int(cnt.sum()) == n
    # the counts agree except for requests within rounding of a target
    if not np.array_equal(met[0], des["met"]):
        slo = np.array([[m.slo[t][j] for j in range(4)] for t in range(m.n_types)])
        near = np.abs(des["lat"] - slo[tr["type"][:n]]) <= 1e-9 * np.maximum(1.0, np.abs(des["lat"]))
        assert near.any()


def _two_node_model():
    return model([comp("E", "ENC", [0.0, 0.0, 0.001], x=["patches"]),
                  comp("G", "GEN", [0.0, 0.0, 0.002], x=["aud_out_ms"])],
                 [rtype("t", ["E", "G"], edges=[("E", "G")], outputs=["G"], slo={"e2e": 10.0})],
                 comm=0.010)


@pytest.mark.parametrize("rep_g,b_e,b_g", [(1, 4, 8), (2, 8, 8), (3, 8, 6)])
def test_effective_batch_by_hand(rep_g, b_e, b_g):
    # per request: E takes k2 = 1 ms of executor time at any batch, G 2 ms, so
    # R_E = 1000 req/s, R_G = rep_g * 500 req/s; R_d = min; b = ceil(8 R_d / R_v)
    m = O.make_model(_two_node_model())
    tab = plan_table_from_list([dict(nodes=[(1, 1, 8, 1), (2, rep_g, 8, 1)], routes=[[(10, {0: 0, 1: 1})]])])
    tr = make_trace([dict(t=0.0, patches=100, aud_out_ms=500)])
    tr["moments"] = np.array([[[1, 0, 0, 100, 0, 500, 0, 0]]], np.uint64)
    rd, bn, fl = O.eval_coarse(m, tab, tr["moments"][0], 64)
    assert rd[0] == pytest.approx(min(1000.0, rep_g * 500.0), rel=1e-12)
    met, cnt, gt, lat = O.eval_mc(m, tab, [0], rd, tr["moments"][0], 1.0, tr, 0, 1, want_lat=True)
    e_end = 0.0 + ((0.0 + 0.0 * float(b_e * 100)) + 0.001 * float(b_e))
    g_end = (e_end + 0.010) + ((0.0 + 0.0 * float(b_g * 500)) + 0.002 * float(b_g))
    assert lat[0, 0, 2] == g_end
    assert lat[0, 0, 3] == g_end  # GEN output: media time
    assert met[0, 0] == 1 and cnt[0, 0] == 1
    assert gt[0, 0] == (1.0 * rd[0]) * 1.0


def test_gated_talker_timeline_by_hand():
    # thinker: prefill 10 ms, 3 tokens, decode steps of 20 ms; talker on another
    # executor (comm 5 ms): prefill 1 ms, 5 tokens, steps of 2 ms
    mc = model([comp("T", "LLM", [0.010, 0.0, 0.0], decode=(0.020, 0.0), n_out="out"),
                comp("A", "LLM", [0.001, 0.0, 0.0], decode=(0.002, 0.0), n_out="aud_out_tok", gate="T")],
               [rtype("t", ["T", "A"], edges=[("T", "A")], outputs=["T", "A"], slo={})], comm=0.005)
    m = O.make_model(mc)
    tab = plan_table_from_list([dict(nodes=[(1, 1, 1, 1), (2, 1, 1, 1)], routes=[[(10, {0: 0, 1: 1})]])])
    tr = make_trace([dict(t=0.0, out=3, aud_out_ms=400)])  # talker tokens ceil(400/80) = 5
    tr["moments"] = np.array([[[1, 0, 3, 0, 0, 400, 0, 5]]], np.uint64)
    rd, _, _ = O.eval_coarse(m, tab, tr["moments"][0], 64)
    met, cnt, gt, lat = O.eval_mc(m, tab, [0], rd, tr["moments"][0], 1.0, tr, 0, 1, want_lat=True)
    th = [0.0 + 0.010]
    for _ in range(2):
        th.append(th[-1] + 0.020)                     # thinker tokens at 10, 30, 50 ms
    vis = [e + 0.005 for e in th]                     # visible at the talker 5 ms later
    ta = [vis[0] + 0.001]                             # talker prefill after token 1 arrives
    for k in range(1, 5):                             # token k+1 needs thinker token min(k+1, 3)
        ta.append(max(ta[-1], vis[min(k + 1, 3) - 1]) + 0.002)
    assert lat[0, 0, 0] == th[0]                      # TTFT: the thinker's first token
    assert lat[0, 0, 1] == (th[2] - th[0]) / 2.0
    assert lat[0, 0, 2] == max(th[2], ta[-1])


def test_goodput_formula_and_conservation():
    cfg = load_config("c2")
    m = O.make_model(cfg["model"])
    from paper_2512_14098_amd.inputs import make_plans
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [1], 700)
    rd, _, fl = O.eval_coarse(m, tab, tr["moments"][0], cfg["gpus"])
    ids = O.select_topk(rd, fl, 40)
    alpha = 0.7
    met, cnt, gt = O.eval_mc(m, tab, ids, rd, tr["moments"][0], alpha, tr, 0, 512)
    w = np.array([t["weight"] for t in cfg["model"]["types"]], np.float64)
    pi = w / w.sum()
    types = np.bincount(tr["type"][:512], minlength=m.n_types)
    for i, p in enumerate(ids):
        assert np.array_equal(cnt[i], types)
        assert np.all(met[i] <= cnt[i])
        for t in range(m.n_types):
            want = ((alpha * rd[p]) * (float(cfg["model"]["types"][t]["weight"]) / w.sum())) * (met[i, t] / cnt[i, t])
            assert gt[i, t] == want
        assert np.allclose(gt[i], alpha * rd[p] * pi * met[i] / cnt[i], rtol=1e-15)


def _dominated_brute(g, i):
    return any(np.all(g[j] >= g[i]) and np.any(g[j] > g[i]) for j in range(len(g)) if j != i)


@pytest.mark.parametrize("seed", range(6))
def test_pareto_against_brute_force(seed):
    rng = np.random.default_rng(seed)
    n, T = int(rng.integers(1, 60)), int(rng.integers(1, 5))
    g = rng.integers(0, 4, size=(n, T)).astype(np.float64)  # many ties and duplicates
    keep = O.pareto(g)
    for i in range(n):
        assert keep[i] == (0 if _dominated_brute(g, i) else 1)
    # the kept set is mutually non-dominated, and every pruned vector is dominated by a kept one
    kept = np.flatnonzero(keep)
    for i, j in itertools.permutations(kept, 2):
        assert not (np.all(g[j] >= g[i]) and np.any(g[j] > g[i]))
    for i in np.flatnonzero(keep == 0):
        assert any(np.all(g[j] >= g[i]) and np.any(g[j] > g[i]) for j in kept)
