"""Pins of the oracle's phase 1 (flow-based throughput, Sec. 4.3, Alg. 2),
top-K selection, rate grid and goodput reduction.

* R_d must be the aggregate rate that saturates the bottleneck: a plan driven
  far above capacity by the simulator completes requests at exactly R_d when
  the per-request work of the latency model does not depend on load (batch 1),
  and close to it otherwise.
* Structural invariants: replicas scale capacity, the budget of Eq. (1).
* Selection and reduction against independent brute force (numpy lexsort,
  bisection on the feasibility predicate).
* The c0 plan set equals an independent itertools enumeration.
"""
import itertools

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans

from .helpers import comp, model, one_plan, rtype


def _saturated_rate(mc, plan, n=6000, seed=0):
    m = O.make_model(mc)
    tr = O.trace_gen(m, [seed], n)
    rd, bn, fl = O.eval_coarse(m, plan, tr["moments"][0], 64)
    o = O.sim_triple(m, plan, 0, 1000.0 * rd[0], tr, 0, want_diag=True)
    a0 = (float(tr["arr_ticks"][0]) * 2.0 ** -32) / (1000.0 * rd[0])
    return rd[0], n / (o["diag"][1] - a0)


def test_rd_is_saturation_throughput_encoder_batch1():
    mc = model([comp("E", "ENC", [0.002, 1e-5, 0.0], x=["patches"])],
               [rtype("i", ["E"], images={"uniform": [1, 4]})])
    rd, thr = _saturated_rate(mc, one_plan([(1, 1, 1)], [[(10, {0: 0})]]))
    assert thr == pytest.approx(rd, rel=1e-9)


def test_rd_is_saturation_throughput_llm_batch1():
    mc = model([comp("L", "LLM", [0.005, 4e-5, 0.0], x=["prompt"], decode=(0.012, 8e-5))],
               [rtype("t", ["L"], prompt={"lognormal": [6.0, 0.5]}, out={"lognormal": [3.0, 0.6]})])
    rd, thr = _saturated_rate(mc, one_plan([(1, 1, 1)], [[(10, {0: 0})]]))
    assert thr == pytest.approx(rd, rel=1e-9)


def test_rd_with_full_batches_and_replicas():
    mc = model([comp("E", "ENC", [0.02, 1e-5, 0.0], x=["patches"])],
               [rtype("i", ["E"], images={"const": 1})])
    rd, thr = _saturated_rate(mc, one_plan([(1, 3, 8)], [[(10, {0: 0})]]), n=24000)
    assert thr == pytest.approx(rd, rel=0.01)


def test_rd_two_nodes_bottleneck():
    cfg = load_config("c1")
    mc = cfg["model"]
    # 1 encoder executor, 2 LLM executors at batch 16: the simulated
    # throughput at overload sits at (not above) the flow bound
    plan = one_plan([(1, 1, 16), (2, 2, 16)], [[(10, {1: 1})], [(10, {0: 0, 1: 1})]])
    m = O.make_model(mc)
    tr = O.trace_gen(m, [0], 8000)
    rd, bn, fl = O.eval_coarse(m, plan, tr["moments"][0], 8)
    o = O.sim_triple(m, plan, 0, 50.0 * rd[0], tr, 0, want_diag=True)
    thr = tr["n_req"] / o["diag"][1]
    assert bn[0] == 1
    assert 0.8 * rd[0] < thr < 1.02 * rd[0]


def test_structural_invariants():
    cfg = load_config("c2")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [0], 3000)
    rd, bn, fl = O.eval_coarse(m, tab, tr["moments"][0], cfg["gpus"])
    # doubling every node's replicas doubles R_d exactly and keeps the bottleneck
    t2 = tab.subset(np.arange(tab.P))
    t2.node_rep = (tab.node_rep.astype(np.int64) * 2).astype(np.uint8)
    rd2, bn2, fl2 = O.eval_coarse(m, t2, tr["moments"][0], 2 * cfg["gpus"])
    ok = (fl & 4) == 0
    assert np.array_equal(rd2[ok], 2 * rd[ok]) and np.array_equal(bn2[ok], bn[ok])
    # budget (Eq. 1): halving the budget flags exactly the plans using more GPUs
    gpus = (tab.node_rep.astype(np.int64) * tab.node_gpus).sum(axis=0)
    rd3, _, fl3 = O.eval_coarse(m, tab, tr["moments"][0], cfg["gpus"] // 2)
    assert np.array_equal((fl3 & 2) != 0, gpus > cfg["gpus"] // 2)
    assert np.all((fl3[(fl3 & 2) != 0] & 1) == 0)
    # keep = not over budget and not redundant
    assert np.array_equal((fl & 1) != 0, (fl & (2 | 4 | 8)) == 0)


def test_redundant_spare_replica_is_pruned():
    cfg = load_config("c1")
    m = O.make_model(cfg["model"])
    tr = O.trace_gen(m, [0], 3000)
    # a lone text type would leave the encoder idle; here: an encoder node with
    # far more replicas than the LLM can feed is redundant, a balanced one is not
    fat = one_plan([(1, 6, 64), (2, 1, 64)], [[(10, {1: 1})], [(10, {0: 0, 1: 1})]])
    lean = one_plan([(1, 1, 64), (2, 1, 64)], [[(10, {1: 1})], [(10, {0: 0, 1: 1})]])
    _, _, ff = O.eval_coarse(m, fat, tr["moments"][0], 8)
    _, _, fl = O.eval_coarse(m, lean, tr["moments"][0], 8)
    assert ff[0] & 8 and not ff[0] & 1
    assert fl[0] & 1


def test_invalid_plan_flag():
    cfg = load_config("c0")
    m = O.make_model(cfg["model"])
    tr = O.trace_gen(m, [0], 100)
    bad = one_plan([(1, 1, 8), (2, 1, 8)], [[(10, {1: 0})], [(10, {0: 0, 1: 1})]])  # node 0 lacks L
    rd, bn, fl = O.eval_coarse(m, bad, tr["moments"][0], 2)
    assert fl[0] == 4 and bn[0] == -1


def test_c0_plans_equal_brute_force_enumeration():
    cfg = load_config("c0")
    tab = make_plans(cfg, cache=False)
    got = set()
    for p in range(tab.P):
        pl = tab.plan(p)
        got.add((tuple((n["comp"], n["rep"], n["batch"]) for n in pl["nodes"]),
                 tuple(tuple(a["node"][:2]) for r in pl["routes"] for a in r)))
    want = set()
    for rep, b in itertools.product((1, 2), (8, 32)):   # E+L colocated on 1 or 2 GPUs
        want.add((((3, rep, b),), ((255, 0), (0, 0))))
    for b in (8, 32):                                   # E and L on one GPU each
        want.add((((1, 1, b), (2, 1, b)), ((255, 1), (0, 1))))
    assert got == want and tab.P == 6


def test_select_topk_matches_lexsort():
    rng = np.random.default_rng(5)
    P = 5000
    rd = rng.choice(np.round(rng.uniform(0, 50, 700), 1), P)   # many ties
    rd[rng.integers(0, P, 20)] = np.inf
    fl = rng.choice(np.array([1, 0, 8, 1, 1], np.uint8), P)
    for k in (1, 7, 100, 5000):
        ids = O.select_topk(rd, fl, k)
        kept = np.nonzero(fl & 1)[0]
        order = kept[np.lexsort((kept, -rd[kept]))]
        assert np.array_equal(ids, order[:k])


def test_rate_grid_ends_at_alpha_rd():
    rd = np.array([3.0, 7.25, 1e-3, 123.456])
    ids = np.array([3, 0, 1], np.int32)
    r = O.rate_grid(rd, ids, 16, 1.0)
    assert np.array_equal(r[:, -1], rd[ids])
    assert np.all(np.diff(r, axis=1) > 0)
    r2 = O.rate_grid(rd, ids, 32, 0.5)
    assert np.array_equal(r2[:, -1], 0.5 * rd[ids])


def test_goodput_reduce_against_bisection():
    rng = np.random.default_rng(6)
    n_plans, K, S, T, n = 40, 16, 3, 4, 1000
    cnt = rng.integers(0, 400, (n_plans, 1, S, T)).astype(np.uint32).repeat(K, axis=1)
    # attainment decreasing with the rate index (monotone, as bisection assumes)
    frac = np.sort(rng.uniform(0.5, 1.0, (n_plans, K)), axis=1)[:, ::-1]
    met = np.floor(cnt * frac[:, :, None, None]).astype(np.uint32)
    rates = np.sort(rng.uniform(0.1, 10, (n_plans, K)), axis=1)
    kstar, gt, g = O.goodput_reduce(met, cnt, rates, (9, 10), n)

    def feasible(i, k):
        M, N = met[i, k].sum(axis=0).astype(np.int64), cnt[i, k].sum(axis=0).astype(np.int64)
        return bool(np.all((N == 0) | (10 * M >= 9 * N)))
    for i in range(n_plans):
        lo, hi = -1, K          # bisection for the last feasible index
        while hi - lo > 1:
            mid = (lo + hi) // 2
            if feasible(i, mid):
                lo = mid
            else:
                hi = mid
        assert kstar[i] == lo
        if lo >= 0:
            M = met[i, lo].sum(axis=0).astype(np.float64)
            assert gt[i] == pytest.approx(rates[i, lo] * M / (S * n), rel=1e-15)
        else:
            assert np.all(gt[i] == 0)
    # a plan meeting every target at every rate has goodput r_max * (sum N)/(S n)
    met_all = cnt.copy()
    ks, gt2, g2 = O.goodput_reduce(met_all, cnt, rates, (9, 10), n)
    assert np.all(ks == K - 1)
    tot = cnt[:, -1].sum(axis=(1, 2)).astype(np.float64)
    assert np.allclose(g2, rates[:, -1] * tot / (S * n), rtol=1e-14)
    assert O.argmax(np.array([1.0, 3.0, 3.0, 2.0])) == 1


def test_failed_simulation_makes_its_rate_infeasible():
    """A rate whose simulation of some seed failed (nonzero status: invalid, deadlock,
    overflow) is infeasible, however good its truncated counts look; the bisection of the
    same counts with that rate failing gives the same answer."""
    rng = np.random.default_rng(7)
    n_plans, K, S, T, n = 12, 16, 4, 3, 500
    cnt = rng.integers(50, 200, (n_plans, 1, S, T)).astype(np.uint32).repeat(K, axis=1)
    met = cnt.copy()  # every rate meets every target on its counts
    rates = np.sort(rng.uniform(0.1, 10, (n_plans, K)), axis=1)
    status = np.zeros((n_plans, K, S), np.uint32)
    fail_at = rng.integers(0, K, n_plans)
    for i in range(n_plans):
        status[i, fail_at[i], rng.integers(0, S)] = [1, 2, 4][i % 3]
    ks, gt, g = O.goodput_reduce(met, cnt, rates, (9, 10), n, status=status)
    assert np.array_equal(ks, fail_at - 1)
    for i in range(n_plans):
        if fail_at[i] == 0:
            assert g[i] == 0.0 and np.all(gt[i] == 0.0)
        else:
            M = met[i, fail_at[i] - 1].sum(axis=0).astype(np.float64)
            assert np.array_equal(gt[i], (rates[i, fail_at[i] - 1] * M) / (S * n))
    # without the status words the same counts are feasible everywhere
    ks0, _, _ = O.goodput_reduce(met, cnt, rates, (9, 10), n)
    assert np.all(ks0 == K - 1)
