"""Pins of the oracle's nodes with executors of two configurations (Eq. (1): a node v holds
n_{v,k} executors of each configuration k; routing between the executors of a node in steps
of 0.1, Sec. 4.2).

A node may hold node_rep executors of one configuration and node_rep2 of a second (another
batch or GPU count); a request reaching the node goes to the first group with probability
node_w / 10, realised by the request's 16-bit replica key for the node: the first group
takes the keys below w * 2^16 / 10, and each group's keys are cut into equal parts for its
executors.  Expected values come from outside the code under test:

* the key space: requests with hand-set keys on both sides of every cut take the executor
  the interval says, seen from their latencies (the second group's executors run on two
  GPUs at half the latency; two requests arriving together on one batch-1 executor queue);
* the binomial law for the share of the second group on seeded traces;
* saturation throughput: with keys stratified over the key space and every request arriving
  at once, each group finishes its share of the requests after n * s_g * w_g / m_g seconds
  of work (full batches of identical requests), so phase 1's R_d must be the smallest
  n / makespan over the groups;
* a node split into two groups of one configuration with w / 10 = m_1 / (m_1 + m_2) has the
  capacity of one group of m_1 + m_2 executors (phase 1 agrees to rounding);
* Eq. (1)'s budget counts both configurations (brute force over random tables);
* phase 2 routes like the simulator (zero-load latencies equal on plans with split nodes).
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import PlanTable, load_config, plan_table_from_list

from .helpers import comp, make_trace, model, rtype

KEYS = 1 << 16


def _enc(tp2=0.5, k=(0.0, 1e-5, 0.0)):
    return model([comp("E", "ENC", list(k), x=["patches"]) | {"tp_scale": {2: tp2}}],
                 [rtype("i", ["E"], slo={"e2e": 1e9}, images={"const": 1})])


def _split_node_plan(rep1, rep2, w, b1=1, b2=1, g2=2):
    return plan_table_from_list([dict(nodes=[(1, rep1, b1, 1, rep2, b2, g2, w)], routes=[[(10, {0: 0})]])])


def _executor_of(key, rep1, rep2, w):
    """The executor the key intervals name (exact rationals): [0, w 2^16 / 10) cut into rep1
    equal parts, the rest of [0, 2^16) into rep2."""
    cut = Fraction(w * KEYS, 10)
    if key < cut:
        return math.floor(key * rep1 / cut)
    return rep1 + math.floor((key - cut) * rep2 / (KEYS - cut))


def _key_inside(j, rep1, rep2, w):
    """An integer key in the middle of executor j's interval."""
    cut = Fraction(w * KEYS, 10)
    if j < rep1:
        return math.floor((j + Fraction(1, 2)) * cut / rep1)
    return math.floor(cut + (j - rep1 + Fraction(1, 2)) * (KEYS - cut) / rep2)


@pytest.mark.parametrize("rep1,rep2,w", [(1, 1, 3), (2, 3, 7), (3, 1, 5), (1, 4, 9), (4, 2, 1)])
def test_group_and_executor_follow_the_key_intervals(rep1, rep2, w):
    m = O.make_model(_enc())
    plan = _split_node_plan(rep1, rep2, w)
    cuts = [w * KEYS / 10.0 * i / rep1 for i in range(1, rep1 + 1)]
    cuts += [w * KEYS / 10.0 + (KEYS - w * KEYS / 10.0) * i / rep2 for i in range(1, rep2)]
    keys = sorted({0, KEYS - 1} | {int(math.floor(c)) for c in cuts} | {int(math.ceil(c)) for c in cuts}
                  | {min(KEYS - 1, int(math.ceil(c)) + 1) for c in cuts})
    keys = [k for k in keys if 0 <= k < KEYS]
    X = 1000
    # each key alone (100 s apart): the second group runs at half the latency
    reqs = [dict(t=100.0 * i, patches=X, rkey0=k) for i, k in enumerate(keys)]
    o = O.sim_triple(m, plan, 0, 1.0, make_trace(reqs), 0, want_lat=True)
    assert o["status"] == 0
    lat1, lat2 = 1e-5 * X, 0.5 * (1e-5 * X)
    for k, e2e in zip(keys, o["lat"][:, 2]):
        second = _executor_of(k, rep1, rep2, w) >= rep1
        assert e2e == pytest.approx(lat2 if second else lat1, rel=1e-9), (k, e2e)
    # pairs arriving together on batch-1 executors queue iff the intervals name one executor
    for k1 in keys[:: max(1, len(keys) // 6)]:
        for k2 in keys[:: max(1, len(keys) // 5)]:
            reqs = [dict(t=0.0, patches=X, rkey0=k1), dict(t=0.0, patches=X, rkey0=k2)]
            o = O.sim_triple(m, plan, 0, 1.0, make_trace(reqs), 0, want_lat=True)
            same = _executor_of(k1, rep1, rep2, w) == _executor_of(k2, rep1, rep2, w)
            one = lat2 if _executor_of(k2, rep1, rep2, w) >= rep1 else lat1
            assert o["lat"][1, 2] == pytest.approx(2 * one if same else one, rel=1e-12), (k1, k2)


@pytest.mark.parametrize("w,seed", [(3, 21), (8, 22)])
def test_second_group_share_follows_the_weight(w, seed):
    m = O.make_model(_enc())
    n = 4000
    tr = O.trace_gen(m, [seed], n)
    tr["arr_ticks"] = np.ascontiguousarray(np.arange(n, dtype=np.uint64) * np.uint64(100 << 32))
    o = O.sim_triple(m, _split_node_plan(2, 3, w), 0, 1.0, tr, 0, want_lat=True)
    assert o["status"] == 0
    lat1 = np.array([1e-5 * int(x) for x in tr["patches"][:n]])
    # arrivals up to 4e5 s: absolute times round at ~1e-10 s
    second = np.abs(o["lat"][:, 2] - 0.5 * lat1) <= 1e-6 * lat1
    first = np.abs(o["lat"][:, 2] - lat1) <= 1e-6 * lat1
    assert np.all(first ^ second)
    p2 = (10 - w) / 10
    k = int(second.sum())
    assert abs(k - n * p2) <= 4.5 * math.sqrt(n * p2 * (1 - p2)), (k, n * p2)


@pytest.mark.parametrize("rep1,rep2,w,b1,b2", [(1, 1, 3, 1, 4), (2, 1, 6, 1, 4), (1, 2, 2, 4, 1), (3, 2, 5, 2, 8)])
def test_phase1_groups_equal_saturation_throughput(rep1, rep2, w, b1, b2):
    a, bpp, X = 0.004, 1e-5, 500
    m = O.make_model(_enc(tp2=1.0, k=(a, bpp, 0.0)))
    plan = _split_node_plan(rep1, rep2, w, b1, b2, g2=1)
    # n requests split exactly in the groups' shares and evenly over a group's executors, in
    # whole batches: keys placed inside each executor's interval in those numbers
    n = 10 * rep1 * rep2 * b1 * b2 * 2
    count = [n * w // (10 * rep1)] * rep1 + [n * (10 - w) // (10 * rep2)] * rep2
    assert sum(count) == n
    keys = [_key_inside(j, rep1, rep2, w) for j in range(rep1 + rep2) for _ in range(count[j])]
    ex = np.array([_executor_of(k, rep1, rep2, w) for k in keys])
    assert list(np.bincount(ex, minlength=rep1 + rep2)) == count
    tr = make_trace([dict(t=0.0, patches=X, rkey0=k) for k in keys])
    o = O.sim_triple(m, plan, 0, 1.0, tr, 0, want_lat=True)
    assert o["status"] == 0
    e2e = o["lat"][:, 2]
    sat = [n / e2e[ex < rep1].max(), n / e2e[ex >= rep1].max()]
    moments = np.zeros((1, 8), np.uint64)
    moments[0, 0], moments[0, 3] = n, n * X
    rd, bn, fl = O.eval_coarse(m, plan, moments, 64)
    assert bn[0] == 0 and fl[0] & 4 == 0
    assert rd[0] == pytest.approx(min(sat), rel=1e-9)


def test_split_of_one_configuration_has_the_capacity_of_one_group():
    cfg = load_config("c1")
    m = O.make_model(cfg["model"])
    tr = O.trace_gen(m, [0], 3000)
    mom = tr["moments"][0]
    for (r1, r2, w) in [(1, 1, 5), (2, 3, 4), (1, 4, 2), (3, 2, 6)]:
        for b in (16, 64):
            split = plan_table_from_list([dict(nodes=[(1, 1, 64, 1), (2, r1, b, 1, r2, b, 1, w)],
                                               routes=[[(10, {1: 1})], [(10, {0: 0, 1: 1})]])])
            whole = plan_table_from_list([dict(nodes=[(1, 1, 64, 1), (2, r1 + r2, b, 1)],
                                               routes=[[(10, {1: 1})], [(10, {0: 0, 1: 1})]])])
            rs, bs, fs = O.eval_coarse(m, split, mom, 8)
            rw, bw, fw = O.eval_coarse(m, whole, mom, 8)
            assert rs[0] == pytest.approx(rw[0], rel=1e-12) and bs[0] == bw[0]
            assert (fs[0] & 2) == (fw[0] & 2)


def test_budget_counts_both_configurations():
    cfg = load_config("c1")
    m = O.make_model(cfg["model"])
    mom = O.trace_gen(m, [0], 2000)["moments"][0]
    rng = np.random.default_rng(5)
    plans, gpus = [], []
    for _ in range(300):
        r1, r2, g1, g2 = (int(v) for v in rng.integers(1, 5, 4))
        re, ge = int(rng.integers(1, 4)), int(rng.integers(1, 3))
        plans.append(dict(nodes=[(1, re, 16, ge), (2, r1, 16, g1, r2, 64, g2, int(rng.integers(1, 10)))],
                          routes=[[(10, {1: 1})], [(10, {0: 0, 1: 1})]]))
        gpus.append(re * ge + r1 * g1 + r2 * g2)
    tab = plan_table_from_list(plans)
    for N in (8, 16, 24):
        _, _, fl = O.eval_coarse(m, tab, mom, N)
        assert np.array_equal((fl & 2) != 0, np.array(gpus) > N), N


def test_invalid_split_weight():
    m = O.make_model(_enc())
    for w in (0, 10, 11):
        plan = _split_node_plan(1, 1, w)
        _, bn, fl = O.eval_coarse(m, plan, np.array([[10, 0, 0, 5000, 0, 0, 0, 0]], np.uint64), 8)
        assert fl[0] == 4 and bn[0] == -1
        o = O.sim_triple(m, plan, 0, 1.0, make_trace([dict(t=0.0, patches=500)]), 0)
        assert o["status"] & O.ST_INVALID


@pytest.mark.parametrize("cfgname", ["c0", "c2"])
def test_monte_carlo_routes_groups_like_the_simulator(cfgname):
    cfg = load_config(cfgname)
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.0
    mc["components"] = [dict(c) | {"tp_scale": {2: 0.5}} for c in mc["components"]]
    m = O.make_model(mc)
    names = [c["name"] for c in mc["components"]]
    n = 300
    tr = O.trace_gen(m, [9], n)
    tr["arr_ticks"] = np.ascontiguousarray(np.arange(n, dtype=np.uint64) * np.uint64(100 << 32))
    # one node per component, batch 1, each split 2 + 2 executors (second group on 2 GPUs)
    nodes = [(1 << c, 2, 1, 1, 2, 1, 2, 3 + c) for c in range(len(names))]
    routes = [[(10, {names.index(c): names.index(c) for c in t["comps"]})] for t in mc["types"]]
    plan = plan_table_from_list([dict(nodes=nodes, routes=routes)])
    des = O.sim_triple(m, plan, 0, 1.0, tr, 0, want_lat=True)
    assert des["status"] == 0
    rd, _, fl = O.eval_coarse(m, plan, tr["moments"][0], 64)
    assert fl[0] & 4 == 0
    met, cnt, gt, lat = O.eval_mc(m, plan, [0], rd, tr["moments"][0], 0.8, tr, 0, n, want_lat=True)
    np.testing.assert_allclose(lat[0], des["lat"], rtol=0, atol=1e-7)


def test_homogeneous_tables_unchanged_by_the_new_fields():
    """A table whose nodes have one configuration gives the same results with the second-group
    arrays present (zeros) as without them."""
    cfg = load_config("c1")
    from paper_2512_14098_amd.inputs import make_plans
    tab = make_plans(cfg)
    m = O.make_model(cfg["model"])
    tr = O.trace_gen(m, [0], 2000)
    a = O.eval_coarse(m, tab, tr["moments"][0], 8)
    bare = PlanTable(tab.P)
    for f in ("n_nodes", "node_comp", "node_rep", "node_batch", "node_gpus", "n_alt", "alt_w", "alt_node"):
        setattr(bare, f, getattr(tab, f))
    for f in ("node_rep2", "node_batch2", "node_gpus2", "node_w"):
        setattr(bare, f, None)
    b = O.eval_coarse(m, bare, tr["moments"][0], 8)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
