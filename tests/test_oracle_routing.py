"""Pins of the oracle's split of a request type between two alternative paths
(routing probabilities between the parallel paths of a logical plan, Sec. 4.2;
a type's load split across them in phase 1, Alg. 2).

The oracle reads a routing weight pair (w0, w1) in tenths as the probability
w0 / (w0 + w1) of alternative 0, realised per request by the trace's 32-bit
alternative key k: the keys sent to alternative 0 must be exactly the first
w0 / (w0 + w1) of the key space, and phase 1 must put the share q_a = w_a /
(w0 + w1) of the type's work on alternative a's nodes.  Expected values come
from outside the code under test:

* the key space itself: with the weights summing to W, a key k goes to
  alternative 0 iff k * W < w0 * 2^32, i.e. the alternative-0 keys are the
  interval [0, b) with b = ceil(w0 * 2^32 / W), whose share of the 2^32 keys
  is w0 / W up to one key; requests with hand-set keys on both sides of b
  must take the alternative the interval says, seen from their zero-load
  latency (alternative 1 crosses two executors and pays the communication
  delay, alternative 0 does not);
* the binomial law: on a seeded trace the number of requests taking
  alternative 1 must lie within 4.5 standard deviations of n * w1 / W;
* saturation throughput: with keys stratified over the key space (so that
  exactly w_a / W of the requests take alternative a) and every request
  arriving at once, node v of a one-component plan finishes its requests
  after n * q_v * w_v seconds of work (full batches of identical requests),
  so the rate at which it completes them is 1 / (q_v w_v) and the plan's
  saturation throughput is the smallest of these: phase 1's R_d and
  bottleneck must match it; the nodes have different per-request work, so
  swapping the alternatives' shares moves both;
* phase 2 (Monte Carlo) routes its sampled requests with the same rule: at
  zero load its per-request latencies equal the simulator's on a
  two-alternative plan.
"""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config

from .helpers import comp, make_trace, model, one_plan, rtype

KEYS = 2 ** 32
COMM = 0.010


def _enc_llm():
    return model([comp("E", "ENC", [0.002, 1e-5, 0.0], x=["patches"]),
                  comp("L", "LLM", [0.005, 2e-5, 0.0], x=["prompt"], decode=(0.008, 5e-5))],
                 [rtype("i", ["E", "L"], edges=[("E", "L")], slo={"e2e": 100.0})], comm=COMM)


def _split_plan(w0, w1):
    # alternative 0: E and L colocated on node 0; alternative 1: E on node 1, L on node 2
    return one_plan([(3, 1, 8), (1, 1, 8), (2, 1, 8)],
                    [[(w0, {0: 0, 1: 0}), (w1, {0: 1, 1: 2})]])


def _first_alt1_key(w0, W):
    """The first key of alternative 1: the alternative-0 keys are [0, b), w0 / W of the space."""
    return -(-w0 * KEYS // W)


def _alternative_from_latency(lat_e2e, reference):
    """1 where the request paid the communication delay of alternative 1, else 0."""
    d = np.asarray(lat_e2e) - np.asarray(reference)
    assert np.all((np.abs(d) < 1e-9) | (np.abs(d - COMM) < 1e-9)), d
    return (d > COMM / 2).astype(int)


@pytest.mark.parametrize("w0,w1", [(3, 7), (1, 9), (9, 1), (5, 5), (2, 3)])
def test_alternative_keys_are_the_first_w0_share_of_the_key_space(w0, w1):
    W = w0 + w1
    b = _first_alt1_key(w0, W)
    assert abs(b / KEYS - w0 / W) <= 1.0 / KEYS
    keys = [0, 1, b - 2, b - 1, b, b + 1, KEYS // 2, KEYS - 1, b // 3, b + (KEYS - b) // 2]
    # every request alone (100 s apart), identical work, so the only difference is the path
    reqs = [dict(t=100.0 * i, patches=400, prompt=50, out=3, akey=k) for i, k in enumerate(keys)]
    m = O.make_model(_enc_llm())
    tr = make_trace(reqs)
    o = O.sim_triple(m, _split_plan(w0, w1), 0, 1.0, tr, 0, want_lat=True)
    assert o["status"] == 0
    e2e = o["lat"][:, 2]
    # a colocated reference: the plan with alternative 0 only
    ref = O.sim_triple(m, one_plan([(3, 1, 8)], [[(10, {0: 0, 1: 0})]]), 0, 1.0, tr, 0, want_lat=True)
    alt = _alternative_from_latency(e2e, ref["lat"][:, 2])
    expect = [0 if k < b else 1 for k in keys]
    assert list(alt) == expect, (w0, w1, b)


@pytest.mark.parametrize("w0,w1,seed", [(3, 7, 11), (8, 2, 12), (1, 9, 13)])
def test_alternative_shares_follow_the_weights(w0, w1, seed):
    W = w0 + w1
    n = 4000
    m = O.make_model(_enc_llm())
    tr = O.trace_gen(m, [seed], n)
    tr["arr_ticks"] = np.ascontiguousarray(np.arange(n, dtype=np.uint64) * np.uint64(100 << 32))
    o = O.sim_triple(m, _split_plan(w0, w1), 0, 1.0, tr, 0, want_lat=True)
    ref = O.sim_triple(m, one_plan([(3, 1, 8)], [[(10, {0: 0, 1: 0})]]), 0, 1.0, tr, 0, want_lat=True)
    assert o["status"] == 0 and ref["status"] == 0
    alt = _alternative_from_latency(o["lat"][:, 2], ref["lat"][:, 2])
    p1 = w1 / W
    k = int(alt.sum())
    assert abs(k - n * p1) <= 4.5 * math.sqrt(n * p1 * (1 - p1)), (k, n * p1)
    # and per request it is the key interval (the trace's alternative key decides)
    b = _first_alt1_key(w0, W)
    assert np.array_equal(alt, (tr["akey"][:n].astype(np.int64) >= b).astype(int))


def _stratified_keys(n):
    # key i at the middle of the i-th of n equal parts of the key space
    return [((2 * i + 1) * KEYS) // (2 * n) for i in range(n)]


@pytest.mark.parametrize("w0,w1,expect_bn", [(3, 7, 1), (8, 2, 0), (2, 8, 1), (5, 5, 0)])
def test_phase1_split_equals_saturation_throughput(w0, w1, expect_bn):
    a, bpp, X = 0.004, 1e-5, 500
    mc = model([comp("E", "ENC", [a, bpp, 0.0], x=["patches"])],
               [rtype("i", ["E"], slo={"e2e": 1e9})])
    m = O.make_model(mc)
    # node 0 runs batches of 1, node 1 batches of 4: per-request work differs
    plan = one_plan([(1, 1, 1), (1, 1, 4)], [[(w0, {0: 0}), (w1, {0: 1})]])
    n = 2000
    keys = _stratified_keys(n)
    b = _first_alt1_key(w0, w0 + w1)
    n0 = sum(1 for k in keys if k < b)
    assert n0 == n * w0 // (w0 + w1)  # the stratified keys realise the shares exactly
    assert (n - n0) % 4 == 0
    # every request arrives at t = 0: both nodes work back to back from the start
    tr = make_trace([dict(t=0.0, patches=X, akey=k) for k in keys])
    o = O.sim_triple(m, plan, 0, 1.0, tr, 0, want_lat=True)
    assert o["status"] == 0
    e2e = o["lat"][:, 2]
    is0 = np.array([k < b for k in keys])
    makespan = [e2e[is0].max(), e2e[~is0].max()]
    # saturation rate of each node = requests of the whole stream per second of its work
    sat = [n / makespan[0], n / makespan[1]]
    moments = np.zeros((1, 8), np.uint64)
    moments[0, 0] = n
    moments[0, 3] = n * X  # sum of patches
    rd, bn, fl = O.eval_coarse(m, plan, moments, 64)
    assert bn[0] == int(np.argmin(sat)) == expect_bn
    assert rd[0] == pytest.approx(min(sat), rel=1e-9)


def test_monte_carlo_routes_like_the_simulator():
    cfg = load_config("c0")
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.0
    m = O.make_model(mc)
    n = 300
    tr = O.trace_gen(m, [7], n)
    tr["arr_ticks"] = np.ascontiguousarray(np.arange(n, dtype=np.uint64) * np.uint64(100 << 32))
    # both types: alternative 0 colocated (node 0), alternative 1 disaggregated (nodes 1, 2);
    # batch 1 everywhere, so every effective batch of phase 2 is 1
    names = [c["name"] for c in mc["components"]]
    iE, iL = names.index("E"), names.index("L")
    routes = []
    for t in mc["types"]:
        comps = [names.index(c) for c in t["comps"]]
        a0 = {c: 0 for c in comps}
        a1 = {c: (1 if c == iE else 2) for c in comps}
        routes.append([(3, a0), (7, a1)])
    plan = one_plan([((1 << iE) | (1 << iL), 1, 1), (1 << iE, 1, 1), (1 << iL, 1, 1)], routes)
    des = O.sim_triple(m, plan, 0, 1.0, tr, 0, want_lat=True)
    assert des["status"] == 0
    rd, _, fl = O.eval_coarse(m, plan, tr["moments"][0], 64)
    assert fl[0] & 4 == 0
    met, cnt, gt, lat = O.eval_mc(m, plan, [0], rd, tr["moments"][0], 0.8, tr, 0, n, want_lat=True)
    np.testing.assert_allclose(lat[0], des["lat"], rtol=0, atol=1e-7)
    # both alternatives were taken
    ref = O.sim_triple(m, one_plan([((1 << iE) | (1 << iL), 1, 1)], [[(10, {c: 0 for c in [names.index(x) for x in t["comps"]]})] for t in mc["types"]]),
                       0, 1.0, tr, 0, want_lat=True)
    alt = _alternative_from_latency(des["lat"][:, 2], ref["lat"][:, 2])
    assert 0 < alt.sum() < n
