"""Pins of the oracle's rate bisection: on every plan whose feasibility over
the grid is monotone (checked on the full grid), bisection returns the
grid's highest feasible rate and the same per-type goodput as the plain
reduction over all K rates (a separate code path); it simulates between
floor(log2(K+1)) and ceil(log2(K+1)) rates, and the request-events it
reports are those of the rates it simulated."""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans


def _monotone(met, cnt, theta):
    n, K, S, T = met.shape
    M, N = met.sum(axis=2).astype(np.uint64), cnt.sum(axis=2).astype(np.uint64)
    feas = np.all((N == 0) | (theta[1] * M >= theta[0] * N), axis=2)
    return [bool(np.all(np.diff(feas[i].astype(int)) <= 0)) for i in range(n)]


@pytest.mark.parametrize("name,n_plans,seeds,n", [("c0", 6, [0], 1000), ("c1", 10, [3, 4], 2000)])
def test_bisection_equals_grid_on_monotone_plans(name, n_plans, seeds, n):
    cfg = load_config(name)
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, seeds, n)
    if "explicit" in cfg["rates"]:
        ids = np.arange(min(n_plans, tab.P), dtype=np.int32)
        rates = np.tile(np.asarray(cfg["rates"]["explicit"], np.float64), (len(ids), 1))
    else:
        rd, _, fl = O.eval_coarse(m, tab, tr["moments"][0], cfg["gpus"])
        ids = O.select_topk(rd, fl, n_plans)
        rates = O.rate_grid(rd, ids, cfg["rates"]["grid"])
    theta = (9, 10)
    met, cnt, events, status = O.eval_fine(m, tab, ids, rates, tr)
    gk, ggt, gg = O.goodput_reduce(met, cnt, rates, theta, n)
    ks, gt, g, ne, ev = O.bisect(m, tab, ids, rates, tr, theta)
    K = rates.shape[1]
    mono = _monotone(met, cnt, theta)
    assert sum(mono) >= len(ids) // 2
    for i in range(len(ids)):
        assert math.floor(math.log2(K + 1)) <= ne[i] <= math.ceil(math.log2(K + 1))
        if mono[i]:
            assert ks[i] == gk[i] and np.array_equal(gt[i], ggt[i]) and g[i] == gg[i]
        assert ev[i] <= events[i].sum() and ev[i] > 0


def test_bisection_single_rate():
    cfg = load_config("c0")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [1], 300)
    rates = np.array([[1.0], [50.0]])
    ks, gt, g, ne, ev = O.bisect(m, tab, [0, 0], rates, tr, (9, 10))
    assert list(ne) == [1, 1]
    met, cnt, _, _ = O.eval_fine(m, tab, [0, 0], rates, tr)
    wk, wgt, wg = O.goodput_reduce(met, cnt, rates, (9, 10), 300)
    assert np.array_equal(ks, wk) and np.array_equal(gt, wgt)


def test_bisection_treats_a_failed_simulation_as_infeasible():
    """Rates below zero make every simulation of a plan invalid (status != 0): its
    truncated counts (no request simulated) would pass the attainment test, but bisection
    must not take them as feasible, and neither does the grid reduction."""
    cfg = load_config("c0")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [1], 200)
    rates = np.array([[-1.0, -0.5, 1.0, 2.0], [1.0, 2.0, 4.0, 8.0]])
    ks, gt, g, ne, ev = O.bisect(m, tab, [0, 0], rates, tr, (9, 10))
    met, cnt, _, st = O.eval_fine(m, tab, [0, 0], rates, tr)
    assert np.all(st[0, :2] != 0) and np.all(st[0, 2:] == 0) and np.all(st[1] == 0)
    wk, wgt, wg = O.goodput_reduce(met, cnt, rates, (9, 10), 200, status=st)
    assert wk[0] == -1 and wg[0] == 0.0
    assert ks[0] == -1 and g[0] == 0.0
    assert ks[1] == wk[1] and g[1] == wg[1]
