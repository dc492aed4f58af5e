"""Pins of the oracle's tensor-parallel latency scaling (the configuration
space's parallelism degree, Sec. 3 and Eq. (1): an executor of g GPUs runs
its component's latency model times tp_scale[c][g]).

Independent check: multiplying every latency coefficient of every component
by 8 (exact in binary) gives a model whose iteration times are exactly 8x
the original's; the original model with tp_scale = 8 on executors of two
GPUs must therefore give identical results on the same plans with two GPUs
per executor -- phase 1's R_d, phase 2's counts, goodput and latencies, and
every phase-3 count, request-event and latency.  A scaling step left out
anywhere breaks the equality.  Executors of one GPU keep the profiled model.
"""
import copy

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans


def _coef_x8(mc):
    mc = copy.deepcopy(mc)
    for c in mc["components"]:
        c["k"] = [v * 8.0 for v in c["k"]]
        if "decode" in c:
            c["decode"] = [v * 8.0 for v in c["decode"]]
    return mc


def _tp8(mc, g=2):
    mc = copy.deepcopy(mc)
    for c in mc["components"]:
        c["tp_scale"] = {str(g): 8.0}
    return mc


def _gpus(tab, g):
    t2 = tab.subset(np.arange(tab.P))
    t2.node_gpus = np.where(t2.node_comp > 0, g, 0).astype(np.uint8)
    return t2


@pytest.mark.parametrize("cfgname", ["c1", "c2", "c3"])
def test_tp_scale_equals_scaled_coefficients(cfgname):
    cfg = load_config(cfgname)
    mc = dict(cfg["model"])
    mc["cpu_pre_s"] = 0.003
    mA, mB = O.make_model(_coef_x8(mc)), O.make_model(_tp8(mc))
    tab = make_plans(cfg)
    tab1, tab2 = _gpus(tab, 1), _gpus(tab, 2)
    tr = O.trace_gen(mA, [6], 1200)
    rdA, bnA, _ = O.eval_coarse(mA, tab1, tr["moments"][0], 4096)
    rdB, bnB, _ = O.eval_coarse(mB, tab2, tr["moments"][0], 4096)
    assert np.array_equal(rdA, rdB) and np.array_equal(bnA, bnB)
    # executors of one GPU keep the profiled latencies
    rd1, _, _ = O.eval_coarse(mB, tab1, tr["moments"][0], 4096)
    rd0, _, _ = O.eval_coarse(O.make_model(mc), tab1, tr["moments"][0], 4096)
    assert np.array_equal(rd1, rd0)
    ids = np.arange(0, tab.P, max(1, tab.P // 40), dtype=np.int32)
    a = O.eval_mc(mA, tab1, ids, rdA, tr["moments"][0], 0.8, tr, 0, 1200, want_lat=True)
    b = O.eval_mc(mB, tab2, ids, rdB, tr["moments"][0], 0.8, tr, 0, 1200, want_lat=True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    for p in (int(ids[0]), int(ids[len(ids) // 2]), int(ids[-1])):
        for rate in (0.2 * rdA[p], 0.9 * rdA[p]):
            if not rate > 0:
                continue
            sa = O.sim_triple(mA, tab1, p, rate, tr, 0, want_lat=True)
            sb = O.sim_triple(mB, tab2, p, rate, tr, 0, want_lat=True)
            assert np.array_equal(sa["met"], sb["met"]) and sa["events"] == sb["events"]
            assert np.array_equal(sa["lat"], sb["lat"])
