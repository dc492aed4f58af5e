"""Pins of the oracle's latency CDFs over target tables (Alg. 2: F_{t,d} is
the CDF of accumulated latencies, evaluated at L_t; goodput against a range
of latency targets, Sec. 6.2 and Appendix B).

Independent checks: with a one-bin table equal to each type's own bounds,
bin 0 holds exactly the requests the SLO counters (a separate code path in
the simulator and in phase 2) call met, and the CDF at that bin is phase 2's
G_t; the goodput reduction over cumulative bins at the SLO bin equals the
plain reduction of the met counts; cumulative counts do not decrease and end
at the type's count; scaling every target by a common factor s moves a
request's bin exactly to the first s whose scaled bounds it meets.
"""
import numpy as np

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans

SCALES = [0.25, 0.5, 0.75, 1.0, 1.5, 2.0, 4.0]


def _c2(n=600):
    cfg = load_config("c2")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [3], n)
    rd, _, fl = O.eval_coarse(m, tab, tr["moments"][0], cfg["gpus"])
    ids = O.select_topk(rd, fl, 30)
    return cfg, m, tab, tr, rd, ids


def test_slo_bin_is_phase_two_met_and_goodput():
    cfg, m, tab, tr, rd, ids = _c2()
    tg = O.scaled_targets(m, [1.0])
    met, cnt, gt, hist, curve = O.mc_curve(m, tab, ids, rd, tr["moments"][0], 0.8, tr, 0, 600, tg)
    met2, cnt2, gt2 = O.eval_mc(m, tab, ids, rd, tr["moments"][0], 0.8, tr, 0, 600)
    assert np.array_equal(met, met2) and np.array_equal(cnt, cnt2) and np.array_equal(gt, gt2)
    assert np.array_equal(hist[:, :, 0], met)
    assert np.array_equal(hist[:, :, 1], cnt - met)
    assert np.array_equal(curve[:, 0, :], gt)


def test_scaled_tables_cumulate_and_bin_exactly():
    cfg, m, tab, tr, rd, ids = _c2()
    tg = O.scaled_targets(m, SCALES)
    met, cnt, gt, hist, curve = O.mc_curve(m, tab, ids[:8], rd, tr["moments"][0], 0.8, tr, 0, 600, tg)
    cum = np.cumsum(hist, axis=2)
    assert np.all(np.diff(cum, axis=2) >= 0)
    assert np.array_equal(cum[:, :, -1], cnt)
    assert np.array_equal(cum[:, :, SCALES.index(1.0)], met)
    # the curve does not decrease with the target and ends at alpha R_d pi_t F_t(inf)
    assert np.all(np.diff(curve, axis=1) >= 0)
    # per request: the bin is the first scale whose scaled bounds hold
    _, _, _, lat = O.eval_mc(m, tab, ids[:8], rd, tr["moments"][0], 0.8, tr, 0, 600, want_lat=True)
    types = tr["type"][:600]
    for i in range(8):
        h = O.latency_hist(lat[i], types, m.n_types, tg)
        assert np.array_equal(h, hist[i])
        r = 17 * i % 600
        t = types[r]
        ok = [all(lat[i, r, j] <= m.slo[t][j] * s for j in range(4)) for s in SCALES]
        first = ok.index(True) if True in ok else len(SCALES)
        one = O.latency_hist(lat[i, r:r + 1], types[r:r + 1], m.n_types, tg)
        assert one[t, first] == 1 and one.sum() == 1


def test_phase_three_histogram_at_the_slo():
    cfg = load_config("c1")
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr = O.trace_gen(m, [2], 3000)
    tg = O.scaled_targets(m, [0.5, 1.0, 2.0])
    for p, rate in ((3, 2.0), (40, 6.0), (200, 12.0)):
        des = O.sim_triple(m, tab, p, rate, tr, 0, want_lat=True)
        h = O.latency_hist(des["lat"], tr["type"][:3000], m.n_types, tg)
        cum = np.cumsum(h, axis=1)
        assert np.array_equal(cum[:, 1], des["met"])
        assert np.array_equal(cum[:, -1], des["cnt"])
