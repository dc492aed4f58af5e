"""GPU parity of the latency CDFs over target tables: phase 2's histograms and
goodput curves (cf_eval_mc_curve), phase 3's per-triple histograms
(cf_eval_fine with targets) and the goodput-against-target reduction
(cf_goodput_curve), against the oracle on the same seeded inputs; counts
bit-exact, fp64 outputs identical (same operations in the same order)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config, make_plans  # noqa: E402

SCALES = [0.25, 0.4, 0.6, 0.8, 1.0, 1.25, 1.6, 2.0, 3.0, 5.0]


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name,n_plans,K,seed", [("c1", 48, 1024, 1), ("c2", 48, 1024, 2), ("c4", 32, 2048, 0)])
def test_mc_curve_parity(cf, name, n_plans, K, seed):
    _say(f"mc curve {name}")
    cfg = load_config(name)
    if name == "c4":
        cfg["plans"]["sampled"]["total"] = 20000
    tab = make_plans(cfg)
    m = O.make_model(cfg["model"])
    otr = O.trace_gen(m, [seed], K)
    rd, _, fl = O.eval_coarse(m, tab, otr["moments"][0], cfg["gpus"])
    ids = O.select_topk(rd, fl, n_plans)
    tg = O.scaled_targets(m, SCALES)
    want = O.mc_curve(m, tab, ids, rd, otr["moments"][0], 0.8, otr, 0, K, tg)
    desc = cf.model_desc(cfg["model"])
    tr, mom = cf.cf_trace_gen(desc, [seed], K)
    plans = cf.DevicePlans(tab)
    grd, _, _ = cf.cf_eval_coarse(desc, plans, mom[0], cfg["gpus"])
    got = cf.cf_eval_mc_curve(desc, plans, torch.as_tensor(ids).cuda(), grd, mom[0], 0.8, tr, 0, K, tg)
    torch.cuda.synchronize()
    for key, w in zip(("met", "cnt", "goodput_t", "hist", "curve"), want):
        g = got[key].cpu().numpy()
        if g.dtype == np.int32:
            g = g.view(np.uint32)
        assert np.array_equal(g, w), key
    assert np.all(np.diff(got["curve"].cpu().numpy(), axis=1) >= 0)


@pytest.mark.parametrize("name,n_plans,seeds,n", [("c1", 5, [0, 9], 5000), ("c2", 2, [4], 4000)])
def test_fine_histograms_and_curves(cf, name, n_plans, seeds, n):
    _say(f"fine hist {name}")
    cfg = load_config(name)
    tab = make_plans(cfg)
    m = O.make_model(cfg["model"])
    otr = O.trace_gen(m, seeds, n)
    rd, _, fl = O.eval_coarse(m, tab, otr["moments"][0], cfg["gpus"])
    ids = O.select_topk(rd, fl, n_plans)
    rates = O.rate_grid(rd, ids, 16)
    tg = O.scaled_targets(m, SCALES)
    desc = cf.model_desc(cfg["model"])
    tr, _ = cf.cf_trace_gen(desc, seeds, n)
    out = cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.as_tensor(ids).cuda(), torch.from_numpy(rates).cuda(),
                          tr, targets=tg)
    torch.cuda.synchronize()
    hist = out["hist"].cpu().numpy().view(np.uint32)
    S, T, nb = len(seeds), m.n_types, len(SCALES)
    assert hist.shape == (len(ids), 16, S, T, nb + 1)
    want = np.zeros_like(hist)
    for i, p in enumerate(ids):
        for k in range(16):
            for s in range(S):
                des = O.sim_triple(m, tab, int(p), float(rates[i, k]), otr, s, want_lat=True)
                want[i, k, s] = O.latency_hist(des["lat"], otr["type"][s * n:(s + 1) * n], T, tg)
    assert np.array_equal(hist, want)
    # the histogram at the SLO bin equals the met counter; all bins sum to the count
    cum = np.cumsum(want, axis=-1).astype(np.uint32)  # the oracle's cumulative counts
    assert np.array_equal(np.cumsum(hist, axis=-1).astype(np.uint32)[..., SCALES.index(1.0)],
                          out["met"].cpu().numpy().view(np.uint32))
    assert np.array_equal(np.cumsum(hist, axis=-1).astype(np.uint32)[..., -1],
                          out["cnt"].cpu().numpy().view(np.uint32))
    # goodput against every target: the plain reduction of the oracle's cumulative counts, bin by bin
    ks, gt, g = cf.cf_goodput_curve(out, torch.from_numpy(rates).cuda(), (9, 10), n)
    ks, gt, g = ks.cpu().numpy(), gt.cpu().numpy(), g.cpu().numpy()
    cnt = np.ascontiguousarray(cum[..., -1])
    for b in range(nb):
        wk, wgt, wg = O.goodput_reduce(np.ascontiguousarray(cum[..., b]), cnt, rates, (9, 10), n)
        assert np.array_equal(ks[:, b], wk) and np.array_equal(gt[:, b], wgt) and np.array_equal(g[:, b], wg), b
    assert np.all(np.diff(g, axis=1) >= 0)


def test_bad_target_tables(cf):
    _say("curve errors")
    cfg = load_config("c1")
    desc = cf.model_desc(cfg["model"])
    m = O.make_model(cfg["model"])
    tab = make_plans(cfg)
    tr, mom = cf.cf_trace_gen(desc, [0], 64)
    plans = cf.DevicePlans(tab)
    rd, _, _ = cf.cf_eval_coarse(desc, plans, mom[0], cfg["gpus"])
    ids = torch.tensor([0, 1], dtype=torch.int32).cuda()
    tg = O.scaled_targets(m, [2.0, 1.0])  # decreasing
    with pytest.raises(cf.CfError):
        cf.cf_eval_mc_curve(desc, plans, ids, rd, mom[0], 0.8, tr, 0, 64, tg)
    tg = O.scaled_targets(m, [1.0])
    tg[0, 0, 1] = np.nan
    with pytest.raises(cf.CfError):
        cf.cf_eval_fine(desc, plans, ids, torch.ones((2, 4), dtype=torch.float64).cuda(), tr, targets=tg)
    with pytest.raises(cf.CfError):
        cf.cf_eval_mc_curve(desc, plans, ids, rd, mom[0], 0.8, tr, 0, 64, np.zeros((2, 65, 4)))
