"""Failure statuses of the request-level simulator (cf_eval_fine), forced from the host.

The capacity limits of cf_fine_out cap, for one call, the queue-chunk pool, the delay line
and the instant budget of every simulation.  A simulation that needs more ends with
CF_ST_OVERFLOW (pool, delay line) or CF_ST_DEADLOCK (instants); the kernel exits
normally.  Every other triple of the same launch must give exactly the counts, events and
status of the unconstrained launch, and a rate with a failed simulation is infeasible in
the goodput reduction.  Invalid rates and plan ids give CF_ST_INVALID, as in the oracle.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config, make_plans  # noqa: E402

ST_INVALID, ST_DEADLOCK, ST_OVERFLOW = 1, 2, 4


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


def _setup(cf, name, ids, n, seeds, K=8, alpha=2.0):
    cfg = load_config(name)
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    tr, mom = cf.cf_trace_gen(desc, seeds, n)
    plans = cf.DevicePlans(tab)
    rd, _, _ = cf.cf_eval_coarse(desc, plans, mom[0], cfg["gpus"])
    ids_t = torch.as_tensor(np.asarray(ids, np.int32)).cuda()
    # rates up to twice the flow bound: the high ones overload the plan and grow its queues
    rates = cf.cf_rate_grid(rd, ids_t, K, alpha)
    return cfg, tab, desc, tr, plans, ids_t, rates


def _np(out):
    return {k: v.cpu().numpy() for k, v in out.items() if k in ("met", "cnt", "events", "status")}


def _check_against_free(got, free, allowed):
    st = got["status"].view(np.uint32)
    assert np.all(np.isin(st, [0, allowed])), np.unique(st)
    ok = st == 0
    for f in ("met", "cnt"):
        assert np.array_equal(got[f][ok], free[f][ok]), f
    assert np.array_equal(got["events"][ok], free["events"][ok])
    return int(ok.sum()), int((~ok).sum())


def _sweep(cf, name, ids, n, seeds, key, values, allowed):
    cfg, tab, desc, tr, plans, ids_t, rates = _setup(cf, name, ids, n, seeds)
    free = _np(cf.cf_eval_fine(desc, plans, ids_t, rates, tr))
    assert np.all(free["status"] == 0)
    mixed = []
    for v in values:
        _say(f"status {name}: {key} = {v}")
        got = _np(cf.cf_eval_fine(desc, plans, ids_t, rates, tr, limits={key: v}))
        n_ok, n_bad = _check_against_free(got, free, allowed)
        if n_ok and n_bad:
            mixed.append((v, got))
    # some limit leaves part of the launch intact and stops the rest
    assert mixed, (key, values)
    # the unconstrained launch is unchanged afterwards (no state left behind)
    again = _np(cf.cf_eval_fine(desc, plans, ids_t, rates, tr))
    for f in free:
        assert np.array_equal(again[f], free[f]), f
    return cfg, rates, free, mixed


def _check_reduce(cf, cfg, rates, free, got, n, S):
    """kstar = min(unconstrained first failure, first rate with a failed simulation) - 1."""
    dev = {k: torch.from_numpy(v).cuda() for k, v in got.items()}
    ks, gt, g = cf.cf_goodput_reduce(dev, rates, (9, 10), n)
    ks0, gt0, g0 = cf.cf_goodput_reduce({k: torch.from_numpy(v).cuda() for k, v in free.items()}, rates,
                                        (9, 10), n)
    ks, ks0 = ks.cpu().numpy(), ks0.cpu().numpy()
    failed = np.any(got["status"] != 0, axis=2)  # [plan, rate]
    K = failed.shape[1]
    first_fail = np.where(failed.any(axis=1), failed.argmax(axis=1), K)
    want = np.minimum(ks0 + 1, first_fail) - 1
    assert np.array_equal(ks, want)
    g, g0 = g.cpu().numpy(), g0.cpu().numpy()
    same = ks == ks0
    assert np.array_equal(g[same], g0[same])
    assert np.all(g[ks < 0] == 0.0)


C1_IDS = [0, 5, 30, 100, 200, 400, 600, 900]
C2_IDS = [0, 3, 50, 400, 2000, 5000]


@pytest.mark.parametrize("name,ids,n", [("c1", C1_IDS, 3000), ("c2", C2_IDS, 2000)])
def test_queue_pool_overflow(cf, name, ids, n):
    cfg, rates, free, mixed = _sweep(cf, name, ids, n, [0, 1], "chunks", [2, 4, 8, 16, 32, 64, 128, 256, 512],
                                     ST_OVERFLOW)
    _check_reduce(cf, cfg, rates, free, mixed[0][1], n, 2)


@pytest.mark.parametrize("name,ids,n", [("c1", C1_IDS, 3000), ("c2", C2_IDS, 2000)])
def test_delay_line_overflow(cf, name, ids, n):
    _sweep(cf, name, ids, n, [0, 1], "delay", [2, 4, 8, 16, 32, 64, 128, 256, 1024], ST_OVERFLOW)


@pytest.mark.parametrize("name,ids,n", [("c1", C1_IDS, 3000), ("c2", C2_IDS, 2000)])
def test_instant_budget_deadlock(cf, name, ids, n):
    cfg, rates, free, mixed = _sweep(cf, name, ids, n, [0, 1], "instants",
                                     [64, 256, 1024, 2048, 4096, 8192, 16384, 65536], ST_DEADLOCK)
    _check_reduce(cf, cfg, rates, free, mixed[len(mixed) // 2][1], n, 2)


def test_invalid_rates_and_plan_ids_match_the_oracle(cf):
    _say("status: invalid rates and plan ids")
    cfg = load_config("c0")
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    n = 500
    tr, _ = cf.cf_trace_gen(desc, [0], n)
    ids = np.array([0, 3, tab.P + 7, -1], np.int32)
    rates = np.array([[1.0, -2.0, 0.0, 4.0], [np.inf, 2.0, 8.0, np.nan], [1.0, 2.0, 4.0, 8.0],
                      [1.0, 2.0, 4.0, 8.0]])
    out = _np(cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.from_numpy(ids).cuda(),
                              torch.from_numpy(rates).cuda(), tr))
    m = O.make_model(cfg["model"])
    otr = O.trace_gen(m, [0], n)
    valid = [(i, k) for i in range(2) for k in range(4) if np.isfinite(rates[i, k]) and rates[i, k] > 0]
    st = out["status"].view(np.uint32)[:, :, 0]
    for i in range(4):
        for k in range(4):
            if (i, k) in valid:
                o = O.sim_triple(m, tab, int(ids[i]), float(rates[i, k]), otr, 0)
                assert st[i, k] == o["status"] == 0
                assert np.array_equal(out["met"][i, k, 0].view(np.uint32), o["met"])
                assert np.array_equal(out["cnt"][i, k, 0].view(np.uint32), o["cnt"])
            else:
                assert st[i, k] == ST_INVALID, (i, k)
                assert np.all(out["cnt"][i, k] == 0) and np.all(out["met"][i, k] == 0)
                if 0 <= ids[i] < tab.P:  # the oracle reads the same rate as invalid
                    assert O.sim_triple(m, tab, int(ids[i]), float(rates[i, k]), otr, 0)["status"] == ST_INVALID
    # the reduction takes a rate with an invalid simulation as infeasible
    ks, _, g = cf.cf_goodput_reduce({k: torch.from_numpy(v).cuda() for k, v in out.items()},
                                    torch.from_numpy(rates).cuda(), (9, 10), n)
    ks = ks.cpu().numpy()
    assert ks[0] == 0 and ks[1] == -1 and ks[2] == -1 and ks[3] == -1
    assert np.all(g.cpu().numpy()[1:] == 0.0)


def test_every_pair_simulated_once_whatever_the_rates(cf):
    """The launch takes a seed's (plan, rate) pairs by ascending rate: repeated rates, signed
    zeros, infinities and NaNs of either sign still give every triple exactly its own result."""
    _say("status: pair order with repeated and non-finite rates")
    cfg = load_config("c0")
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    n = 300
    tr, _ = cf.cf_trace_gen(desc, [0, 1], n)
    neg_nan = np.frombuffer(np.uint64(0xFFF8000000000001).tobytes(), np.float64)[0]
    ids = np.array([0, 1, 2, 3, 4, 5, 0], np.int32)
    rates = np.array([[2.0, 2.0, np.nan, 4.0, -0.0],
                      [0.0, 2.0, 2.0, neg_nan, 8.0],
                      [np.inf, -np.inf, 1.0, 1.0, 1.0],
                      [np.nan, np.nan, 4.0, 4.0, 2.0],
                      [1.0, 2.0, 4.0, 8.0, 16.0],
                      [-1.0, 1e-300, 2.0, neg_nan, 2.0],
                      [2.0, 2.0, np.nan, 4.0, -0.0]])
    out = _np(cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.from_numpy(ids).cuda(),
                              torch.from_numpy(rates).cuda(), tr))
    m = O.make_model(cfg["model"])
    otr = O.trace_gen(m, [0, 1], n)
    st = out["status"].view(np.uint32)
    for i in range(len(ids)):
        for k in range(rates.shape[1]):
            for s_ in range(2):
                r = float(rates[i, k])
                if np.isfinite(r) and r > 0:
                    o = O.sim_triple(m, tab, int(ids[i]), r, otr, s_)
                    assert st[i, k, s_] == o["status"], (i, k, s_)
                    assert np.array_equal(out["met"][i, k, s_].view(np.uint32), o["met"]), (i, k, s_)
                    assert np.array_equal(out["cnt"][i, k, s_].view(np.uint32), o["cnt"]), (i, k, s_)
                    assert out["events"][i, k, s_].view(np.uint64) == o["events"], (i, k, s_)
                else:
                    assert st[i, k, s_] == ST_INVALID, (i, k, s_)
    # the first and last rows are the same plan at the same rates
    for key in ("met", "cnt", "events", "status"):
        assert np.array_equal(out[key][0], out[key][6])


def test_launch_above_the_ordered_pair_limit(cf):
    """Above 2^17 (plan, rate) pairs per seed the launch takes them by rate index, then plan:
    8,200 copies of c0's plans x 16 rates, every copy equal to its first occurrence, the first
    occurrences equal to the oracle."""
    _say("status: launch of 131,200 pairs (unordered)")
    cfg = load_config("c0")
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    n, P, K = 40, 8200, 16
    tr, _ = cf.cf_trace_gen(desc, [3], n)
    ids = (np.arange(P) % tab.P).astype(np.int32)
    base = np.array([0.5 * 1.25 ** k for k in range(K)])
    rates = np.tile(base, (P, 1))
    out = _np(cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.from_numpy(ids).cuda(),
                              torch.from_numpy(rates).cuda(), tr))
    assert P * K > (1 << 17)
    for key in ("met", "cnt", "events", "status"):
        first = out[key][: tab.P]
        assert np.array_equal(out[key], np.concatenate([first] * (P // tab.P) + [first[: P % tab.P]])), key
    m = O.make_model(cfg["model"])
    want = O.eval_fine(m, tab, ids[: tab.P], np.ascontiguousarray(rates[: tab.P]), O.trace_gen(m, [3], n))
    assert np.array_equal(out["met"][: tab.P].view(np.uint32), want[0])
    assert np.array_equal(out["cnt"][: tab.P].view(np.uint32), want[1])
    assert np.array_equal(out["events"][: tab.P].view(np.uint64), want[2])
    assert np.array_equal(out["status"][: tab.P].view(np.uint32), want[3])


def test_bad_limits_and_flags_are_rejected(cf):
    cfg = load_config("c0")
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    tr, _ = cf.cf_trace_gen(desc, [0], 100)
    ids = torch.zeros(1, dtype=torch.int32).cuda()
    rates = torch.ones((1, 1), dtype=torch.float64).cuda()
    for lim in ({"delay": 3}, {"delay": 1}, {"chunks": -1}):
        with pytest.raises(cf.CfError):
            cf.cf_eval_fine(desc, cf.DevicePlans(tab), ids, rates, tr, limits=lim)
    # every trace array the simulation reads must be given
    for f in ("aud_out_ms", "prompt", "akey"):
        saved = getattr(tr.c, f + "_dev")
        setattr(tr.c, f + "_dev", None)
        try:
            with pytest.raises(cf.CfError, match="NULL trace array"):
                cf.cf_eval_fine(desc, cf.DevicePlans(tab), ids, rates, tr)
        finally:
            setattr(tr.c, f + "_dev", saved)
    cf.cf_eval_fine(desc, cf.DevicePlans(tab), ids, rates, tr)
