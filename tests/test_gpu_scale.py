"""GPU parity at the configurations' own scale: full trace lengths and full seed counts.

* Per-request latencies (TTFT, TPOT, E2E, MEDIA) of whole triples at full trace length on
  c1, c3 and c4, one triple per quarter of the rate grid: bit-identical to the oracle (the
  stated bar is 1e-9 relative; both sides evaluate every formula in the same order).
* Goodput at full seed count: two plans of phase 1's selection (its first and its middle
  one), every grid rate, every
  seed of the configuration (c1 32 x 10^4, c2 32 x 2.10^4, c3 64 x 5.10^4, c4 64 x 10^5
  requests): the counts, events and status of every triple bit-exact, and the GPU's goodput
  reduction of its own counts equal to the oracle's reduction of the oracle's counts (the
  stated bar is 1e-6 relative).  The oracle side runs in worker processes over the host's
  cores (tests/oracle_pool.py); c4's 4,096 triples are split over four tests so that none
  runs silent for long.
* c4's trace at 10^5 requests on three of its 64 seeds, field by field.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config, make_plans, seeds_of  # noqa: E402

from . import oracle_pool  # noqa: E402


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


_SEL = {}


def _selection(name):
    """The oracle's own phase 1 on seed 0 of the configuration: the first and the middle plan of
    its top-K selection (top plans can be copies of one another up to node order) and their grid."""
    if name not in _SEL:
        cfg = load_config(name)
        tab = make_plans(cfg)
        m = O.make_model(cfg["model"])
        mom = O.trace_gen(m, [seeds_of(cfg)[0]], int(cfg["n_req"]))["moments"][0]
        rd, _, fl = O.eval_coarse(m, tab, mom, cfg["gpus"])
        kept = O.select_topk(rd, fl, int(cfg.get("top_k") or tab.P))
        ids = np.asarray([kept[0], kept[len(kept) // 2]], np.int32)
        rates = O.rate_grid(rd, ids, cfg["rates"]["grid"], cfg["rates"].get("alpha_max", 1.0))
        _SEL[name] = (cfg, tab, m, ids, rates)
    return _SEL[name]


@pytest.mark.parametrize("name", ["c1", "c3", "c4"])
def test_latencies_at_full_trace_length(cf, name):
    cfg, tab, m, ids, rates = _selection(name)
    ids, rates = ids[:1], rates[:1]
    n = int(cfg["n_req"])
    K = rates.shape[1]
    ks = [0, K // 4, K // 2, (3 * K) // 4]  # one rate per quarter of the grid
    r = np.ascontiguousarray(rates[:, ks])
    _say(f"latencies {name}: plan {int(ids[0])}, rates {list(r[0])}, {n} requests")
    seed = seeds_of(cfg)[0]
    desc = cf.model_desc(cfg["model"])
    tr, _ = cf.cf_trace_gen(desc, [seed], n)
    out = cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.as_tensor(ids).cuda(), torch.from_numpy(r).cuda(),
                          tr, lat_triples=list(range(len(ks))))
    torch.cuda.synchronize()
    lat = out["lat"].cpu().numpy()
    otr = O.trace_gen(m, [seed], n)
    for j in range(len(ks)):
        o = O.sim_triple(m, tab, int(ids[0]), float(r[0, j]), otr, 0, want_lat=True)
        assert out["status"][0, j, 0].item() == o["status"] == 0
        assert np.array_equal(out["met"][0, j, 0].cpu().numpy().view(np.uint32), o["met"])
        np.testing.assert_allclose(lat[j], o["lat"], rtol=1e-9, atol=0)
        assert np.array_equal(lat[j], o["lat"]), (name, j)


def _goodput_case(cf, name, seed_idx):
    """GPU and oracle on the two top plans, every rate, the given seed indices."""
    cfg, tab, m, ids, rates = _selection(name)
    n = int(cfg["n_req"])
    seeds = seeds_of(cfg)
    desc = cf.model_desc(cfg["model"])
    tr, _ = cf.cf_trace_gen(desc, [seeds[s] for s in seed_idx], n)
    out = cf.cf_eval_fine(desc, cf.DevicePlans(tab), torch.as_tensor(ids).cuda(), torch.from_numpy(rates).cuda(), tr)
    torch.cuda.synchronize()
    got = {k: out[k].cpu().numpy() for k in ("met", "cnt", "events", "status")}
    sub = tab.subset(ids)
    want = oracle_pool.eval_fine_seeds(cfg["model"], sub, seeds, n, rates, list(seed_idx))
    assert np.array_equal(got["status"].view(np.uint32), want[3])
    assert np.array_equal(got["cnt"].view(np.uint32), want[1])
    assert np.array_equal(got["met"].view(np.uint32), want[0])
    assert np.array_equal(got["events"].view(np.uint64), want[2])
    return got, want


def _assert_goodput(cf, name, got, want):
    cfg, tab, m, ids, rates = _selection(name)
    n = int(cfg["n_req"])
    theta = cfg["model"].get("theta", [9, 10])
    ks, gt, g = cf.cf_goodput_reduce({k: torch.from_numpy(v).cuda() for k, v in got.items()},
                                     torch.from_numpy(rates).cuda(), theta, n)
    wk, wgt, wg = O.goodput_reduce(want[0], want[1], rates, theta, n, status=want[3])
    assert np.array_equal(ks.cpu().numpy(), wk)
    np.testing.assert_allclose(g.cpu().numpy(), wg, rtol=1e-6, atol=0)
    assert np.array_equal(gt.cpu().numpy(), wgt) and np.array_equal(g.cpu().numpy(), wg)
    _say(f"  {name}: kstar {list(wk)}, goodput {list(wg)}")


@pytest.mark.parametrize("name", ["c1", "c2", "c3"])
def test_goodput_at_full_seed_count(cf, name):
    cfg = load_config(name)
    S = len(seeds_of(cfg))
    _say(f"goodput {name}: 2 plans x {cfg['rates']['grid']} rates x {S} seeds x {cfg['n_req']} requests")
    got, want = _goodput_case(cf, name, list(range(S)))
    _assert_goodput(cf, name, got, want)


_C4 = {}


@pytest.mark.parametrize("part", [0, 1, 2, 3])
def test_goodput_c4_full_seed_count(cf, part):
    """c4 in four parts of 16 seeds (GPU and oracle both), reduced over all 64 after the last."""
    cfg = load_config("c4")
    S = len(seeds_of(cfg))
    idx = list(range(part * S // 4, (part + 1) * S // 4))
    _say(f"goodput c4 part {part}: seeds {idx[0]}..{idx[-1]}")
    _C4[part] = _goodput_case(cf, "c4", idx)
    if part == 3:
        assert sorted(_C4) == [0, 1, 2, 3], "run the four parts together"
        got = {k: np.concatenate([_C4[p][0][k] for p in range(4)], axis=2) for k in _C4[0][0]}
        want = tuple(np.concatenate([_C4[p][1][j] for p in range(4)], axis=2) for j in range(4))
        _assert_goodput(cf, "c4", got, want)


def test_c4_trace_at_full_length(cf):
    cfg = load_config("c4")
    n = int(cfg["n_req"])
    seeds = [seeds_of(cfg)[s] for s in (0, 17, 63)]
    _say(f"trace c4 seeds {seeds} n={n}")
    desc = cf.model_desc(cfg["model"])
    tr, mom = cf.cf_trace_gen(desc, seeds, n)
    torch.cuda.synchronize()
    got = tr.to_numpy()
    want = O.trace_gen(O.make_model(cfg["model"]), seeds, n)
    for f, _ in O.TRACE_FIELDS:
        assert np.array_equal(got[f], want[f]), f
    assert np.array_equal(mom.cpu().numpy().view(np.uint64), want["moments"])
