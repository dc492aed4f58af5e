"""GPU parity with tensor-parallel latency scaling: plans enumerated on the
device with 1, 2 and 4 GPUs per executor, models whose components run faster
on more GPUs (multipliers that are not powers of two), every phase against
the oracle -- phase 1 R_d and flags, phase 2 counts, goodput and latencies,
phase 3 counts, request-events, status and latencies -- bit-identical."""
import copy

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config  # noqa: E402

TP = {"1": 1.0, "2": 0.55, "4": 0.32}


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name,N,seeds,n", [("c1", 8, [2, 3], 3000), ("c2", 16, [4], 3000)])
def test_tp_scaling_all_phases(cf, name, N, seeds, n):
    _say(f"tp {name}")
    cfg = load_config(name)
    mc = copy.deepcopy(cfg["model"])
    for c in mc["components"]:
        c["tp_scale"] = dict(TP)
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: [16, 64] for c in mc["components"]},
            "gpus": {c["name"]: [1, 2, 4] for c in mc["components"]}}
    desc, opts = cf.model_desc(mc), cf.enum_opts(mc, spec, N)
    ldev = torch.from_numpy(cf.cf_enum_logical(desc, opts)).cuda()
    offsets, total = cf.cf_enum_count(desc, opts, ldev)
    m = O.make_model(mc)
    oo = O.enum_opts(mc, spec, N)
    Ls = O.enum_logical(m, oo)
    first = sum(O.enum_count(m, oo, L) for L in Ls[:4])  # from the fifth logical plan: windows with kept plans
    assert first == int(offsets[4].item())
    plans = cf.cf_enum_plans(desc, opts, ldev, offsets, total, first, 30000)
    tab = O.enum_plans(m, oo, Ls, first, 30000)
    assert len(np.unique(tab.node_gpus[tab.node_comp > 0])) >= 2
    tr, mom = cf.cf_trace_gen(desc, seeds, n)
    otr = O.trace_gen(m, seeds, n)
    rd, bn, fl = cf.cf_eval_coarse(desc, plans, mom[0], N)
    want = O.eval_coarse(m, tab, otr["moments"][0], N)
    assert np.array_equal(rd.cpu().numpy(), want[0]) and np.array_equal(fl.cpu().numpy(), want[2])
    ids = cf.cf_select_topk(rd, fl, 24)
    ids_h = O.select_topk(want[0], want[2], 24)  # the oracle's own selection drives its side
    assert len(ids_h) == 24
    assert np.array_equal(ids.cpu().numpy(), ids_h)
    # phase 2
    g2 = cf.cf_eval_mc(desc, plans, ids, rd, mom[0], 0.8, tr, 0, 1024, want_lat=True)
    w2 = O.eval_mc(m, tab, ids_h, want[0], otr["moments"][0], 0.8, otr, 0, 1024, want_lat=True)
    assert np.array_equal(g2["met"].cpu().numpy().view(np.uint32), w2[0])
    assert np.array_equal(g2["goodput_t"].cpu().numpy(), w2[2])
    assert np.array_equal(g2["lat"].cpu().numpy(), w2[3])
    # phase 3 on a few plans at rates around their R_d, with latencies of some triples
    sel = ids[:6]
    rates = cf.cf_rate_grid(rd, sel, 8, 1.0)
    rates_h = O.rate_grid(want[0], ids_h[:6], 8, 1.0)
    assert np.array_equal(rates.cpu().numpy(), rates_h)
    K, S = 8, len(seeds)
    lat_tr = [0, K * S // 2, 6 * K * S - 1]
    g3 = cf.cf_eval_fine(desc, plans, sel, rates, tr, lat_triples=lat_tr)
    w3 = O.eval_fine(m, tab, ids_h[:6], rates_h, otr)
    assert np.array_equal(g3["met"].cpu().numpy().view(np.uint32), w3[0])
    assert np.array_equal(g3["events"].cpu().numpy().view(np.uint64), w3[2])
    assert np.array_equal(g3["status"].cpu().numpy().view(np.uint32), w3[3])
    for j, tid in enumerate(lat_tr):
        i, rem = divmod(tid, K * S)
        k, s = divmod(rem, S)
        o = O.sim_triple(m, tab, int(ids_h[i]), float(rates_h[i, k]), otr, s, want_lat=True)
        assert np.array_equal(g3["lat"][j].cpu().numpy(), o["lat"])
