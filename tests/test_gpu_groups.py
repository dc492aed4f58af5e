"""GPU parity on plans whose nodes hold executors of two configurations (Eq. (1)'s
n_{v,k}: a node's executors split between two batches, optionally two GPU counts, the
node's requests split between them in tenths).

Plan tables come from the workloads' sampler with second configurations switched on
(``het``), some nodes given two-GPU second configurations under a tensor-parallel
multiplier; phase 1 (R_d, bottleneck, flags), phase 2 (counts, goodput, every sampled
latency) and phase 3 (counts, events, status of every triple, latencies of whole triples)
are compared with the oracle bit for bit, for a model without gating (c1, k_fine<false>)
and the omni model (c2, k_fine<true>).
"""
import copy

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config, make_plans  # noqa: E402


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


def _workload(name, total):
    cfg = copy.deepcopy(load_config(name))
    cfg["plans"].pop("families", None)  # sampled plans only
    cfg["plans"]["sampled"]["total"] = total
    cfg["plans"]["sampled"]["het"] = 0.5
    tab = make_plans(cfg, cache=False)
    # every third split node runs its second configuration on two GPUs, 0.6 times as long
    k = 0
    for p in range(tab.P):
        for v in range(tab.n_nodes[p]):
            if tab.node_rep2[v, p]:
                if k % 3 == 0:
                    tab.node_gpus2[v, p] = 2
                k += 1
    cfg["model"] = copy.deepcopy(cfg["model"])
    for c in cfg["model"]["components"]:
        c["tp_scale"] = {2: 0.6}
    return cfg, tab


@pytest.mark.parametrize("name,total,n", [("c1", 3000, 3000), ("c2", 3000, 2000)])
def test_split_nodes_all_phases(cf, name, total, n):
    cfg, tab = _workload(name, total)
    split = np.array([bool(np.any(tab.node_rep2[:, p])) for p in range(tab.P)])
    _say(f"groups {name}: {tab.P} plans, {int(split.sum())} with a split node")
    assert split.sum() > tab.P // 5
    m = O.make_model(cfg["model"])
    desc = cf.model_desc(cfg["model"])
    plans = cf.DevicePlans(tab)
    tr, mom = cf.cf_trace_gen(desc, [0, 1], n)
    otr = O.trace_gen(m, [0, 1], n)
    # phase 1
    rd, bn, fl = cf.cf_eval_coarse(desc, plans, mom[0], cfg["gpus"])
    want = O.eval_coarse(m, tab, otr["moments"][0], cfg["gpus"])
    assert np.array_equal(rd.cpu().numpy(), want[0])
    assert np.array_equal(bn.cpu().numpy(), want[1])
    assert np.array_equal(fl.cpu().numpy(), want[2])
    kept = O.select_topk(want[0], want[2], tab.P)
    kept_split = [int(p) for p in kept if split[p]]
    assert len(kept_split) >= 8
    ids = np.asarray(kept_split[:: max(1, len(kept_split) // 8)][:8], np.int32)
    # phase 2
    met, cnt, gt, lat = O.eval_mc(m, tab, ids, want[0], otr["moments"][0], 0.8, otr, 0, n, want_lat=True)
    out = cf.cf_eval_mc(desc, plans, torch.from_numpy(ids).cuda(), rd, mom[0], 0.8, tr, 0, n, want_lat=True)
    torch.cuda.synchronize()
    assert np.array_equal(out["met"].cpu().numpy().view(np.uint32), met)
    assert np.array_equal(out["cnt"].cpu().numpy().view(np.uint32), cnt)
    assert np.array_equal(out["goodput_t"].cpu().numpy(), gt)
    assert np.array_equal(out["lat"].cpu().numpy(), lat)
    # phase 3: every 4th rate of the grid, both seeds, latencies of four whole triples
    rates = np.ascontiguousarray(O.rate_grid(want[0], ids, cfg["rates"]["grid"])[:, 1::4])
    K = rates.shape[1]
    lat_tr = [0, (K * 2) * 3 + 1, (K * 2) * 5 + 2, (K * 2) * len(ids) - 1]
    g = cf.cf_eval_fine(desc, plans, torch.from_numpy(ids).cuda(), torch.from_numpy(rates).cuda(), tr,
                        lat_triples=lat_tr)
    torch.cuda.synchronize()
    wm, wc, we, ws = O.eval_fine(m, tab, ids, rates, otr)
    assert np.array_equal(g["status"].cpu().numpy().view(np.uint32), ws)
    assert np.all(ws == 0)
    assert np.array_equal(g["cnt"].cpu().numpy().view(np.uint32), wc)
    assert np.array_equal(g["met"].cpu().numpy().view(np.uint32), wm)
    assert np.array_equal(g["events"].cpu().numpy().view(np.uint64), we)
    gl = g["lat"].cpu().numpy()
    for j, tid in enumerate(lat_tr):
        i, rem = divmod(tid, K * 2)
        k, s = divmod(rem, 2)
        o = O.sim_triple(m, tab, int(ids[i]), float(rates[i, k]), otr, s, want_lat=True)
        assert np.array_equal(gl[j], o["lat"]), tid


def test_split_weight_out_of_range_is_invalid(cf):
    cfg, tab = _workload("c1", 200)
    p = next(p for p in range(tab.P) if np.any(tab.node_rep2[:, p]))
    v = int(np.argmax(tab.node_rep2[:, p] > 0))
    bad = tab.subset([p, p])
    bad.node_w[v, 1] = 10
    desc = cf.model_desc(cfg["model"])
    m = O.make_model(cfg["model"])
    tr, mom = cf.cf_trace_gen(desc, [0], 500)
    rd, bn, fl = cf.cf_eval_coarse(desc, cf.DevicePlans(bad), mom[0], cfg["gpus"])
    want = O.eval_coarse(m, bad, O.trace_gen(m, [0], 500)["moments"][0], cfg["gpus"])
    assert np.array_equal(fl.cpu().numpy(), want[2]) and fl[1].item() == 4 and fl[0].item() != 4
    out = cf.cf_eval_fine(desc, cf.DevicePlans(bad), torch.tensor([0, 1], dtype=torch.int32).cuda(),
                          torch.tensor([[5.0], [5.0]], dtype=torch.float64).cuda(), tr)
    st = out["status"].cpu().numpy().view(np.uint32)
    assert st[0, 0, 0] == 0 and st[1, 0, 0] == 1
