"""GPU parity of plan enumeration (cf_enum_count, cf_enum_plans) against the
oracle: totals and offsets exact, plan-table columns byte-identical over
whole spaces (the E->L graph) and over windows of the omni graph's 5e13-plan
space, including windows that start and end inside logical plans."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import oracle as O  # noqa: E402
from paper_2512_14098_amd.inputs import load_config  # noqa: E402
from paper_2512_14098_amd.inputs.plans import PlanTable  # noqa: E402

KNOBS = [16, 64, 256]


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


def _setup(cf, name, N, **extra):
    cfg = load_config(name)
    mc = cfg["model"]
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: KNOBS for c in mc["components"]}}
    spec.update(extra)
    desc, opts = cf.model_desc(mc), cf.enum_opts(mc, spec, N)
    logical = cf.cf_enum_logical(desc, opts)
    ldev = torch.from_numpy(logical).cuda()
    offsets, total = cf.cf_enum_count(desc, opts, ldev)
    m, oo = O.make_model(mc), O.enum_opts(mc, spec, N)
    Ls = O.enum_logical(m, oo)
    return desc, opts, ldev, offsets, total, m, oo, Ls


def _check_window(cf, desc, opts, ldev, offsets, total, m, oo, Ls, first, count):
    got = cf.cf_enum_plans(desc, opts, ldev, offsets, total, first, count).to_host()
    want = O.enum_plans(m, oo, Ls, first, count)
    for f in PlanTable.FIELDS:
        assert np.array_equal(getattr(got, f), getattr(want, f)), (f, first, count)


@pytest.mark.parametrize("N,extra", [(8, {}), (9, {"gpus": {"E": [1, 2], "L": [1, 4]}}), (1, {}),
                                     (5, {"share": False}), (6, {"k_s": 1})])
def test_enum_two_type_graph_whole_space(cf, N, extra):
    _say(f"enum c1 N={N} {extra}")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, "c1", N, **extra)
    counts = [O.enum_count(m, oo, L) for L in Ls]
    assert total == sum(counts)
    assert np.array_equal(offsets.cpu().numpy().view(np.uint64), np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64))
    if total:
        _check_window(cf, desc, opts, ldev, offsets, total, m, oo, Ls, 0, total)


def test_enum_omni_graph_windows(cf):
    _say("enum c2 windows")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, "c2", 16)
    counts = [O.enum_count(m, oo, L) for L in Ls]
    assert total == sum(counts) == 50378648407914
    offs = np.concatenate([[0], np.cumsum(counts)])  # the oracle's own offsets place the windows
    rng = np.random.default_rng(7)
    starts = [0, int(offs[1]) - 1000, int(offs[37]) - 17, total // 3, total - 5000]
    starts += [int(x) for x in rng.integers(0, total - 5000, size=4)]
    for s in starts:
        _check_window(cf, desc, opts, ldev, offsets, total, m, oo, Ls, s, 5000)
    # a count that is not a multiple of four in a table whose width is (the last thread's tail)
    out = cf.DevicePlans.empty(5000)
    got = cf.cf_enum_plans(desc, opts, ldev, offsets, total, starts[3], 4997, out).to_host()
    want = O.enum_plans(m, oo, Ls, starts[3], 4997)
    for f in PlanTable.FIELDS:
        assert np.array_equal(getattr(got, f)[..., :4997], getattr(want, f)), f


def test_enum_large_budget_single_subplans(cf):
    _say("enum c4 k_s=1")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, "c4", 64, k_s=1)
    assert total == sum(O.enum_count(m, oo, L) for L in Ls)
    for s in (0, total // 2, total - 3000):
        _check_window(cf, desc, opts, ldev, offsets, total, m, oo, Ls, s, 3000)


def test_enum_errors_and_overflow(cf):
    _say("enum errors")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, "c1", 4)
    with pytest.raises(cf.CfError):
        cf.cf_enum_plans(desc, opts, ldev, offsets, total, total - 2, 3)
    out = cf.cf_enum_plans(desc, opts, ldev, offsets, total, 0, 0)
    assert out.P == 0
    # the omni graph on 64 GPUs with two subplans has more than 2^64 plans
    cfg = load_config("c4")
    mc = cfg["model"]
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: KNOBS for c in mc["components"]}}
    o4 = cf.enum_opts(mc, spec, 64)
    lg = torch.from_numpy(cf.cf_enum_logical(cf.model_desc(mc), o4)).cuda()
    with pytest.raises(cf.CfError):
        cf.cf_enum_count(cf.model_desc(mc), o4, lg)


def test_enumerated_plans_screen_like_the_oracle(cf):
    """Phase 1 on a window of enumerated plans: the device table feeds cf_eval_coarse directly."""
    _say("enum + coarse c2")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, "c2", 16)
    first = total // 7
    plans = cf.cf_enum_plans(desc, opts, ldev, offsets, total, first, 20000)
    tr, mom = cf.cf_trace_gen(desc, [0], 2000)
    rd, bn, fl = cf.cf_eval_coarse(desc, plans, mom[0], 16)
    want = O.eval_coarse(m, O.enum_plans(m, oo, Ls, first, 20000), O.trace_gen(m, [0], 2000)["moments"][0], 16)
    assert np.array_equal(rd.cpu().numpy(), want[0])
    assert np.array_equal(fl.cpu().numpy(), want[2])
    assert not np.any(fl.cpu().numpy() & 6)  # none invalid or over budget


@pytest.mark.parametrize("name,N,extra", [("c1", 8, {}), ("c2", 16, {}),
                                          ("c2", 16, {"gpus": {"E_img": [1, 2], "E_aud": [1], "L_th": [1, 2, 4],
                                                               "L_ta": [1, 2], "G": [1]}})])
def test_enum_screen_fused_equals_table_path(cf, name, N, extra):
    """Phase 1 of enumerated plans without their table: identical to cf_eval_coarse on the
    enumerated table and to the oracle on its own enumeration, over windows of the space."""
    _say(f"enum screen {name} {bool(extra)}")
    cfg = load_config(name)
    mc = dict(cfg["model"])
    if extra:
        mc["components"] = [dict(c, tp_scale={"2": 0.55, "4": 0.3}) for c in mc["components"]]
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: KNOBS for c in mc["components"]}}
    spec.update(extra)
    desc, opts = cf.model_desc(mc), cf.enum_opts(mc, spec, N)
    ldev = torch.from_numpy(cf.cf_enum_logical(desc, opts)).cuda()
    offsets, total = cf.cf_enum_count(desc, opts, ldev)
    m, oo = O.make_model(mc), O.enum_opts(mc, spec, N)
    Ls = O.enum_logical(m, oo)
    tr, mom = cf.cf_trace_gen(desc, [0], 3000)
    mom_h = O.trace_gen(m, [0], 3000)["moments"][0]
    for first in (0, total // 5, total - 7000):
        cnt = min(7000, total - first)
        rd, bn, fl = cf.cf_enum_screen(desc, opts, ldev, offsets, total, first, cnt, mom[0], N)
        plans = cf.cf_enum_plans(desc, opts, ldev, offsets, total, first, cnt)
        rd2, bn2, fl2 = cf.cf_eval_coarse(desc, plans, mom[0], N)
        assert np.array_equal(rd.cpu().numpy(), rd2.cpu().numpy())
        assert np.array_equal(bn.cpu().numpy(), bn2.cpu().numpy())
        assert np.array_equal(fl.cpu().numpy(), fl2.cpu().numpy())
        want = O.eval_coarse(m, O.enum_plans(m, oo, Ls, first, cnt), mom_h, N)
        assert np.array_equal(rd.cpu().numpy(), want[0]) and np.array_equal(fl.cpu().numpy(), want[2])


@pytest.mark.parametrize("name,N,logical,count,window,k", [
    ("c1", 8, 0, 60000, 997, 50),
    ("c2", 16, 400, 50000, 4096, 300),
    ("c2", 16, 100, 9000, 1 << 24, 20000),
])
def test_space_screened_in_windows_keeps_the_top_k(cf, name, N, logical, count, window, k):
    """A range of an enumerated space screened window by window (cf_enum_screen, then
    cf_select_topk per window and cf_topk_merge across windows) keeps the same k plans, in
    the same order, as the oracle's selection over the whole range at once; R_d ties (plans
    that differ off their bottleneck) are broken by plan number across windows too."""
    _say(f"screen space {name} window={window} k={k}")
    from paper_2512_14098_amd import pipeline
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, name, N)
    first = sum(O.enum_count(m, oo, L) for L in Ls[:logical])  # from the start of a logical plan
    tr, mom = cf.cf_trace_gen(desc, [0], 3000)
    rd, gid = pipeline.screen_space(desc, opts, ldev, offsets, total, mom[0], N, k, first, count, window)
    torch.cuda.synchronize()
    ord_rd, _, fl = O.eval_coarse(m, O.enum_plans(m, oo, Ls, first, count), O.trace_gen(m, [0], 3000)["moments"][0], N)
    want = O.select_topk(ord_rd, fl, count)[:k]
    assert np.array_equal(gid.cpu().numpy(), first + np.asarray(want, np.int64))
    assert np.array_equal(rd.cpu().numpy().view(np.uint64), ord_rd[want].view(np.uint64))
    kept = ord_rd[fl & 1 != 0]
    assert len(kept) > 0 and len(np.unique(kept)) < len(kept)  # the range holds R_d ties


def test_topk_merge_edges(cf):
    dev = "cuda"
    rd = torch.tensor([3.0, 2.0, 2.0, 1.0], dtype=torch.float64, device=dev)
    e = torch.empty(0, dtype=torch.float64, device=dev)
    eg = torch.empty(0, dtype=torch.int64, device=dev)
    ids = torch.tensor([0, 1, 2, 3], dtype=torch.int32, device=dev)
    # an empty running list takes the window's first k
    r, g = cf.cf_topk_merge(e, eg, rd, ids, 100, 3)
    assert g.cpu().tolist() == [100, 101, 102] and r.cpu().tolist() == [3.0, 2.0, 2.0]
    # ties with the running list: the smaller plan number first
    r2, g2 = cf.cf_topk_merge(r, g, torch.tensor([2.0, 0.5], dtype=torch.float64, device=dev),
                              torch.tensor([0, 1], dtype=torch.int32, device=dev), 50, 4)
    assert g2.cpu().tolist() == [100, 50, 101, 102] and r2.cpu().tolist() == [3.0, 2.0, 2.0, 2.0]
    # an empty window keeps the running list
    r3, g3 = cf.cf_topk_merge(r2, g2, rd, ids[:0], 7, 4)
    assert g3.cpu().tolist() == g2.cpu().tolist()
    # a window longer than k keeps its first k
    r4, g4 = cf.cf_topk_merge(e, eg, rd, ids, 0, 2)
    assert g4.cpu().tolist() == [0, 1]
    with pytest.raises(cf.CfError):
        cf.cf_topk_merge(e, eg, rd, ids, 0, 0)       # k below 1
    buf = torch.empty(4, dtype=torch.float64, device=dev)
    bg = torch.empty(4, dtype=torch.int64, device=dev)
    rc = cf._lib.cf_topk_merge(cf._p(buf), cf._p(bg), 2, cf._p(rd), cf._p(ids), 2, 0, 4, cf._p(buf), cf._p(bg), None)
    assert rc == -1                                  # outputs alias the running list
    rc = cf._lib.cf_topk_merge(cf._p(r2), cf._p(g2), -1, cf._p(rd), cf._p(ids), 2, 0, 4, cf._p(buf), cf._p(bg), None)
    assert rc == -1                                  # a negative count


@pytest.mark.parametrize("name,N,extra,window", [
    ("c1", 4, {"gpus": {"E": [1, 2], "L": [1]}, "batch": {"E": [16, 64], "L": [16, 64, 256]}}, None),
    ("c1", 8, {}, 20000),
    ("c2", 10, {}, 5000),
])
def test_enum_two_configuration_nodes(cf, name, N, extra, window):
    """Nodes of two configurations (het): counts and offsets, plan tables byte-identical to
    the oracle's (whole space, or windows at evenly spaced starts of a large one), phase 1 of
    the device table equal to the oracle's; the fused screen refuses het."""
    _say(f"enum het {name} N={N}")
    desc, opts, ldev, offsets, total, m, oo, Ls = _setup(cf, name, N, het=True, **extra)
    counts = [O.enum_count(m, oo, L) for L in Ls]
    assert total == sum(counts)
    assert np.array_equal(offsets.cpu().numpy().view(np.uint64), np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64))
    starts = [0] if window is None else [0, total // 5, (2 * total) // 5, total // 2 + 3, total - window]
    count = total if window is None else window
    for s in starts:
        got = cf.cf_enum_plans(desc, opts, ldev, offsets, total, s, count)
        want = O.enum_plans(m, oo, Ls, s, count)
        host = got.to_host()
        for f in PlanTable.FIELDS:
            assert np.array_equal(getattr(host, f), getattr(want, f)), (f, s)
        assert np.any(want.node_rep2) or s == 0
        mom = cf.cf_trace_gen(desc, [0], 2000)[1]
        mom0 = O.trace_gen(m, [0], 2000)["moments"][0]
        rd, bn, fl = cf.cf_eval_coarse(desc, got, mom[0], N)
        w = O.eval_coarse(m, want, mom0, N)
        assert np.array_equal(rd.cpu().numpy(), w[0]) and np.array_equal(fl.cpu().numpy(), w[2])
    with pytest.raises(cf.CfError):
        cf.cf_enum_screen(desc, opts, ldev, offsets, total, 0, 64, mom[0], N)
