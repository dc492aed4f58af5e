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
    offs = offsets.cpu().numpy().view(np.uint64)
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
    want = O.eval_coarse(m, O.enum_plans(m, oo, Ls, first, 20000), mom[0].cpu().numpy().view(np.uint64), 16)
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
    mom_h = mom[0].cpu().numpy().view(np.uint64)
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
