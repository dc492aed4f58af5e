"""The allocation-free entry point cf_eval_fine_noalloc against cf_eval_fine.

Both are called through the C ABI on the same inputs; every output (counts, events,
status words, per-request latencies, latency histograms) must be identical, on two calls
in a row where the second is smaller than the first (it runs in the fixed array the first
left dirty).  The call must not allocate device memory: with the library's cached scratch
released, the device's free memory is the same before and after it.
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2512_14098_amd.inputs import load_config, make_plans  # noqa: E402


@pytest.fixture(scope="module")
def cf():
    from paper_2512_14098_amd import cf as _cf
    return _cf


def _say(msg):
    print(msg, flush=True)


def _inputs(cf, name, ids, n, seeds, K, alpha):
    cfg = load_config(name)
    tab = make_plans(cfg)
    desc = cf.model_desc(cfg["model"])
    tr, mom = cf.cf_trace_gen(desc, seeds, n)
    plans = cf.DevicePlans(tab)
    ids_t = torch.as_tensor(np.asarray(ids, np.int32)).cuda()
    if "explicit" in cfg["rates"]:
        rates = torch.as_tensor(np.tile(np.asarray(cfg["rates"]["explicit"], np.float64), (len(ids), 1))).cuda()
    else:
        rd, _, _ = cf.cf_eval_coarse(desc, plans, mom[0], cfg["gpus"])
        rates = cf.cf_rate_grid(rd, ids_t, K, alpha)
    return desc, plans, ids_t, rates, tr


def _compare(cf, name, ids, n, seeds, K=4, alpha=1.2, lat=False, targets=None):
    _say(f"no-alloc {name}: {len(ids)} plans, {n} requests, seeds {seeds}")
    desc, plans, ids_t, rates, tr = _inputs(cf, name, ids, n, seeds, K, alpha)
    S = len(seeds)
    lt = [0, (len(ids) * rates.shape[1] * S) // 2] if lat else None
    want = cf.cf_eval_fine(desc, plans, ids_t, rates, tr, lat_triples=lt, targets=targets)
    got = cf.cf_eval_fine_noalloc(desc, plans, ids_t, rates, tr, lat_triples=lt, targets=targets)
    torch.cuda.synchronize()
    for k in ("met", "cnt", "events", "status", "lat", "hist"):
        if want[k] is None:
            assert got[k] is None, k
            continue
        assert torch.equal(got[k], want[k]), (name, k)
    assert int(want["status"].abs().sum().item()) == 0
    return want


def test_noalloc_equals_cf_eval_fine_on_two_calls(cf):
    # a gated omni workload first, then a smaller E->L one in the array it left behind
    _compare(cf, "c2", [0, 3, 50, 400, 2000, 5000], 3000, [0, 1], K=4, lat=True)
    scales = [0.5, 1.0, 2.0]
    tg = [[[s * 0.5, s * 0.05, np.inf, np.inf] for s in scales] for _ in range(2)]
    _compare(cf, "c0", [0, 1, 2, 3, 4, 5], 500, [0], lat=True, targets=tg)


def test_noalloc_allocates_no_device_memory(cf):
    desc, plans, ids_t, rates, tr = _inputs(cf, "c1", [0, 5, 30, 100], 2000, [0], 4, 1.0)
    n_plans, K = rates.shape
    T = desc.n_types
    met = torch.empty((n_plans, K, 1, T), dtype=torch.int32, device="cuda")
    cnt = torch.empty_like(met)
    events = torch.empty((n_plans, K, 1), dtype=torch.int64, device="cuda")
    status = torch.empty((n_plans, K, 1), dtype=torch.int32, device="cuda")
    out = cf.cf_fine_out()
    out.met_dev, out.cnt_dev = met.data_ptr(), cnt.data_ptr()
    out.events_dev, out.status_dev = events.data_ptr(), status.data_ptr()
    lib = cf.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    args = (C.byref(desc), C.byref(plans.c), C.c_void_p(ids_t.data_ptr()), n_plans, C.c_void_p(rates.data_ptr()),
            K, C.byref(tr.c), 0, C.byref(out), stream)
    assert lib.cf_eval_fine_noalloc(*args) == 0  # the library's code objects are loaded by now
    torch.cuda.synchronize()
    first = (met.clone(), events.clone())
    for _ in range(2):
        assert lib.cf_release_scratch() == 0
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        assert lib.cf_eval_fine_noalloc(*args) == 0
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info()[0] == free0
        assert torch.equal(met, first[0]) and torch.equal(events, first[1])
        assert int(status.abs().sum().item()) == 0
    # the plain entry point on the same arguments allocates its scratch (the check can see it)
    assert lib.cf_release_scratch() == 0
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    assert lib.cf_eval_fine(*args) == 0
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] < free0
    assert torch.equal(met, first[0]) and torch.equal(events, first[1])


def test_noalloc_rejects_a_simulation_larger_than_its_array(cf):
    desc, plans, ids_t, rates, tr = _inputs(cf, "c0", [0], 1 << 20, [0], 4, 1.0)
    with pytest.raises(cf.CfError, match="capacity"):
        cf.cf_eval_fine_noalloc(desc, plans, ids_t, rates, tr)
