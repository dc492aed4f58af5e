"""The library's host-side logical-plan enumeration (cf_enum_logical, no
device work) against the oracle's, byte for byte, on every workload's model
and on option variants (no sharing, one subplan, restricted colocatable
edges, GPU options).  Runs without a GPU."""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2512_14098_amd", "libcf.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libcf.so not built")

KNOBS = [16, 64, 256]


def _spec(mc, **kw):
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: KNOBS for c in mc["components"]}}
    spec.update(kw)
    return spec


def _oracle_bytes(mc, spec, N):
    Ls = O.enum_logical(O.make_model(mc), O.enum_opts(mc, spec, N))
    return np.frombuffer(bytes(O.logical_array(Ls)), np.uint8).reshape(-1, 153)[: len(Ls)]


CASES = [("c0", {}), ("c1", {}), ("c2", {}), ("c3", {}), ("c4", {}),
         ("c2", {"share": False}), ("c2", {"k_s": 1}), ("c1", {"gpus": {"E": [1, 2], "L": [1, 4]}}),
         ("c2", {"colocatable": [["L_th", "L_ta"], ["L_ta", "G"]]}), ("c2", {"colocatable": []})]


@pytest.mark.parametrize("name,extra", CASES)
def test_logical_plans_match_the_oracle(name, extra):
    from paper_2512_14098_amd import cf
    cfg = load_config(name)
    mc = cfg["model"]
    spec = _spec(mc, **extra)
    N = min(int(cfg["gpus"]), 64)
    got = cf.cf_enum_logical(cf.model_desc(mc), cf.enum_opts(mc, spec, N))
    want = _oracle_bytes(mc, spec, N)
    assert got.shape == want.shape and np.array_equal(got, want)
    assert len(got) >= 1


def test_bad_options_are_rejected():
    from paper_2512_14098_amd import cf
    mc = load_config("c1")["model"]
    desc = cf.model_desc(mc)
    for bad in ({"n_gpus": 0}, {"n_gpus": 65}, {"k_s": 3}):
        o = cf.enum_opts(mc, _spec(mc), 8)
        for k, v in bad.items():
            setattr(o, k, v)
        with pytest.raises(cf.CfError):
            cf.cf_enum_logical(desc, o)
    o = cf.enum_opts(mc, _spec(mc), 8)
    o.batch[0][0] = 0
    with pytest.raises(cf.CfError):
        cf.cf_enum_logical(desc, o)
    with pytest.raises(cf.CfError):  # capacity
        cf.cf_enum_logical(desc, cf.enum_opts(mc, _spec(mc), 8), cap=3)
