"""Pins of the oracle's trace generator against the distributions it must draw.

The workload (Sec. 3.1) is a mix of request types with fractions pi_t;
arrivals are Poisson (Sec. 6.4 uses Poisson intervals).  Here the
inter-arrival gap in units of the mean is Exp(1); type counts follow the
weights; image counts and patches are uniform integers; lengths are
lognormal (tokens, and seconds of audio scaled to milliseconds) after
rounding and clamping.  Each check is a statistical test at a fixed seed or
an exact identity.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config

from .helpers import model, rtype, comp


@pytest.fixture(scope="module")
def omni_trace():
    cfg = load_config("c2")
    m = O.make_model(cfg["model"])
    return cfg, m, O.trace_gen(m, [0, 1], 100000)


def test_gaps_are_exponential(omni_trace):
    _, _, tr = omni_trace
    n = tr["n_req"]
    for s in range(2):
        ticks = tr["arr_ticks"][s * n:(s + 1) * n].astype(np.float64)
        gaps = np.diff(np.concatenate([[0.0], ticks])) / 2 ** 32
        assert stats.kstest(gaps, "expon").pvalue > 1e-3
        assert np.all(np.diff(tr["arr_ticks"][s * n:(s + 1) * n].astype(np.int64)) >= 0)


def test_type_mix_follows_weights(omni_trace):
    cfg, _, tr = omni_trace
    w = np.array([t["weight"] for t in cfg["model"]["types"]], float)
    counts = np.bincount(tr["type"], minlength=len(w))
    exp = w / w.sum() * counts.sum()
    assert stats.chisquare(counts, exp).pvalue > 1e-3


def test_moments_equal_direct_sums(omni_trace):
    _, m, tr = omni_trace
    n = tr["n_req"]
    for s in range(2):
        sl = slice(s * n, (s + 1) * n)
        ty = tr["type"][sl]
        for t in range(m.n_types):
            sel = ty == t
            mo = tr["moments"][s, t]
            assert mo[0] == sel.sum()
            assert mo[1] == tr["prompt"][sl][sel].astype(np.uint64).sum()
            assert mo[2] == tr["out"][sl][sel].astype(np.uint64).sum()
            assert mo[3] == tr["patches"][sl][sel].astype(np.uint64).sum()
            assert mo[4] == tr["aud_in_ms"][sl][sel].astype(np.uint64).sum()
            assert mo[5] == tr["aud_out_ms"][sl][sel].astype(np.uint64).sum()
            assert mo[6] == ((tr["aud_in_ms"][sl][sel].astype(np.uint64) + 79) // 80).sum()
            assert mo[7] == ((tr["aud_out_ms"][sl][sel].astype(np.uint64) + 79) // 80).sum()


def test_lognormal_lengths(omni_trace):
    _, _, tr = omni_trace
    # prompt ~ round(exp(N(6, 0.5))), out ~ round(exp(N(5, 0.6))) on every type
    for field, mu, sig in (("prompt", 6.0, 0.5), ("out", 5.0, 0.6)):
        x = np.log(tr[field].astype(np.float64))
        se = sig / np.sqrt(len(x))
        assert abs(x.mean() - mu) < 5 * se + 2e-4, field
        assert abs(x.std() - sig) < 0.01, field
    # audio (types 2, 3): ms = round(1000 * exp(N(1.5, 0.5)))
    aud = tr["type"] >= 2
    for field in ("aud_in_ms", "aud_out_ms"):
        x = np.log(tr[field][aud].astype(np.float64) / 1000.0)
        assert abs(x.mean() - 1.5) < 5 * 0.5 / np.sqrt(len(x)), field
        assert abs(x.std() - 0.5) < 0.01, field
        assert np.all(tr[field][~aud] == 0)


def test_images_and_patches():
    cfg = load_config("c1")
    m = O.make_model(cfg["model"])
    tr = O.trace_gen(m, [5], 100000)
    img = tr["type"] == 1
    nimg = tr["n_img"][img]
    assert set(np.unique(nimg)) == {1, 2, 3, 4}
    assert stats.chisquare(np.bincount(nimg)[1:]).pvalue > 1e-3
    assert np.all(tr["n_img"][~img] == 0) and np.all(tr["patches"][~img] == 0)
    one = tr["patches"][img][nimg == 1].astype(np.int64)
    assert one.min() >= 256 and one.max() <= 1024
    # uniform on 769 values: mean 640, variance (769^2 - 1) / 12
    assert abs(one.mean() - 640) < 5 * np.sqrt((769 ** 2 - 1) / 12 / len(one))
    assert stats.chisquare(np.bincount(one - 256, minlength=769)).pvalue > 1e-4


def test_exponential_and_const_lengths():
    mc = model([comp("S", "ENC", [0, 1e-3, 0], x=["aud_in_ms"])],
               [rtype("a", ["S"], aud_in={"exp": 1000}, aud_out={"const": 777}, prompt={"const": 12})])
    m = O.make_model(mc)
    tr = O.trace_gen(m, [3], 100000)
    x = tr["aud_in_ms"].astype(np.float64)
    assert abs(x.mean() - 1000) < 5 * 1000 / np.sqrt(len(x))
    assert stats.kstest(x / 1000.0, "expon").statistic < 0.01  # rounding to 1 ms, clamp at 1
    assert np.all(tr["aud_out_ms"] == 777) and np.all(tr["prompt"] == 12) and np.all(tr["out"] == 0)


def test_trace_is_keyed_by_seed_and_request():
    cfg = load_config("c0")
    m = O.make_model(cfg["model"])
    a = O.trace_gen(m, [7, 8], 500)
    b = O.trace_gen(m, [8], 300)
    # request i of seed 8 does not depend on how many requests or seeds were drawn
    for f in ("type", "prompt", "out", "patches", "rkey0", "rkey1", "akey"):
        assert np.array_equal(a[f][500:800], b[f][:300]), f
    assert np.array_equal(a["arr_ticks"][500:800], b["arr_ticks"][:300])
    assert not np.array_equal(a["prompt"][:300], b["prompt"][:300])


def test_route_keys_are_uniform(omni_trace):
    _, _, tr = omni_trace
    for word in ("rkey0", "rkey1"):
        for k in range(4):
            key = (tr[word] >> np.uint64(16 * k)) & np.uint64(0xFFFF)
            rep = (key.astype(np.uint64) * np.uint64(5)) >> np.uint64(16)
            assert stats.chisquare(np.bincount(rep.astype(np.int64), minlength=5)).pvalue > 1e-3
    alt = (tr["akey"].astype(np.uint64) * np.uint64(10)) >> np.uint64(32)
    assert stats.chisquare(np.bincount(alt.astype(np.int64), minlength=10)).pvalue > 1e-3
