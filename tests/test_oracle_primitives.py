"""Pins of the oracle's primitives against independent references.

* Philox4x64-10 (Salmon et al., SC'11) against numpy's own implementation:
  numpy increments the counter before producing a block, so block(c) equals
  ``Philox(counter=c-1, key=k).random_raw(4)``.
* The open-interval uniform is exact: (2m+1) 2^-53 for the top 52 bits m.
* The pinned log / exp against mpmath at 200 bits (error bound in ulp).
"""
import math
import struct

import mpmath
import numpy as np
import pytest

from oracle import oracle as O


def _numpy_block(ctr, key):
    # numpy adds one to the 256-bit counter before the first block: start from ctr - 1
    v = sum(int(w) << (64 * i) for i, w in enumerate(ctr))
    v = (v - 1) % 2 ** 256
    words = [(v >> (64 * i)) & (2 ** 64 - 1) for i in range(4)]
    g = np.random.Philox(counter=np.array(words, dtype=np.uint64), key=np.array(key, dtype=np.uint64))
    return [int(w) for w in g.random_raw(4)]


def test_philox_matches_numpy():
    rng = np.random.default_rng(1234)
    cases = [((0, 0, 0, 0), (0, 0)), ((1, 0, 0, 0), (0, 0)), ((2 ** 64 - 1, 5, 7, 9), (3, 4))]
    for _ in range(300):
        ctr = tuple(int(v) for v in rng.integers(0, 2 ** 63, size=4, dtype=np.uint64))
        key = tuple(int(v) for v in rng.integers(0, 2 ** 63, size=2, dtype=np.uint64))
        cases.append((ctr, key))
    for ctr, key in cases:
        got = [int(v) for v in O.philox(ctr, key)]
        assert got == _numpy_block(ctr, key), (ctr, key)


def test_uniform_exact_open_interval():
    for x in [0, 1, 2 ** 12 - 1, 2 ** 12, 2 ** 64 - 1, 0x8000000000000000, 123456789123456789]:
        u = O.uniform(x)
        m = x >> 12
        assert u == (2 * m + 1) / 2 ** 53
        assert 0.0 < u < 1.0


def _ulp_err(got, exact):
    exact_f = float(exact)
    ulp = math.ulp(exact_f)
    return abs(mpmath.mpf(got) - exact) / ulp


@pytest.mark.parametrize("lo,hi", [(1e-300, 1e-10), (1e-10, 0.5), (0.5, 2.0), (2.0, 1e300)])
def test_log_accuracy(lo, hi):
    mpmath.mp.prec = 200
    rng = np.random.default_rng(7)
    xs = np.exp(rng.uniform(np.log(lo), np.log(hi), 4000))
    xs = np.concatenate([xs, [1.0, 2.0, 0.5, math.sqrt(2), np.nextafter(1.0, 2), np.nextafter(1.0, 0)]])
    worst = 0.0
    for x in xs:
        x = float(x)
        if not (lo <= x <= hi) and x not in (1.0, 2.0, 0.5):
            continue
        exact = mpmath.log(mpmath.mpf(x))
        got = O.cf_log(x)
        if exact == 0:
            assert got == 0.0
            continue
        worst = max(worst, float(_ulp_err(got, exact)))
    assert worst <= 2.0, worst


def test_log_of_uniforms_is_accurate():
    """The arrival gaps use -log(u) for u = (2m+1) 2^-53; check the whole range of u."""
    mpmath.mp.prec = 200
    rng = np.random.default_rng(8)
    worst = 0.0
    for x in rng.integers(0, 2 ** 64, size=3000, dtype=np.uint64):
        u = O.uniform(int(x))
        worst = max(worst, float(_ulp_err(O.cf_log(u), mpmath.log(mpmath.mpf(u)))))
    assert worst <= 2.0, worst


@pytest.mark.parametrize("lo,hi", [(-700.0, -1.0), (-1.0, 1.0), (1.0, 20.0), (20.0, 700.0)])
def test_exp_accuracy(lo, hi):
    mpmath.mp.prec = 200
    rng = np.random.default_rng(9)
    worst = 0.0
    for x in np.concatenate([rng.uniform(lo, hi, 4000), [0.0, math.log(2), -math.log(2)]]):
        x = float(x)
        exact = mpmath.exp(mpmath.mpf(x))
        worst = max(worst, float(_ulp_err(O.cf_exp(x), exact)))
    assert worst <= 2.0, worst


def test_exp_special_values():
    assert O.cf_exp(0.0) == 1.0
    # the scaling by 2^n goes through the exponent field: exp(x + n ln2) = 2^n exp(x)
    # holds to the accuracy of the reduced argument
    for n in (-10, -1, 1, 10, 100):
        assert O.cf_exp(n * math.log(2)) == pytest.approx(2.0 ** n, rel=n * n * 1e-16 + 4e-16)


def test_log_exp_inverse():
    rng = np.random.default_rng(11)
    for x in rng.uniform(-50, 50, 2000):
        assert O.cf_log(O.cf_exp(float(x))) == pytest.approx(float(x), rel=1e-14, abs=1e-15)
