"""Pins of the pre-copy occupancy model (App. H, the coupon-law derivation:
w uniformly random chunk writes over N chunks dirty N(1 - e^(-w/N)) distinct
chunks in expectation) and of its round recursion."""
import itertools
import math

import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("n", [1, 2, 3, 4])
@pytest.mark.parametrize("w", [0, 1, 2, 3, 4])
def test_occupancy_by_enumeration(n, w):
    counts = [len(set(seq)) for seq in itertools.product(range(n), repeat=w)]
    mean = sum(counts) / len(counts)
    var = sum(c * c for c in counts) / len(counts) - mean * mean
    assert oracle.occupancy_mean(n, w) == pytest.approx(mean, abs=1e-12)
    assert oracle.occupancy_var(n, w) == pytest.approx(var, abs=1e-9)


def test_occupancy_by_simulation():
    rng = np.random.default_rng(5)
    n, w, trials = 1000, 700, 4000
    d = np.array([np.unique(rng.integers(0, n, w)).size for _ in range(trials)])
    mean, var = oracle.occupancy_mean(n, w), oracle.occupancy_var(n, w)
    assert abs(d.mean() - mean) < 4 * math.sqrt(var / trials)
    assert d.var() == pytest.approx(var, rel=0.1)


def test_large_n_form():
    # the paper's form with w counted in chunks
    for n, w in ((25536, 19152), (6144, 3000), (10**6, 10**6)):
        assert oracle.occupancy_mean(n, w) == pytest.approx(n * (1 - math.exp(-w / n)),
                                                            rel=2.0 / n)


def test_recursion_regimes():
    n = 25536
    # writes below one chunk per chunk shipped: the dirty set decays about
    # geometrically (rate rho when it is small)
    d = oracle.precopy_recursion(n, 0.5, n, 40)
    assert d[-1] < 1e-3 * n
    assert d[-1] / d[-2] == pytest.approx(0.5, rel=1e-3)
    # above one: it saturates at the nonzero root of f = 1 - e^(-rho f)
    for rho in (1.5, 1.93, 3.0):
        f = oracle.precopy_recursion(n, rho, n, 300)[-1] / n
        assert f > 0.5 and abs(f - (1 - math.exp(-rho * f))) < 1e-9
    # the saturation the paper measured while generating, 0.777 of the
    # cache, is the fixed point for rho of about 1.93 chunk writes per
    # chunk shipped
    f = oracle.precopy_recursion(n, 1.93, n, 300)[-1] / n
    assert f == pytest.approx(0.777, abs=0.002)
