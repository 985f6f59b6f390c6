"""Pins of the oracle's index refresh for running requests (attained service).

Sec. 3.3: a running request's index is refreshed with the distribution of
its remaining cost, at bucket boundaries (bucket size 200 by default, Sec. 4).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2603_07917_amd import workloads
from tests import brute


def test_attained_service_at_bucket_boundaries():
    # o = bucket * floor(generated / bucket); a = o^2/2 + I*o (the Sec. 3.2 cost model)
    a = oracle.attained_service([100, 100, 100, 7], [450, 199, 200, 3], 200)
    assert list(a) == [400 * 400 / 2 + 100 * 400, 0.0, 200 * 200 / 2 + 100 * 200, 0.0]
    assert oracle.attained_service([7], [3], 1)[0] == 3 * 3 / 2 + 7 * 3
    with pytest.raises(ValueError):
        oracle.attained_service([1], [1], 0)


def test_zero_attained_is_the_arrival_index():
    rng = np.random.default_rng(4)
    p = rng.dirichlet(np.full(50, 0.3), size=20)
    _, r = workloads.log_bins(8192, 50)
    x = oracle.cost(rng.integers(8, 4000, size=20), r)
    G, arg = oracle.gittins(p, x)
    Ga, arga = oracle.gittins_attained(p, x, np.zeros(20))
    assert np.array_equal(G, Ga) and np.array_equal(arg, arga)


def test_exact_rational_example():
    # p = (1/4, 1/4, 1/2) on x = (1, 4, 10), served a = 2: the remaining cost is
    # 2 w.p. 1/4 and 8 w.p. 1/2 (unnormalised); both candidates give 6.
    p = [Fraction(1, 4), Fraction(1, 4), Fraction(1, 2)]
    x = [Fraction(1), Fraction(4), Fraction(10)]
    assert brute.gittins_attained_by_delta(p, x, Fraction(2)) == 6
    G, arg = oracle.gittins_attained(np.array([[0.25, 0.25, 0.5]]), np.array([1.0, 4.0, 10.0]), [2.0])
    assert G[0] == 6.0 and arg[0] == 1                    # tie: the smaller bin


def test_point_mass_left_is_its_remaining_cost():
    x = np.array([10.0, 20.0, 35.0, 70.0])
    for a in [0.0, 5.0, 19.0, 34.5]:
        G, _ = oracle.gittins_attained(np.array([[0.0, 0.0, 1.0, 0.0]]), x, [a])
        assert G[0] == 35.0 - a
    # a two-point law with the first point already passed leaves a point mass
    G, arg = oracle.gittins_attained(np.array([[0.9, 0.0, 0.0, 0.1]]), x, [12.0])
    assert abs(G[0] - (70.0 - 12.0)) <= 1e-14 * 58.0 and arg[0] == 3


def test_no_mass_above_the_attained_service():
    x = np.array([10.0, 20.0, 35.0])
    G, arg = oracle.gittins_attained(np.array([[0.5, 0.5, 0.0]]), x, [20.0])   # x <= a ruled out
    assert np.isinf(G[0]) and arg[0] == -1


@pytest.mark.parametrize("seed", range(12))
def test_equals_direct_delta_scan(seed):
    rng = np.random.default_rng(100 + seed)
    B = int(rng.integers(1, 9))
    num = rng.integers(0, 5, size=B)
    if num.sum() == 0:
        num[-1] = 1
    p = [Fraction(int(v)) for v in num]
    x = sorted(set(Fraction(int(v)) for v in rng.integers(1, 60, size=B)))
    p = p[:len(x)]
    # attained service: below, between and exactly at support points
    for a in [Fraction(0), x[0], (x[0] + x[-1]) / 2, x[-1] - Fraction(1, 3), Fraction(int(rng.integers(0, 60)))]:
        want = brute.gittins_attained_by_delta(
            p, x, a, extra_points=[Fraction(int(v), 7) for v in rng.integers(1, 500, size=20)])
        G, arg = oracle.gittins_attained(np.array([[float(v) for v in p]]),
                                         np.array([float(v) for v in x]), [float(a)])
        if want is None:
            assert np.isinf(G[0]) and arg[0] == -1
        else:
            assert abs(G[0] - float(want)) <= 1e-12 * float(want)


def test_scale_invariance_and_order_shift():
    rng = np.random.default_rng(9)
    p = rng.dirichlet(np.full(30, 0.5), size=8)
    x = np.sort(rng.uniform(1, 1e5, size=30))
    a = rng.uniform(0, 5e4, size=8)
    G1, _ = oracle.gittins_attained(p, x, a)
    G2, _ = oracle.gittins_attained(p * 7.0, x, a)
    assert np.allclose(G1, G2, rtol=1e-14)
    # shifting both the support and the attained service leaves the index unchanged
    G3, _ = oracle.gittins_attained(p, x + 1000.0, a + 1000.0)
    assert np.allclose(G1, G3, rtol=1e-9)
