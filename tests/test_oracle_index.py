"""Pins of the oracle's cost, index and rank stages (CPU only)."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2603_07917_amd import workloads
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_gittins():
    rows = []
    for line in open(os.path.join(GOLDEN, "gittins_cases.txt")):
        if line.startswith("#") or not line.strip():
            continue
        p, x, g, mean, _ = [f.strip() for f in line.split("|")]
        rows.append(([Fraction(v) for v in p.split()], [Fraction(v) for v in x.split()],
                     Fraction(g), Fraction(mean)))
    return rows


# ------------------------------------------------------------------ cost
def test_cost_closed_form_and_sum_form():
    # Sec. 3.2 adopts C = O^2/2 + I*O; the printed sum over l = I..I+O of l
    # equals that plus I + O/2 (the adopted form drops lower-order terms).
    for I in [0, 1, 10, 517]:
        for O in [1, 2, 4, 1000]:
            s = sum(range(I, I + O + 1))
            c = oracle.cost(np.array([I]), np.array([float(O)]))[0, 0]
            assert c == O * O / 2 + I * O
            assert Fraction(s) - Fraction(c) == I + Fraction(O, 2)


def test_cost_monotone():
    _, r = workloads.log_bins(32768, 1024)
    x = oracle.cost(np.array([0, 8, 9, 30000]), r)
    assert np.all(np.diff(x, axis=1) > 0)            # increasing in O
    assert np.all(np.diff(x, axis=0) > 0)            # increasing in I
    assert np.allclose(x[0], r * r / 2, rtol=0, atol=0)


# ----------------------------------------------------------------- index
def test_gittins_golden_cases():
    for p, x, g, mean in _golden_gittins():
        G, arg = oracle.gittins(np.array([[float(v) for v in p]]), np.array([float(v) for v in x]))
        assert abs(G[0] - float(g)) <= 1e-12 * float(g)
        bf, _ = brute.gittins_by_delta(p, x)
        assert bf == g
        assert sum(pi * xi for pi, xi in zip(p, x)) / sum(p) == mean


def test_gittins_fig6_ordering():
    # a request that finishes early half of the time (cost 1) but is long
    # otherwise (cost 100) is served before a certain cost-5 request, although
    # its mean (50.5) is ten times larger (Sec. 3.3, Fig. 6 discussion).
    G, _ = oracle.gittins(np.array([[0.5, 0.5], [1.0, 0.0]]), np.array([[1.0, 100.0], [5.0, 6.0]]))
    assert G[0] == 2.0 and G[1] == 5.0
    assert list(oracle.rank(G)) == [0, 1]
    means = np.array([50.5, 5.0])
    assert list(np.argsort(means)) == [1, 0]


@pytest.mark.parametrize("seed", range(10))
def test_gittins_equals_direct_delta_scan(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 9))
    num = rng.integers(0, 5, size=B)
    if num.sum() == 0:
        num[0] = 1
    p = [Fraction(int(v)) for v in num]
    x = sorted(Fraction(int(v)) for v in rng.integers(1, 60, size=B))
    want, evals = brute.gittins_by_delta(
        p, x, extra_points=[Fraction(int(v), 7) for v in rng.integers(1, 500, size=20)])
    G, arg = oracle.gittins(np.array([[float(v) for v in p]]), np.array([float(v) for v in x]))
    assert abs(G[0] - float(want)) <= 1e-12 * float(want)
    # the minimiser is a support point, and the oracle's argmin bin attains it
    a = int(arg[0])
    F = sum(p[: a + 1]); S = sum(pi * xi for pi, xi in zip(p[: a + 1], x[: a + 1]))
    T = sum(p[a + 1:])
    assert (S + T * x[a]) / F == want


def test_gittins_point_mass_is_cost():
    B = 64
    x = np.sort(np.random.default_rng(1).uniform(1, 1e6, size=B))
    for b in [0, 5, 63]:
        p = np.zeros((1, B)); p[0, b] = 0.37
        G, arg = oracle.gittins(p, x)
        assert G[0] == x[b] and arg[0] == b


def test_gittins_two_point_closed_form():
    rng = np.random.default_rng(2)
    for _ in range(200):
        a, b = np.sort(rng.uniform(1, 1000, size=2))
        pa = rng.uniform(0.01, 0.99)
        G, _ = oracle.gittins(np.array([[pa, 1 - pa]]), np.array([a, b]))
        want = min(a / pa, pa * a + (1 - pa) * b)
        assert abs(G[0] - want) <= 1e-12 * want


def test_gittins_bounds_scale_and_empty():
    w = workloads.small_index(Q=300, B=64, seed=4)
    x = oracle.cost(w.prompt_len, w.bin_repr)
    G, _ = oracle.gittins(w.mass, x)
    p = w.mass.astype(np.float64)
    mean = (p * x).sum(1) / p.sum(1)
    xmin = np.array([x[q][p[q] > 0].min() for q in range(300)])
    assert np.all(G >= xmin * (1 - 1e-12)) and np.all(G <= mean * (1 + 1e-12))
    G2, _ = oracle.gittins(p * 7.5, x)
    assert np.allclose(G2, G, rtol=1e-12, atol=0)
    G3, _ = oracle.gittins(p, x * 3.0)
    assert np.allclose(G3, 3 * G, rtol=1e-12, atol=0)
    Gz, az = oracle.gittins(np.zeros((2, 64)), x[:2])
    assert np.all(np.isinf(Gz)) and np.all(az == -1)


def test_gittins_stochastic_dominance():
    # moving mass to larger costs can only raise the index
    rng = np.random.default_rng(5)
    x = np.sort(rng.uniform(1, 1e4, size=32))
    for _ in range(200):
        p = rng.dirichlet(np.full(32, 0.3))
        q = p.copy()
        i = int(rng.integers(0, 31)); j = int(rng.integers(i + 1, 32))
        move = q[i] * rng.uniform(0, 1)
        q[i] -= move; q[j] += move
        G, _ = oracle.gittins(np.stack([p, q]), x)
        assert G[0] <= G[1] * (1 + 1e-12)


def test_gittins_monotone_in_prompt_length():
    w = workloads.small_index(Q=50, B=128, seed=6)
    G1, _ = oracle.gittins(w.mass, oracle.cost(w.prompt_len, w.bin_repr))
    G2, _ = oracle.gittins(w.mass, oracle.cost(w.prompt_len + 100, w.bin_repr))
    assert np.all(G2 > G1)


def test_gittins_last_bin_gives_mean():
    # the candidate at the last support point is the mean
    rng = np.random.default_rng(8)
    p = rng.dirichlet(np.ones(10))[None, :]
    x = np.sort(rng.uniform(1, 100, size=10))
    F = np.cumsum(p[0]); S = np.cumsum(p[0] * x)
    assert abs(S[-1] / F[-1] - (p[0] * x).sum()) < 1e-12


def test_gittins_rejects_unsorted_support():
    with pytest.raises(ValueError):
        oracle.gittins(np.ones((1, 3)), np.array([1.0, 3.0, 2.0]))


# ------------------------------------------------------------------ rank
def test_rank_is_stable_ascending():
    rng = np.random.default_rng(9)
    G = np.round(rng.uniform(0, 10, size=500)).astype(np.float32)
    G[::17] = np.inf
    order = oracle.rank(G)
    assert list(order) == brute.stable_order(list(G))


def test_schedule_pipeline():
    w = workloads.small_index(Q=200, B=32, seed=10)
    G, arg, order = oracle.schedule(w.mass, w.prompt_len, w.bin_repr)
    assert sorted(order) == list(range(200))
    assert np.all(np.diff(G[order]) >= 0)
