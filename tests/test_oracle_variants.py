"""Pins of the oracle's variants of the method (the paper's ablations, Sec. 4):
cost models, the Mean index, uniform-noise mixing, unweighted histogram."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2603_07917_amd import workloads
from tests import brute


def test_cost_models():
    _, r = workloads.log_bins(8192, 64)
    I = np.array([0, 8, 1000])
    assert np.array_equal(oracle.cost_variant(I, r, "resource"), oracle.cost(I, r))
    assert np.array_equal(oracle.cost_variant(I, r, "output"), np.broadcast_to(r, (3, 64)))
    assert np.array_equal(oracle.cost_variant(I, r, "overall"), I[:, None] + 2.0 * r[None, :])
    # every model is increasing in the output length, so the Gittins scan applies
    for m in ("resource", "output", "overall"):
        assert np.all(np.diff(oracle.cost_variant(I, r, m), axis=1) > 0)
    with pytest.raises(ValueError):
        oracle.cost_variant(I, r, "tokens")


def test_mean_index_exact_and_bounds():
    p = np.array([[0.25, 0.25, 0.5], [0.0, 0.0, 0.0], [2.0, 0.0, 6.0]])
    x = np.array([1.0, 4.0, 10.0])
    m = oracle.mean_index(p, x)
    assert m[0] == 6.25 and np.isinf(m[1]) and m[2] == (2 * 1 + 6 * 10) / 8
    # the Gittins index never exceeds the mean (Delta = the largest support point)
    rng = np.random.default_rng(3)
    P = rng.dirichlet(np.full(40, 0.2), size=50)
    X = np.sort(rng.uniform(1, 1e4, size=40))
    G, _ = oracle.gittins(P, X)
    assert np.all(G <= oracle.mean_index(P, X) * (1 + 1e-12))
    assert np.allclose(oracle.mean_index(P * 3.0, X), oracle.mean_index(P, X), rtol=1e-14)


def test_mean_and_gittins_order_differently():
    # Fig. 6's point: a likely-short request with a long tail vs a certain medium one
    p = np.array([[0.5, 0.0, 0.5], [0.0, 1.0, 0.0]])
    x = np.array([1.0, 5.0, 100.0])
    G, _ = oracle.gittins(p, x)
    assert list(oracle.rank(G)) == [0, 1]
    assert list(oracle.rank(oracle.mean_index(p, x))) == [1, 0]


def test_uniform_mixing():
    p = np.array([[1.0, 3.0], [0.0, 0.0]])
    mixed = oracle.mix_uniform(p, 0.2)                 # 1 : 4
    want = [Fraction(4, 5) * Fraction(1, 4) + Fraction(1, 10), Fraction(4, 5) * Fraction(3, 4) + Fraction(1, 10)]
    assert np.allclose(mixed[0], [float(v) for v in want], rtol=0, atol=1e-15)
    assert np.array_equal(mixed[1], [0.0, 0.0])        # no prediction: stays empty
    rng = np.random.default_rng(5)
    P = rng.dirichlet(np.full(16, 0.5), size=10) * 7.0
    assert np.allclose(oracle.mix_uniform(P, 0.0), P / P.sum(1, keepdims=True), rtol=1e-15)
    assert np.allclose(oracle.mix_uniform(P, 1.0), 1.0 / 16, rtol=1e-15)
    assert np.allclose(oracle.mix_uniform(P, 0.2).sum(1), 1.0, rtol=1e-15)


@pytest.mark.parametrize("seed", range(6))
def test_unweighted_histogram_matches_exact(seed):
    rng = np.random.default_rng(seed)
    N, k, B = 200, 12, 9
    edges, _ = workloads.log_bins(1000, B)
    lengths = rng.integers(1, 1001, size=N)
    ids = rng.choice(N, size=(4, k), replace=False).astype(np.int32)
    ids[3, 8:] = -1
    sims = np.round(rng.uniform(0.6, 1.0, size=(4, k)), 3).astype(np.float32)
    sims[2] = 0.5                                      # nobody above tau: counts fallback
    counts, mass = oracle.histogram(ids, sims, lengths, edges, 0.8, weighting="uniform")
    for q in range(4):
        c, m = brute.histogram_exact(ids[q], sims[q].astype(np.float64), lengths, edges, 0.8, uniform=True)
        assert list(counts[q]) == c
        assert np.allclose(mass[q], [float(v) for v in m], rtol=0, atol=1e-15)
    # with every neighbour above tau, the unweighted masses are the counts' shares
    sims_hi = np.full((4, k), 0.9, dtype=np.float32)
    c2, m2 = oracle.histogram(ids, sims_hi, lengths, edges, 0.8, weighting="uniform")
    valid = (ids >= 0).sum(1, keepdims=True)
    assert np.allclose(m2, c2 / valid, rtol=0, atol=1e-15)
    with pytest.raises(ValueError):
        oracle.histogram(ids, sims, lengths, edges, 0.8, weighting="rank")


GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_cost_models_golden():
    """The three cost models against hand-derived values (golden/cost_models.txt)."""
    n = 0
    for line in open(os.path.join(GOLDEN, "cost_models.txt")):
        if line.startswith("#") or not line.strip():
            continue
        I, O, res, out, overall, _ = [f.strip() for f in line.split("|")]
        I, O = np.array([int(I)]), np.array([float(O)])
        for model, want in (("resource", res), ("output", out), ("overall", overall)):
            assert oracle.cost_variant(I, O, model)[0, 0] == float(Fraction(want)), (model, I, O)
        n += 1
    assert n == 5


def _policy_golden():
    kv = {}
    for line in open(os.path.join(GOLDEN, "policy_orders.txt")):
        if line.startswith("#") or not line.strip():
            continue
        key, val = line.split(":", 1)
        kv[key.strip()] = val.strip()
    return kv


def test_policy_orders_golden():
    """Each policy's queue order (FCFS, Mean, Gittins at arrival, Gittins
    refreshed) and the index values behind it, against hand-derived values
    (golden/policy_orders.txt)."""
    from oracle import sage_sim
    kv = _policy_golden()
    frac = lambda s: [Fraction(v) for v in s.split()]
    mass = np.array([[float(v) for v in frac(row)] for row in kv["masses"].split(";")])
    repr_ = np.array([float(v) for v in frac(kv["repr"])])
    plen = np.array([int(v) for v in kv["prompt_len"].split()], dtype=np.int32)
    arrival = np.array([float(v) for v in kv["arrival"].split()])
    out_len = np.array([int(v) for v in kv["output_len"].split()], dtype=np.int32)
    x = oracle.cost(plen, repr_)
    G, _ = oracle.gittins(mass, x)
    assert np.allclose(G, [float(v) for v in frac(kv["gittins"])], rtol=1e-15, atol=0)
    assert np.allclose(oracle.mean_index(mass, x), [float(v) for v in frac(kv["mean"])], rtol=1e-15, atol=0)
    a1 = oracle.attained_service(plen, np.ones(4), 1)
    g1, _ = oracle.gittins_attained(mass, x, a1)
    assert np.allclose(g1, [float(v) for v in frac(kv["refreshed_level1"])], rtol=1e-15, atol=0)
    for policy in ("fcfs", "mean", "gittins-static", "gittins"):
        order, levels, informed = sage_sim.policy_order(policy, arrival, mass, plen, repr_, out_len, bucket=1)
        want = [int(v) for v in kv[f"order {policy}"].split()]
        assert list(order) == want, policy
        assert levels == (2 if policy == "gittins" else 1) and informed == len(want)
